// Internal launch interfaces of the decoder kernels (GEMM, attention).
#pragma once

#include "common.h"

namespace spider {

// One GEMM problem of a grouped launch: out = A[rows] x W^T (nn.Linear layout).
struct GemmGroup {
  const void* A;          // activations [*, K] row-major, row stride lda
  const int32_t* a_rows;  // optional: A row of output row m (gather); null = identity
  int M;                  // output rows
  const void* W;          // weights [N, K] row-major
  const void* W2;         // second weights for the dual (SwiGLU) epilogue, else null
  int N;                  // output columns
  void* out;              // see GemmArgs::epilogue
  int64_t ldo;            // row stride of out (elements)
  int64_t split_stride;   // elements between split-K slabs of out
  int tiles_m, tiles_n;   // filled by the launcher
  int tile_begin;         // filled by the launcher
  int kind;               // EPI_QKV_BF16 only: 1 = RoPE'd rows (Q, K), 2 = transposed rows (V^T)
  // Optional device row count: the kernel takes min(M, *m_dev) rows (M is then
  // the bound the launch is sized for).  Streaming, LDS-staged and fp32
  // kernels only; the launcher rejects it where it would pick another kernel.
  const int32_t* m_dev;
};

enum GemmEpilogue {
  EPI_PARTIAL_F32 = 0,  // out fp32 [split][M][N]: this split's partial sums
  EPI_SWIGLU = 1,       // out act dtype [M][N] = silu(A W^T) * (A W2^T); split must be 1
  EPI_LENS_STATS = 2,   // out fp32 [M][N/128][4]: per row and 128-column tile of z = A W^T,
                        // (max z, sum e^(z-max), sum e^(z-max) (z-max), 0); bf16 only,
                        // M <= 256, N % 128 == 0, K % 64 == 0, no split
  EPI_RESIDUAL_F32 = 3,  // out fp32 [M][N] += A W^T; bf16, M <= 4 only (decode), no split
  EPI_QKV_BF16 = 4,      // bf16 out per group kind: 1 = rotate-half RoPE at pos[row] (row = a_rows[m]
                         // or m) then out [M][ldo]; 2 = out^T [N][ldvt]; head size 128, more than
                         // 256 rows, the tile kernel without split only (gemm_tile_unsplit_blocks)
  EPI_DECODE_QKV = 5     // bf16, M <= 4 (decode rows, row m = sample m), head size 128: kind bit 0 =
                         // rotate-half RoPE at pos[m], bit 1 = row m goes to the cache slot
                         // out + (m * kv_cap + pos[m]) * ldo instead of out + m * ldo
};

struct GemmArgs {
  GemmGroup g[3];
  int ngroups;
  int K;
  int64_t lda;
  int split;
  int k_per_split;
  int epilogue;
  int total_tiles;
  // Optional fp32 scratch the launcher may use (SwiGLU with more than 256 rows:
  // the tiles of a nearly empty last wave of blocks are split along k, their
  // gate and up partial sums go here and a reduction applies the epilogue).
  void* scratch;
  size_t scratch_bytes;
  // filled by the launcher for those split tiles
  int tail_tiles, tail_split, tail_kps;
  // Optional (bf16, M <= 4): A rows are RMSNorm(norm_h rows) * norm_w rounded
  // to bf16, computed by the GEMM itself (norm_h fp32 [*, K], same row gather)
  const float* norm_h;
  const float* norm_w;
  float norm_eps;
  // EPI_QKV_BF16: RoPE table [positions][64] (cos, sin), packed-row positions, V^T row stride
  const float2* rope;
  const int32_t* pos;
  int64_t ldvt;
  int kv_cap;  // EPI_DECODE_QKV: cache slots per sample
};

// Blocks of the launch when launch_gemm_bf16 would run these groups through
// the tile kernel without split-K (the condition of EPI_QKV_BF16), else 0.
int gemm_tile_unsplit_blocks(const GemmArgs& a, int split_max);

// The rotate-half RoPE of the pair (x0, x1) with (cos, sin): one rounding
// order shared by every kernel that applies it.
__device__ __forceinline__ float2 rope_rotate(float x0, float x1, float c, float s) {
  return make_float2(fmaf(x0, c, -(x1 * s)), fmaf(x1, c, x0 * s));
}

// Chooses tiles and split-K for the groups (all with the same K) and launches.
// `split_max` bounds split-K (partial buffers are sized for it).
hipError_t launch_gemm_bf16(GemmArgs& a, int split_max, hipStream_t st);
hipError_t launch_gemm_f32(GemmArgs& a, int split_max, hipStream_t st);

// Split-K factor the launcher will use for a group of M rows, N columns, K depth.
int gemm_split_for(int M, int N, int K, bool dual, bool bf16, int split_max);

// Causal attention over packed samples for a compacted list of query rows.
struct AttnArgs {
  const void* q;           // [nq, d] (row a = query a)
  const int32_t* q_rows;   // [nq] packed row of query a
  const void* k;           // [rows, d]
  const void* v;           // bf16: V^T [d][ldvt] (rows >= `rows` zero); fp32: [rows, d]
  int64_t ldvt;            // row stride of V^T (a multiple of 32); 0 for row-major V
  const int32_t* row_start;  // [rows] first row of the sample that owns the row
  void* o;                 // [nq, d]
  int nq, rows, H, dh, d;
  float scale;             // 1/sqrt(dh)
  const int32_t* nq_dev;   // optional device query count: min(nq, *nq_dev) queries (nq = the bound)
};
hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t st);
hipError_t launch_attention_f32(const AttnArgs& a, int max_seq, hipStream_t st);

// Online skip controller (Sec. 4.2.1, Eq. 4, Eq. 6).  Candidates are visual
// rows not yet in skip mode: cand[c] = packed row, cand_sample[c] = its sample.
// tmean[b] = mean hidden state of sample b's last n_text rows.
hipError_t launch_text_mean(const float* h, int d, const int32_t* cu, int B, int n_text, float* tmean,
                            hipStream_t st);
// hc[c] = h[cand[c]] in the activation dtype, F[c] = (1 + cos(h[cand[c]], tmean[b])) / 2.
// With nc_dev non-null the launch is sized for nc candidates and
// min(nc, *nc_dev) of them are processed (also for the two admission launches).
hipError_t launch_lens_prep(bool bf16, const float* h, int d, const int32_t* cand,
                            const int32_t* cand_sample, int nc, const int32_t* nc_dev, const float* tmean,
                            void* hc, double* F, hipStream_t st);
struct LensAdmitArgs {
  double log_v;      // ln V
  double w1;         // weight of S_sa
  double w2_sel;     // w2 * SLC_sel(l), formed on the host in double
  double t_skip;     // admission threshold
  double* acc;       // [rows] accumulated skip score (indexed by packed row)
  int32_t* flag;     // [nc] 1 = admitted at this layer
  float* s_out;      // [rows] S_sa of this layer, or null
  uint32_t ablation; // SPIDER_ONLINE_* bits: E_ii or F_itc left out, no accumulation
};
// Per candidate c (logits row c of [nc, V]): E_ii, S_sa, acc update, flag.
hipError_t launch_lens_admit(const float* logits, int V, const int32_t* cand, int nc, const int32_t* nc_dev,
                             const double* F, const LensAdmitArgs& p, hipStream_t st);
// The same from EPI_LENS_STATS tiles: stats [nc][ntiles][4].
hipError_t launch_lens_admit_stats(const float* stats, int ntiles, const int32_t* cand, int nc,
                                   const int32_t* nc_dev, const double* F, const LensAdmitArgs& p,
                                   hipStream_t st);
// Zero `bytes` (a multiple of 4) of device memory with a kernel.
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st);

}  // namespace spider
