// MSV-Prune scoring (Sec. 4.1): anchor scores, anchor top-k (Eq. 1),
// K-means on last-layer features (Sec. 4.1.2), anchor max-similarity and the
// per-token multi-layer similarity score of Eq. 3 in its factored form:
//   mean_{j in C} S_ij = sum_l u^l_i . mu^l_C + m_i + mean_{j in C} m_j,
//   u^l_i = F^l_i / |F^l_i|,  mu^l_C = mean_{j in C} u^l_j.
//
// Kernels (all per tile g, enqueued in this order):
//   score_prep     grid (ceil(n/16), G) x 256: a_i (sequential fp32 head sum,
//                  then one IEEE division) and 1/|F^l_i| for every tapped layer.
//   anchor_topk    grid G x 1024: LDS bitonic sort of 64-bit keys
//                  (~order(a), i); the first n_anchor are the anchors; block
//                  scans write the ascending anchor and non-anchor lists.
//   anchor_maxsim  m_i = max_p u_i . u_p.  bf16: grid (ceil(n/128), G) x 256,
//                  v_mfma_f32_32x32x16_bf16 on the raw rows (exact products,
//                  fp32 accumulation; anchors staged in LDS per 64-dimension
//                  chunk) scaled by the two inverse norms; fp32: grid
//                  (ceil(n/4), G), a wave-per-row FMA loop.
//   kmeans         grid G x (512|256): Lloyd passes; each wave keeps every
//                  centroid's slice of dimensions in registers, processes
//                  rows round-robin, and the per-wave partial sums are
//                  combined in LDS in fixed wave order (deterministic).
//   score_final    grid G x (512|256): cluster means of unit rows per tapped
//                  layer (same fixed-order reduction), cluster mean of m, and
//                  the factored score of every non-anchor row.
//
// Lane-to-dimension map used by kmeans/score_final: lane l owns VPL
// dimensions, in chunks of 8: dims {c*512 + 8*l + e : c < VPL/8, e < 8}.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <mutex>

#include "common.h"

namespace spider {
namespace {

template <typename FT>
struct Feat;
template <>
struct Feat<float> {
  static constexpr spider_dtype dt = SPIDER_F32;
  // 8 consecutive elements -> fp32
  __device__ static inline void load8(const float* p, float* o) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
  __device__ static inline float load1(const float* p) { return *p; }
  // 8 consecutive elements kept raw while in flight
  struct Raw {
    floatx4 a, b;
  };
  __device__ static inline Raw load8_raw(const float* p) {
    return {*reinterpret_cast<const floatx4*>(p), *reinterpret_cast<const floatx4*>(p + 4)};
  }
  __device__ static inline float raw_at(const Raw& v, int e) { return e < 4 ? v.a[e] : v.b[e - 4]; }
  __device__ static inline Raw load8_nt(const float* p) {
    return {__builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p)),
            __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(p + 4))};
  }
  static constexpr int kPrepRowBatch = 2;
};
template <>
struct Feat<uint16_t> {
  static constexpr spider_dtype dt = SPIDER_BF16;
  __device__ static inline void load8(const uint16_t* p, float* o) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = __uint_as_float(w[i] << 16);
      o[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ static inline float load1(const uint16_t* p) { return bf16_bits_to_f32(*p); }
  typedef u32x4 Raw;
  __device__ static inline Raw load8_raw(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
  __device__ static inline Raw load8_nt(const uint16_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  }
  __device__ static inline float raw_at(const Raw& v, int e) {
    return __uint_as_float((e & 1) ? (v[e >> 1] & 0xFFFF0000u) : (v[e >> 1] << 16));
  }
  static constexpr int kPrepRowBatch = 4;
};

struct FeatArgs {
  const void* ptr[8];
  int64_t stride_g, stride_row;
  int row0;
};

template <typename FT>
__device__ inline const FT* feat_row(const FeatArgs& fa, int l, int g, int i) {
  return reinterpret_cast<const FT*>(fa.ptr[l]) + (int64_t)g * fa.stride_g +
         (int64_t)(fa.row0 + i) * fa.stride_row;
}

// Load this lane's VPL dims of a row (zeros beyond d).
template <typename FT, int VPL>
__device__ inline void load_slice(const FT* row, int d, int lane, float* x) {
#pragma unroll
  for (int c = 0; c < VPL / 8; ++c) {
    const int base = c * 512 + lane * 8;
    if (base + 8 <= d) {
      Feat<FT>::load8(row + base, x + 8 * c);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[8 * c + e] = (base + e < d) ? Feat<FT>::load1(row + base + e) : 0.f;
    }
  }
}

__device__ inline int slice_dim(int v, int lane) { return (v >> 3) * 512 + lane * 8 + (v & 7); }

// ------------------------------------------------------------- score_prep
// Row norms of every tapped layer and the head-mean anchor scores, 16 patches
// per block (the compulsory single read of the features and the CLS rows).
// Each wave owns 4 patches; per tapped layer it issues the 16-byte loads of
// a batch of rows (4 bf16 / 2 fp32 rows, NCH chunks of 512 elements each)
// before reducing any of them.  Small batches keep the kernel at ~58 VGPRs,
// 8 waves per SIMD: more waves in flight moved more bytes than more loads per
// wave (8-row batches at 97 VGPRs ran 35 % slower).  A lane sums its chunks
// in ascending order and the wave sum is a fixed butterfly.  The last 16
// threads own one patch's head mean each, after their rows: all head loads
// are issued (8 at a time) before the sum, which runs over h = 0..H-1 in
// order, then one IEEE division.  Loads are non-temporal when the features
// exceed the last-level cache (kPrepNtBytes): the later passes re-read the
// same rows, from that cache while the tiles fit in it, and from HBM anyway
// once they do not.
constexpr int kPrepRows = 16;
constexpr int64_t kPrepNtBytes = 256ll << 20;  // MI355X Infinity Cache

template <typename FT, int NCH, bool NT>
__global__ void __launch_bounds__(256) score_prep_kernel(
    int n, int H, int d, int n_layers, const float* __restrict__ attn, int64_t as_g,
    int64_t as_h, int col0, FeatArgs fa, float* __restrict__ a_out, float* __restrict__ nu) {
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i0 = blockIdx.x * kPrepRows;
  constexpr int RW = kPrepRows / 4;  // rows per wave, in batches of RB
  constexpr int RB = Feat<FT>::kPrepRowBatch;
  const int r0 = i0 + RW * wave;
  for (int l = 0; l < n_layers; ++l) {
#pragma unroll
    for (int rb = 0; rb < RW; rb += RB) {
      typename Feat<FT>::Raw x[RB][NCH];
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const FT* row = feat_row<FT>(fa, l, g, min(r0 + rb + r, n - 1));
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const int e0 = lane * 8 + 512 * c;
          if (e0 < d) x[r][c] = NT ? Feat<FT>::load8_nt(row + e0) : Feat<FT>::load8_raw(row + e0);
        }
      }
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        float ss = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; ++c)
          if (lane * 8 + 512 * c < d) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float v = Feat<FT>::raw_at(x[r][c], e);
              ss = fmaf(v, v, ss);
            }
          }
        ss = wave_sum(ss);
        const int i = r0 + rb + r;
        if (lane == 0 && i < n) nu[((int64_t)g * n_layers + l) * n + i] = ss > 0.f ? 1.0f / sqrtf(ss) : 0.f;
      }
    }
  }
  const int t = threadIdx.x - (256 - kPrepRows);
  if (attn && t >= 0 && i0 + t < n) {  // null: scores given in a_out
    const int i = i0 + t;
    const float* col = attn + (int64_t)g * as_g + col0 + i;
    float acc = 0.f;
    for (int h0 = 0; h0 < H; h0 += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = h0 + u < H ? col[(int64_t)(h0 + u) * as_h] : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (h0 + u < H) acc = __fadd_rn(acc, v[u]);
    }
    a_out[(int64_t)g * n + i] = __fdiv_rn(acc, (float)H);
  }
}

template <typename FT>
void launch_score_prep(int G, int n, int H, int d, int n_layers, const float* attn, int64_t as_g, int64_t as_h,
                       int col0, const FeatArgs& fa, float* a_out, float* nu, hipStream_t st) {
  const dim3 grid(ceil_div(n, kPrepRows), G);
  const bool nt = (int64_t)G * n * d * (int64_t)sizeof(FT) * n_layers > kPrepNtBytes;
#define SPIDER_PREP(NCH_, NT_) \
  score_prep_kernel<FT, NCH_, NT_><<<grid, 256, 0, st>>>(n, H, d, n_layers, attn, as_g, as_h, col0, fa, a_out, nu)
  if (d <= 512) {
    if (nt) SPIDER_PREP(1, true); else SPIDER_PREP(1, false);
  } else if (d <= 1024) {
    if (nt) SPIDER_PREP(2, true); else SPIDER_PREP(2, false);
  } else {
    if (nt) SPIDER_PREP(4, true); else SPIDER_PREP(4, false);
  }
#undef SPIDER_PREP
}

// ------------------------------------------------------------- anchor_topk
constexpr int kMaxN = 4096;

__device__ inline void block_bitonic_sort(uint64_t* keys, int N) {
  for (int k = 2; k <= N; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int t = threadIdx.x; t < N / 2; t += blockDim.x) {
        const int i = (t / j) * 2 * j + (t % j);
        const int p = i + j;
        const bool up = (i & k) == 0;
        const uint64_t x = keys[i], y = keys[p];
        if ((x > y) == up) {
          keys[i] = y;
          keys[p] = x;
        }
      }
      __syncthreads();
    }
  }
}

// Exclusive scan of flags[0..n) (values 0/1) into pos[], returns the total.
// Uses `scratch` (>= blockDim/64 + 1 ints of LDS).
template <typename IT>
__device__ inline int block_scan_flags(const IT* flags, IT* pos, int n, int* scratch) {
  // each thread handles a contiguous chunk
  const int T = blockDim.x;
  const int per = (n + T - 1) / T;
  const int beg = threadIdx.x * per;
  const int end = min(n, beg + per);
  int local = 0;
  for (int i = beg; i < end; ++i) local += flags[i];
  // inclusive scan across the block of `local`
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int v = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  if (lane == 63) scratch[wave] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < T / 64; ++w) {
      const int t = scratch[w];
      scratch[w] = run;
      run += t;
    }
    scratch[T / 64] = run;
  }
  __syncthreads();
  int run = scratch[wave] + v - local;
  for (int i = beg; i < end; ++i) {
    pos[i] = (IT)run;
    run += flags[i];
  }
  const int total = scratch[T / 64];
  __syncthreads();
  return total;
}

__global__ void __launch_bounds__(1024) anchor_topk_kernel(int n, int n_anchor,
                                                           const float* __restrict__ a,
                                                           int32_t* __restrict__ cluster_out,
                                                           float* __restrict__ s_out,
                                                           int32_t* __restrict__ anc_list,
                                                           int32_t* __restrict__ rest_list,
                                                           int32_t* __restrict__ conv) {
  __shared__ uint64_t keys[kMaxN];
  __shared__ uint16_t flag[kMaxN];
  __shared__ uint16_t pos[kMaxN];
  __shared__ int scratch[17];
  const int g = blockIdx.x;
  if (threadIdx.x == 0) conv[g] = 0;
  int N = 1;
  while (N < n) N <<= 1;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    uint64_t k = ~0ull;
    if (i < n) k = ((uint64_t)(~float_order_key(a[(int64_t)g * n + i])) << 32) | (uint32_t)i;
    keys[i] = k;
  }
  __syncthreads();
  block_bitonic_sort(keys, N);
  for (int p = threadIdx.x; p < n; p += blockDim.x)
    flag[(int)(keys[p] & 0xFFFFFFFFu)] = (uint16_t)(p < n_anchor);
  __syncthreads();
  const int na = block_scan_flags(flag, pos, n, scratch);
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int64_t o = (int64_t)g * n;
    if (flag[i]) {
      anc_list[o + pos[i]] = i;
      cluster_out[o + i] = -1;
      s_out[o + i] = INFINITY;
    } else {
      rest_list[o + (i - pos[i])] = i;
      cluster_out[o + i] = 0;
    }
  }
  (void)na;
}

// ------------------------------------------------------------- anchor_maxsim
// m_i = max_p u_i . u_p over the anchors p of the tile (bf16 features):
// one block per 128 rows, one 32-row tile per wave (B operand: lane % 32 owns
// a row and its output), the anchors in tiles of 32 (A operand), up to 8 tiles
// per pass over the rows.  The anchors go through LDS one 64-dimension chunk
// at a time (double buffered; 16-byte chunk q of anchor a at slot
// q ^ ((a >> 1) & 7), so a 16-lane read of 16 anchors hits distinct banks)
// and serve all four waves; each wave reads its own rows once, the next
// chunk's loads in flight while the current chunk's MFMAs run.  A lane
// covers k in [k0 + 32 hi, k0 + 32 hi + 32) as 4 chunks of 8 for both
// operands (v_mfma_f32_32x32x16_bf16, exact products, fp32 accumulation in
// chunk order), then acc * nu_row * nu_anchor, maxed.
constexpr int kMaxAnchorTiles = 8;

__global__ void __launch_bounds__(256) anchor_maxsim_bf16_kernel(
    int n, int d, int n_anchor, FeatArgs fa, int last, const float* __restrict__ nu_last,
    int64_t nu_stride_g, const int32_t* __restrict__ anc_list, float* __restrict__ mvec) {
  __shared__ __attribute__((aligned(16))) uint8_t abuf[2][kMaxAnchorTiles * 32 * 128];
  const int g = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, hi = lane >> 5, lo = lane & 31;
  const int my_row = blockIdx.x * 128 + 32 * wave + lo;
  const bool row_ok = my_row < n;
  const uint16_t* rowp = feat_row<uint16_t>(fa, last, g, row_ok ? my_row : 0);
  const float* nu_g = nu_last + (int64_t)g * nu_stride_g;
  const int32_t* anc = anc_list + (int64_t)g * n;
  const float nu_r = row_ok ? nu_g[my_row] : 0.f;
  float best = -INFINITY;
  const int n_at = (n_anchor + 31) / 32;
  const int nkc = (d + 63) / 64;
  // staging: thread (anchor a = tid / 8 + 32 j of the pass, chunk q = tid % 8)
  const int sq = tid & 7, sa0 = tid >> 3;
  for (int t0 = 0; t0 < n_at; t0 += kMaxAnchorTiles) {
    const int nt = min(kMaxAnchorTiles, n_at - t0);
    const uint16_t* sp[kMaxAnchorTiles];
#pragma unroll
    for (int j = 0; j < kMaxAnchorTiles; ++j) {
      const int p = 32 * (t0 + j) + sa0;
      sp[j] = (j < nt && p < n_anchor) ? feat_row<uint16_t>(fa, last, g, anc[p]) : nullptr;
    }
    u32x4 ast[kMaxAnchorTiles], bv[4], bn[4];
    auto load_anchors = [&](int k0) {
      const int kk = k0 + 8 * sq;
#pragma unroll
      for (int j = 0; j < kMaxAnchorTiles; ++j)
        ast[j] = (sp[j] && kk + 8 <= d) ? *reinterpret_cast<const u32x4*>(sp[j] + kk) : u32x4{0, 0, 0, 0};
    };
    auto store_anchors = [&](int buf) {
#pragma unroll
      for (int j = 0; j < kMaxAnchorTiles; ++j)
        if (j < nt) {
          const int a = sa0 + 32 * j;
          *reinterpret_cast<u32x4*>(&abuf[buf][a * 128 + 16 * (sq ^ ((a >> 1) & 7))]) = ast[j];
        }
    };
    auto load_rows = [&](int k0, u32x4* dst) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int kk = k0 + 32 * hi + 8 * c;
        dst[c] = (row_ok && kk + 8 <= d) ? *reinterpret_cast<const u32x4*>(rowp + kk) : u32x4{0, 0, 0, 0};
      }
    };
    floatx16 acc[kMaxAnchorTiles];
#pragma unroll
    for (int j = 0; j < kMaxAnchorTiles; ++j) acc[j] = floatx16{};
    load_anchors(0);
    load_rows(0, bv);
    store_anchors(0);
    __syncthreads();
    for (int kc = 0; kc < nkc; ++kc) {
      const bool more = kc + 1 < nkc;
      if (more) {
        load_anchors(64 * (kc + 1));
        load_rows(64 * (kc + 1), bn);
      }
      const uint8_t* ab = abuf[kc & 1];
#pragma unroll
      for (int j = 0; j < kMaxAnchorTiles; ++j)
        if (j < nt) {
          const int a = 32 * j + lo;
          bf16x8 av[4];
#pragma unroll
          for (int c = 0; c < 4; ++c)
            av[c] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(ab + a * 128 + 16 * ((4 * hi + c) ^ ((a >> 1) & 7))));
#pragma unroll
          for (int c = 0; c < 4; ++c)
            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[c], __builtin_bit_cast(bf16x8, bv[c]), acc[j], 0, 0, 0);
        }
      if (more) store_anchors((kc + 1) & 1);  // that buffer was last read before the previous barrier
      __syncthreads();
#pragma unroll
      for (int c = 0; c < 4; ++c) bv[c] = bn[c];
    }
    // acc[j][r]: anchor 32 (t0 + j) + 8 (r / 4) + 4 hi + r % 4, data row my_row
#pragma unroll
    for (int j = 0; j < kMaxAnchorTiles; ++j)
      if (j < nt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int pa = 32 * (t0 + j) + 8 * (r >> 2) + 4 * hi + (r & 3);
          if (pa < n_anchor) best = fmaxf(best, acc[j][r] * nu_r * nu_g[anc[pa]]);
        }
      }
  }
  best = fmaxf(best, __shfl_xor(best, 32, 64));
  if (hi == 0 && row_ok) mvec[(int64_t)g * n + my_row] = n_anchor > 0 ? best : 0.f;
}

// fp32 features: one wave per data row, loop over anchors.
__global__ void __launch_bounds__(256) anchor_maxsim_f32_kernel(
    int n, int d, int n_anchor, FeatArgs fa, int last, const float* __restrict__ nu_last,
    int64_t nu_stride_g, const int32_t* __restrict__ anc_list, float* __restrict__ mvec) {
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + wave;
  if (i >= n) return;
  const float* row = feat_row<float>(fa, last, g, i);
  const float* nu_g = nu_last + (int64_t)g * nu_stride_g;
  float best = -INFINITY;
  for (int q = 0; q < n_anchor; ++q) {
    const int p = anc_list[(int64_t)g * n + q];
    const float* pr = feat_row<float>(fa, last, g, p);
    float dot = 0.f;
    for (int c = lane; c < d; c += 64) dot = fmaf(row[c], pr[c], dot);
    dot = wave_sum(dot);
    best = fmaxf(best, dot * nu_g[i] * nu_g[p]);
  }
  if (lane == 0) mvec[(int64_t)g * n + i] = n_anchor > 0 ? best : 0.f;
}

// ------------------------------------------------------------- clustering
// Multi-workgroup Lloyd iterations.  Each tile's m non-anchor rows are split
// into NB contiguous row ranges, one 256-thread block per range.  One Lloyd
// pass = kmeans_assign (assign rows to the nearest centroid, per-block
// per-cluster partial sums) + kmeans_update (fixed-order sum of the NB
// partials, new centroids in place; empty clusters keep theirs).  The host
// enqueues max_iter passes; once a pass changes no assignment, update sets a
// per-tile flag and the remaining launches return at once.  Centroids live
// in global memory and are staged in LDS; every reduction runs in a fixed
// order, so results are bitwise reproducible.

// Per-cluster partial sums over this block's rows [j0, j1) of layer `l`
// (optionally scaled by w[i]): out[k*d + c] for k < K.  The block makes one
// pass per cluster over its rows (they stay in L1/L2), one wave per row; the 4
// wave partials are combined in a fixed order through LDS, 512 dimensions at
// a time (red: 4 * 512 floats).
template <typename FT, int VPL>
__device__ inline void block_cluster_sums(const FeatArgs& fa, int l, int g, int d, int K,
                                          const int32_t* U, int j0, int j1, const int32_t* lab,
                                          const float* w, float* red, float* out) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int k = 0; k < K; ++k) {
    float acc[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) acc[v] = 0.f;
    for (int j = j0 + wave; j < j1; j += 4) {
      if (lab[j - j0] != k) continue;
      const int i = U[j];
      float x[VPL];
      load_slice<FT, VPL>(feat_row<FT>(fa, l, g, i), d, lane, x);
      const float sc = w ? w[i] : 1.0f;
#pragma unroll
      for (int v = 0; v < VPL; ++v) acc[v] = fmaf(x[v], sc, acc[v]);
    }
#pragma unroll
    for (int q = 0; q < VPL / 8; ++q) {
#pragma unroll
      for (int e = 0; e < 8; ++e) red[wave * 512 + lane * 8 + e] = acc[8 * q + e];
      __syncthreads();
      for (int c = threadIdx.x; c < 512; c += blockDim.x) {
        const int dim = q * 512 + c;
        if (dim < d) out[k * d + dim] = ((red[c] + red[512 + c]) + red[1024 + c]) + red[1536 + c];
      }
      __syncthreads();
    }
  }
}

// Fixed-order combine of the 4 waves' per-cluster sums acc[k] (k < K) into
// out[k*d + c], 512 dimensions at a time through LDS (red: 4 * 512 floats).
template <int KM, int VPL>
__device__ __forceinline__ void block_combine_cluster_sums(const float (&acc)[KM][VPL], int K, int d, float* red,
                                                           float* out) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 0; k < KM; ++k) {
    if (k >= K) break;
#pragma unroll
    for (int q = 0; q < VPL / 8; ++q) {
#pragma unroll
      for (int e = 0; e < 8; ++e) red[wave * 512 + lane * 8 + e] = acc[k][8 * q + e];
      __syncthreads();
      for (int c = threadIdx.x; c < 512; c += blockDim.x) {
        const int dim = q * 512 + c;
        if (dim < d) out[k * d + dim] = ((red[c] + red[512 + c]) + red[1024 + c]) + red[1536 + c];
      }
      __syncthreads();
    }
  }
}

// Adds row x (scaled by sc) to the accumulator of its cluster.  fmaf(x, 1, a)
// rounds like a + x, and each cluster receives its rows in increasing row
// order, the order block_cluster_sums uses: both paths give the same bits.
// (Written as per-element selects: a branch per cluster gets merged by the
// compiler into one dynamically indexed update, which lives in scratch.)
template <int KM, int VPL>
__device__ __forceinline__ void add_to_cluster(float (&acc)[KM][VPL], int k_row, const float* x, float sc) {
#pragma unroll
  for (int k = 0; k < KM; ++k) {
    const bool mine = k_row == k;
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const float t = fmaf(x[v], sc, acc[k][v]);
      acc[k][v] = mine ? t : acc[k][v];
    }
  }
}

// Cluster counts up to this size keep one accumulator per cluster in
// registers and read every row once per pass.
constexpr int kFusedClusters = 4;

constexpr int kMaxRowsPerBlock = 128;

struct ClusterWs {
  float* cent;      // [G][K][d]
  float* psum;      // [G][NB][K][d]    (kmeans) / [G][NB][L][K][d] (means)
  int32_t* pcnt;    // [G][NB][K]
  float* pm;        // [G][NB][K]       partial sums of m
  int32_t* pchg;    // [G][NB]
  int32_t* conv;    // [G]
  int32_t* assign;  // [G][n]  assignment of non-anchor row j (index into U)
  float* mu;        // [G][L][K][d]
  float* mbar;      // [G][K]
  int NB, RB;       // blocks per tile, rows per block
};

template <typename FT, int VPL>
__global__ void __launch_bounds__(256) kmeans_assign_kernel(int n, int d, int n_anchor, int K,
                                                            int first, FeatArgs fa, int last,
                                                            const int32_t* __restrict__ rest_list,
                                                            ClusterWs cw, int32_t* __restrict__ cluster_out) {
  extern __shared__ __attribute__((aligned(16))) float smem[];  // 16-byte centroid reads
  float* cs = smem;                 // [K*d] centroids
  float* red = cs + K * d;          // [4*512]
  __shared__ int lab[kMaxRowsPerBlock];
  __shared__ int sidx[kMaxRowsPerBlock];  // U[j0..j1): one dependent load less per row
  __shared__ int chg;
  const int g = blockIdx.y, b = blockIdx.x;
  const int m = n - n_anchor;
  const int j0 = b * cw.RB, j1 = min(m, j0 + cw.RB);
  if (j0 >= j1 || cw.conv[g]) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int32_t* U = rest_list + (int64_t)g * n;
  for (int j = j0 + threadIdx.x; j < j1; j += blockDim.x) sidx[j - j0] = U[j];
  float* cent = cw.cent + (int64_t)g * K * d;
  if (first) {
    // centroids at rows floor(k*m/K) of the non-anchor list
    for (int t = threadIdx.x; t < K * d; t += blockDim.x) {
      const int k = t / d, c = t - k * d;
      const FT* row = feat_row<FT>(fa, last, g, U[(int)(((int64_t)k * m) / K)]);
      const float v = Feat<FT>::load1(row + c);
      cs[t] = v;
      if (b == 0) cent[t] = v;
    }
  } else {
    for (int t = threadIdx.x; t < K * d; t += blockDim.x) cs[t] = cent[t];
  }
  if (threadIdx.x == 0) chg = first;
  __syncthreads();
  int32_t* asg = cw.assign + (int64_t)g * n;
  const bool fused = K <= kFusedClusters;
  float acc[kFusedClusters][VPL];
#pragma unroll
  for (int k = 0; k < kFusedClusters; ++k)
#pragma unroll
    for (int v = 0; v < VPL; ++v) acc[k][v] = 0.f;
  // d % 8 == 0: every 8-dimension chunk of a lane is whole, and its centroid
  // values are read as two 16-byte LDS vectors (lane l reads bytes 32 l ..,
  // no bank conflicts; scalar reads at 8-float lane strides conflict 8 ways).
  // Same terms in the same order as the scalar loop, so the same bits.
  const bool d8 = (d & 7) == 0;
  for (int j = j0 + wave; j < j1; j += 4) {
    float x[VPL];
    load_slice<FT, VPL>(feat_row<FT>(fa, last, g, sidx[j - j0]), d, lane, x);
    int best = 0;
    float bd = 0.f;
    for (int k = 0; k < K; ++k) {
      float s = 0.f;
      if (d8) {
#pragma unroll
        for (int c = 0; c < VPL / 8; ++c) {
          const int base = c * 512 + lane * 8;
          if (base < d) {
            const float4 c0 = *reinterpret_cast<const float4*>(cs + k * d + base);
            const float4 c1 = *reinterpret_cast<const float4*>(cs + k * d + base + 4);
            const float cc[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float t = x[8 * c + e] - cc[e];
              s = fmaf(t, t, s);
            }
          }
        }
      } else {
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          const int dim = slice_dim(v, lane);
          const float t = dim < d ? x[v] - cs[k * d + dim] : 0.f;
          s = fmaf(t, t, s);
        }
      }
      s = wave_sum(s);
      if (k == 0 || s < bd) {
        bd = s;
        best = k;
      }
    }
    if (fused) add_to_cluster<kFusedClusters, VPL>(acc, best, x, 1.0f);
    if (lane == 0) {
      if (!first && asg[j] != best) chg = 1;
      asg[j] = best;
      lab[j - j0] = best;
      cluster_out[(int64_t)g * n + sidx[j - j0]] = best;
    }
  }
  __syncthreads();
  const int64_t slot = (int64_t)g * cw.NB + b;
  if (fused)
    block_combine_cluster_sums<kFusedClusters, VPL>(acc, K, d, red, cw.psum + slot * K * d);
  else
    block_cluster_sums<FT, VPL>(fa, last, g, d, K, U, j0, j1, lab, nullptr, red, cw.psum + slot * K * d);
  if (threadIdx.x < K) {
    int c = 0;
    for (int j = j0; j < j1; ++j) c += lab[j - j0] == (int)threadIdx.x;
    cw.pcnt[slot * K + threadIdx.x] = c;
  }
  if (threadIdx.x == 0) cw.pchg[slot] = chg;
}

// grid (ceil(K*d/256), G): new centroids = fixed-order sums of the partials.
__global__ void __launch_bounds__(256) kmeans_update_kernel(int d, int K, ClusterWs cw, int nb_used) {
  const int g = blockIdx.y;
  if (cw.conv[g]) return;
  int any = 0;
  for (int b = 0; b < nb_used; ++b) any |= cw.pchg[(int64_t)g * cw.NB + b];
  if (!any) {
    if (blockIdx.x == 0 && threadIdx.x == 0) cw.conv[g] = 1;
    return;
  }
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= K * d) return;
  const int k = t / d;
  float s = 0.f;
  int c = 0;
  for (int b = 0; b < nb_used; ++b) {
    const int64_t slot = (int64_t)g * cw.NB + b;
    s += cw.psum[slot * K * d + t];
    c += cw.pcnt[slot * K + k];
  }
  if (c > 0) cw.cent[(int64_t)g * K * d + t] = __fdiv_rn(s, (float)c);
}

// Partial per-cluster sums of unit rows (every tapped layer) and of m.
template <typename FT, int VPL>
__global__ void __launch_bounds__(256) cluster_sum_kernel(int n, int d, int n_anchor, int K,
                                                          int n_layers, FeatArgs fa,
                                                          const float* __restrict__ nu,
                                                          const int32_t* __restrict__ rest_list,
                                                          const float* __restrict__ mvec, ClusterWs cw) {
  __shared__ float red[4 * 512];
  __shared__ int lab[kMaxRowsPerBlock];
  __shared__ int sidx[kMaxRowsPerBlock];  // U[j0..j1), then m of those rows: no dependent
  __shared__ float sm_m[kMaxRowsPerBlock];  // index loads inside the row loops
  const int g = blockIdx.y, b = blockIdx.x;
  const int m = n - n_anchor;
  const int j0 = b * cw.RB, j1 = min(m, j0 + cw.RB);
  if (j0 >= j1) return;
  const int32_t* U = rest_list + (int64_t)g * n;
  const int32_t* asg = cw.assign + (int64_t)g * n;
  for (int j = j0 + threadIdx.x; j < j1; j += blockDim.x) {
    lab[j - j0] = asg[j];
    const int i = U[j];
    sidx[j - j0] = i;
    sm_m[j - j0] = mvec[(int64_t)g * n + i];
  }
  __syncthreads();
  const int64_t slot = (int64_t)g * cw.NB + b;
  for (int l = 0; l < n_layers; ++l) {
    const float* nul = nu + ((int64_t)g * n_layers + l) * n;
    float* out = cw.psum + (slot * n_layers + l) * K * d;
    if (K <= kFusedClusters) {
      // one read of every row: each goes to its cluster's accumulator
      const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
      float acc[kFusedClusters][VPL];
#pragma unroll
      for (int k = 0; k < kFusedClusters; ++k)
#pragma unroll
        for (int v = 0; v < VPL; ++v) acc[k][v] = 0.f;
      for (int j = j0 + wave; j < j1; j += 4) {
        const int i = sidx[j - j0];
        float x[VPL];
        load_slice<FT, VPL>(feat_row<FT>(fa, l, g, i), d, lane, x);
        add_to_cluster<kFusedClusters, VPL>(acc, lab[j - j0], x, nul[i]);
      }
      block_combine_cluster_sums<kFusedClusters, VPL>(acc, K, d, red, out);
    } else {
      block_cluster_sums<FT, VPL>(fa, l, g, d, K, U, j0, j1, lab, nul, red, out);
    }
  }
  if (threadIdx.x < K) {
    int c = 0;
    float sm = 0.f;
    for (int j = j0; j < j1; ++j)
      if (lab[j - j0] == (int)threadIdx.x) {
        ++c;
        sm += sm_m[j - j0];
      }
    cw.pcnt[slot * K + threadIdx.x] = c;
    cw.pm[slot * K + threadIdx.x] = sm;
  }
}

// grid (ceil(L*K*d/256), G): mu = fixed-order sums / counts; mbar likewise.
__global__ void __launch_bounds__(256) cluster_mean_kernel(int d, int K, int n_layers, ClusterWs cw,
                                                           int nb_used) {
  const int g = blockIdx.y;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int per = K * d;
  if (t < n_layers * per) {
    const int l = t / per, r = t - l * per, k = r / d;
    float s = 0.f;
    int c = 0;
    for (int b = 0; b < nb_used; ++b) {
      const int64_t slot = (int64_t)g * cw.NB + b;
      s += cw.psum[(slot * n_layers + l) * per + r];
      c += cw.pcnt[slot * K + k];
    }
    cw.mu[((int64_t)g * n_layers + l) * per + r] = c ? __fdiv_rn(s, (float)c) : 0.f;
  }
  if (blockIdx.x == 0 && threadIdx.x < K) {
    const int k = threadIdx.x;
    float s = 0.f;
    int c = 0;
    for (int b = 0; b < nb_used; ++b) {
      const int64_t slot = (int64_t)g * cw.NB + b;
      s += cw.pm[slot * K + k];
      c += cw.pcnt[slot * K + k];
    }
    cw.mbar[(int64_t)g * K + k] = c ? __fdiv_rn(s, (float)c) : 0.f;
  }
}

// One wave per non-anchor row (fallback where the cluster means do not fit in LDS): s = sum_l nu_l * (F^l_i . mu^l_c) + m_i + mbar_c.
template <typename FT, int VPL>
__global__ void __launch_bounds__(256) score_rows_wave_kernel(int n, int d, int n_anchor, int K,
                                                              int n_layers, FeatArgs fa,
                                                         const float* __restrict__ nu,
                                                         const int32_t* __restrict__ rest_list,
                                                         const float* __restrict__ mvec, ClusterWs cw,
                                                         float* __restrict__ s_out,
                                                         float* __restrict__ m_out) {
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = n - n_anchor;
  if (m_out && blockIdx.x == 0)
    for (int i = threadIdx.x; i < n; i += blockDim.x) m_out[(int64_t)g * n + i] = mvec[(int64_t)g * n + i];
  const int j = blockIdx.x * 4 + wave;
  if (j >= m) return;
  const int i = rest_list[(int64_t)g * n + j];
  const int k = cw.assign[(int64_t)g * n + j];
  float s = 0.f;
  for (int l = 0; l < n_layers; ++l) {
    float x[VPL];
    load_slice<FT, VPL>(feat_row<FT>(fa, l, g, i), d, lane, x);
    const float* mu = cw.mu + (((int64_t)g * n_layers + l) * K + k) * d;
    float dot = 0.f;
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const int dim = slice_dim(v, lane);
      if (dim < d) dot = fmaf(x[v], mu[dim], dot);
    }
    dot = wave_sum(dot);
    s += dot * nu[((int64_t)g * n_layers + l) * n + i];
  }
  if (lane == 0) s_out[(int64_t)g * n + i] = s + mvec[(int64_t)g * n + i] + cw.mbar[(int64_t)g * K + k];
}

// The same scores, 64 rows per block and 16 per wave in batches of RB rows
// whose feature loads (two tapped layers at a time) are all issued before
// any is used; the tile's cluster means mu[l][k] (n_layers * K * d floats, at
// most kMuLdsFloats) are staged in LDS once per block.  Per row and layer a
// lane adds its dimensions in ascending order, then the wave sum, then
// s += dot * nu_l in layer order: the arithmetic of score_rows_wave_kernel in
// the same order, so the same bits.
constexpr int kScoreRowsPerBlock = 64;
constexpr int kMuLdsFloats = 8192;

template <typename FT, int VPL>
__global__ void __launch_bounds__(256) score_rows_kernel(int n, int d, int n_anchor, int K, int n_layers,
                                                         FeatArgs fa, const float* __restrict__ nu,
                                                         const int32_t* __restrict__ rest_list,
                                                         const float* __restrict__ mvec, ClusterWs cw,
                                                         float* __restrict__ s_out, float* __restrict__ m_out) {
  __shared__ __attribute__((aligned(16))) float smu[kMuLdsFloats];
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m = n - n_anchor;
  if (m_out && blockIdx.x == 0)
    for (int i = threadIdx.x; i < n; i += blockDim.x) m_out[(int64_t)g * n + i] = mvec[(int64_t)g * n + i];
  if (m <= 0) return;
  const int lkd = n_layers * K * d;  // a multiple of 8 (d is)
  const float* mug = cw.mu + (int64_t)g * lkd;
  for (int t = threadIdx.x * 4; t < lkd; t += 1024)
    *reinterpret_cast<float4*>(smu + t) = *reinterpret_cast<const float4*>(mug + t);
  __syncthreads();
  constexpr int RB = Feat<FT>::kPrepRowBatch;
  constexpr int NCH = VPL / 8;
  const int32_t* U = rest_list + (int64_t)g * n;
  const int32_t* asg = cw.assign + (int64_t)g * n;
  const int jw = blockIdx.x * kScoreRowsPerBlock + 16 * wave;
  for (int jb = 0; jb < 16; jb += RB) {
    if (jw + jb >= m) break;
    int ii[RB], kc[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int j = min(jw + jb + r, m - 1);
      ii[r] = U[j];
      kc[r] = asg[j];
    }
    float sacc[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) sacc[r] = 0.f;
    for (int l0 = 0; l0 < n_layers; l0 += 2) {
      const bool two = l0 + 1 < n_layers;
      typename Feat<FT>::Raw x[2][RB][NCH];
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          const FT* row = feat_row<FT>(fa, q == 0 || !two ? l0 : l0 + 1, g, ii[r]);
#pragma unroll
          for (int c = 0; c < NCH; ++c) {
            const int e0 = lane * 8 + 512 * c;
            if (e0 < d && (q == 0 || two)) x[q][r][c] = Feat<FT>::load8_raw(row + e0);
          }
        }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        if (q == 1 && !two) break;
        const int l = l0 + q;
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          const float* mu = smu + (l * K + kc[r]) * d;
          float dot = 0.f;
#pragma unroll
          for (int c = 0; c < NCH; ++c) {
            const int e0 = lane * 8 + 512 * c;
            if (e0 < d) {
              const float4 m0 = *reinterpret_cast<const float4*>(mu + e0);
              const float4 m1 = *reinterpret_cast<const float4*>(mu + e0 + 4);
              const float mv[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
#pragma unroll
              for (int e = 0; e < 8; ++e) dot = fmaf(Feat<FT>::raw_at(x[q][r][c], e), mv[e], dot);
            }
          }
          dot = wave_sum(dot);
          sacc[r] += dot * nu[((int64_t)g * n_layers + l) * n + ii[r]];
        }
      }
    }
    if (lane == 0)
#pragma unroll
      for (int r = 0; r < RB; ++r)
        if (jw + jb + r < m)
          s_out[(int64_t)g * n + ii[r]] = sacc[r] + mvec[(int64_t)g * n + ii[r]] + cw.mbar[(int64_t)g * K + kc[r]];
  }
}

struct ScoreWs {
  float* nu;
  int32_t* anc;
  int32_t* rest;
  float* mvec;
  ClusterWs cw;
};

// Blocks per tile: about 32 rows each (at most 16 per tile, never more than
// kMaxRowsPerBlock rows per block).  It depends on n only, so a tile gets the
// same partial-sum order, hence the same bits, whatever the batch size G.
int blocks_per_tile(int G, int n) {
  (void)G;
  const int need = (n + kMaxRowsPerBlock - 1) / kMaxRowsPerBlock;
  const int want = std::min(16, (n + 31) / 32);
  return std::max(need, std::max(1, want));
}

size_t score_ws_layout(int G, int n, int d, int n_layers, int K, ScoreWs* w, char* base) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return base ? base + o : nullptr;
  };
  const int NB = blocks_per_tile(G, n);
  const int L1 = std::max(1, n_layers);
  char* p_nu = take((size_t)G * n_layers * n * 4);
  char* p_anc = take((size_t)G * n * 4);
  char* p_rest = take((size_t)G * n * 4);
  char* p_mvec = take((size_t)G * n * 4);
  char* p_cent = take((size_t)G * K * d * 4);
  char* p_psum = take((size_t)G * NB * L1 * K * d * 4);
  char* p_pcnt = take((size_t)G * NB * K * 4);
  char* p_pm = take((size_t)G * NB * K * 4);
  char* p_pchg = take((size_t)G * NB * 4);
  char* p_conv = take((size_t)G * 4);
  char* p_asg = take((size_t)G * n * 4);
  char* p_mu = take((size_t)G * L1 * K * d * 4);
  char* p_mbar = take((size_t)G * K * 4);
  if (w) {
    w->nu = reinterpret_cast<float*>(p_nu);
    w->anc = reinterpret_cast<int32_t*>(p_anc);
    w->rest = reinterpret_cast<int32_t*>(p_rest);
    w->mvec = reinterpret_cast<float*>(p_mvec);
    w->cw.cent = reinterpret_cast<float*>(p_cent);
    w->cw.psum = reinterpret_cast<float*>(p_psum);
    w->cw.pcnt = reinterpret_cast<int32_t*>(p_pcnt);
    w->cw.pm = reinterpret_cast<float*>(p_pm);
    w->cw.pchg = reinterpret_cast<int32_t*>(p_pchg);
    w->cw.conv = reinterpret_cast<int32_t*>(p_conv);
    w->cw.assign = reinterpret_cast<int32_t*>(p_asg);
    w->cw.mu = reinterpret_cast<float*>(p_mu);
    w->cw.mbar = reinterpret_cast<float*>(p_mbar);
    w->cw.NB = NB;
  }
  return off;
}

template <typename FT, int VPL>
hipError_t launch_cluster_kernels(int G, int n, int d, int n_anchor, int K, int max_iter,
                                  int n_layers, const FeatArgs& fa, ScoreWs ws,
                                  int32_t* cluster_out, float* s_out, float* m_out, hipStream_t st) {
  const int m = n - n_anchor;
  const int NB = ws.cw.NB;
  ws.cw.RB = m > 0 ? (m + NB - 1) / NB : 1;
  const int nb_used = m > 0 ? (m + ws.cw.RB - 1) / ws.cw.RB : 0;
  // NB >= ceil(n / kMaxRowsPerBlock) guarantees these; checked before any launch
  if (ws.cw.RB > kMaxRowsPerBlock || nb_used > NB) return hipErrorInvalidValue;
  if (m > 0) {
    ProfScope ps(KC_KMEANS, st);
    const size_t sh = ((size_t)K * d + 4 * 512) * 4;
    for (int it = 0; it < max_iter; ++it) {
      kmeans_assign_kernel<FT, VPL><<<dim3(nb_used, G), 256, sh, st>>>(
          n, d, n_anchor, K, it == 0, fa, n_layers - 1, ws.rest, ws.cw, cluster_out);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      if (it + 1 < max_iter) {
        kmeans_update_kernel<<<dim3(ceil_div(K * d, 256), G), 256, 0, st>>>(d, K, ws.cw, nb_used);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
      }
    }
  }
  {
    ProfScope ps(KC_SCORE_FINAL, st);
    if (m > 0) {
      cluster_sum_kernel<FT, VPL><<<dim3(nb_used, G), 256, 0, st>>>(
          n, d, n_anchor, K, n_layers, fa, ws.nu, ws.rest, ws.mvec, ws.cw);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      cluster_mean_kernel<<<dim3(ceil_div(n_layers * K * d, 256), G), 256, 0, st>>>(d, K, n_layers,
                                                                                  ws.cw, nb_used);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    if ((int64_t)n_layers * K * d <= kMuLdsFloats)
      score_rows_kernel<FT, VPL><<<dim3(std::max(1, ceil_div(m, kScoreRowsPerBlock)), G), 256, 0, st>>>(
          n, d, n_anchor, K, n_layers, fa, ws.nu, ws.rest, ws.mvec, ws.cw, s_out, m_out);
    else
      score_rows_wave_kernel<FT, VPL><<<dim3(std::max(1, ceil_div(m, 4)), G), 256, 0, st>>>(
          n, d, n_anchor, K, n_layers, fa, ws.nu, ws.rest, ws.mvec, ws.cw, s_out, m_out);
    return hipGetLastError();
  }
}

template <typename FT>
hipError_t dispatch_cluster(int G, int n, int d, int n_anchor, int K, int max_iter, int n_layers,
                            const FeatArgs& fa, const ScoreWs& ws, int32_t* cl, float* s,
                            float* mo, hipStream_t st) {
  if (d <= 512)
    return launch_cluster_kernels<FT, 8>(G, n, d, n_anchor, K, max_iter, n_layers, fa, ws, cl, s, mo, st);
  if (d <= 1024)
    return launch_cluster_kernels<FT, 16>(G, n, d, n_anchor, K, max_iter, n_layers, fa, ws, cl, s, mo, st);
  return launch_cluster_kernels<FT, 32>(G, n, d, n_anchor, K, max_iter, n_layers, fa, ws, cl, s, mo, st);
}

}  // namespace
}  // namespace spider

using namespace spider;

extern "C" size_t spider_score_workspace_size(int G, int n, int d_v, int n_layers, int K) {
  if (G <= 0 || n <= 0 || d_v <= 0 || n_layers <= 0 || K <= 0) return 0;
  return score_ws_layout(G, n, d_v, n_layers, K, nullptr, nullptr);
}

extern "C" spider_status spider_score(int G, int n, int H, int d_v, int n_layers,
                                      const float* cls_attn, int64_t attn_stride_g,
                                      int64_t attn_stride_h, int attn_col0,
                                      const void* const* feats, spider_dtype feat_dtype,
                                      int64_t feat_stride_g, int64_t feat_stride_row, int feat_row0,
                                      int n_anchor, int K, int kmeans_max_iter, float* a_out,
                                      int32_t* cluster_out, float* s_out, float* m_out,
                                      void* workspace, size_t workspace_bytes,
                                      spider_stream stream) {
  clear_error();
  SPIDER_REQUIRE(G >= 1 && n >= 1 && d_v >= 1 && n_layers >= 1, SPIDER_ERR_INVALID_ARG,
                 "spider_score: G, n, d_v and n_layers must be >= 1");
  // cls_attn == NULL with H == 0: a_out already holds the anchor scores (input)
  const bool given_a = cls_attn == nullptr;
  SPIDER_REQUIRE(given_a ? H == 0 : H >= 1, SPIDER_ERR_INVALID_ARG,
                 "spider_score: H must be >= 1 with CLS attention, 0 with given anchor scores");
  SPIDER_REQUIRE(n <= kMaxN, SPIDER_ERR_UNSUPPORTED, "spider_score: n = %d exceeds 4096", n);
  SPIDER_REQUIRE(d_v <= 2048, SPIDER_ERR_UNSUPPORTED, "spider_score: d_v = %d exceeds 2048", d_v);
  SPIDER_REQUIRE(n_layers <= 8, SPIDER_ERR_UNSUPPORTED, "spider_score: at most 8 tapped layers");
  SPIDER_REQUIRE(K >= 1 && K <= 8, SPIDER_ERR_UNSUPPORTED, "spider_score: K must be in [1, 8]");
  SPIDER_REQUIRE(!(d_v > 1024 && K > 4), SPIDER_ERR_UNSUPPORTED,
                 "spider_score: K > 4 needs d_v <= 1024");
  SPIDER_REQUIRE(n_anchor >= 0 && n_anchor <= n, SPIDER_ERR_SHAPE,
                 "spider_score: n_anchor = %d outside [0, n = %d]", n_anchor, n);
  SPIDER_REQUIRE(kmeans_max_iter >= 1, SPIDER_ERR_INVALID_ARG,
                 "spider_score: kmeans_max_iter must be >= 1");
  SPIDER_REQUIRE(feats && a_out && cluster_out && s_out, SPIDER_ERR_INVALID_ARG,
                 "spider_score: null pointer argument");
  SPIDER_REQUIRE(feat_dtype == SPIDER_F32 || feat_dtype == SPIDER_BF16, SPIDER_ERR_INVALID_ARG,
                 "spider_score: bad feature dtype");
  SPIDER_REQUIRE(given_a || (attn_col0 >= 0 && attn_stride_h >= attn_col0 + n &&
                              attn_stride_g >= (int64_t)H * attn_stride_h),
                 SPIDER_ERR_SHAPE, "spider_score: attention strides do not cover [H, col0 + n]");
  SPIDER_REQUIRE(feat_row0 >= 0, SPIDER_ERR_SHAPE, "spider_score: feat_row0 must be >= 0");
  SPIDER_REQUIRE(feat_stride_row >= d_v && feat_stride_g >= (int64_t)(feat_row0 + n) * feat_stride_row,
                 SPIDER_ERR_SHAPE, "spider_score: feature strides do not cover [row0 + n, d_v]");
  SPIDER_REQUIRE(feat_stride_row % 8 == 0 && feat_stride_g % 8 == 0 && d_v % 8 == 0,
                 SPIDER_ERR_UNSUPPORTED,
                 "spider_score: d_v and the feature strides must be multiples of 8 elements");
  for (int l = 0; l < n_layers; ++l) {
    SPIDER_REQUIRE(feats[l] != nullptr, SPIDER_ERR_INVALID_ARG, "spider_score: feats[%d] is null", l);
    SPIDER_REQUIRE(((uintptr_t)feats[l] % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                   "spider_score: feats[%d] must be 16-byte aligned", l);
  }
  const size_t need = score_ws_layout(G, n, d_v, n_layers, K, nullptr, nullptr);
  SPIDER_REQUIRE(workspace && workspace_bytes >= need, SPIDER_ERR_WORKSPACE,
                 "spider_score: workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  SPIDER_REQUIRE(((uintptr_t)workspace % 256) == 0, SPIDER_ERR_WORKSPACE,
                 "spider_score: workspace must be 256-byte aligned");

  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  ScoreWs ws;
  score_ws_layout(G, n, d_v, n_layers, K, &ws, reinterpret_cast<char*>(workspace));
  FeatArgs fa;
  for (int l = 0; l < 8; ++l) fa.ptr[l] = l < n_layers ? feats[l] : nullptr;
  fa.stride_g = feat_stride_g;
  fa.stride_row = feat_stride_row;
  fa.row0 = feat_row0;
  const int last = n_layers - 1;

  {
    ProfScope ps(KC_SCORE_PREP, st);
    if (feat_dtype == SPIDER_BF16)
      launch_score_prep<uint16_t>(G, n, H, d_v, n_layers, cls_attn, attn_stride_g, attn_stride_h, attn_col0, fa,
                                  a_out, ws.nu, st);
    else
      launch_score_prep<float>(G, n, H, d_v, n_layers, cls_attn, attn_stride_g, attn_stride_h, attn_col0, fa,
                               a_out, ws.nu, st);
    SPIDER_LAUNCHED("score_prep");
  }
  {
    ProfScope ps(KC_ANCHOR_TOPK, st);
    anchor_topk_kernel<<<G, 1024, 0, st>>>(n, n_anchor, a_out, cluster_out, s_out, ws.anc, ws.rest,
                                            ws.cw.conv);
    SPIDER_LAUNCHED("anchor_topk");
  }
  {
    ProfScope ps(KC_MAXSIM, st);
    const float* nu_last = ws.nu + (size_t)last * n;
    const int64_t nu_stride = (int64_t)n_layers * n;
    if (feat_dtype == SPIDER_BF16)
      anchor_maxsim_bf16_kernel<<<dim3(ceil_div(n, 128), G), 256, 0, st>>>(
          n, d_v, n_anchor, fa, last, nu_last, nu_stride, ws.anc, ws.mvec);
    else
      anchor_maxsim_f32_kernel<<<dim3(ceil_div(n, 4), G), 256, 0, st>>>(
          n, d_v, n_anchor, fa, last, nu_last, nu_stride, ws.anc, ws.mvec);
    SPIDER_LAUNCHED("anchor_maxsim");
  }
  hipError_t e = feat_dtype == SPIDER_BF16
                     ? dispatch_cluster<uint16_t>(G, n, d_v, n_anchor, K, kmeans_max_iter, n_layers,
                                                  fa, ws, cluster_out, s_out, m_out, st)
                     : dispatch_cluster<float>(G, n, d_v, n_anchor, K, kmeans_max_iter, n_layers, fa,
                                               ws, cluster_out, s_out, m_out, st);
  SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "spider_score: cluster kernels failed: %s",
                 hipGetErrorString(e));
  return SPIDER_OK;
}

// ------------------------------------------------------------------ no-allocation variant
// Scratch of spider_score_noalloc: a file-scope device array, so the call needs
// no device allocation (for callers that cannot allocate, e.g. under graph
// capture or in a serving loop).  Every GPU the library runs on holds its own
// copy until the process ends.  Host code never uses the array's name as an
// address: the device address is looked up once per device with
// hipGetSymbolAddress and kept in g_scratch_ptr.
static __device__ __align__(256) uint8_t scratch[SPIDER_SCORE_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of the scratch array (looked up on the
// first call made with that device current).
spider_status scratch_of_current_device(void** out) {
  int dev = -1;
  SPIDER_HIP(hipGetDevice(&dev));
  SPIDER_REQUIRE(dev >= 0 && dev < kMaxDevices, SPIDER_ERR_UNSUPPORTED,
                 "spider_score_noalloc: device %d beyond the %d the library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    SPIDER_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    SPIDER_REQUIRE(p != nullptr && ((uintptr_t)p % 256) == 0, SPIDER_ERR_HIP,
                   "spider_score_noalloc: scratch address of device %d is not usable", dev);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SPIDER_OK;
}
}  // namespace

extern "C" spider_status spider_score_noalloc(int G, int n, int H, int d_v, int n_layers,
                                              const float* cls_attn, int64_t attn_stride_g,
                                              int64_t attn_stride_h, int attn_col0,
                                              const void* const* feats, spider_dtype feat_dtype,
                                              int64_t feat_stride_g, int64_t feat_stride_row,
                                              int feat_row0, int n_anchor, int K, int kmeans_max_iter,
                                              float* a_out, int32_t* cluster_out, float* s_out,
                                              float* m_out, spider_stream stream) {
  clear_error();
  SPIDER_REQUIRE(G >= 1 && n >= 1 && d_v >= 1 && n_layers >= 1 && K >= 1, SPIDER_ERR_INVALID_ARG,
                 "spider_score_noalloc: G, n, d_v, n_layers and K must be >= 1");
  const size_t need = score_ws_layout(G, n, d_v, n_layers, K, nullptr, nullptr);
  SPIDER_REQUIRE(need <= (size_t)SPIDER_SCORE_SCRATCH_BYTES, SPIDER_ERR_WORKSPACE,
                 "spider_score_noalloc: these sizes need %zu bytes of scratch, the static scratch "
                 "holds %zu (use spider_score with a workspace)",
                 need, (size_t)SPIDER_SCORE_SCRATCH_BYTES);
  void* ws = nullptr;
  const spider_status st = scratch_of_current_device(&ws);
  if (st != SPIDER_OK) return st;
  // the kernels write every scratch element they read: stale contents from an
  // earlier call on this device need no clearing
  return spider_score(G, n, H, d_v, n_layers, cls_attn, attn_stride_g, attn_stride_h, attn_col0, feats,
                      feat_dtype, feat_stride_g, feat_stride_row, feat_row0, n_anchor, K, kmeans_max_iter,
                      a_out, cluster_out, s_out, m_out, ws, SPIDER_SCORE_SCRATCH_BYTES, stream);
}
