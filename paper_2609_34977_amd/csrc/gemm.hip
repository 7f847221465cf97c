// Decoder GEMMs: out = A[rows] x W^T with W in nn.Linear layout [N, K].
//
// bf16 path (gemm_bf16_kernel): built for the weight-streaming regime of a
// pruned prefill (a few hundred rows against multi-MB weight matrices), and
// for large row counts.  256 threads = 4 waves; block tile BM x BN x 32 with
// v_mfma_f32_16x16x32_bf16 (fp32 accumulation); a wave owns a
// (BM/WGM) x (BN/WGN) sub-tile.  For up to 256 rows one block covers every
// row (BM = rows rounded up to 64), so each weight element is read from HBM
// exactly once; the activations (a few MB) stay in L2.  The k-loop keeps a
// ring of PF register stages of 16-byte global loads in flight (PF tiles
// ahead), double-buffers LDS (row pitch 40 bf16: the 16 rows x 16 bytes of a
// fragment read hit distinct banks) and needs one barrier per k-tile.  A rows
// may be gathered through a row list.  Grouped launch: up to three problems
// sharing K (Q over the query rows, K and V over all rows) in one grid.
// Logical tiles are ordered (group, n-tile, k-split, m-tile) and the hardware
// block id is remapped so consecutive logical tiles run on the same XCD
// (blocks are dispatched round-robin over the 8 XCDs) and share its L2.
// Epilogues: fp32 split-K partials (summed by the consumer kernel in fixed
// order: deterministic without atomics), or the fused SwiGLU
// silu(A Wg^T) * (A Wu^T) rounded to bf16 (dual weights, no split).
//
// fp32 path (gemm_f32_kernel): 16x16 FMA tiles through LDS with the same
// group/gather/split/epilogue semantics (used by fp32 workloads).
#include <algorithm>
#include <type_traits>

#include "kernels.h"

namespace spider {
namespace {

constexpr int kNumXcd = 8;

__device__ inline int xcd_remap(int b, int total) {
  const int q = total / kNumXcd, r = total % kNumXcd;
  const int xcd = b % kNumXcd, idx = b / kNumXcd;
  return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

template <typename T>
__device__ __forceinline__ T sel3(int gi, T x0, T x1, T x2) {
  return gi == 0 ? x0 : (gi == 1 ? x1 : x2);
}

struct TileCoord {
  int gi, m0, n0, s;
};

__device__ inline TileCoord decode_tile(const GemmArgs& a, int t, int BM, int BN) {
  int gi = 0;
  if (a.ngroups > 1 && t >= a.g[1].tile_begin) gi = 1;
  if (a.ngroups > 2 && t >= a.g[2].tile_begin) gi = 2;
  const int tb = sel3(gi, a.g[0].tile_begin, a.g[1].tile_begin, a.g[2].tile_begin);
  const int tm = sel3(gi, a.g[0].tiles_m, a.g[1].tiles_m, a.g[2].tiles_m);
  int local = t - tb;
  const int m_tile = local % tm;
  local /= tm;
  const int s = local % a.split;
  const int n_tile = local / a.split;
  return {gi, m_tile * BM, n_tile * BN, s};
}

__device__ inline float silu(float g) { return g / (1.0f + __expf(-g)); }

// Fields of group gi, read with constant offsets from the kernel arguments
// (a dynamic index into the argument array would be materialised in scratch).
struct GroupView {
  const void* A;
  const int32_t* rows;
  int M;
  const void* W;
  const void* W2;
  void* out;
  int N;
  int64_t ldo, sstride;
};

__device__ __forceinline__ GroupView group_view(const GemmArgs& a, int gi) {
  GroupView v;
  v.A = sel3(gi, a.g[0].A, a.g[1].A, a.g[2].A);
  v.rows = sel3(gi, a.g[0].a_rows, a.g[1].a_rows, a.g[2].a_rows);
  v.M = sel3(gi, a.g[0].M, a.g[1].M, a.g[2].M);
  v.W = sel3(gi, a.g[0].W, a.g[1].W, a.g[2].W);
  v.W2 = sel3(gi, a.g[0].W2, a.g[1].W2, a.g[2].W2);
  v.out = sel3(gi, a.g[0].out, a.g[1].out, a.g[2].out);
  v.N = sel3(gi, a.g[0].N, a.g[1].N, a.g[2].N);
  v.ldo = sel3(gi, a.g[0].ldo, a.g[1].ldo, a.g[2].ldo);
  v.sstride = sel3(gi, a.g[0].split_stride, a.g[1].split_stride, a.g[2].split_stride);
  return v;
}

template <int BM, int BN, int WGM, int WGN, int PF, bool DUAL, bool NT = false>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(GemmArgs a) {
  constexpr int BK = 32, PITCH = BK + 8;
  constexpr int BROWS = DUAL ? 2 * BN : BN;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int A_CH = BM * (BK / 8) / 256;
  constexpr int B_CH = BROWS * (BK / 8) / 256;
  static_assert(WGM * WGN == 4, "4 waves");
  static_assert(TM >= 1 && TN >= 1 && WTM % 16 == 0 && WTN % 16 == 0, "wave tile");
  static_assert(A_CH >= 1 && B_CH >= 1 && A_CH * 256 == BM * 4 && B_CH * 256 == BROWS * 4, "chunks");
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BROWS * PITCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, lg = lane >> 4;
  const int wm = wave / WGN, wn = wave % WGN;
  const TileCoord tc = decode_tile(a, xcd_remap(blockIdx.x, a.total_tiles), BM, BN);
  const GroupView G = group_view(a, tc.gi);
  const int M = G.M;
  const int kbeg = tc.s * a.k_per_split;
  const int kend = min(a.K, kbeg + a.k_per_split);
  const int nt = kend > kbeg ? (kend - kbeg) / BK : 0;

  // per-thread global sources and LDS slots of its chunks (fixed across k)
  const uint16_t* pa[A_CH];
  int ca[A_CH];
#pragma unroll
  for (int c = 0; c < A_CH; ++c) {
    const int lin = c * 256 + tid;
    const int row = lin >> 2, col = (lin & 3) * 8;
    const int gm = tc.m0 + row;
    ca[c] = row * PITCH + col;
    pa[c] = nullptr;
    if (gm < M) {
      const int src = G.rows ? G.rows[gm] : gm;
      pa[c] = reinterpret_cast<const uint16_t*>(G.A) + (int64_t)src * a.lda + kbeg + col;
    }
  }
  const uint16_t* pb[B_CH];
  int cb[B_CH];
#pragma unroll
  for (int c = 0; c < B_CH; ++c) {
    const int lin = c * 256 + tid;
    const int row = lin >> 2, col = (lin & 3) * 8;
    cb[c] = row * PITCH + col;
    const bool second = DUAL && row >= BN;
    const uint16_t* W = reinterpret_cast<const uint16_t*>(second ? G.W2 : G.W);
    pb[c] = W + (int64_t)(tc.n0 + (second ? row - BN : row)) * a.K + kbeg + col;
  }

  floatx4 acc[TM][TN];
  floatx4 acc2[DUAL ? TM : 1][DUAL ? TN : 1];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      acc[i][j] = floatx4{};
      if constexpr (DUAL) acc2[i][j] = floatx4{};
    }

  u32x4 ra[PF][A_CH], rb[PF][B_CH];
  auto load = [&](int t, u32x4 (&xa)[A_CH], u32x4 (&xb)[B_CH]) {
    const int ko = t * BK;
#pragma unroll
    for (int c = 0; c < A_CH; ++c)
      xa[c] = pa[c] ? *reinterpret_cast<const u32x4*>(pa[c] + ko) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      const u32x4* src = reinterpret_cast<const u32x4*>(pb[c] + ko);
      xb[c] = NT ? __builtin_nontemporal_load(src) : *src;
    }
  };
  auto store = [&](int buf, const u32x4 (&xa)[A_CH], const u32x4 (&xb)[B_CH]) {
#pragma unroll
    for (int c = 0; c < A_CH; ++c) *reinterpret_cast<u32x4*>(&sA[buf][ca[c]]) = xa[c];
#pragma unroll
    for (int c = 0; c < B_CH; ++c) *reinterpret_cast<u32x4*>(&sB[buf][cb[c]]) = xb[c];
  };
  auto compute = [&](int buf) {
    const uint16_t* A = sA[buf];
    const uint16_t* B = sB[buf];
    bf16x8 af[TM], bfr[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
      af[i] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(&A[(wm * WTM + i * 16 + l16) * PITCH + lg * 8]));
#pragma unroll
    for (int j = 0; j < TN; ++j)
      bfr[j] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(&B[(wn * WTN + j * 16 + l16) * PITCH + lg * 8]));
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    if constexpr (DUAL) {
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = __builtin_bit_cast(
            bf16x8,
            *reinterpret_cast<const u32x4*>(&B[(BN + wn * WTN + j * 16 + l16) * PITCH + lg * 8]));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc2[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc2[i][j], 0, 0, 0);
    }
  };

  // prologue: tiles 0..PF-1 in flight (tile t lives in register set t % PF),
  // tile 0 in LDS buffer 0
  static_for<0, PF>([&](auto P) {
    if (P.value < nt) load(P.value, ra[P.value], rb[P.value]);
  });
  if (nt > 0) {
    store(0, ra[0], rb[0]);
    if (PF < nt) load(PF, ra[0], rb[0]);
  }
  __syncthreads();
  for (int i0 = 0; i0 < nt; i0 += PF) {
    static_for<0, PF>([&](auto J) {
      constexpr int nx = (J.value + 1) % PF;
      const int i = i0 + J.value;
      if (i < nt) {
        compute(i & 1);
        if (i + 1 < nt) {
          store((i + 1) & 1, ra[nx], rb[nx]);
          if (i + 1 + PF < nt) load(i + 1 + PF, ra[nx], rb[nx]);
        }
        __syncthreads();
      }
    });
  }

  // epilogue: 16x16 D layout, n = lane%16 (weight row), m = 4*(lane/16) + r
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = tc.n0 + wn * WTN + j * 16 + l16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = tc.m0 + wm * WTM + i * 16 + 4 * lg + r;
        if (m < M) {
          if constexpr (DUAL) {
            const float v = silu(acc[i][j][r]) * acc2[i][j][r];
            reinterpret_cast<uint16_t*>(G.out)[(int64_t)m * G.ldo + n] = f32_to_bf16_bits(v);
          } else {
            reinterpret_cast<float*>(G.out)[tc.s * G.sstride + (int64_t)m * G.ldo + n] =
                acc[i][j][r];
          }
        }
      }
    }
}

// ------------------------------------------------------------------ weight streaming
// gemm_ws_kernel: for M <= 32*MT rows (the pruned-prefill regime).  4 waves per
// block; wave w owns NWT consecutive 32-column tiles (dual: NWT/2 tiles of
// each weight matrix over the same columns).  Each lane streams one weight
// row (n = lane % 32 of a tile) straight into MFMA B registers: per 64-wide
// k-block it loads 64 contiguous bytes (k = 32*(lane/32) .. +32) and feeds
// them to four v_mfma_f32_32x32x16_bf16 steps, so weights never touch LDS.
// The activations (all M rows) are shared through a double-buffered LDS tile
// of 64 k; their k order inside a block is the same permutation as the
// weights' (a consistent permutation of k leaves the dot products unchanged).
// Software pipeline with one barrier per k-block: at iteration kb the block
// multiplies k-block kb, issues the global loads of k-block kb+LEAD for both
// operands together (A into a register ring, W into the MFMA register ring),
// and writes k-block kb+1's activations (loaded LEAD-1 iterations earlier)
// to LDS.  Loads of one k-block are issued in the order they are consumed,
// so the in-order vector-memory counter never makes a wait for near data
// also wait for far data.
template <int MT, int NWT, int LEAD, bool DUAL, bool NT = false>
__global__ void __launch_bounds__(256) gemm_ws_kernel(GemmArgs a) {
  constexpr int KB = 64, PITCH = KB + 8;
  constexpr int BM = 32 * MT;
  constexpr int NCOLW = DUAL ? 32 * NWT / 2 : 32 * NWT;  // output columns per wave
  constexpr int BN = 4 * NCOLW;
  constexpr int A_CH = BM * (KB / 8) / 256;
  static_assert(A_CH * 256 == BM * (KB / 8), "A tile split");
  static_assert(!DUAL || NWT % 2 == 0, "dual needs pairs of tiles");
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * PITCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hi = lane >> 5, lo = lane & 31;
  const TileCoord tc = decode_tile(a, xcd_remap(blockIdx.x, a.total_tiles), BM, BN);
  const GroupView G = group_view(a, tc.gi);
  const int M = G.M;
  const int kbeg = tc.s * a.k_per_split;
  const int kend = min(a.K, kbeg + a.k_per_split);
  const int nkb = kend > kbeg ? (kend - kbeg) / KB : 0;
  const int col0 = tc.n0 + wave * NCOLW;  // first output column of this wave

  // weight row streamed by this lane for each of its tiles
  const uint16_t* pw[NWT];
#pragma unroll
  for (int t = 0; t < NWT; ++t) {
    const bool second = DUAL && t >= NWT / 2;
    const int col = col0 + 32 * (DUAL ? (t % (NWT / 2)) : t) + lo;
    const uint16_t* W = reinterpret_cast<const uint16_t*>(second ? G.W2 : G.W);
    pw[t] = W + (int64_t)col * a.K + kbeg + 32 * hi;
  }
  const uint16_t* pa[A_CH];
  int ca[A_CH];
#pragma unroll
  for (int c = 0; c < A_CH; ++c) {
    const int lin = c * 256 + tid;
    const int row = lin >> 3, col = (lin & 7) * 8;
    ca[c] = row * PITCH + col;
    pa[c] = nullptr;
    if (tc.m0 + row < M) {
      const int gm = tc.m0 + row;
      const int src = G.rows ? G.rows[gm] : gm;
      pa[c] = reinterpret_cast<const uint16_t*>(G.A) + (int64_t)src * a.lda + kbeg + col;
    }
  }

  floatx16 acc[MT][NWT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int t = 0; t < NWT; ++t) acc[i][t] = floatx16{};

  u32x4 wr[LEAD][NWT][4];
  u32x4 ar[LEAD][A_CH];
  auto issue = [&](int kb, u32x4 (&xa)[A_CH], u32x4 (&xw)[NWT][4]) {
#pragma unroll
    for (int c = 0; c < A_CH; ++c)
      xa[c] = pa[c] ? *reinterpret_cast<const u32x4*>(pa[c] + kb * KB) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int t = 0; t < NWT; ++t)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const u32x4* src = reinterpret_cast<const u32x4*>(pw[t] + kb * KB + 8 * q);
        // weights are read once: stream them past L2 so the activations stay resident
        xw[t][q] = NT ? __builtin_nontemporal_load(src) : *src;
      }
  };
  auto store_a = [&](int buf, const u32x4 (&xa)[A_CH]) {
#pragma unroll
    for (int c = 0; c < A_CH; ++c) *reinterpret_cast<u32x4*>(&sA[buf][ca[c]]) = xa[c];
  };
  // One k-block = 4 MFMA steps.  A fragments of step q+1 are read from LDS
  // while the MFMAs of step q issue (one wave per SIMD: nothing else would
  // hide the LDS latency).
  auto compute = [&](int buf, const u32x4 (&w)[NWT][4]) {
    const uint16_t* A = sA[buf];
    bf16x8 af[2][MT];
    auto frags = [&](int q, bf16x8 (&dst)[MT]) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
        dst[i] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&A[(32 * i + lo) * PITCH + 32 * hi + 8 * q]));
    };
    frags(0, af[0]);
    static_for<0, 4>([&](auto Q) {
      constexpr int q = Q.value;
      if constexpr (q + 1 < 4) frags(q + 1, af[(q + 1) & 1]);
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int t = 0; t < NWT; ++t)
          acc[i][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              af[q & 1][i], __builtin_bit_cast(bf16x8, w[t][q]), acc[i][t], 0, 0, 0);
    });
  };

  // prologue: k-blocks 0..LEAD-1 in flight (k-block j in ring slot j % LEAD),
  // k-block 0's activations in LDS buffer 0
  static_for<0, LEAD>([&](auto P) {
    if (P.value < nkb) issue(P.value, ar[P.value], wr[P.value]);
  });
  if (nkb > 0) store_a(0, ar[0]);
  __syncthreads();
  for (int k0 = 0; k0 < nkb; k0 += LEAD) {
    static_for<0, LEAD>([&](auto J) {
      constexpr int slot = J.value;
      constexpr int nxt = (J.value + 1) % LEAD;
      const int kb = k0 + J.value;
      if (kb < nkb) {
        compute(kb & 1, wr[slot]);
        if (kb + LEAD < nkb) issue(kb + LEAD, ar[slot], wr[slot]);
        if (kb + 1 < nkb) store_a((kb + 1) & 1, ar[nxt]);
        __syncthreads();
      }
    });
  }

  // epilogue: D[m][n], n = lane%32 (this lane's weight row), m = 8*(r/4) + 4*hi + r%4
  constexpr int NOUT = DUAL ? NWT / 2 : NWT;
#pragma unroll
  for (int t = 0; t < NOUT; ++t) {
    const int ncol = col0 + 32 * t + lo;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = tc.m0 + 32 * i + 8 * (r >> 2) + 4 * hi + (r & 3);
        if (m < M) {
          if constexpr (DUAL) {
            const float v = silu(acc[i][t][r]) * acc[i][t + NWT / 2][r];
            reinterpret_cast<uint16_t*>(G.out)[(int64_t)m * G.ldo + ncol] = f32_to_bf16_bits(v);
          } else {
            reinterpret_cast<float*>(G.out)[tc.s * G.sstride + (int64_t)m * G.ldo + ncol] =
                acc[i][t][r];
          }
        }
      }
  }
}

// ------------------------------------------------------------------ fp32
template <bool DUAL>
__global__ void __launch_bounds__(256) gemm_f32_kernel(GemmArgs a) {
  constexpr int T = 16;
  __shared__ float sA[T][T + 1];
  __shared__ float sB[T][T + 1];
  __shared__ float sB2[DUAL ? T : 1][T + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const TileCoord tc = decode_tile(a, blockIdx.x, T, T);
  const GroupView G = group_view(a, tc.gi);
  const int kbeg = tc.s * a.k_per_split;
  const int kend = min(a.K, kbeg + a.k_per_split);
  const int m = tc.m0 + ty, n = tc.n0 + tx;
  const float* A = reinterpret_cast<const float*>(G.A);
  const float* W = reinterpret_cast<const float*>(G.W);
  const float* W2 = reinterpret_cast<const float*>(G.W2);
  // A tile row loaded by this thread: row tc.m0 + ty, column k0 + tx
  const int am = tc.m0 + ty;
  const float* arow = nullptr;
  if (am < G.M) arow = A + (int64_t)(G.rows ? G.rows[am] : am) * a.lda;
  const int bn = tc.n0 + ty;
  float acc = 0.f, acc2 = 0.f;
  for (int k0 = kbeg; k0 < kend; k0 += T) {
    const int k = k0 + tx;
    sA[ty][tx] = (arow && k < kend) ? arow[k] : 0.f;
    sB[ty][tx] = (bn < G.N && k < kend) ? W[(int64_t)bn * a.K + k] : 0.f;
    if constexpr (DUAL) sB2[ty][tx] = (bn < G.N && k < kend) ? W2[(int64_t)bn * a.K + k] : 0.f;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < T; ++kk) {
      acc = fmaf(sA[ty][kk], sB[tx][kk], acc);
      if constexpr (DUAL) acc2 = fmaf(sA[ty][kk], sB2[tx][kk], acc2);
    }
    __syncthreads();
  }
  if (m < G.M && n < G.N) {
    if constexpr (DUAL) {
      reinterpret_cast<float*>(G.out)[(int64_t)m * G.ldo + n] = silu(acc) * acc2;
    } else {
      reinterpret_cast<float*>(G.out)[tc.s * G.sstride + (int64_t)m * G.ldo + n] = acc;
    }
  }
}

struct TileCfg {
  int BM, BN;
  bool ws;  // weight-streaming kernel
};

// Tile shape.  Up to 256 rows one M-tile covers every row so each weight
// element is read from HBM once.  Non-dual skinny GEMMs use the
// weight-streaming kernel (4 waves x 32 columns, BM = rows rounded up to 64,
// at most 192); the dual SwiGLU GEMM and everything with more rows use the
// LDS-staged kernel.
TileCfg pick_bf16_tile(int maxM, bool dual) {
  if (maxM <= 192 && !dual) {
    const int bm = std::max(64, (maxM + 63) / 64 * 64);
    return TileCfg{bm, 128, true};
  }
  if (maxM <= 256) {
    const int bm = std::max(64, (maxM + 63) / 64 * 64);
    return dual ? TileCfg{bm, 32, false} : TileCfg{bm, 64, false};
  }
  return dual ? TileCfg{128, 64, false} : TileCfg{128, 128, false};
}

constexpr int kTargetBlocks = 256;

int choose_split(int tiles, int K, int split_max, int kgran) {
  int split = 1;
  while (split < split_max && tiles * split < kTargetBlocks && K / (kgran * split * 2) >= 4) split *= 2;
  return split;
}

void fill_tiles(GemmArgs& a, int BM, int BN) {
  int t = 0;
  for (int i = 0; i < a.ngroups; ++i) {
    GemmGroup& g = a.g[i];
    g.tiles_m = ceil_div(g.M, BM);
    g.tiles_n = g.N / BN;
    g.tile_begin = t;
    t += g.tiles_m * g.tiles_n * a.split;
  }
  a.total_tiles = t;
}

int tiles_for(const GemmArgs& a, int BM, int BN) {
  int t = 0;
  for (int i = 0; i < a.ngroups; ++i) t += ceil_div(a.g[i].M, BM) * (a.g[i].N / BN);
  return t;
}

template <int BM, int BN, int WGM, int WGN, bool DUAL>
void launch_cfg(const GemmArgs& a, hipStream_t st) {
  gemm_bf16_kernel<BM, BN, WGM, WGN, 4, DUAL><<<a.total_tiles, 256, 0, st>>>(a);
}

template <int MT>
void launch_ws(const GemmArgs& a, hipStream_t st) {
  gemm_ws_kernel<MT, 1, 3, false><<<a.total_tiles, 256, 0, st>>>(a);
}

}  // namespace

int gemm_split_for(int M, int N, int K, bool dual, bool bf16, int split_max) {
  if (dual || !bf16) return 1;
  TileCfg tc = pick_bf16_tile(M, false);
  return choose_split(ceil_div(M, tc.BM) * (N / tc.BN), K, split_max, tc.ws ? 64 : 32);
}

hipError_t launch_gemm_bf16(GemmArgs& a, int split_max, hipStream_t st) {
  int maxM = 0;
  for (int i = 0; i < a.ngroups; ++i) maxM = std::max(maxM, a.g[i].M);
  const bool dual = a.epilogue == EPI_SWIGLU;
  TileCfg tc = pick_bf16_tile(maxM, dual);
  for (int i = 0; i < a.ngroups; ++i)
    if (a.g[i].N % tc.BN) {
      if (tc.ws) tc = TileCfg{std::max(64, (maxM + 63) / 64 * 64), 64, false};
      if (a.g[i].N % tc.BN) return hipErrorInvalidValue;
    }
  const int kgran = tc.ws ? 64 : 32;
  if (a.K % kgran) return hipErrorInvalidValue;
  a.split = dual ? 1 : choose_split(tiles_for(a, tc.BM, tc.BN), a.K, split_max, kgran);
  a.k_per_split = ceil_div(ceil_div(a.K, kgran), a.split) * kgran;
  fill_tiles(a, tc.BM, tc.BN);
  if (a.total_tiles == 0) return hipSuccess;
  if (tc.ws) {
    switch (tc.BM) {
      case 64: launch_ws<2>(a, st); break;
      case 128: launch_ws<4>(a, st); break;
      default: launch_ws<6>(a, st); break;
    }
  } else if (dual) {
    switch (tc.BM * 1000 + tc.BN) {
      case 64032: launch_cfg<64, 32, 4, 1, true>(a, st); break;
      case 128032: launch_cfg<128, 32, 4, 1, true>(a, st); break;
      case 192032: launch_cfg<192, 32, 4, 1, true>(a, st); break;
      case 256032: launch_cfg<256, 32, 4, 1, true>(a, st); break;
      default: launch_cfg<128, 64, 2, 2, true>(a, st); break;
    }
  } else {
    switch (tc.BM * 1000 + tc.BN) {
      case 64064: launch_cfg<64, 64, 2, 2, false>(a, st); break;
      case 128064: launch_cfg<128, 64, 2, 2, false>(a, st); break;
      case 192064: launch_cfg<192, 64, 2, 2, false>(a, st); break;
      case 256064: launch_cfg<256, 64, 2, 2, false>(a, st); break;
      default: launch_cfg<128, 128, 2, 2, false>(a, st); break;
    }
  }
  return hipGetLastError();
}

hipError_t launch_gemm_f32(GemmArgs& a, int split_max, hipStream_t st) {
  (void)split_max;
  a.split = 1;
  a.k_per_split = a.K;
  int t = 0;
  for (int i = 0; i < a.ngroups; ++i) {
    GemmGroup& g = a.g[i];
    g.tiles_m = ceil_div(g.M, 16);
    g.tiles_n = ceil_div(g.N, 16);
    g.tile_begin = t;
    t += g.tiles_m * g.tiles_n;
  }
  a.total_tiles = t;
  if (t == 0) return hipSuccess;
  if (a.epilogue == EPI_SWIGLU) gemm_f32_kernel<true><<<t, 256, 0, st>>>(a);
  else gemm_f32_kernel<false><<<t, 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace spider
