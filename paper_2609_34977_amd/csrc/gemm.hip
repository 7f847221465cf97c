// Decoder GEMMs: out = A[rows] x W^T with W in nn.Linear layout [N, K].
//
// bf16 path (gemm_bf16_kernel): 256 threads = 4 waves in a 2x2 grid, block
// tile BM x BN x 64, each wave a (BM/2) x (BN/2) tile of 32x32 MFMA blocks
// (v_mfma_f32_32x32x16_bf16, fp32 accumulation).  A and W k-slices go
// global -> registers (16-byte loads; A rows optionally gathered through a
// row list) -> LDS (row pitch 72 bf16 to spread banks), with the next slice's
// global loads in flight while the current one is multiplied.  Grouped
// launch: up to three problems sharing K (e.g. Q over the query rows, K and
// V over all rows) in one grid.  Logical tiles are ordered
// (group, n-tile, k-split, m-tile) so that the m-tiles sharing a weight tile
// are consecutive, and the hardware block id is remapped so that consecutive
// logical tiles run on the same XCD (blocks are dispatched round-robin over
// the 8 XCDs) and share its L2.
// Epilogues: fp32 split-K partials (summed by the consumer kernel, in fixed
// order, so the result is deterministic without atomics), or the fused
// SwiGLU silu(A Wg^T) * (A Wu^T) rounded to bf16 (dual weights).
//
// fp32 path (gemm_f32_kernel): 16x16 FMA tiles through LDS with the same
// group/gather/split/epilogue semantics (used by fp32 workloads).
#include <algorithm>

#include "kernels.h"

namespace spider {
namespace {

constexpr int kNumXcd = 8;

__device__ inline int xcd_remap(int b, int total) {
  const int q = total / kNumXcd, r = total % kNumXcd;
  const int xcd = b % kNumXcd, idx = b / kNumXcd;
  return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

struct TileCoord {
  int gi, m0, n0, s;
};

__device__ inline TileCoord decode_tile(const GemmArgs& a, int t, int BM, int BN) {
  int gi = 0;
  if (a.ngroups > 1 && t >= a.g[1].tile_begin) gi = 1;
  if (a.ngroups > 2 && t >= a.g[2].tile_begin) gi = 2;
  int local = t - a.g[gi].tile_begin;
  const int tm = a.g[gi].tiles_m;
  const int m_tile = local % tm;
  local /= tm;
  const int s = local % a.split;
  const int n_tile = local / a.split;
  return {gi, m_tile * BM, n_tile * BN, s};
}

__device__ inline float silu(float g) { return g / (1.0f + __expf(-g)); }

template <int BM, int BN, bool DUAL>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(GemmArgs a) {
  constexpr int BK = 64, PITCH = BK + 8;
  constexpr int BROWS = DUAL ? 2 * BN : BN;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int A_CH = BM * (BK / 8) / 256;
  constexpr int B_CH = BROWS * (BK / 8) / 256;
  static_assert(A_CH >= 1 && B_CH >= 1, "tile too small");
  __shared__ __attribute__((aligned(16))) uint16_t sA[BM * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sB[BROWS * PITCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hi = lane >> 5, lo = lane & 31;
  const int wm = wave >> 1, wn = wave & 1;
  const TileCoord tc = decode_tile(a, xcd_remap(blockIdx.x, a.total_tiles), BM, BN);
  const GemmGroup& G = a.g[tc.gi];
  const int M = G.M;
  const int kbeg = tc.s * a.k_per_split;
  const int kend = min(a.K, kbeg + a.k_per_split);

  // per-thread source pointers of its A and B chunks (row fixed across k)
  const uint16_t* pa[A_CH];
  int ca[A_CH];
#pragma unroll
  for (int c = 0; c < A_CH; ++c) {
    const int lin = c * 256 + tid;
    const int row = lin >> 3, col = (lin & 7) * 8;
    const int gm = tc.m0 + row;
    ca[c] = row * PITCH + col;
    if (gm < M) {
      const int src = G.a_rows ? G.a_rows[gm] : gm;
      pa[c] = reinterpret_cast<const uint16_t*>(G.A) + (int64_t)src * a.lda + col;
    } else {
      pa[c] = nullptr;
    }
  }
  const uint16_t* pb[B_CH];
  int cb[B_CH];
#pragma unroll
  for (int c = 0; c < B_CH; ++c) {
    const int lin = c * 256 + tid;
    const int row = lin >> 3, col = (lin & 7) * 8;
    cb[c] = row * PITCH + col;
    const uint16_t* W = reinterpret_cast<const uint16_t*>((DUAL && row >= BN) ? G.W2 : G.W);
    const int wr = tc.n0 + ((DUAL && row >= BN) ? row - BN : row);
    pb[c] = W + (int64_t)wr * a.K + col;
  }

  floatx16 acc[TM][TN];
  floatx16 acc2[DUAL ? TM : 1][DUAL ? TN : 1];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      acc[i][j] = floatx16{};
      if constexpr (DUAL) acc2[i][j] = floatx16{};
    }

  uint4 ra[A_CH], rb[B_CH];
  auto load = [&](int k0) {
#pragma unroll
    for (int c = 0; c < A_CH; ++c)
      ra[c] = pa[c] ? *reinterpret_cast<const uint4*>(pa[c] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int c = 0; c < B_CH; ++c) rb[c] = *reinterpret_cast<const uint4*>(pb[c] + k0);
  };
  if (kbeg < kend) load(kbeg);
  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    __syncthreads();
#pragma unroll
    for (int c = 0; c < A_CH; ++c) *reinterpret_cast<uint4*>(&sA[ca[c]]) = ra[c];
#pragma unroll
    for (int c = 0; c < B_CH; ++c) *reinterpret_cast<uint4*>(&sB[cb[c]]) = rb[c];
    __syncthreads();
    if (k0 + BK < kend) load(k0 + BK);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int kc = kk * 16 + hi * 8;
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const uint4*>(&sA[(wm * WM + i * 32 + lo) * PITCH + kc]));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const uint4*>(&sB[(wn * WN + j * 32 + lo) * PITCH + kc]));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      if constexpr (DUAL) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[j] = __builtin_bit_cast(
              bf16x8,
              *reinterpret_cast<const uint4*>(&sB[(BN + wn * WN + j * 32 + lo) * PITCH + kc]));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc2[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc2[i][j], 0, 0, 0);
      }
    }
  }

  // epilogue: D[m][n] with n = lane%32 (weight row), m = 8*(r/4) + 4*hi + r%4
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = tc.n0 + wn * WN + j * 32 + lo;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = tc.m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
        if (m < M) {
          if constexpr (DUAL) {
            const float v = silu(acc[i][j][r]) * acc2[i][j][r];
            reinterpret_cast<uint16_t*>(G.out)[(int64_t)m * G.ldo + n] = f32_to_bf16_bits(v);
          } else {
            reinterpret_cast<float*>(G.out)[tc.s * G.split_stride + (int64_t)m * G.ldo + n] =
                acc[i][j][r];
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
  const GemmGroup& G = a.g[tc.gi];
  const int kbeg = tc.s * a.k_per_split;
  const int kend = min(a.K, kbeg + a.k_per_split);
  const int m = tc.m0 + ty, n = tc.n0 + tx;
  const float* A = reinterpret_cast<const float*>(G.A);
  const float* W = reinterpret_cast<const float*>(G.W);
  const float* W2 = reinterpret_cast<const float*>(G.W2);
  // A tile row loaded by this thread: row tc.m0 + ty, column k0 + tx
  const int am = tc.m0 + ty;
  const float* arow = nullptr;
  if (am < G.M) arow = A + (int64_t)(G.a_rows ? G.a_rows[am] : am) * a.lda;
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
      reinterpret_cast<float*>(G.out)[tc.s * G.split_stride + (int64_t)m * G.ldo + n] = acc;
    }
  }
}

struct TileCfg {
  int BM, BN;
};

TileCfg pick_bf16_tile(int maxM, bool dual) {
  if (maxM >= 512) return dual ? TileCfg{128, 64} : TileCfg{128, 128};
  return TileCfg{64, 64};
}

int choose_split(int tiles, int K, int split_max) {
  int split = 1;
  while (split < split_max && tiles * split < 512 && K / (64 * split * 2) >= 4) split *= 2;
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

}  // namespace

int gemm_split_for(int M, int N, int K, bool dual, bool bf16, int split_max) {
  if (dual) return 1;
  if (!bf16) return 1;
  TileCfg tc = pick_bf16_tile(M, false);
  return choose_split(ceil_div(M, tc.BM) * (N / tc.BN), K, split_max);
}

hipError_t launch_gemm_bf16(GemmArgs& a, int split_max, hipStream_t st) {
  int maxM = 0;
  for (int i = 0; i < a.ngroups; ++i) maxM = std::max(maxM, a.g[i].M);
  const bool dual = a.epilogue == EPI_SWIGLU;
  TileCfg tc = pick_bf16_tile(maxM, dual);
  // every group's N must be a multiple of BN
  for (int i = 0; i < a.ngroups; ++i)
    if (a.g[i].N % tc.BN) tc = TileCfg{tc.BM, 64};
  a.split = dual ? 1 : choose_split(tiles_for(a, tc.BM, tc.BN), a.K, split_max);
  a.k_per_split = ceil_div(ceil_div(a.K, 64), a.split) * 64;
  fill_tiles(a, tc.BM, tc.BN);
  if (a.total_tiles == 0) return hipSuccess;
  dim3 grid(a.total_tiles), block(256);
  if (dual) {
    if (tc.BM == 128) gemm_bf16_kernel<128, 64, true><<<grid, block, 0, st>>>(a);
    else gemm_bf16_kernel<64, 64, true><<<grid, block, 0, st>>>(a);
  } else {
    if (tc.BM == 128 && tc.BN == 128) gemm_bf16_kernel<128, 128, false><<<grid, block, 0, st>>>(a);
    else if (tc.BM == 128) gemm_bf16_kernel<128, 64, false><<<grid, block, 0, st>>>(a);
    else gemm_bf16_kernel<64, 64, false><<<grid, block, 0, st>>>(a);
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
