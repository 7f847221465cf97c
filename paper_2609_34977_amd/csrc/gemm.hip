// Decoder GEMMs: out = A[rows] x W^T with W in nn.Linear layout [N, K].
//
// Up to 4 rows (decoding) gemv_kernel streams the weights against the few
// activation rows.  Up to 256 rows (the pruned-prefill regime: a few hundred
// rows against multi-MB weight matrices) gemm_stream_kernel streams every
// weight element from HBM once through an LDS ring into the MFMAs.  More rows
// use gemm_tile_kernel (256-column tiles of 128-256 rows).  Shapes neither of
// the last two takes (N not a multiple of their column tiles, unaligned
// outputs) use gemm_bf16_kernel: 256 threads = 4 waves, block tile BM x BN x
// 32 with v_mfma_f32_16x16x32_bf16 (fp32 accumulation), a wave owning a
// (BM/WGM) x (BN/WGN) sub-tile; a ring of PF register stages of 16-byte
// global loads in flight, double-buffered LDS (row pitch 40 bf16: the
// 16 rows x 16 bytes of a fragment read hit distinct banks), one barrier per
// k-tile.  The kernels may gather A rows through a row list and take a
// grouped launch: up to three problems sharing K (Q over the query rows, K and
// V over all rows) in one grid.  Logical tiles are ordered (group, n-tile,
// k-split, m-tile) and the hardware block id is remapped so consecutive
// logical tiles run on the same XCD (blocks are dispatched round-robin over
// the 8 XCDs) and share its L2.  Epilogues: fp32 split-K partials (summed by
// the consumer kernel in fixed order: deterministic without atomics), or the
// fused SwiGLU silu(A Wg^T) * (A Wu^T) rounded to bf16 (dual weights, no split).
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

// silu(g) = g / (1 + e^-g) with the hardware reciprocal (1 ulp): the result is
// rounded to bf16 or summed in fp32 afterwards, far coarser than that.
__device__ inline float silu(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

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
  const int32_t* md = sel3(gi, a.g[0].m_dev, a.g[1].m_dev, a.g[2].m_dev);
  if (md) v.M = min(v.M, *md);
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
  if (tc.m0 >= M) return;  // a device row count below the launch's bound
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
// gemm_stream_kernel: up to 32*MT (<= 256) rows, the pruned-prefill regime.
// 4 waves per block, one per SIMD, each owning 32 weight rows: non-dual, the
// block covers 128 output columns; dual (SwiGLU), waves 0-1 take gate rows and
// waves 2-3 up rows of the same 64 output columns, the up sums are handed over
// through LDS and the epilogue writes bf16 silu(g) * u.
//
// Both operands go global -> LDS with global_load_lds (no register round
// trip) into a ring of LEAD+1 stages; a stage holds BM activation rows and the
// block's 128 weight rows, 64 k each.  Every row is 128 B = eight 16-B chunks;
// chunk c of row r sits in slot c ^ (r & 7), so the DMA writes (1 KB per
// instruction, 8 rows of 8 lanes: a whole cache line per 8 lanes) and the MFMA
// fragment reads (32 rows, one chunk) are both free of bank conflicts.  Each
// k-block is four v_mfma_f32_32x32x16_bf16 steps; step q takes chunk
// 4*(lane/32) + q on both operands (a consistent permutation of k leaves every
// dot product unchanged).
//
// Pipeline: at iteration kb the block multiplies k-block kb, issues the DMA of
// k-block kb+LEAD, waits until k-block kb+1 has landed and passes one barrier.
// Every iteration issues the same loads (the tail re-reads the last k-block
// into a slot never consumed), so the wait is an exact count of outstanding
// loads; ring slots are compile-time (k-block kb lives in slot kb % (LEAD+1)).
// Rows past M read row M-1 (their outputs are never stored).
//
// Why this shape: at a few hundred rows the activation tile is 1.5x the
// weight bytes of a block per k-block, and both streams compete for the
// per-CU limit on outstanding L1 requests; whole-line weight requests (8
// lanes per 128-B line) need a quarter of the L1 accesses of lane-per-row
// register loads, and one block per column tile with the full row range reads
// every weight once.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Softmax statistics of one row piece: max, sum e^(z-max), sum e^(z-max) (z-max).
struct SoftStat {
  float m, s, t;
};

// Merge of two pieces (b.m and a.m finite): rescale both to the larger max.
__device__ __forceinline__ SoftStat soft_merge(SoftStat a, SoftStat b) {
  const float m = fmaxf(a.m, b.m);
  const float da = a.m - m, db = b.m - m;
  const float ea = expf(da), eb = expf(db);
  return {m, ea * a.s + eb * b.s, ea * fmaf(a.s, da, a.t) + eb * fmaf(b.s, db, b.t)};
}

// Tile layout shared by the GEMM kernels: 16-byte chunk c of a 128-byte tile
// row r is stored in slot c ^ ((r >> 1) & 7).  An LDS pass of a 16-byte read
// serves 16 lanes; a fragment read has those lanes on 16 consecutive rows, so
// even and odd rows each cover the 8 slots and the 16 lanes hit 16 distinct
// bank groups (with c ^ (r & 7), rows r and r + 8 collide).
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

template <int MT, int LEAD, bool DUAL, bool LENS = false>
__global__ void __launch_bounds__(256) gemm_stream_kernel(GemmArgs a) {
  constexpr int KB = 64;
  // weights are read once: the SwiGLU and lens launches (split 1, whole K per
  // block) load them non-temporal (measured 2-6 % faster there, no gain with split-K)
  constexpr bool kWeightNT = DUAL || LENS;
  constexpr int BM = 32 * MT;
  constexpr int BN = DUAL ? 64 : 128;  // output columns per block
  constexpr int STAGES = LEAD + 1;
  constexpr int A_BYTES = BM * 128;
  constexpr int STAGE_BYTES = A_BYTES + 128 * 128;  // activations, then the 128 weight rows
  constexpr int PER_IT = 4 + MT;  // DMA instructions per wave per k-block: 4 weight, MT activation
  // epilogue staging reuses the ring: dual hand-over + bf16 tile, or the fp32 tile (pitch 132)
  constexpr int EPI_BYTES = DUAL ? 4 * (MT / 2) * 64 * 16 * 4 + BM * 72 * 2 : BM * 132 * 4;
  constexpr int RING_BYTES = STAGES * STAGE_BYTES > EPI_BYTES ? STAGES * STAGE_BYTES : EPI_BYTES;
  static_assert(RING_BYTES <= 160 * 1024, "LDS of one CU");
  __shared__ __attribute__((aligned(1024))) uint8_t ring[RING_BYTES];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hi = lane >> 5, lo = lane & 31;
  constexpr int MH = MT / 2;
  static_assert(MT % 2 == 0, "row tiles split over two waves");
  const int mh = wave >> 1, nh = wave & 1;
  // row of accumulator register r of row tile i, in the block (MMA D layout:
  // column = lane % 32, row = 8 (r / 4) + 4 (lane / 32) + r % 4)
  auto acc_row = [&](int i, int r) { return 32 * (MH * mh + i) + 8 * (r >> 2) + 4 * hi + (r & 3); };
  const TileCoord tc = decode_tile(a, xcd_remap(blockIdx.x, a.total_tiles), BM, BN);
  const GroupView G = group_view(a, tc.gi);
  const int M = G.M;
  if (tc.m0 >= M) return;  // a device row count below the launch's bound
  const int kbeg = tc.s * a.k_per_split;
  const int kend = min(a.K, kbeg + a.k_per_split);
  const int nkb = kend > kbeg ? (kend - kbeg) / KB : 0;
  const int wrow0 = tc.n0 + 32 * (DUAL ? (wave & 1) : wave);  // first weight row of this wave
  const uint16_t* W = reinterpret_cast<const uint16_t*>(DUAL && wave >= 2 ? G.W2 : G.W);
  // weight DMA: instruction q fills the wave's rows 8q..8q+7; lane l takes row
  // 8q + l/8, slot l%8
  const uint16_t* pw[4];
#pragma unroll
  for (int q = 0; q < 4; ++q)  // LDS weight row 32 wave + 8q + l/8
    pw[q] = W + (int64_t)(wrow0 + 8 * q + (lane >> 3)) * a.K + kbeg + 8 * ((lane & 7) ^ swz(8 * q + (lane >> 3)));

  // activation DMA: instruction j of this wave fills tile rows 8g..8g+7,
  // g = wave*MT + j; lane l takes row 8g + l/8, slot l%8
  const uint16_t* pa[MT];
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    const int g = wave * MT + j;
    const int r = min(tc.m0 + 8 * g + (lane >> 3), M - 1);
    const int src = G.rows ? G.rows[r] : r;
    const int c = (lane & 7) ^ swz(8 * g + (lane >> 3));
    pa[j] = reinterpret_cast<const uint16_t*>(G.A) + (int64_t)src * a.lda + kbeg + 8 * c;
  }

  floatx16 acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = floatx16{};

  const uint32_t ring_lds = lds_offset(ring);
  auto issue = [&](int kb, auto S) {
    constexpr int st = decltype(S)::value;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      dma16<kWeightNT>(pw[q] + kb * KB, ring_lds + st * STAGE_BYTES + A_BYTES + (wave * 4 + q) * 1024);
#pragma unroll
    for (int j = 0; j < MT; ++j) dma16(pa[j] + kb * KB, ring_lds + st * STAGE_BYTES + (wave * MT + j) * 1024);
  };
  // Wave tile (2 x 2 over the block): rows [32 MH mh, 32 MH (mh + 1)) against LDS
  // weight rows [64 nh, 64 nh + 64) -- output columns n0 + 64 nh.. (dual: nh 0
  // the gate rows, 1 the up rows of the block's 64 columns).  Accumulator
  // 2 i + t holds row tile i and column tile t.  Per k-step a wave reads MH + 2
  // fragments from LDS for 2 MH MMAs.
  auto compute = [&](auto S) {
    constexpr int st = decltype(S)::value;
    const uint8_t* tile = ring + st * STAGE_BYTES;
    const uint8_t* wt = tile + A_BYTES + (64 * nh + lo) * 128;
    const uint8_t* at = tile + (32 * MH * mh + lo) * 128;
    bf16x8 wf[2][2], af[2][MH];
    auto frags = [&](int q, bf16x8 (&w)[2], bf16x8 (&x)[MH]) {
      const int c = 16 * ((4 * hi + q) ^ swz(lo));
#pragma unroll
      for (int t = 0; t < 2; ++t)
        w[t] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wt + t * 32 * 128 + c));
#pragma unroll
      for (int i = 0; i < MH; ++i)
        x[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(at + i * 32 * 128 + c));
    };
    frags(0, wf[0], af[0]);
    static_for<0, 4>([&](auto Q) {
      constexpr int q = Q.value;
      if constexpr (q + 1 < 4) frags(q + 1, wf[(q + 1) & 1], af[(q + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < MH; ++i)
#pragma unroll
        for (int t = 0; t < 2; ++t)
          acc[2 * i + t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[q & 1][i], wf[q & 1][t], acc[2 * i + t], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  if (nkb > 0) {
    static_for<0, LEAD>([&](auto P) { issue(min((int)P.value, nkb - 1), P); });
    dma_wait_barrier<(LEAD - 1) * PER_IT>();
    // k-block kb+LEAD goes to the slot that iteration kb-1 consumed (free since
    // its barrier), before the MMAs of kb, so the loads overlap them; every
    // iteration issues the same DMAs (the last k-block again at the end), so
    // the count of DMAs still in flight is exact
    auto body = [&](int kb, auto J) {
      constexpr int j = decltype(J)::value;
      issue(min(kb + LEAD, nkb - 1), std::integral_constant<int, (j + LEAD) % STAGES>{});
      compute(J);
      dma_wait_barrier<(LEAD - 1) * PER_IT>();
    };
    int k0 = 0;
    for (; k0 + STAGES <= nkb; k0 += STAGES)
      static_for<0, STAGES>([&](auto J) { body(k0 + J.value, J); });
    const int rem = nkb - k0;
    static_for<0, STAGES>([&](auto J) {
      if (J.value < rem) body(k0 + J.value, J);
    });
    dma_wait_all();
  }

  // D layout of 32x32 MFMA: n = lane % 32, m = 8*(r/4) + 4*(lane/32) + r%4
  if constexpr (DUAL) {
    // Waves (mh, 0) hold the gate sums of rows half mh, waves (mh, 1) the up sums
    // of the same rows and columns.  Each pair splits the work by column tile:
    // the gate wave finishes tile t = 0, the up wave t = 1, after trading the
    // other tile through LDS.  The bf16 results are staged as a BM x 64
    // row-major tile (pitch 72) and written with 16-byte stores, a whole
    // 128-byte line per row.
    constexpr int OPITCH = 72;
    constexpr int XFER_BYTES = 4 * MH * 64 * 16 * 4;
    static_assert(XFER_BYTES + BM * OPITCH * 2 <= RING_BYTES, "dual epilogue fits");
    __syncthreads();  // ring free
    float* xfer = reinterpret_cast<float*>(ring);
    uint16_t* ot = reinterpret_cast<uint16_t*>(ring + XFER_BYTES);
    // (dir, i): dir 0 carries up tile (i, 0) to the gate wave, dir 1 gate tile (i, 1) to the up wave
    auto slot = [&](int dir, int i) { return xfer + (((mh * 2 + dir) * MH + i) * 64 + lane) * 16; };
    auto put = [&](float* dst, const floatx16& v) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<floatx4*>(dst + 4 * q) = floatx4{v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
    };
    if (nh == 0) {
#pragma unroll
      for (int i = 0; i < MH; ++i) put(slot(1, i), acc[2 * i + 1]);
    } else {
#pragma unroll
      for (int i = 0; i < MH; ++i) put(slot(0, i), acc[2 * i]);
    }
    __syncthreads();
    if (nh == 0) {
#pragma unroll
      for (int i = 0; i < MH; ++i) {
        const float* up = slot(0, i);
#pragma unroll
        for (int r = 0; r < 16; ++r)
          ot[acc_row(i, r) * OPITCH + lo] = f32_to_bf16_bits(silu(acc[2 * i][r]) * up[r]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < MH; ++i) {
        const float* gp = slot(1, i);
#pragma unroll
        for (int r = 0; r < 16; ++r)
          ot[acc_row(i, r) * OPITCH + 32 + lo] = f32_to_bf16_bits(silu(gp[r]) * acc[2 * i + 1][r]);
      }
    }
    __syncthreads();
    const int rows = min(BM, M - tc.m0);
    uint16_t* op = reinterpret_cast<uint16_t*>(G.out) + (int64_t)tc.m0 * G.ldo + tc.n0;
    for (int c = tid; c < rows * 8; c += 256) {
      const int row = c >> 3, ch = c & 7;
      *reinterpret_cast<u32x4*>(op + (int64_t)row * G.ldo + 8 * ch) =
          *reinterpret_cast<const u32x4*>(ot + row * OPITCH + 8 * ch);
    }
  } else if constexpr (LENS) {
    // the block's BM x 128 logits go through LDS (row pitch 132 floats); each
    // row is reduced by 256/BM threads (64 rows: 4, 128: 2, 192/256: 1) over
    // consecutive column ranges, merged across those threads in fixed order
    constexpr int PITCH = 132;
    constexpr int TPR = BM <= 64 ? 4 : (BM <= 128 ? 2 : 1);
    constexpr int CPT = 128 / TPR;
    static_assert(BM * PITCH * 4 <= RING_BYTES, "lens tile fits the ring");
    __syncthreads();
    float* sm = reinterpret_cast<float*>(ring);
#pragma unroll
    for (int i = 0; i < MH; ++i)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) sm[acc_row(i, r) * PITCH + 64 * nh + 32 * t + lo] = acc[2 * i + t][r];
    __syncthreads();
    const int row = tid / TPR, part = tid % TPR;
    SoftStat st{-INFINITY, 0.f, 0.f};
    if (row < BM) {
      const float* z = sm + row * PITCH + part * CPT;
      float mx = -INFINITY;
#pragma unroll
      for (int c = 0; c < CPT; c += 4) {
        const floatx4 v = *reinterpret_cast<const floatx4*>(z + c);
        mx = fmaxf(mx, fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
      }
      float se = 0.f, te = 0.f;
#pragma unroll
      for (int c = 0; c < CPT; c += 4) {
        const floatx4 v = *reinterpret_cast<const floatx4*>(z + c);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float u = v[e] - mx;
          const float x = expf(u);
          se += x;
          te = fmaf(x, u, te);
        }
      }
      st = {mx, se, te};
    }
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) {
      const SoftStat other{__shfl_xor(st.m, o, 64), __shfl_xor(st.s, o, 64), __shfl_xor(st.t, o, 64)};
      st = (part & o) ? soft_merge(other, st) : soft_merge(st, other);
    }
    const int m = tc.m0 + row;
    if (row < BM && part == 0 && m < M)
      *reinterpret_cast<floatx4*>(reinterpret_cast<float*>(G.out) +
                                  ((int64_t)m * G.ldo + tc.n0 / 128) * 4) = floatx4{st.m, st.s, st.t, 0.f};
  } else {
    // fp32 partial sums go through LDS (row pitch 132 floats) so that every
    // thread stores 16-byte pieces: 32 threads cover a 512-byte row segment
    constexpr int PITCH = 132;
    static_assert(BM * PITCH * 4 <= RING_BYTES, "partial tile fits the ring");
    __syncthreads();
    float* sm = reinterpret_cast<float*>(ring);
#pragma unroll
    for (int i = 0; i < MH; ++i)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) sm[acc_row(i, r) * PITCH + 64 * nh + 32 * t + lo] = acc[2 * i + t][r];
    __syncthreads();
    const int rows = min(BM, M - tc.m0);
    float* op = reinterpret_cast<float*>(G.out) + tc.s * G.sstride + (int64_t)tc.m0 * G.ldo + tc.n0;
    for (int c = tid; c < rows * 32; c += 256) {
      const int row = c >> 5, ch = c & 31;
      *reinterpret_cast<floatx4*>(op + (int64_t)row * G.ldo + 4 * ch) =
          *reinterpret_cast<const floatx4*>(sm + row * PITCH + 4 * ch);
    }
  }
}

// ------------------------------------------------------------------ large row counts
// gemm_tile_kernel: the compute-bound regime (more than 256 rows).  A block
// computes BM = 64*MH rows against 256 weight rows (non-dual: 256 output
// columns; dual: the gate and up rows of 128 output columns) over its k range,
// in k-blocks of 64.  4 waves in 2 x 2, wave (mh, nh) owning rows
// [32 MH mh, 32 MH (mh + 1)) and 128 weight rows: non-dual LDS weight rows
// [128 nh, 128 nh + 128); dual output columns [64 nh, 64 nh + 64), i.e. gate
// rows [64 nh, +64) and up rows [128 + 64 nh, +64) of the stage, so every wave
// holds the gate and up sums of the same outputs and the SwiGLU epilogue needs
// no exchange.  Per k-step a wave reads MH + 4 fragments from LDS for 4 MH
// v_mfma_f32_32x32x16_bf16 (acc[i][t]: row tile i, weight tile t).
//
// Operands go global -> LDS by global_load_lds into two stages (BM + 256 rows
// of 128 B each); chunk c of row r sits in slot c ^ (r & 7) as in the
// streaming kernel.  The DMA of k-block kb+1 is interleaved with the first
// half of the MMAs of kb, then the wave waits for all its loads and the block
// passes one barrier.  What bounds it: operand bytes from L2 (a block tile of
// 256 x 256 needs 32 B per clock per CU at the MFMA rate; L2 hits measured
// ~20 B per clock per CU), hence the large tile and the L2-friendly order.
// Row tiles entirely past M skip their MMAs; their rows read row M-1.
//
// Tile order: per group, split-major, then GM = 8 row tiles x all column
// tiles in column-major groups, so that the 32 blocks one XCD runs at a time
// (after the XCD remap) share 4 weight tiles and 8 activation tiles in its L2.
// Origin (first row, first output column) of logical tile `local` of a group
// with tm x tn tiles: groups of GM = 8 row tiles, column-major inside a group.
__device__ __forceinline__ int2 tile_origin(int local, int tm, int tn, int BM, int BN) {
  constexpr int GM = 8;
  const int grp = local / (GM * tn);
  const int first_m = grp * GM;
  const int gm = min(tm - first_m, GM);
  const int within = local - grp * GM * tn;
  return make_int2((first_m + within % gm) * BM, (within / gm) * BN);
}

template <int MH, bool DUAL, bool QKV = false>
__global__ void __launch_bounds__(256) gemm_tile_kernel(GemmArgs a) {
  constexpr int KB = 64;
  constexpr int BM = 64 * MH;
  constexpr int A_BYTES = BM * 128;
  constexpr int STAGE_BYTES = A_BYTES + 256 * 128;
  constexpr int OPITCH = 136;  // dual epilogue: bf16 tile BM x 128, padded rows
  constexpr int RING_BYTES = 2 * STAGE_BYTES > BM * OPITCH * 2 ? 2 * STAGE_BYTES : BM * OPITCH * 2;
  // QKV epilogue: RoPE positions of the block's rows past the ring.  They
  // share its LDS array on purpose: with a second __shared__ object the
  // compiler can no longer tell the fragment reads from the in-flight
  // global_load_lds writes and waits for all loads before them.
  constexpr int POS_BYTES = QKV ? BM * 4 : 0;
  static_assert(RING_BYTES + POS_BYTES <= 144 * 1024, "LDS of one block");
  constexpr int A_PER_WAVE = BM / 32;  // DMA instructions (8 rows each) per wave and k-block
  __shared__ __attribute__((aligned(1024))) uint8_t ring[RING_BYTES + POS_BYTES];

  // wave-derived values are uniform: keep them (and the branches on them) scalar
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hi = lane >> 5, lo = lane & 31;
  const int mh = wave >> 1, nh = wave & 1;

  // Block -> (group, split, row tile, column tile).  SwiGLU launches may
  // start with tail pieces: blocks [0, tail_tiles * tail_split) compute piece
  // b % tail_split of the k range of tile (total_tiles + b / tail_split), the
  // rest the whole tiles [0, total_tiles).
  const int n_tail = a.tail_tiles * a.tail_split;
  const bool tail = (int)blockIdx.x < n_tail;
  int gi = 0, s, local, kps;
  if (tail) {
    s = blockIdx.x % a.tail_split;
    local = a.total_tiles + blockIdx.x / a.tail_split;
    kps = a.tail_kps;
  } else {
    const int t = xcd_remap(blockIdx.x - n_tail, a.total_tiles);
    if (a.ngroups > 1 && t >= a.g[1].tile_begin) gi = 1;
    if (a.ngroups > 2 && t >= a.g[2].tile_begin) gi = 2;
    const int tm = sel3(gi, a.g[0].tiles_m, a.g[1].tiles_m, a.g[2].tiles_m);
    const int tn = sel3(gi, a.g[0].tiles_n, a.g[1].tiles_n, a.g[2].tiles_n);
    local = t - sel3(gi, a.g[0].tile_begin, a.g[1].tile_begin, a.g[2].tile_begin);
    s = local / (tm * tn);
    local -= s * tm * tn;
    kps = a.k_per_split;
  }
  const GroupView G = group_view(a, gi);
  const int2 mn = tile_origin(local, sel3(gi, a.g[0].tiles_m, a.g[1].tiles_m, a.g[2].tiles_m),
                              sel3(gi, a.g[0].tiles_n, a.g[1].tiles_n, a.g[2].tiles_n), BM, DUAL ? 128 : 256);
  const int m0 = mn.x, n0 = mn.y;  // first row, first output column

  const int M = G.M;
  const int kbeg = s * kps;
  const int kend = min(a.K, kbeg + kps);
  const int nkb = kend > kbeg ? (kend - kbeg) / KB : 0;
  auto chunk_of = [&](int r) { return 8 * ((lane & 7) ^ swz(r)); };

  // activation DMA: instruction j of this wave fills tile rows 8g..8g+7,
  // g = wave*A_PER_WAVE + j; lane l takes row 8g + l/8, slot l%8
  const uint16_t* pa[A_PER_WAVE];
#pragma unroll
  for (int j = 0; j < A_PER_WAVE; ++j) {
    const int tr = 8 * (wave * A_PER_WAVE + j) + (lane >> 3);
    const int r = min(m0 + tr, M - 1);
    const int src = G.rows ? G.rows[r] : r;
    pa[j] = reinterpret_cast<const uint16_t*>(G.A) + (int64_t)src * a.lda + kbeg + chunk_of(tr);
  }
  // weight DMA: instruction j of this wave fills stage weight rows 8g..8g+7, g = 8*wave + j
  const uint16_t* pw[8];
  // QKV epilogue: RoPE positions of the block's rows, read once at the start
  int* spos = reinterpret_cast<int*>(ring + RING_BYTES);
  const int kind = sel3(gi, a.g[0].kind, a.g[1].kind, a.g[2].kind);
  if constexpr (QKV) {
    if (kind == 1 && tid < BM) {
      const int m = min(m0 + tid, M - 1);
      spos[tid] = a.pos[G.rows ? G.rows[m] : m];
    }
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int wr = 8 * (8 * wave + j) + (lane >> 3);  // 0..255
    const uint16_t* W;
    int row;
    if constexpr (DUAL) {
      W = reinterpret_cast<const uint16_t*>(wr < 128 ? G.W : G.W2);
      row = n0 + (wr & 127);
    } else {
      W = reinterpret_cast<const uint16_t*>(G.W);
      row = n0 + wr;
    }
    pw[j] = W + (int64_t)row * a.K + kbeg + chunk_of(wr);
  }

  // row tiles of this wave that hold rows < M (the rest skip their MMAs)
  const int live = __builtin_amdgcn_readfirstlane(min(MH, max(0, (M - m0 - 32 * MH * mh + 31) / 32)));

  floatx16 acc[MH][4];
#pragma unroll
  for (int i = 0; i < MH; ++i)
#pragma unroll
    for (int u = 0; u < 4; ++u) acc[i][u] = floatx16{};

  // DMA instruction p (of NP per wave and k-block) of k-block kb into stage S
  constexpr int NP = A_PER_WAVE + 8;
  // LDS offset of the ring (the DMA takes its LDS destination from M0)
  const uint32_t ring_lds = lds_offset(ring);
  auto issue_piece = [&](int kb, auto S, auto Pc) {
    constexpr int st = decltype(S)::value;
    constexpr int p = decltype(Pc)::value;
    const uint32_t base = ring_lds + st * STAGE_BYTES;
    if constexpr (p < A_PER_WAVE)
      dma16(pa[p] + kb * KB, base + (wave * A_PER_WAVE + p) * 1024);
    else
      dma16(pw[p - A_PER_WAVE] + kb * KB, base + A_BYTES + (8 * wave + p - A_PER_WAVE) * 1024);
  };

  // weight tile u of the wave: LDS weight rows wrow(u) .. +31
  auto wrow = [&](int u) {
    if constexpr (DUAL) return (u < 2 ? 64 * nh + 32 * u : 128 + 64 * nh + 32 * (u - 2));
    else return 128 * nh + 32 * u;
  };

  // MMAs of the k-block in stage S.  The DMA of k-block kbn into stage SN is
  // issued between the MMA groups of the first two k-steps (a burst of all of
  // them at once stalls the wave before its MMAs; spread over all four k-steps
  // the last ones land too late), measured 10-15 % faster than either.
  // fragments of k-step q of the k-block in stage S
  auto frags = [&](auto S, int q, bf16x8 (&w)[4], bf16x8 (&x)[MH]) __attribute__((always_inline)) {
    constexpr int st = decltype(S)::value;
    const uint8_t* tile = ring + st * STAGE_BYTES;
    const uint8_t* at = tile + (32 * MH * mh + lo) * 128;
    const uint8_t* wt = tile + A_BYTES + lo * 128;
    const int c = 16 * ((4 * hi + q) ^ swz(lo));
#pragma unroll
    for (int u = 0; u < 4; ++u)
      w[u] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(wt + wrow(u) * 128 + c));
#pragma unroll
    for (int i = 0; i < MH; ++i)
      x[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(at + i * 32 * 128 + c));
  };
  bf16x8 wf[2][4], af[2][MH];
  constexpr int HALF = NP / 2;  // DMA pieces issued in step 3, the rest in the next step 0

  // One k-block in stage S.  On entry buffer 0 holds its step-0 fragments and
  // the first half of the DMA of the next k-block (stage SN) is in flight.
  // Step 0 issues the other half; the barrier comes after step 2's MMAs, once
  // step 3's fragments are in registers: then stage S is free (DMA of k-block
  // kdma goes there, interleaved with step 3's MMAs) and stage SN has landed
  // (the next k-block's step-0 fragments are read while step 3's MMAs run).
  auto kblock = [&](auto S, auto SN, int knext, int kdma, auto FULL) __attribute__((always_inline)) {
    auto mmas = [&](auto Q, auto P0, auto P1, auto SD, int kd) __attribute__((always_inline)) {
      constexpr int q = decltype(Q)::value;
      constexpr int p0 = decltype(P0)::value, p1 = decltype(P1)::value;
      static_for<0, MH>([&](auto I) {
        constexpr int i = I.value;
        if (decltype(FULL)::value || i < live) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            acc[i][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[q & 1][u], af[q & 1][i], acc[i][u], 0, 0, 0);
        }
        constexpr int a0 = p0 + i * (p1 - p0) / MH, a1 = p0 + (i + 1) * (p1 - p0) / MH;
        static_for<a0, a1>([&](auto P) { issue_piece(kd, SD, P); });
        __builtin_amdgcn_sched_barrier(0);
      });
    };
    using Z = std::integral_constant<int, 0>;
    frags(S, 1, wf[1], af[1]);
    __builtin_amdgcn_sched_barrier(0);
    mmas(std::integral_constant<int, 0>{}, std::integral_constant<int, HALF>{}, std::integral_constant<int, NP>{}, SN, knext);
    frags(S, 2, wf[0], af[0]);
    __builtin_amdgcn_sched_barrier(0);
    mmas(std::integral_constant<int, 1>{}, Z{}, Z{}, SN, knext);
    frags(S, 3, wf[1], af[1]);
    __builtin_amdgcn_sched_barrier(0);
    mmas(std::integral_constant<int, 2>{}, Z{}, Z{}, SN, knext);
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    frags(SN, 0, wf[0], af[0]);
    __builtin_amdgcn_sched_barrier(0);
    mmas(std::integral_constant<int, 3>{}, Z{}, std::integral_constant<int, HALF>{}, S, kdma);
  };

  if (nkb > 0) {
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    static_for<0, NP>([&](auto P) { issue_piece(0, S0{}, P); });
    dma_wait_barrier();
    frags(S0{}, 0, wf[0], af[0]);
    static_for<0, HALF>([&](auto P) { issue_piece(min(1, nkb - 1), S1{}, P); });
    // Waves whose row tiles all hold rows < M (every block but the last row
    // tile) run a copy of the loop without the per-tile guards: a branch
    // inside the MMA groups splits the loop into basic blocks, across which
    // the compiler can only wait for every outstanding LDS read.
    auto run = [&](auto FULL) __attribute__((always_inline)) {
      int kb = 0;
      for (; kb + 2 <= nkb; kb += 2) {
        kblock(S0{}, S1{}, min(kb + 1, nkb - 1), min(kb + 2, nkb - 1), FULL);
        kblock(S1{}, S0{}, min(kb + 2, nkb - 1), min(kb + 3, nkb - 1), FULL);
      }
      if (kb < nkb) kblock(S0{}, S1{}, min(kb + 1, nkb - 1), min(kb + 2, nkb - 1), FULL);
    };
    if (live == MH) run(std::true_type{});
    else run(std::false_type{});
    dma_wait_all();
  }

  // The MMA takes the weight fragment as A and the activation fragment as B,
  // so its D layout puts one activation row in each lane (row lane % 32 of the
  // 32-row tile) and, in registers 4g..4g+3, the four consecutive output
  // columns 8 g + 4 (lane / 32) + [0, 4) of the 32-column tile: every lane
  // writes 16-byte (fp32) or 8-byte (bf16) row pieces.
  const int lrow = 32 * MH * mh + lo;  // tile row of acc[0][*]; acc[i][*] is 32 i further
  auto quad = [&](const floatx16& v, int g) { return floatx4{v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]}; };
  if constexpr (DUAL) {
    if (tail) {
      // fp32 partial sums of piece s: scratch[s][tail tile][BM][256], gate
      // columns 0..127 then up columns 128..255 of the tile's 128 outputs
      float* sp = reinterpret_cast<float*>(a.scratch) +
                  ((int64_t)s * a.tail_tiles + (local - a.total_tiles)) * BM * 256;
#pragma unroll
      for (int i = 0; i < MH; ++i) {
        const int row = lrow + 32 * i;
        if (m0 + row < M) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int g = 0; g < 4; ++g)
              *reinterpret_cast<floatx4*>(sp + row * 256 + (u >> 1) * 128 + 64 * nh + 32 * (u & 1) + 8 * g + 4 * hi) =
                  quad(acc[i][u], g);
        }
      }
      return;
    }
    // bf16 silu(g) * u staged as a BM x 128 tile, written as 16-byte row pieces
    __syncthreads();
    uint16_t* ot = reinterpret_cast<uint16_t*>(ring);
#pragma unroll
    for (int i = 0; i < MH; ++i)
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint32_t w[2];
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const int r = 4 * g + 2 * e;
            w[e] = (uint32_t)f32_to_bf16_bits(silu(acc[i][u][r]) * acc[i][u + 2][r]) |
                   ((uint32_t)f32_to_bf16_bits(silu(acc[i][u][r + 1]) * acc[i][u + 2][r + 1]) << 16);
          }
          *reinterpret_cast<uint2*>(ot + (lrow + 32 * i) * OPITCH + 64 * nh + 32 * u + 8 * g + 4 * hi) =
              make_uint2(w[0], w[1]);
        }
    __syncthreads();
    const int rows = min(BM, M - m0);
    uint16_t* op = reinterpret_cast<uint16_t*>(G.out) + (int64_t)m0 * G.ldo + n0;
    for (int c = tid; c < rows * 16; c += 256) {
      const int row = c >> 4, ch = c & 15;
      *reinterpret_cast<u32x4*>(op + (int64_t)row * G.ldo + 8 * ch) =
          *reinterpret_cast<const u32x4*>(ot + row * OPITCH + 8 * ch);
    }
  } else if constexpr (QKV) {
    // bf16 Q, K or V^T.  The wave's 128 output columns are one head, so the
    // rotate-half partner of column 32u + lo (u = 0, 1) is the same lane's
    // column 32(u + 2) + lo.  First RoPE in place on the accumulators, then
    // one 32-row tile at a time through the wave's own LDS area and out
    // as 16-byte pieces: [row][column] rows of Q and K, or [column][row] for
    // V^T whose rows M..ldvt-1 are written zero.  That loop and its barriers
    // run the same number of times in every wave.
    if (kind == 1) {
      // cos/sin rows of the block's BM rows into the ring (512 B per row, row
      // j at byte 512 j): one burst of global_load_lds, 2 rows per wave
      // instruction, then one wait instead of one table latency per tile
      static_assert(BM * 512 <= RING_BYTES, "RoPE rows fit in the ring");
      __syncthreads();  // spos written, every wave done with the last stage
#pragma unroll
      for (int t = 0; t < BM / 8; ++t) {
        const int row = 2 * (wave + 4 * t) + hi;
        const int p = spos[row];
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(a.rope + (int64_t)p * 64 + 2 * lo),
                                         (__attribute__((address_space(3))) void*)(ring + 2 * (wave + 4 * t) * 512),
                                         16, 0, 0);
      }
      wait_vmcnt<0>();
      __syncthreads();
#pragma unroll
      for (int i = 0; i < MH; ++i) {
        if (i < live) {
          const uint8_t* cs = ring + (lrow + 32 * i) * 512;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              const int col = 32 * u + 8 * (r >> 2) + 4 * hi + (r & 3);
              const float2 c = *reinterpret_cast<const float2*>(cs + col * 8);
              const float2 y = rope_rotate(acc[i][u][r], acc[i][u + 2][r], c.x, c.y);
              acc[i][u][r] = y.x;
              acc[i][u + 2][r] = y.y;
            }
          }
        }
      }
    }
    constexpr int QP = 136, VP = 40;  // pitches (bf16) of the two layouts
    constexpr int WAREA = 32 * QP > 128 * VP ? 32 * QP : 128 * VP;
    static_assert(4 * WAREA * 2 <= RING_BYTES, "epilogue staging fits");
    uint16_t* sw = reinterpret_cast<uint16_t*>(ring) + wave * WAREA;
    const int col0 = n0 + 128 * nh;
    uint16_t* out = reinterpret_cast<uint16_t*>(G.out);
#pragma unroll
    for (int i = 0; i < MH; ++i) {
      const int rb = m0 + 32 * (MH * mh + i);  // first row of the tile
      __syncthreads();
      if (i < live) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int col = 32 * u + 8 * g + 4 * hi;
            if (kind == 1) {
              *reinterpret_cast<uint2*>(sw + lo * QP + col) =
                  make_uint2((uint32_t)f32_to_bf16_bits(acc[i][u][4 * g]) |
                                 ((uint32_t)f32_to_bf16_bits(acc[i][u][4 * g + 1]) << 16),
                             (uint32_t)f32_to_bf16_bits(acc[i][u][4 * g + 2]) |
                                 ((uint32_t)f32_to_bf16_bits(acc[i][u][4 * g + 3]) << 16));
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                sw[(col + e) * VP + lo] = f32_to_bf16_bits(rb + lo < M ? acc[i][u][4 * g + e] : 0.f);
            }
          }
      }
      __syncthreads();
      if (i < live) {
        if (kind == 1) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int row = (lane >> 4) + 4 * j, ch = lane & 15;
            if (rb + row < M)
              *reinterpret_cast<u32x4*>(out + (int64_t)(rb + row) * G.ldo + col0 + 8 * ch) =
                  *reinterpret_cast<const u32x4*>(sw + row * QP + 8 * ch);
          }
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int c = (lane >> 2) + 16 * j, ch = lane & 3;
            if (rb + 8 * ch < a.ldvt)
              *reinterpret_cast<u32x4*>(out + (int64_t)(col0 + c) * a.ldvt + rb + 8 * ch) =
                  *reinterpret_cast<const u32x4*>(sw + c * VP + 8 * ch);
          }
        }
      }
    }
  } else {
    // fp32 partial sums as 16-byte row pieces
    float* op = reinterpret_cast<float*>(G.out) + s * G.sstride;
#pragma unroll
    for (int i = 0; i < MH; ++i) {
      const int m = m0 + lrow + 32 * i;
      if (m < M) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int g = 0; g < 4; ++g)
            *reinterpret_cast<floatx4*>(op + (int64_t)m * G.ldo + n0 + wrow(u) + 8 * g + 4 * hi) = quad(acc[i][u], g);
      }
    }
  }
}

// Tail pieces of a SwiGLU launch: gate and up summed over the pieces in
// piece order, out = bf16(silu(g) * u).  Grid (rows of a tile, tail tiles) x 128.
__global__ void __launch_bounds__(128) swiglu_tail_reduce_kernel(GemmArgs a, int BM) {
  const int row = blockIdx.x, tt = blockIdx.y, c = threadIdx.x;
  const int2 mn = tile_origin(a.total_tiles + tt, a.g[0].tiles_m, a.g[0].tiles_n, BM, 128);
  const int m = mn.x + row;
  if (m >= a.g[0].M) return;
  const float* sp = reinterpret_cast<const float*>(a.scratch) + ((int64_t)tt * BM + row) * 256;
  const int64_t piece = (int64_t)a.tail_tiles * BM * 256;
  float g = 0.f, u = 0.f;
  for (int s = 0; s < a.tail_split; ++s) {
    g += sp[s * piece + c];
    u += sp[s * piece + 128 + c];
  }
  reinterpret_cast<uint16_t*>(a.g[0].out)[(int64_t)m * a.g[0].ldo + mn.y + c] = f32_to_bf16_bits(silu(g) * u);
}

// ------------------------------------------------------------------ decode rows
// gemv_kernel: at most 4 rows (greedy decoding, one row per sample).  The
// GEMM is then a stream of weight rows against a few activation rows: one
// block of 4 waves, the MB activation rows staged in LDS once (bf16), each
// wave owning NR weight rows (SwiGLU: NR/2 outputs, their gate and up rows)
// for the whole K.  Lane l takes the 16-byte chunks l, l + 64, ... of every
// row (1 KB per wave instruction, non-temporal: weights are read once), U
// chunks of each row in flight per iteration; fp32 FMAs, then one fixed-order
// wave sum per (row, activation row).  No split-K: the fp32 output is the
// finished sum.  A lane adds its chunks in ascending order whatever NR and U
// are, so they change the speed, not the bits.
// QKV (EPI_DECODE_QKV): NR = 2, the wave's rows are the rotate-half pair
// (c, c + 64) of one head, c = 128 (w / 64) + w % 64 for wave w of the launch.
template <int MB, bool DUAL, int NR, int U, bool QKV = false>
__global__ void __launch_bounds__(256) gemv_kernel(GemmArgs a) {
  static_assert(!QKV || (NR == 2 && !DUAL), "QKV: one rotate-half pair per wave");
  constexpr int NO = DUAL ? NR / 2 : NR;      // outputs per wave
  extern __shared__ __attribute__((aligned(16))) uint16_t xs[];  // [MB][K]
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int gi = 0;
  if (a.ngroups > 1 && (int)blockIdx.x >= a.g[1].tile_begin) gi = 1;
  if (a.ngroups > 2 && (int)blockIdx.x >= a.g[2].tile_begin) gi = 2;
  const GroupView G = group_view(a, gi);
  const int blk = blockIdx.x - sel3(gi, a.g[0].tile_begin, a.g[1].tile_begin, a.g[2].tile_begin);
  const int K = a.K, K8 = K / 8;
  if (a.norm_h) {
    // rows = bf16(h * rsqrt(mean(h^2) + eps) * w), summed in the order of the
    // RMSNorm kernel (float4 pieces tid + 256 j, wave sums, waves (0+1)+(2+3))
    __shared__ float red[4];
    const int K4 = K / 4;
    for (int m = 0; m < MB; ++m) {
      float4 v[8];
      const float4* hr = reinterpret_cast<const float4*>(a.norm_h + (int64_t)(m < G.M ? (G.rows ? G.rows[m] : m) : 0) * K);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int c = threadIdx.x + 256 * j;
        v[j] = (m < G.M && c < K4) ? hr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      float ss = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        ss = fmaf(v[j].x, v[j].x, fmaf(v[j].y, v[j].y, fmaf(v[j].z, v[j].z, fmaf(v[j].w, v[j].w, ss))));
      ss = wave_sum(ss);
      if (lane == 0) red[wave] = ss;
      __syncthreads();
      const float tot = (red[0] + red[1]) + (red[2] + red[3]);
      const float inv = 1.0f / sqrtf(tot / (float)K + a.norm_eps);
      const float4* w4 = reinterpret_cast<const float4*>(a.norm_w);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int c = threadIdx.x + 256 * j;
        if (c < K4) {
          const float4 ww = w4[c];
          uint16_t* o = xs + (int64_t)m * K + 4 * c;
          o[0] = f32_to_bf16_bits(v[j].x * inv * ww.x);
          o[1] = f32_to_bf16_bits(v[j].y * inv * ww.y);
          o[2] = f32_to_bf16_bits(v[j].z * inv * ww.z);
          o[3] = f32_to_bf16_bits(v[j].w * inv * ww.w);
        }
      }
      __syncthreads();  // red is reused by the next row
    }
  } else {
    // activation rows (rows past M are zero)
    for (int c = threadIdx.x; c < MB * K8; c += 256) {
      const int m = c / K8, k8 = c - m * K8;
      u32x4 v = {0, 0, 0, 0};
      if (m < G.M) {
        const int src = G.rows ? G.rows[m] : m;
        v = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(G.A) + (int64_t)src * a.lda + 8 * k8);
      }
      *reinterpret_cast<u32x4*>(xs + (int64_t)m * K + 8 * k8) = v;
    }
    __syncthreads();
  }
  const int gw = blk * 4 + wave;  // wave of the group
  const int o0 = QKV ? 128 * (gw >> 6) + (gw & 63) : gw * NO;  // first output column of this wave
  if (o0 >= G.N) return;
  const uint16_t* wrow[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int o = QKV ? o0 + 64 * r : min(o0 + (DUAL ? r % NO : r), G.N - 1);
    const uint16_t* W = reinterpret_cast<const uint16_t*>(DUAL && r >= NO ? G.W2 : G.W);
    wrow[r] = W + (int64_t)o * K;
  }
  float acc[NR][MB];
#pragma unroll
  for (int r = 0; r < NR; ++r)
#pragma unroll
    for (int m = 0; m < MB; ++m) acc[r][m] = 0.f;
  for (int c0 = lane; c0 < K8; c0 += 64 * U) {
    u32x4 wv[U][NR];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        const int c = c0 + 64 * u;
        wv[u][r] = c < K8 ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wrow[r] + 8 * c))
                          : u32x4{0, 0, 0, 0};
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + 64 * u;
      if (c >= K8) break;
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        const u32x4 xv = *reinterpret_cast<const u32x4*>(xs + (int64_t)m * K + 8 * c);
        float x[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[2 * e] = __uint_as_float(xv[e] << 16);
          x[2 * e + 1] = __uint_as_float(xv[e] & 0xFFFF0000u);
        }
#pragma unroll
        for (int r = 0; r < NR; ++r)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[r][m] = fmaf(__uint_as_float(wv[u][r][e] << 16), x[2 * e], acc[r][m]);
            acc[r][m] = fmaf(__uint_as_float(wv[u][r][e] & 0xFFFF0000u), x[2 * e + 1], acc[r][m]);
          }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < NR; ++r)
#pragma unroll
    for (int m = 0; m < MB; ++m) acc[r][m] = wave_sum(acc[r][m]);
  if (lane != 0) return;
  if constexpr (QKV) {
    const int kind = sel3(gi, a.g[0].kind, a.g[1].kind, a.g[2].kind);
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      if (m >= G.M) break;
      const int p = a.pos[m];
      float y0 = acc[0][m], y1 = acc[1][m];
      if (kind & 1) {
        const float2 cs = a.rope[(int64_t)p * 64 + (o0 & 63)];
        const float2 y = rope_rotate(y0, y1, cs.x, cs.y);
        y0 = y.x;
        y1 = y.y;
      }
      uint16_t* dst = reinterpret_cast<uint16_t*>(G.out) + ((kind & 2) ? (int64_t)m * a.kv_cap + p : m) * G.ldo;
      dst[o0] = f32_to_bf16_bits(y0);
      dst[o0 + 64] = f32_to_bf16_bits(y1);
    }
    return;
  }
#pragma unroll
  for (int q = 0; q < NO; ++q) {
    const int o = o0 + q;
    if (o >= G.N) break;
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      if (m >= G.M) break;
      if constexpr (DUAL)
        reinterpret_cast<uint16_t*>(G.out)[(int64_t)m * G.ldo + o] =
            f32_to_bf16_bits(silu(acc[q][m]) * acc[q + NO][m]);
      else if (a.epilogue == EPI_RESIDUAL_F32)
        reinterpret_cast<float*>(G.out)[(int64_t)m * G.ldo + o] += acc[q][m];
      else
        reinterpret_cast<float*>(G.out)[(int64_t)m * G.ldo + o] = acc[q][m];
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
  if (tc.m0 >= G.M) return;  // a device row count below the launch's bound
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
  bool stream;  // weight-streaming kernel
};

// Tile shape.  Up to 256 rows the weight-streaming kernel covers every row in
// one tile (BM = rows rounded up to 64), so each weight element is read from
// HBM once; more rows use the LDS-staged kernel.
TileCfg pick_bf16_tile(int maxM, bool dual) {
  if (maxM <= 256) {
    const int bm = std::max(64, (maxM + 63) / 64 * 64);
    return TileCfg{bm, dual ? 64 : 128, true};
  }
  return dual ? TileCfg{128, 64, false} : TileCfg{128, 128, false};
}

constexpr int kTargetBlocks = 256;

// LDS-staged kernel: split until the grid covers the chip.  Streaming kernel
// (one block per CU): the largest split whose grid still fits in one wave of
// blocks; a second partial wave costs more than it hides.
int choose_split(int tiles, int K, int split_max, int kgran, bool stream) {
  int split = 1;
  if (stream) {
    while (split < split_max && tiles * split * 2 <= kTargetBlocks && K / (kgran * split * 2) >= 4) split *= 2;
  } else {
    while (split < split_max && tiles * split < kTargetBlocks && K / (kgran * split * 2) >= 4) split *= 2;
  }
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

template <int MT, bool DUAL, bool LENS = false>
void launch_stream(const GemmArgs& a, hipStream_t st) {
  constexpr int LEAD = MT <= 2 ? 3 : 2;
  gemm_stream_kernel<MT, LEAD, DUAL, LENS><<<a.total_tiles, 256, 0, st>>>(a);
}

// More than 256 rows: gemm_tile_kernel when the shapes fit it (N a multiple of
// the block's output columns, K of 64, 16-byte aligned bf16 output rows for
// the SwiGLU epilogue).  The row tile (256, 192 or 128) minimises the number
// of waves of blocks (one block per CU) times the cost of a block; split-K
// only fills a grid that would leave CUs idle.
bool tile_path_fits(const GemmArgs& a, bool dual) {
  if (a.K % 64) return false;
  for (int i = 0; i < a.ngroups; ++i) {
    const GemmGroup& g = a.g[i];
    if (g.N % (dual ? 128 : 256)) return false;
    if (dual && (reinterpret_cast<uintptr_t>(g.out) % 16 || g.ldo % 8)) return false;
    // fp32 partial sums leave as 16-byte row pieces
    if (!dual && a.epilogue != EPI_QKV_BF16 &&
        (reinterpret_cast<uintptr_t>(g.out) % 16 || g.ldo % 4 || g.split_stride % 4))
      return false;
  }
  return true;
}

struct TileChoice {
  int mh, split, tail, tail_split;
};

TileChoice tile_choice(const GemmArgs& a, int split_max, bool dual) {
  const int bn = dual ? 128 : 256;
  TileChoice best{4, 1, 0, 0};
  double best_cost = 1e300;
  for (int mh : {4, 3, 2}) {
    const int bm = 64 * mh;
    const int tiles = tiles_for(a, bm, bn);
    const int split = dual ? 1 : choose_split(tiles, a.K, split_max, 64, true);
    double cost = (double)ceil_div(tiles * split, kTargetBlocks) * (bm + 64) / split;
    int tail = 0, ts = 0;
    // SwiGLU, one group: a last wave at most a quarter full is split along k
    // into pieces that run beside the first wave (fp32 partials in scratch)
    const int r = tiles % kTargetBlocks;
    if (dual && a.ngroups == 1 && tiles > kTargetBlocks && r > 0 && r <= kTargetBlocks / 4 && a.scratch) {
      const int nkb = a.K / 64;
      int s = std::min(16, std::min(nkb / 2, kTargetBlocks / r));
      while (s >= 2 && (size_t)r * s * bm * 256 * 4 > a.scratch_bytes) --s;
      if (s >= 2) {
        const double c2 = (double)(tiles / kTargetBlocks) * (bm + 64) + (bm + 64) * (1.0 / s + 0.1);
        if (c2 < cost) {
          cost = c2;
          tail = r;
          ts = s;
        }
      }
    }
    if (cost < best_cost) {
      best_cost = cost;
      best = TileChoice{mh, split, tail, ts};
    }
  }
  return best;
}

hipError_t launch_tile(GemmArgs& a, int split_max, bool dual, hipStream_t st) {
  const int bn = dual ? 128 : 256;
  const TileChoice tc = tile_choice(a, split_max, dual);
  const int best_mh = tc.mh, best_split = tc.split, best_tail = tc.tail, best_ts = tc.tail_split;
  const bool qkv = a.epilogue == EPI_QKV_BF16;
  if (qkv && best_split != 1) return hipErrorInvalidValue;
  a.split = best_split;
  a.k_per_split = ceil_div(a.K / 64, a.split) * 64;
  fill_tiles(a, 64 * best_mh, bn);
  a.tail_tiles = best_tail;
  a.tail_split = best_ts;
  a.tail_kps = best_ts ? ceil_div(a.K / 64, best_ts) * 64 : 0;
  a.total_tiles -= best_tail;  // whole tiles; the tail tiles follow them in logical order
  const int blocks = a.total_tiles + best_tail * best_ts;
  if (blocks == 0) return hipSuccess;
  switch (best_mh * 2 + (dual ? 1 : 0)) {
    case 8: qkv ? gemm_tile_kernel<4, false, true><<<blocks, 256, 0, st>>>(a)
                : gemm_tile_kernel<4, false><<<blocks, 256, 0, st>>>(a); break;
    case 9: gemm_tile_kernel<4, true><<<blocks, 256, 0, st>>>(a); break;
    case 6: qkv ? gemm_tile_kernel<3, false, true><<<blocks, 256, 0, st>>>(a)
                : gemm_tile_kernel<3, false><<<blocks, 256, 0, st>>>(a); break;
    case 7: gemm_tile_kernel<3, true><<<blocks, 256, 0, st>>>(a); break;
    case 4: qkv ? gemm_tile_kernel<2, false, true><<<blocks, 256, 0, st>>>(a)
                : gemm_tile_kernel<2, false><<<blocks, 256, 0, st>>>(a); break;
    default: gemm_tile_kernel<2, true><<<blocks, 256, 0, st>>>(a); break;
  }
  if (best_tail) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    swiglu_tail_reduce_kernel<<<dim3(64 * best_mh, best_tail), 128, 0, st>>>(a, 64 * best_mh);
  }
  return hipGetLastError();
}

// At most 4 rows: gemv_kernel, no split (the output holds the finished sums).
// Decode rows: one weight row per wave with 16 chunks in flight (SwiGLU: the
// gate and up rows of one output, 8 chunks each), four waves per block.  With
// 4 rows (2 outputs) and 4 chunks per wave, a wave fetched its rows in several
// dependent rounds and the O and down projections filled only 256 blocks:
// 3.40 ms per decode step then, 3.13 now; 32 / 16 chunks (more registers,
// fewer waves per SIMD) measured 3.55 ms.
hipError_t launch_gemv(GemmArgs& a, int maxM, bool dual, hipStream_t st) {
  a.split = 1;
  a.k_per_split = a.K;
  const bool qkv = a.epilogue == EPI_DECODE_QKV;
  const int per_block = qkv ? 8 : 4;  // outputs per block
  int t = 0;
  for (int i = 0; i < a.ngroups; ++i) {
    a.g[i].tile_begin = t;
    t += ceil_div(a.g[i].N, per_block);
  }
  a.total_tiles = t;
  if (t == 0 || maxM == 0) return hipSuccess;
  const int mb = maxM <= 1 ? 1 : (maxM <= 2 ? 2 : 4);
  const size_t sh = (size_t)mb * a.K * 2;
  if (qkv) {
    switch (mb) {
      case 1: gemv_kernel<1, false, 2, 8, true><<<t, 256, sh, st>>>(a); break;
      case 2: gemv_kernel<2, false, 2, 8, true><<<t, 256, sh, st>>>(a); break;
      default: gemv_kernel<4, false, 2, 8, true><<<t, 256, sh, st>>>(a); break;
    }
    return hipGetLastError();
  }
  if (!dual) {
    switch (mb) {
      case 1: gemv_kernel<1, false, 1, 16><<<t, 256, sh, st>>>(a); break;
      case 2: gemv_kernel<2, false, 1, 16><<<t, 256, sh, st>>>(a); break;
      default: gemv_kernel<4, false, 1, 16><<<t, 256, sh, st>>>(a); break;
    }
    return hipGetLastError();
  }
  switch (mb) {
    case 1: gemv_kernel<1, true, 2, 8><<<t, 256, sh, st>>>(a); break;
    case 2: gemv_kernel<2, true, 2, 8><<<t, 256, sh, st>>>(a); break;
    default: gemv_kernel<4, true, 2, 8><<<t, 256, sh, st>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace

namespace {
bool gemv_fits(int maxM, int K) { return maxM <= 4 && K % 8 == 0 && (size_t)4 * K * 2 <= 160 * 1024; }
int max_rows(const GemmArgs& a) {
  int maxM = 0;
  for (int i = 0; i < a.ngroups; ++i) maxM = std::max(maxM, a.g[i].M);
  return maxM;
}
// a group whose rows come from a device count (streaming, LDS-staged, fp32 kernels only)
bool has_row_count(const GemmArgs& a) {
  for (int i = 0; i < a.ngroups; ++i)
    if (a.g[i].m_dev) return true;
  return false;
}
}  // namespace

int gemm_tile_unsplit_blocks(const GemmArgs& a, int split_max) {
  const int maxM = max_rows(a);
  if (gemv_fits(maxM, a.K) || maxM <= 256 || !tile_path_fits(a, false)) return 0;
  const TileChoice tc = tile_choice(a, split_max, false);
  return tc.split == 1 ? tiles_for(a, 64 * tc.mh, 256) : 0;
}

int gemm_split_for(int M, int N, int K, bool dual, bool bf16, int split_max) {
  if (dual || !bf16) return 1;
  TileCfg tc = pick_bf16_tile(M, false);
  return choose_split(ceil_div(M, tc.BM) * (N / tc.BN), K, split_max, tc.stream ? 64 : 32, tc.stream);
}

hipError_t launch_gemm_bf16(GemmArgs& a, int split_max, hipStream_t st) {
  const int maxM = max_rows(a);
  if (a.epilogue == EPI_LENS_STATS) {
    if (maxM > 256 || a.K % 64) return hipErrorInvalidValue;
    for (int i = 0; i < a.ngroups; ++i)
      if (a.g[i].N % 128) return hipErrorInvalidValue;
    a.split = 1;
    a.k_per_split = a.K;
    const int bm = std::max(64, (maxM + 63) / 64 * 64);
    fill_tiles(a, bm, 128);
    if (a.total_tiles == 0) return hipSuccess;
    switch (bm) {
      case 64: launch_stream<2, false, true>(a, st); break;
      case 128: launch_stream<4, false, true>(a, st); break;
      case 192: launch_stream<6, false, true>(a, st); break;
      default: launch_stream<8, false, true>(a, st); break;
    }
    return hipGetLastError();
  }
  const bool dual = a.epilogue == EPI_SWIGLU;
  const bool gemv_ok = gemv_fits(maxM, a.K);
  if (a.epilogue == EPI_QKV_BF16 && has_row_count(a)) return hipErrorInvalidValue;
  if (a.epilogue == EPI_QKV_BF16) {
    // the tile kernel without split, one head of 128 columns per wave, 16-byte stores
    if (gemm_tile_unsplit_blocks(a, split_max) == 0 || !a.rope || !a.pos) return hipErrorInvalidValue;
    for (int i = 0; i < a.ngroups; ++i) {
      const GemmGroup& g = a.g[i];
      if (reinterpret_cast<uintptr_t>(g.out) % 16) return hipErrorInvalidValue;
      if (g.kind == 1 ? g.ldo % 8 != 0 : (g.kind != 2 || a.ldvt % 32 || a.ldvt < g.M)) return hipErrorInvalidValue;
    }
    return launch_tile(a, split_max, false, st);
  }
  if (a.epilogue == EPI_RESIDUAL_F32 || a.epilogue == EPI_DECODE_QKV || a.norm_h) {
    // only the decode-row kernel applies a residual or cache epilogue or a
    // fused norm (the norm holds a row of at most 8192 floats in registers)
    if (!gemv_ok || (a.norm_h && (!a.norm_w || a.K > 8192))) return hipErrorInvalidValue;
  }
  if (a.epilogue == EPI_DECODE_QKV) {
    if (!a.rope || !a.pos || a.kv_cap < 1) return hipErrorInvalidValue;
    for (int i = 0; i < a.ngroups; ++i)
      if (a.g[i].N % 128 || a.g[i].a_rows) return hipErrorInvalidValue;
  }
  if ((gemv_ok || (maxM > 256 && tile_path_fits(a, dual))) && has_row_count(a)) return hipErrorInvalidValue;
  if (gemv_ok) return launch_gemv(a, maxM, dual, st);
  if (maxM > 256 && tile_path_fits(a, dual)) return launch_tile(a, split_max, dual, st);
  TileCfg tc = pick_bf16_tile(maxM, dual);
  // the streaming kernel's epilogue stores 16-byte pieces of output rows
  auto vec_out = [&](const GemmGroup& g) {
    const int per16 = dual ? 8 : 4;
    return reinterpret_cast<uintptr_t>(g.out) % 16 == 0 && g.ldo % per16 == 0 && g.split_stride % per16 == 0;
  };
  // Shapes the streaming and tile kernels do not take go to the LDS-staged kernel
  // (up to 256 rows a tile of all rows, non-dual; the SwiGLU launch fits the
  // streaming kernel whenever K and N are multiples of 64 and its output is
  // aligned, so its fallback is the 128 x 64 tile at any row count)
  for (int i = 0; i < a.ngroups; ++i)
    if (a.g[i].N % tc.BN || (tc.stream && (a.K % 64 || !vec_out(a.g[i])))) {
      tc = maxM <= 256 && !dual ? TileCfg{std::max(64, (maxM + 63) / 64 * 64), 64, false}
                                : TileCfg{128, dual ? 64 : 128, false};
      break;
    }
  for (int i = 0; i < a.ngroups; ++i)
    if (a.g[i].N % tc.BN) return hipErrorInvalidValue;
  const int kgran = tc.stream ? 64 : 32;
  if (a.K % kgran) return hipErrorInvalidValue;
  a.split = dual ? 1 : choose_split(tiles_for(a, tc.BM, tc.BN), a.K, split_max, kgran, tc.stream);
  a.k_per_split = ceil_div(ceil_div(a.K, kgran), a.split) * kgran;
  fill_tiles(a, tc.BM, tc.BN);
  if (a.total_tiles == 0) return hipSuccess;
  if (tc.stream) {
    switch (tc.BM) {
      case 64: dual ? launch_stream<2, true>(a, st) : launch_stream<2, false>(a, st); break;
      case 128: dual ? launch_stream<4, true>(a, st) : launch_stream<4, false>(a, st); break;
      case 192: dual ? launch_stream<6, true>(a, st) : launch_stream<6, false>(a, st); break;
      default: dual ? launch_stream<8, true>(a, st) : launch_stream<8, false>(a, st); break;
    }
  } else if (dual) {
    launch_cfg<128, 64, 2, 2, true>(a, st);
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
  if (a.epilogue != EPI_PARTIAL_F32 && a.epilogue != EPI_SWIGLU) return hipErrorInvalidValue;
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
