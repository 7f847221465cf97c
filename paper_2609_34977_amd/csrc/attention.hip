// Causal prefill attention over packed samples for a compacted list of query
// rows (the rows that do not bypass attention).  Keys/values are every row of
// the query's sample up to the query's own position (VSkip-Attn rows still
// serve as keys and values, Sec. 3.2).
//
// bf16, dh = 128 (attention_bf16_kernel): one block of 4 waves per (block of
// 32 queries, head).  The key range of the 32 queries is cut into 32-key
// blocks aligned to multiples of 32, dealt round-robin to the 4 waves; each
// wave keeps its own online softmax and the four partial results are merged
// through LDS in fixed wave order at the end.  S^T = K Q^T is computed with
// v_mfma_f32_32x32x16_bf16 so that each lane owns one query (lane % 32) and
// 16 of the 32 keys (the other 16 are in lane ^ 32); the softmax runs per lane
// in fp32 (exp2 with the 1/sqrt(dh)*log2(e) scale folded in) plus one
// cross-half exchange; O^T += V^T P^T with P taken straight from the S^T
// registers (the key order inside an MFMA k-block is any permutation as long
// as both operands use it), split into bf16 hi + lo parts so the product sees
// P to ~16 bits, and V^T fragments read from the transposed V
// written by the QKV finalize (8 bytes = 4 keys per load, no LDS staging).
// Masking: key row j is visible to query row q iff start(q) <= j <= q.
//
// fp32 (attention_f32_kernel): one wave per (query, head), scores in LDS,
// wave reductions; any even dh <= 256.
#include "kernels.h"

namespace spider {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
// The online softmax keeps a stale running max until a key block's max
// exceeds it by this much in the base-2 exponent (weights <= 2^kLazyLog2).
constexpr float kLazyLog2 = 8.0f;

// Lane l and lane l ^ 32 of a value, as (lower-half lane's, upper-half lane's)
// in both lanes of the pair: one v_permlane32_swap, no LDS round trip (a
// ds_bpermute's lgkmcnt wait would also wait for every fragment read in flight).
__device__ __forceinline__ float2 lane_pair(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

typedef float float2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

// 16-byte-per-lane DMA into LDS like dma16, from a wave-uniform base kept in
// SGPRs plus a per-lane byte offset: moving the base each key block is two
// scalar adds instead of 64-bit lane address arithmetic.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16_at(const void* base, uint32_t off, uint32_t lds) {
  lds = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
#pragma clang diagnostic pop

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__global__ void __launch_bounds__(256) attention_bf16_kernel(AttnArgs a) {
  constexpr int DH = 128;
  constexpr int NW = 4;
  __shared__ float xm[NW - 1][32], xl[NW - 1][32];
  __shared__ __attribute__((aligned(16))) float xo[NW - 1][64 * 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hi = lane >> 5, lo = lane & 31;
  const int h = blockIdx.y;
  const int nq = a.nq_dev ? min(a.nq, *a.nq_dev) : a.nq;
  if ((int)blockIdx.x * 32 >= nq) return;
  const int qa = blockIdx.x * 32 + lo;
  const bool qok = qa < nq;
  const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
  const uint16_t* Kp = reinterpret_cast<const uint16_t*>(a.k);
  const uint16_t* VT = reinterpret_cast<const uint16_t*>(a.v);
  const int qrow = qok ? a.q_rows[qa] : -1;
  const int qstart = qok ? a.row_start[qrow] : 0x7FFFFFFF;

  // Q fragments: step t covers dh 16t + 8*hi + [0, 8)
  bf16x8 qf[DH / 16];
#pragma unroll
  for (int t = 0; t < DH / 16; ++t) {
    u32x4 u = {0, 0, 0, 0};
    if (qok) u = *reinterpret_cast<const u32x4*>(Q + (int64_t)qa * a.d + h * DH + 16 * t + 8 * hi);
    qf[t] = __builtin_bit_cast(bf16x8, u);
  }
  // key range of the 32 queries (every block holds at least one query)
  int lo_row = qstart, hi_row = qrow;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    lo_row = min(lo_row, __shfl_xor(lo_row, o, 64));
    hi_row = max(hi_row, __shfl_xor(hi_row, o, 64));
  }
  const int jb0 = lo_row & ~31;
  const int nblk = (hi_row - jb0) / 32 + 1;
  // a key block [j0, j0 + 31] is fully visible to every valid query iff
  // j0 >= st_max and j0 + 31 <= q_min (invalid lanes store nothing)
  int st_max = qok ? qstart : -1, q_min = qok ? qrow : 0x7FFFFFFF;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    st_max = max(st_max, __shfl_xor(st_max, o, 64));
    q_min = min(q_min, __shfl_xor(q_min, o, 64));
  }
  st_max = __builtin_amdgcn_readfirstlane(st_max);
  q_min = __builtin_amdgcn_readfirstlane(q_min);
  const float sc = a.scale * kLog2e;
  const float lazy = kLazyLog2 / sc;  // in raw score units
  float m_run = -INFINITY, l_run = 0.f;
  floatx16 o[DH / 32];
#pragma unroll
  for (int c = 0; c < DH / 32; ++c) o[c] = floatx16{};

  for (int bi = wave; bi < nblk; bi += NW) {
    const int j0 = jb0 + 32 * bi;
    // ---- loads of this key block: K rows j0 + lane%32, V^T keys j0 .. j0+31
    const int kr = j0 + lo;
    const bool kok = kr <= hi_row;
    u32x4 kf[DH / 16];
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) {
      kf[t] = u32x4{0, 0, 0, 0};
      if (kok) kf[t] = *reinterpret_cast<const u32x4*>(Kp + (int64_t)kr * a.d + h * DH + 16 * t + 8 * hi);
    }
    // V^T fragment (c, u): dh column 32c + lane%32, keys 16u + 4hi + [0,4) and 16u + 8 + 4hi + [0,4)
    uint2 vf[DH / 32][2][2];
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint16_t* base = VT + (int64_t)(h * DH + 32 * c + lo) * a.ldvt + j0 + 16 * u + 4 * hi;
        vf[c][u][0] = *reinterpret_cast<const uint2*>(base);
        vf[c][u][1] = *reinterpret_cast<const uint2*>(base + 8);
      }
    // ---- S^T = K Q^T (this lane: query lo, keys 8*(r/4) + 4*hi + r%4).  As in
    // attention_wide_kernel, keys some query of the block cannot see enter as
    // -inf through the first MMA's accumulator, only in key blocks that hold
    // such keys.
    floatx16 s;
    if (j0 >= st_max && j0 + 31 <= q_min) {
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[0]), qf[0], floatx16{}, 0, 0, 0);
    } else {
      floatx16 bias;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = j0 + 8 * (r >> 2) + 4 * hi + (r & 3);
        const bool vis = qok && key >= qstart && key <= qrow;
        bias[r] = vis ? 0.f : -INFINITY;
      }
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[0]), qf[0], bias, 0, 0, 0);
    }
#pragma unroll
    for (int t = 1; t < DH / 16; ++t)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kf[t]), qf[t], s, 0, 0, 0);
    // ---- online softmax on the raw scores, as in attention_wide_kernel: the
    // scale folded into the exponent's FMA, a lazily moved running max and a
    // vote before any rescale.
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[r]);
    {
      const float2 pm = lane_pair(mx);
      mx = fmaxf(pm.x, pm.y);
    }
    const bool move = mx > m_run + lazy;
    const float m_new = move ? mx : m_run;
    const float msc = m_new == -INFINITY ? 0.f : m_new * sc;  // no visible key yet: weights 0
    const float alpha = move ? __builtin_amdgcn_exp2f(fmaf(m_run, sc, -msc)) : 1.f;
    float p[16], s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int r = 0; r < 16; r += 2) {
      p[r] = __builtin_amdgcn_exp2f(fmaf(s[r], sc, -msc));
      p[r + 1] = __builtin_amdgcn_exp2f(fmaf(s[r + 1], sc, -msc));
      s0 += p[r];
      s1 += p[r + 1];
    }
    const float2 ps = lane_pair(s0 + s1);
    const float sum = ps.x + ps.y;
    l_run = l_run * alpha + sum;
    m_run = m_new;
    if (__any(move)) {
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[c][r] *= alpha;
    }
    // ---- O^T += V^T P^T, two k-blocks of 16 keys.  The fp32 weights enter the
    // bf16 MFMA as hi + lo parts (hi = bf16(p), lo = bf16(p - hi), hardware
    // round to nearest even), so P keeps ~16 significant bits and the softmax
    // stays fp32 up to that split.
    bf16x8 pf[2][2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      uint32_t wh[4], wl[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a0 = p[8 * u + 2 * e], a1 = p[8 * u + 2 * e + 1];
        wh[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(float2v{a0, a1}, bf16x2v));
        const float2v rest{a0 - __uint_as_float(wh[e] << 16), a1 - __uint_as_float(wh[e] & 0xFFFF0000u)};
        wl[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(rest, bf16x2v));
      }
      pf[u][0] = __builtin_bit_cast(bf16x8, u32x4{wh[0], wh[1], wh[2], wh[3]});
      pf[u][1] = __builtin_bit_cast(bf16x8, u32x4{wl[0], wl[1], wl[2], wl[3]});
    }
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const bf16x8 v8 = __builtin_bit_cast(
            bf16x8, u32x4{vf[c][u][0].x, vf[c][u][0].y, vf[c][u][1].x, vf[c][u][1].y});
        o[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v8, pf[u][0], o[c], 0, 0, 0);
        o[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v8, pf[u][1], o[c], 0, 0, 0);
      }
  }

  // ---- merge the waves' partial softmax states (fixed order 0..3)
  if (wave > 0) {
    if (hi == 0) {
      xm[wave - 1][lo] = m_run;
      xl[wave - 1][lo] = l_run;
    }
    float* dst = xo[wave - 1] + lane * 64;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        *reinterpret_cast<floatx4*>(dst + 16 * c + 4 * v) =
            floatx4{o[c][4 * v], o[c][4 * v + 1], o[c][4 * v + 2], o[c][4 * v + 3]};
  }
  __syncthreads();
  if (wave != 0 || !qok) return;
  float M = m_run;
#pragma unroll
  for (int w = 0; w < NW - 1; ++w) M = fmaxf(M, xm[w][lo]);
  const float Msc = M * sc;  // maxima are raw scores; weights exp2((m - M) sc)
  const float f0 = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(fmaf(m_run, sc, -Msc));
  float L = f0 * l_run;
#pragma unroll
  for (int c = 0; c < DH / 32; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[c][r] *= f0;
#pragma unroll
  for (int w = 0; w < NW - 1; ++w) {
    const float mw = xm[w][lo];
    const float fw = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(fmaf(mw, sc, -Msc));
    L += fw * xl[w][lo];
    const float* srcp = xo[w] + lane * 64;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const floatx4 x = *reinterpret_cast<const floatx4*>(srcp + 16 * c + 4 * v);
#pragma unroll
        for (int e = 0; e < 4; ++e) o[c][4 * v + e] += fw * x[e];
      }
  }
  const float inv = L > 0.f ? 1.0f / L : 0.f;
  uint16_t* O = reinterpret_cast<uint16_t*>(a.o) + (int64_t)qa * a.d + h * DH;
#pragma unroll
  for (int c = 0; c < DH / 32; ++c)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int dh0 = c * 32 + 8 * r4 + 4 * hi;
      uint32_t w0 = (uint32_t)f32_to_bf16_bits(o[c][4 * r4] * inv) |
                    ((uint32_t)f32_to_bf16_bits(o[c][4 * r4 + 1] * inv) << 16);
      uint32_t w1 = (uint32_t)f32_to_bf16_bits(o[c][4 * r4 + 2] * inv) |
                    ((uint32_t)f32_to_bf16_bits(o[c][4 * r4 + 3] * inv) << 16);
      *reinterpret_cast<uint2*>(O + dh0) = make_uint2(w0, w1);
    }
}

// bf16, dh = 128, many queries (attention_wide_kernel): one block of 4 waves
// per (128 QT compacted queries, head); wave w owns QT tiles of 32 queries.
// The 32-key blocks of K and V^T are staged once per block in LDS by DMA
// (two stages) and shared by the four waves, so every key read serves 128 QT
// queries (the per-query-block kernel above re-reads them per 32 queries).
// K rows enter the tile in the order sigma(i) = i with bits 2 and 3 swapped:
// then the S^T registers of a lane hold, for MFMA k-block u of P V, the 8
// consecutive keys 16u + 8 hi + [0, 8), and the V^T operand is one 16-byte
// read.  LDS chunks are swizzled (K: chunk c of row r at c ^ (r & 15), rows of
// 256 B; V^T: c ^ ((r >> 2) & 3), rows of 64 B) so the 16 lanes an LDS pass of
// a 16-byte read serves (16 consecutive rows) hit distinct banks: fragment reads are free of
// bank conflicts.  Key rows past the last row read the last row (masked).  A
// wave skips the MMAs of a key block that none of its queries can see.
template <int QT>
__global__ void __launch_bounds__(256, QT == 1 ? 2 : 1) attention_wide_kernel(AttnArgs a) {
  constexpr int DH = 128;
  constexpr int KT_BYTES = 32 * 256, STAGE = KT_BYTES + 128 * 64;
  __shared__ __attribute__((aligned(1024))) uint8_t ring[2 * STAGE];
  __shared__ int red[2][4];
  const int tid = threadIdx.x, lane = tid & 63, hi = lane >> 5, lo = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // One-dimensional grid, heads innermost, query tiles from the last one down.
  // The compacted queries are packed by sample in ascending position, so
  // within a sample a later tile sees more keys: the causal tiles start
  // longest first and the blocks that start last are short ones.
  const int ntiles = (a.nq + 128 * QT - 1) / (128 * QT);
  const int tile = ntiles - 1 - (int)blockIdx.x / a.H;
  const int h = (int)blockIdx.x % a.H;
  const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
  const uint16_t* Kp = reinterpret_cast<const uint16_t*>(a.k);
  const uint16_t* VT = reinterpret_cast<const uint16_t*>(a.v);

  int qrow[QT], qst[QT], qa[QT];
  bool qok[QT];
  bf16x8 qf[QT][DH / 16];
  int wlo = 0x7FFFFFFF, whi = -1;
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    qa[t] = tile * (128 * QT) + wave * (32 * QT) + 32 * t + lo;
    qok[t] = qa[t] < a.nq;
    qrow[t] = qok[t] ? a.q_rows[qa[t]] : -1;
    qst[t] = qok[t] ? a.row_start[qrow[t]] : 0x7FFFFFFF;
    wlo = min(wlo, qst[t]);
    whi = max(whi, qrow[t]);
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) {
      u32x4 u = {0, 0, 0, 0};
      if (qok[t]) u = *reinterpret_cast<const u32x4*>(Q + (int64_t)qa[t] * a.d + h * DH + 16 * s + 8 * hi);
      qf[t][s] = __builtin_bit_cast(bf16x8, u);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    wlo = min(wlo, __shfl_xor(wlo, o, 64));
    whi = max(whi, __shfl_xor(whi, o, 64));
  }
  wlo = __builtin_amdgcn_readfirstlane(wlo);
  whi = __builtin_amdgcn_readfirstlane(whi);
  // a key block [j0, j0 + 31] is fully visible to every valid query of the wave
  // iff j0 >= wst_max and j0 + 31 <= wq_min (invalid lanes store nothing)
  int wst_max = -1, wq_min = 0x7FFFFFFF;
#pragma unroll
  for (int t = 0; t < QT; ++t)
    if (qok[t]) {
      wst_max = max(wst_max, qst[t]);
      wq_min = min(wq_min, qrow[t]);
    }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    wst_max = max(wst_max, __shfl_xor(wst_max, o, 64));
    wq_min = min(wq_min, __shfl_xor(wq_min, o, 64));
  }
  wst_max = __builtin_amdgcn_readfirstlane(wst_max);
  wq_min = __builtin_amdgcn_readfirstlane(wq_min);
  if (lane == 0) {
    red[0][wave] = wlo;
    red[1][wave] = whi;
  }
  __syncthreads();
  const int blo = min(min(red[0][0], red[0][1]), min(red[0][2], red[0][3]));
  const int bhi = max(max(red[1][0], red[1][1]), max(red[1][2], red[1][3]));
  const int jb0 = blo & ~31;
  const int nblk = (bhi - jb0) / 32 + 1;  // every block holds at least one query

  // DMA of the key block at j0 into stage S: K tile rows 4i..4i+3 and V^T rows
  // 16i..16i+15 for i = 2 wave + e (e = 0, 1); lane l writes 16 bytes at l*16.
  // Each lane's byte offset from the key block's first K row / V^T column is
  // fixed, so a key block moves two scalar bases (the launcher keeps d * ldvt
  // below 2^31); only a block reaching past the last row clamps per lane.
  const uint32_t ring_lds = lds_offset(ring);
  uint32_t koff[2], voff[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int i = 2 * wave + e;
    const int row = 4 * i + (lane >> 4);
    const int sig = (row & ~12) | ((row & 4) << 1) | ((row & 8) >> 1);
    const int c = (lane & 15) ^ (row & 15);
    koff[e] = (uint32_t)(sig * a.d + h * DH + 8 * c) * 2u;
    const int rv = 16 * i + (lane >> 2);
    const int cv = (lane & 3) ^ ((rv >> 2) & 3);
    voff[e] = ((uint32_t)(h * DH + rv) * (uint32_t)a.ldvt + 8u * cv) * 2u;
  }
  auto issue = [&](int j0, auto S) {
    constexpr int st = decltype(S)::value;
    const uint32_t base = ring_lds + st * STAGE;
    if (j0 + 31 <= a.rows - 1) {
      const uint16_t* kb = Kp + (int64_t)j0 * a.d;
#pragma unroll
      for (int e = 0; e < 2; ++e) dma16_at(kb, koff[e], base + (2 * wave + e) * 1024);
    } else {
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int i = 2 * wave + e;
        const int row = 4 * i + (lane >> 4);
        const int sig = (row & ~12) | ((row & 4) << 1) | ((row & 8) >> 1);
        const int key = min(j0 + sig, a.rows - 1);
        const int c = (lane & 15) ^ (row & 15);
        dma16(Kp + (int64_t)key * a.d + h * DH + 8 * c, base + i * 1024);
      }
    }
    const uint16_t* vb = VT + j0;
#pragma unroll
    for (int e = 0; e < 2; ++e) dma16_at(vb, voff[e], base + KT_BYTES + (2 * wave + e) * 1024);
  };

  const float sc = a.scale * kLog2e;
  const float lazy = kLazyLog2 / sc;  // in raw score units
  float m_run[QT], l_run[QT];
  floatx16 o[QT][DH / 32];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c) o[t][c] = floatx16{};
  }

  auto compute = [&](int j0, auto S) {
    constexpr int st = decltype(S)::value;
    if (j0 > whi || j0 + 31 < wlo) return;
    const uint8_t* kt = ring + st * STAGE;
    const uint8_t* vt = kt + KT_BYTES;
    // S^T = K Q^T: lane (query lo) holds keys j0 + 16 (r >> 3) + 8 hi + (r & 7)
    floatx16 s[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) s[t] = floatx16{};
    // every K fragment of the block first (one LDS latency for all of them),
    // then the V^T fragments, whose latency the softmax below covers
    bf16x8 kf[DH / 16], vf[DH / 32][2];
#pragma unroll
    for (int k = 0; k < DH / 16; ++k)
      kf[k] = __builtin_bit_cast(bf16x8,
                                 *reinterpret_cast<const u32x4*>(kt + lo * 256 + 16 * ((2 * k + hi) ^ (lo & 15))));
    __builtin_amdgcn_sched_barrier(0);
    // keys some query of the wave cannot see enter as -inf through the first
    // MMA's accumulator (exactly 0 elsewhere), so the softmax below needs no
    // masking branch and the scores stay in the MMA's registers
    const bool full = j0 >= wst_max && j0 + 31 <= wq_min;
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      if (full) {
        s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[0], qf[t][0], s[t], 0, 0, 0);
      } else {
        floatx16 bias;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = j0 + 16 * (r >> 3) + 8 * hi + (r & 7);
          const bool vis = qok[t] && key >= qst[t] && key <= qrow[t];
          bias[r] = vis ? 0.f : -INFINITY;
        }
        s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[0], qf[t][0], bias, 0, 0, 0);
      }
    }
#pragma unroll
    for (int k = 1; k < DH / 16; ++k)
#pragma unroll
      for (int t = 0; t < QT; ++t) s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[k], qf[t][k], s[t], 0, 0, 0);
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int row = 32 * c + lo;
        vf[c][u] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(vt + row * 64 + 16 * ((2 * u + hi) ^ ((row >> 2) & 3))));
      }
    __builtin_amdgcn_sched_barrier(0);
    // Online softmax on the raw (already masked) scores: the scale enters the
    // exponent through one FMA, exp2 is the hardware instruction.  The running
    // max moves only when the block's max exceeds it by more than kLazyLog2 in
    // the exponent (weights then stay below 2^kLazyLog2), so the accumulators
    // are rescaled a few times per query instead of at almost every key block;
    // a rescale runs when some lane's max moved (wave vote).
    bf16x8 pf[QT][2][2];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[t][r]);
      {
        const float2 pm = lane_pair(mx);
        mx = fmaxf(pm.x, pm.y);
      }
      const bool move = mx > m_run[t] + lazy;
      const float m_new = move ? mx : m_run[t];
      // no visible key yet: every weight is exp2(-inf) = 0
      const float msc = m_new == -INFINITY ? 0.f : m_new * sc;
      const float alpha = move ? __builtin_amdgcn_exp2f(fmaf(m_run[t], sc, -msc)) : 1.f;
      float p[16], s0 = 0.f, s1 = 0.f;
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        p[r] = __builtin_amdgcn_exp2f(fmaf(s[t][r], sc, -msc));
        p[r + 1] = __builtin_amdgcn_exp2f(fmaf(s[t][r + 1], sc, -msc));
        s0 += p[r];
        s1 += p[r + 1];
      }
      const float2 ps = lane_pair(s0 + s1);
      const float sum = ps.x + ps.y;
      l_run[t] = l_run[t] * alpha + sum;
      m_run[t] = m_new;
      if (__any(move)) {
#pragma unroll
        for (int c = 0; c < DH / 32; ++c)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[t][c][r] *= alpha;
      }
      // hi + lo bf16 parts of the fp32 weights (hardware round to nearest even)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        uint32_t wh[4], wl[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float a0 = p[8 * u + 2 * e], a1 = p[8 * u + 2 * e + 1];
          wh[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(float2v{a0, a1}, bf16x2v));
          const float2v rest{a0 - __uint_as_float(wh[e] << 16), a1 - __uint_as_float(wh[e] & 0xFFFF0000u)};
          wl[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(rest, bf16x2v));
        }
        pf[t][u][0] = __builtin_bit_cast(bf16x8, u32x4{wh[0], wh[1], wh[2], wh[3]});
        pf[t][u][1] = __builtin_bit_cast(bf16x8, u32x4{wl[0], wl[1], wl[2], wl[3]});
      }
    }
    // O^T += V^T P^T: V^T operand = dh row 32c + lo, keys 16u + 8 hi + [0, 8)
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int t = 0; t < QT; ++t) {
          o[t][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[c][u], pf[t][u][0], o[t][c], 0, 0, 0);
          o[t][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[c][u], pf[t][u][1], o[t][c], 0, 0, 0);
        }
  };

  issue(jb0, std::integral_constant<int, 0>{});
  dma_wait_barrier();
  auto body = [&](int bi, auto J) {
    constexpr int j = decltype(J)::value;
    const int nb = min(bi + 1, nblk - 1);
    issue(jb0 + 32 * nb, std::integral_constant<int, j ^ 1>{});
    compute(jb0 + 32 * bi, J);
    dma_wait_barrier();
  };
  int bi = 0;
  for (; bi + 2 <= nblk; bi += 2) {
    body(bi, std::integral_constant<int, 0>{});
    body(bi + 1, std::integral_constant<int, 1>{});
  }
  if (bi < nblk) body(bi, std::integral_constant<int, 0>{});

  // D layout: lane holds query lo, dh rows 32c + 8 (r / 4) + 4 hi + r % 4
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    if (!qok[t]) continue;
    const float inv = l_run[t] > 0.f ? 1.0f / l_run[t] : 0.f;
    uint16_t* O = reinterpret_cast<uint16_t*>(a.o) + (int64_t)qa[t] * a.d + h * DH;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int dh0 = c * 32 + 8 * r4 + 4 * hi;
        uint32_t w0 = (uint32_t)f32_to_bf16_bits(o[t][c][4 * r4] * inv) |
                      ((uint32_t)f32_to_bf16_bits(o[t][c][4 * r4 + 1] * inv) << 16);
        uint32_t w1 = (uint32_t)f32_to_bf16_bits(o[t][c][4 * r4 + 2] * inv) |
                      ((uint32_t)f32_to_bf16_bits(o[t][c][4 * r4 + 3] * inv) << 16);
        *reinterpret_cast<uint2*>(O + dh0) = make_uint2(w0, w1);
      }
  }
}

__global__ void __launch_bounds__(64) attention_f32_kernel(AttnArgs a) {
  extern __shared__ float sc[];  // [max_seq]
  const int lane = threadIdx.x;
  const int qa = blockIdx.x, h = blockIdx.y;
  if (a.nq_dev && qa >= *a.nq_dev) return;
  const int qrow = a.q_rows[qa];
  const int st = a.row_start[qrow];
  const int nk = qrow - st + 1;
  const float* Q = reinterpret_cast<const float*>(a.q) + (int64_t)qa * a.d + h * a.dh;
  const float* Kp = reinterpret_cast<const float*>(a.k);
  const float* Vp = reinterpret_cast<const float*>(a.v);
  float qv[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int c = lane + 64 * e;
    qv[e] = c < a.dh ? Q[c] : 0.f;
  }
  float mx = -INFINITY;
  for (int j = 0; j < nk; ++j) {
    const float* kr = Kp + (int64_t)(st + j) * a.d + h * a.dh;
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int c = lane + 64 * e;
      if (c < a.dh) dot = fmaf(qv[e], kr[c], dot);
    }
    dot = wave_sum(dot) * a.scale;
    if (lane == 0) sc[j] = dot;
    mx = fmaxf(mx, dot);
  }
  __syncthreads();
  float sum = 0.f;
  for (int j = lane; j < nk; j += 64) {
    const float p = expf(sc[j] - mx);
    sc[j] = p;
    sum += p;
  }
  sum = wave_sum(sum);
  __syncthreads();
  float ov[4] = {0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < nk; ++j) {
    const float p = sc[j];
    const float* vr = Vp + (int64_t)(st + j) * a.d + h * a.dh;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int c = lane + 64 * e;
      if (c < a.dh) ov[e] = fmaf(p, vr[c], ov[e]);
    }
  }
  float* O = reinterpret_cast<float*>(a.o) + (int64_t)qa * a.d + h * a.dh;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int c = lane + 64 * e;
    if (c < a.dh) O[c] = ov[e] / sum;
  }
}

}  // namespace

hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t st) {
  if (a.nq == 0) return hipSuccess;
  if (a.dh != 128 || a.ldvt < ((a.rows + 31) / 32) * 32 || a.ldvt % 32) return hipErrorInvalidValue;
  // a device query count is honoured by the per-32-query kernel only
  // (the shared-tile kernel's per-lane DMA offsets are 32-bit byte offsets)
  const bool wide = (int64_t)ceil_div(a.nq, 128) * a.H >= 128 && (int64_t)a.d * a.ldvt < (int64_t(1) << 31);
  if (wide && a.nq_dev) return hipErrorInvalidValue;
  // At least 128 blocks of 128 queries: the shared-tile kernel (one query tile
  // per wave: two waves per SIMD overlap one's softmax with the other's MMAs;
  // two tiles per wave measured 1.7x slower at one wave per SIMD).  Fewer
  // queries: the per-32-query kernel, whose waves split the keys.
  if (wide) {
    attention_wide_kernel<1><<<ceil_div(a.nq, 128) * a.H, 256, 0, st>>>(a);
  } else {
    attention_bf16_kernel<<<dim3(ceil_div(a.nq, 32), a.H), 256, 0, st>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_attention_f32(const AttnArgs& a, int max_seq, hipStream_t st) {
  if (a.nq == 0) return hipSuccess;
  dim3 grid(a.nq, a.H);
  attention_f32_kernel<<<grid, 64, (size_t)std::max(1, max_seq) * 4, st>>>(a);
  return hipGetLastError();
}

}  // namespace spider
