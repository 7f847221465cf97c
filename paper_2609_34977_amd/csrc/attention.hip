// Causal prefill attention over packed samples for a compacted list of query
// rows (the rows that do not bypass attention).  Keys/values are every row of
// the query's sample up to the query's own position (VSkip-Attn rows still
// serve as keys and values, Sec. 3.2).
//
// bf16, dh = 128 (attention_bf16_kernel): one wave per (block of 32 queries,
// head).  S^T = K Q^T is computed 32 keys at a time with
// v_mfma_f32_32x32x16_bf16 so that each lane owns one query (lane % 32) and
// 16 of the 32 keys (the other 16 are in lane ^ 32); the online softmax is
// per lane (fp32, exp2 with the 1/sqrt(dh)*log2(e) scale folded in) plus one
// cross-half exchange; O^T += V^T P^T with P taken straight from the S^T
// registers (the key order inside an MFMA k-block is any permutation as long
// as both operands use it).  V tiles are transposed through LDS so every lane
// reads its 8 keys of a dh column as two 8-byte words.  Masking: key row j is
// visible to query row q iff start(q) <= j <= q.
//
// fp32 (attention_f32_kernel): one wave per (query, head), scores in LDS,
// wave reductions; any even dh <= 256.
#include "kernels.h"

namespace spider {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

__global__ void __launch_bounds__(64) attention_bf16_kernel(AttnArgs a) {
  constexpr int DH = 128;
  constexpr int VP = 32 + 4;  // key pitch of the transposed V tile (bf16)
  __shared__ __attribute__((aligned(16))) uint16_t sV[DH * VP];
  const int lane = threadIdx.x, hi = lane >> 5, lo = lane & 31;
  const int h = blockIdx.y;
  const int qa = blockIdx.x * 32 + lo;
  const bool qok = qa < a.nq;
  const uint16_t* Q = reinterpret_cast<const uint16_t*>(a.q);
  const uint16_t* Kp = reinterpret_cast<const uint16_t*>(a.k);
  const uint16_t* Vp = reinterpret_cast<const uint16_t*>(a.v);
  const int qrow = qok ? a.q_rows[qa] : -1;
  const int qstart = qok ? a.row_start[qrow] : 0x7FFFFFFF;

  // Q fragments: step t covers dh 16t + 8*hi + [0, 8)
  bf16x8 qf[DH / 16];
#pragma unroll
  for (int t = 0; t < DH / 16; ++t) {
    uint4 u = make_uint4(0, 0, 0, 0);
    if (qok) u = *reinterpret_cast<const uint4*>(Q + (int64_t)qa * a.d + h * DH + 16 * t + 8 * hi);
    qf[t] = __builtin_bit_cast(bf16x8, u);
  }
  // key range of the block
  int lo_row = qstart, hi_row = qrow;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    lo_row = min(lo_row, __shfl_xor(lo_row, o, 64));
    hi_row = max(hi_row, __shfl_xor(hi_row, o, 64));
  }
  const float sc = a.scale * kLog2e;
  float m_run = -INFINITY, l_run = 0.f;
  floatx16 o[DH / 32];
#pragma unroll
  for (int c = 0; c < DH / 32; ++c) o[c] = floatx16{};

  for (int j0 = lo_row; j0 <= hi_row; j0 += 32) {
    // ---- S^T = K Q^T for keys j0 .. j0+31
    const int kr = j0 + lo;
    const bool kok = kr <= hi_row && kr < a.rows;
    floatx16 s = {};
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) {
      uint4 u = make_uint4(0, 0, 0, 0);
      if (kok) u = *reinterpret_cast<const uint4*>(Kp + (int64_t)kr * a.d + h * DH + 16 * t + 8 * hi);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, u), qf[t], s, 0, 0, 0);
    }
    // ---- stage V^T tile in LDS: sV[dh][key]
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int lin = c * 64 + lane;  // 512 chunks of 8 dh
      const int key = lin >> 4, ch = lin & 15;
      const int vr = j0 + key;
      uint4 u = make_uint4(0, 0, 0, 0);
      if (vr <= hi_row && vr < a.rows)
        u = *reinterpret_cast<const uint4*>(Vp + (int64_t)vr * a.d + h * DH + ch * 8);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sV[(ch * 8 + 2 * e) * VP + key] = (uint16_t)(w[e] & 0xFFFFu);
        sV[(ch * 8 + 2 * e + 1) * VP + key] = (uint16_t)(w[e] >> 16);
      }
    }
    // ---- online softmax (this lane: query lo, keys 8*(r/4) + 4*hi + r%4)
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = j0 + 8 * (r >> 2) + 4 * hi + (r & 3);
      const bool vis = qok && key >= qstart && key <= qrow;
      s[r] = vis ? s[r] * sc : -INFINITY;
      mx = fmaxf(mx, s[r]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    float alpha = 1.f, sum = 0.f;
    float p[16];
    if (m_new == -INFINITY) {
#pragma unroll
      for (int r = 0; r < 16; ++r) p[r] = 0.f;
    } else {
      alpha = exp2f(m_run - m_new);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        // P enters the MFMA in bf16; normalise with the same rounded weights
        p[r] = bf16_bits_to_f32(f32_to_bf16_bits(exp2f(s[r] - m_new)));
        sum += p[r];
      }
    }
    sum += __shfl_xor(sum, 32, 64);
    l_run = l_run * alpha + sum;
    m_run = m_new;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[c][r] *= alpha;
    // ---- O^T += V^T P^T, two k-blocks of 16 keys
    bf16x8 pf[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = (uint32_t)f32_to_bf16_bits(p[8 * u + 2 * e]) |
               ((uint32_t)f32_to_bf16_bits(p[8 * u + 2 * e + 1]) << 16);
      pf[u] = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < DH / 32; ++c) {
      const int dcol = c * 32 + lo;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        // keys 16u + 4hi + [0,4) and 16u + 8 + 4hi + [0,4), matching p[8u .. 8u+7]
        const uint2 v0 = *reinterpret_cast<const uint2*>(&sV[dcol * VP + 16 * u + 4 * hi]);
        const uint2 v1 = *reinterpret_cast<const uint2*>(&sV[dcol * VP + 16 * u + 8 + 4 * hi]);
        const bf16x8 vf = __builtin_bit_cast(bf16x8, make_uint4(v0.x, v0.y, v1.x, v1.y));
        o[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[u], o[c], 0, 0, 0);
      }
    }
  }
  if (!qok) return;
  const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
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

__global__ void __launch_bounds__(64) attention_f32_kernel(AttnArgs a) {
  extern __shared__ float sc[];  // [max_seq]
  const int lane = threadIdx.x;
  const int qa = blockIdx.x, h = blockIdx.y;
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
  dim3 grid(ceil_div(a.nq, 32), a.H);
  attention_bf16_kernel<<<grid, 64, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_attention_f32(const AttnArgs& a, int max_seq, hipStream_t st) {
  if (a.nq == 0) return hipSuccess;
  dim3 grid(a.nq, a.H);
  attention_f32_kernel<<<grid, 64, (size_t)std::max(1, max_seq) * 4, st>>>(a);
  return hipGetLastError();
}

}  // namespace spider
