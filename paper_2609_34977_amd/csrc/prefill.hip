// Skip-aware decoder prefill driver (the per-layer forward of Algorithm 1
// with VSkip-Attn / VSkip-FFN rows, Sec. 3.2) and its small kernels.
//
// Per layer l (host loop; row lists built on the host from the codes):
//   A_l = rows that do not bypass attention (queries), F_l = rows that do not
//   bypass the FFN.
//   if A_l non-empty:
//     rmsnorm   every row: h += pending residual partials; xn = bf16(norm(h))
//     gemm_qkv  one grouped launch: Q over A_l (gathered rows of xn), K and V
//               over every row (bypassing rows still provide keys/values)
//     qkv_fin   sum split-K partials, RoPE (table built in double), round
//     attention causal, compacted queries A_l
//     gemm_o    O rows of A_l -> fp32 split-K partials (pending residual)
//   if F_l non-empty:
//     rmsnorm   every row: h += pending; rows of F_l -> compact xf
//     gemm_gateup fused SwiGLU over F_l -> act
//     gemm_down act -> fp32 split-K partials (pending residual)
//   Nothing is launched for an empty set.  After the last layer a residual
//   kernel applies what is still pending.  Residual partials are summed in
//   fixed split order by the consuming kernel (deterministic, no atomics).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "kernels.h"

namespace spider {
namespace {

template <typename AT>
struct Act;
template <>
struct Act<float> {
  __device__ static inline void store(float* p, float v) { *p = v; }
  __device__ static inline float load(const float* p) { return *p; }
  // 4 consecutive values, p 16-byte aligned
  __device__ static inline void store4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
};
template <>
struct Act<uint16_t> {
  __device__ static inline void store(uint16_t* p, float v) { *p = f32_to_bf16_bits(v); }
  __device__ static inline float load(const uint16_t* p) { return bf16_bits_to_f32(*p); }
  // 4 consecutive values, p 8-byte aligned
  __device__ static inline void store4(uint16_t* p, float4 v) {
    *reinterpret_cast<uint2*>(p) = make_uint2((uint32_t)f32_to_bf16_bits(v.x) | ((uint32_t)f32_to_bf16_bits(v.y) << 16),
                                              (uint32_t)f32_to_bf16_bits(v.z) | ((uint32_t)f32_to_bf16_bits(v.w) << 16));
  }
};

// h = float(x)
template <typename AT>
__global__ void __launch_bounds__(256) embed_kernel(const AT* __restrict__ x, float* __restrict__ h,
                                                    int64_t total) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < total) h[i] = Act<AT>::load(x + i);
}

// cos/sin table for RoPE: tab[p*half + i] = (cos, sin)(p * theta^(-2i/dh)), double math.
__global__ void __launch_bounds__(256) rope_table_kernel(float2* __restrict__ tab, int max_pos,
                                                         int half, int dh, double log2_theta) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)max_pos * half) return;
  const int p = (int)(t / half), i = (int)(t % half);
  const double inv = exp2(-(2.0 * i / dh) * log2_theta);
  const double ang = (double)p * inv;
  tab[t] = make_float2((float)cos(ang), (float)sin(ang));
}

// One block per row: apply pending residual partials (h[r] += sum_s P[s][pslot[r]],
// summed in split order) then, if the row is selected,
// out[nslot[r]] = round(h * rsqrt(mean(h^2) + eps) * w).  Each thread owns up to
// 8 float4 of the row (d <= 8192, d % 4 == 0) and issues all of its loads at once.
template <typename AT, int MAXV>
__global__ void __launch_bounds__(256) norm_kernel(float* __restrict__ h, int d,
                                                   const float* __restrict__ P, int psplit,
                                                   int64_t pstride, const int32_t* __restrict__ pslot,
                                                   const float* __restrict__ w, float eps,
                                                   const int32_t* __restrict__ nslot, int all_rows,
                                                   AT* __restrict__ out) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const int d4 = d >> 2;
  // the row of h and the norm weights first: neither depends on the slot
  // lookups, so their latency overlaps those and the partial sums' (w is
  // null for a residual-only pass, which never reaches the normalisation)
  float4* hr = reinterpret_cast<float4*>(h + (int64_t)r * d);
  const float4* w4 = reinterpret_cast<const float4*>(w);
  float4 v[MAXV], ww[MAXV];
#pragma unroll
  for (int k = 0; k < MAXV; ++k) {
    const int c = threadIdx.x + k * 256;
    v[k] = c < d4 ? hr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    ww[k] = (w && c < d4) ? w4[c] : make_float4(0.f, 0.f, 0.f, 0.f);  // no weights: residual only
  }
  const int ps = (P && pslot) ? pslot[r] : -1;
  const int ns = all_rows ? r : (nslot ? nslot[r] : -1);
  if (ps < 0 && ns < 0) return;
  if (ps >= 0) {
    const float4* pr = reinterpret_cast<const float4*>(P + (int64_t)ps * d);
    const int64_t ps4 = pstride >> 2;
    // SB splits' loads in flight at a time (all of them up to 8 splits when
    // rows are at most 4096 wide), summed in split order
    constexpr int SB = MAXV <= 4 ? 8 : 4;
    for (int s0 = 0; s0 < psplit; s0 += SB) {
      float4 add[SB][MAXV];
#pragma unroll
      for (int q = 0; q < SB; ++q)
#pragma unroll
        for (int k = 0; k < MAXV; ++k) {
          const int c = threadIdx.x + k * 256;
          add[q][k] = (c < d4 && s0 + q < psplit) ? pr[(s0 + q) * ps4 + c] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
      for (int q = 0; q < SB; ++q)
#pragma unroll
        for (int k = 0; k < MAXV; ++k) {
          v[k].x += add[q][k].x;
          v[k].y += add[q][k].y;
          v[k].z += add[q][k].z;
          v[k].w += add[q][k].w;
        }
    }
#pragma unroll
    for (int k = 0; k < MAXV; ++k) {
      const int c = threadIdx.x + k * 256;
      if (c < d4) hr[c] = v[k];
    }
  }
  if (ns < 0) return;
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < MAXV; ++k)
    ss = fmaf(v[k].x, v[k].x, fmaf(v[k].y, v[k].y, fmaf(v[k].z, v[k].z, fmaf(v[k].w, v[k].w, ss))));
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  AT* o = out + (int64_t)ns * d;
#pragma unroll
  for (int k = 0; k < MAXV; ++k) {
    const int c = threadIdx.x + k * 256;
    if (c < d4)
      Act<AT>::store4(o + 4 * c, make_float4(v[k].x * inv * ww[k].x, v[k].y * inv * ww[k].y,
                                             v[k].z * inv * ww[k].z, v[k].w * inv * ww[k].w));
  }
}

// d <= 4096 uses 4 float4 per thread, larger rows 8.
template <typename AT>
void launch_norm(int R, float* h, int d, const float* P, int psplit, int64_t pstride,
                 const int32_t* pslot, const float* w, float eps, const int32_t* nslot,
                 int all_rows, AT* out, hipStream_t st) {
  if (d <= 4096)
    norm_kernel<AT, 4><<<R, 256, 0, st>>>(h, d, P, psplit, pstride, pslot, w, eps, nslot, all_rows, out);
  else
    norm_kernel<AT, 8><<<R, 256, 0, st>>>(h, d, P, psplit, pstride, pslot, w, eps, nslot, all_rows, out);
}

// Blocks [0, nq): Q rows, [nq, nq+R): K rows; then V.  Sums split partials,
// applies rotate-half RoPE to Q and K, stores act dtype.  V: with ldvt == 0
// one block per row, row-major [R, d]; with ldvt > 0 (bf16) V is stored
// transposed, V^T [d][ldvt] with ldvt = R rounded up to 32 and rows R..ldvt-1
// zero, one block per 32-row x 64-column tile (transposed through LDS).
template <typename AT>
__global__ void __launch_bounds__(256) qkv_finalize_kernel(
    const float* __restrict__ Pq, const float* __restrict__ Pk, const float* __restrict__ Pv,
    int split, int64_t pstride, int nq, int R, int d, int dh, const int32_t* __restrict__ q_rows,
    const int32_t* __restrict__ pos, const float2* __restrict__ rope, AT* __restrict__ Q,
    AT* __restrict__ K, AT* __restrict__ V, int64_t ldvt, const int32_t* __restrict__ nq_dev) {
  int b = blockIdx.x;
  // nq is the bound the grid is sized for; with a device count the Q blocks
  // past it have nothing to do
  if (nq_dev && b < nq && b >= *nq_dev) return;
  if (ldvt > 0 && b >= nq + R) {
    // one 32 x 64 tile of V, written transposed
    __shared__ __attribute__((aligned(16))) uint16_t tT[64 * 40];  // [column][row], pitch 40
    const int vb = b - nq - R, ntc = d / 64;
    const int rt = vb / ntc, ct = vb - rt * ntc;
    const int t = threadIdx.x;
    {
      const int r = t >> 3, c8 = (t & 7) * 8;
      const int row = rt * 32 + r, col = ct * 64 + c8;
      float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (row < R) {
        for (int s = 0; s < split; ++s) {
          const float4* src = reinterpret_cast<const float4*>(Pv + s * pstride + (int64_t)row * d + col);
          const float4 v0 = src[0], v1 = src[1];
          x[0] += v0.x; x[1] += v0.y; x[2] += v0.z; x[3] += v0.w;
          x[4] += v1.x; x[5] += v1.y; x[6] += v1.z; x[7] += v1.w;
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) tT[(c8 + e) * 40 + r] = f32_to_bf16_bits(x[e]);
    }
    __syncthreads();
    {
      const int cidx = t >> 2, k8 = (t & 3) * 8;
      const u32x4 w = *reinterpret_cast<const u32x4*>(&tT[cidx * 40 + k8]);
      *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(V) + (int64_t)(ct * 64 + cidx) * ldvt + rt * 32 + k8) = w;
    }
    return;
  }
  const float* P;
  AT* out;
  int prow, p = -1;
  if (b < nq) {
    P = Pq;
    out = Q;
    prow = b;
    p = pos[q_rows[b]];
  } else if (b < nq + R) {
    P = Pk;
    out = K;
    prow = b - nq;
    p = pos[prow];
  } else {
    P = Pv;
    out = V;
    prow = b - nq - R;
  }
  const int half = dh / 2;
  const float* src = P + (int64_t)prow * d;
  AT* dst = out + (int64_t)prow * d;
  if (half % 4 == 0 && split <= 2 && d <= 8192) {
    // each thread: up to 4 groups of 4 consecutive rotate-half pairs (float4
    // loads), every load issued before any use
    constexpr int NG = 4;
    const int ngroups = d / 8;  // pairs / 4
    float4 x0[NG][2], x1[NG][2];
    float4 cs[NG][2];
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      const int gi = threadIdx.x + 256 * q;
      if (gi < ngroups) {
        const int pair = 4 * gi, head = pair / half, i = pair - head * half;
        const int c0 = head * dh + i, c1 = c0 + half;
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          x0[q][s2] = s2 < split ? *reinterpret_cast<const float4*>(src + s2 * pstride + c0) : make_float4(0.f, 0.f, 0.f, 0.f);
          x1[q][s2] = s2 < split ? *reinterpret_cast<const float4*>(src + s2 * pstride + c1) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        if (p >= 0) {
          const float4* rp = reinterpret_cast<const float4*>(rope + (int64_t)p * half + i);
          cs[q][0] = rp[0];
          cs[q][1] = rp[1];
        }
      }
    }
#pragma unroll
    for (int q = 0; q < NG; ++q) {
      const int gi = threadIdx.x + 256 * q;
      if (gi >= ngroups) continue;
      const int pair = 4 * gi, head = pair / half, i = pair - head * half;
      const int c0 = head * dh + i, c1 = c0 + half;
      // split-order sums (split 0 first), as the scalar loop below
      float a[4] = {x0[q][0].x + x0[q][1].x, x0[q][0].y + x0[q][1].y, x0[q][0].z + x0[q][1].z,
                    x0[q][0].w + x0[q][1].w};
      float b[4] = {x1[q][0].x + x1[q][1].x, x1[q][0].y + x1[q][1].y, x1[q][0].z + x1[q][1].z,
                    x1[q][0].w + x1[q][1].w};
      if (p >= 0) {
        const float cx[4] = {cs[q][0].x, cs[q][0].z, cs[q][1].x, cs[q][1].z};
        const float sy[4] = {cs[q][0].y, cs[q][0].w, cs[q][1].y, cs[q][1].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float2 y = rope_rotate(a[e], b[e], cx[e], sy[e]);
          a[e] = y.x;
          b[e] = y.y;
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Act<AT>::store(dst + c0 + e, a[e]);
        Act<AT>::store(dst + c1 + e, b[e]);
      }
    }
    return;
  }
  for (int t = threadIdx.x; t < d / 2; t += 256) {
    const int head = t / half, i = t - head * half;
    const int c0 = head * dh + i, c1 = c0 + half;
    float x0 = 0.f, x1 = 0.f;
    for (int s = 0; s < split; ++s) {
      x0 += src[s * pstride + c0];
      x1 += src[s * pstride + c1];
    }
    if (p >= 0) {
      const float2 cs = rope[(int64_t)p * half + i];
      const float2 y = rope_rotate(x0, x1, cs.x, cs.y);
      x0 = y.x;
      x1 = y.y;
    }
    Act<AT>::store(dst + c0, x0);
    Act<AT>::store(dst + c1, x1);
  }
}

// ------------------------------------------------------------------ KV cache and decode
// Cache layout: keys (after RoPE) and values [L][B][cap][d] in the activation
// dtype; token at position p of sample b in layer l at ((l*B + b)*cap + p)*d.

// Copies one prefill layer's keys and values into the cache.  Values are
// summed again from the split partials in the order the finalize kernel sums
// them, so the cached values equal the ones the prefill's attention read.
template <typename AT>
__global__ void __launch_bounds__(256) kv_store_kernel(const AT* __restrict__ K, const float* __restrict__ Pv,
                                                       int split, int64_t pstride, int d,
                                                       const int32_t* __restrict__ row_sample,
                                                       const int32_t* __restrict__ pos, AT* __restrict__ ck,
                                                       AT* __restrict__ cv, int64_t layer_off, int cap) {
  const int r = blockIdx.x;
  const int64_t dst = layer_off + ((int64_t)row_sample[r] * cap + pos[r]) * d;
  const AT* ks = K + (int64_t)r * d;
  for (int c = threadIdx.x; c < d; c += 256) {
    ck[dst + c] = ks[c];
    float x = 0.f;
    for (int s = 0; s < split; ++s) x += Pv[s * pstride + (int64_t)r * d + c];
    Act<AT>::store(cv + dst + c, x);
  }
}

// Decode step, grid (B, 3): the new token of sample b at position lens[b].
// Kind 0 sums the query partials and applies RoPE into Q[b]; kind 1 the key
// (RoPE) and kind 2 the value, both written into the cache at lens[b].
template <typename AT>
__global__ void __launch_bounds__(256) decode_qkv_kernel(const float* __restrict__ Pq, const float* __restrict__ Pk,
                                                         const float* __restrict__ Pv, int split, int64_t pstride,
                                                         int d, int dh, const int32_t* __restrict__ lens,
                                                         const float2* __restrict__ rope, AT* __restrict__ Q,
                                                         AT* __restrict__ ck, AT* __restrict__ cv,
                                                         int64_t layer_off, int cap) {
  const int b = blockIdx.x, kind = blockIdx.y;
  const float* src = (kind == 0 ? Pq : (kind == 1 ? Pk : Pv)) + (int64_t)b * d;
  const int p = lens[b];
  AT* dst = kind == 0 ? Q + (int64_t)b * d : (kind == 1 ? ck : cv) + layer_off + ((int64_t)b * cap + p) * d;
  const int half = dh / 2;
  for (int t = threadIdx.x; t < d / 2; t += 256) {
    const int head = t / half, i = t - head * half;
    const int c0 = head * dh + i, c1 = c0 + half;
    float x0 = 0.f, x1 = 0.f;
    for (int s = 0; s < split; ++s) {
      x0 += src[s * pstride + c0];
      x1 += src[s * pstride + c1];
    }
    if (kind < 2) {
      const float2 cs = rope[(int64_t)p * half + i];
      const float2 y = rope_rotate(x0, x1, cs.x, cs.y);
      x0 = y.x;
      x1 = y.y;
    }
    Act<AT>::store(dst + c0, x0);
    Act<AT>::store(dst + c1, x1);
  }
}

constexpr int kDecodeMaxKeys = 8192;
constexpr int kDecodeMaxDh = 256;

template <typename AT>
__device__ __forceinline__ float act_load(const AT* p) {
  if constexpr (std::is_same<AT, float>::value) return *p;
  else return bf16_bits_to_f32(*p);
}

// A 16-byte vector of activations as floats (8 bf16 or 4 fp32).
template <typename AT>
__device__ __forceinline__ void unpack16(const uint4& v, float* x) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  if constexpr (sizeof(AT) == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(w[i]);
  }
}

// grid (H, B): one query (the new token) against the cache rows 0..lens[b].
// Logits fp32 (dot products over c ascending), softmax with the block max,
// exponentials summed per thread in key order then in a fixed tree; P.V in
// fp32: thread t sums keys j = g, g + G, ... (g = t / dh, G = 256 / dh) for
// column t % dh, the G partial sums added in order, one division.
template <typename AT>
__global__ void __launch_bounds__(256) decode_attention_kernel(const AT* __restrict__ Q, const AT* __restrict__ ck,
                                                               const AT* __restrict__ cv, int64_t layer_off, int cap,
                                                               const int32_t* __restrict__ lens, int d, int dh,
                                                               float scale, AT* __restrict__ O) {
  // One block per (head, sample).  Scores: a thread per cached key, its row
  // read as 16-byte vectors all in flight (dh <= 256).  P V: a thread per
  // (group of VE columns, key group), its keys strided by the number of key
  // groups; the key groups are combined in fixed order through LDS.
  constexpr int VE = 16 / sizeof(AT);  // elements per 16-byte vector
  __shared__ float qs[kDecodeMaxDh];
  __shared__ float z[kDecodeMaxKeys];
  __shared__ float red[4];
  __shared__ float part[256 * VE];
  const int h = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lens[b] + 1;
  const int nv = dh / VE;  // vectors per row
  for (int c = tid; c < dh; c += 256) qs[c] = act_load<AT>(Q + (int64_t)b * d + h * dh + c);
  __syncthreads();
  const AT* kb = ck + layer_off + (int64_t)b * cap * d + h * dh;
  const AT* vb = cv + layer_off + (int64_t)b * cap * d + h * dh;
  // P V work split (below); this thread's first PF value vectors are loaded
  // now, so their latency overlaps the scores and the softmax
  constexpr int PF = 16;
  const int ng = 256 / nv;  // key groups
  const int cg = tid % nv, kg = tid / nv;
  uint4 vpre[PF];
#pragma unroll
  for (int u = 0; u < PF; ++u) {
    const int j = kg + u * ng;
    vpre[u] = (kg < ng && j < n) ? reinterpret_cast<const uint4*>(vb + (int64_t)j * d)[cg] : make_uint4(0, 0, 0, 0);
  }
  float mx = -INFINITY;
  for (int j = tid; j < n; j += 256) {
    const uint4* kr = reinterpret_cast<const uint4*>(kb + (int64_t)j * d);
    float acc = 0.f;
    for (int q0 = 0; q0 < nv; q0 += 16) {  // 16 vectors (256 B) of the row in flight
      uint4 kv[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) kv[u] = q0 + u < nv ? kr[q0 + u] : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        if (q0 + u >= nv) break;
        float x[VE];
        unpack16<AT>(kv[u], x);
#pragma unroll
        for (int e = 0; e < VE; ++e) acc = fmaf(qs[(q0 + u) * VE + e], x[e], acc);
      }
    }
    const float v = acc * scale;
    z[j] = v;
    mx = fmaxf(mx, v);
  }
  mx = wave_max(mx);
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float s = 0.f;
  for (int j = tid; j < n; j += 256) {
    const float e = expf(z[j] - mx);
    z[j] = e;
    s += e;
  }
  s = wave_sum(s);
  if (lane == 0) red[wave] = s;
  __syncthreads();
  s = (red[0] + red[1]) + (red[2] + red[3]);
  float acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.f;
  if (kg < ng) {
    // keys kg, kg + ng, ... in increasing order: the prefetched ones first
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int j = kg + u * ng;
      if (j >= n) break;
      float x[VE];
      unpack16<AT>(vpre[u], x);
      const float p = z[j];
#pragma unroll
      for (int e = 0; e < VE; ++e) acc[e] = fmaf(p, x[e], acc[e]);
    }
    for (int j0 = kg + PF * ng; j0 < n; j0 += 4 * ng) {
      uint4 vv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = j0 + u * ng;
        if (j < n) vv[u] = reinterpret_cast<const uint4*>(vb + (int64_t)j * d)[cg];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = j0 + u * ng;
        if (j >= n) break;
        float x[VE];
        unpack16<AT>(vv[u], x);
        const float p = z[j];
#pragma unroll
        for (int e = 0; e < VE; ++e) acc[e] = fmaf(p, x[e], acc[e]);
      }
    }
  }
  if (kg < ng) {
#pragma unroll
    for (int e = 0; e < VE; ++e) part[kg * dh + cg * VE + e] = acc[e];
  }
  __syncthreads();
  for (int c = tid; c < dh; c += 256) {
    float o = part[c];
    for (int g = 1; g < ng; ++g) o += part[g * dh + c];
    Act<AT>::store(O + (int64_t)b * d + h * dh + c, __fdiv_rn(o, s));
  }
}

// One block per row: logits = the split partials summed in order; the arg max
// (ties to the lowest id) by a per-thread scan in id order and a fixed tree.
__global__ void __launch_bounds__(256) logits_argmax_kernel(const float* __restrict__ P, int split, int64_t pstride,
                                                            int V, float* __restrict__ logits,
                                                            int32_t* __restrict__ next) {
  __shared__ float bv[256];
  __shared__ int bi[256];
  const int b = blockIdx.x, tid = threadIdx.x;
  float best = -INFINITY;
  int arg = 0x7fffffff;
  if (split == 1 && V % 4 == 0) {
    // float4 pieces 4t, 4t + 1024, ...: four in flight, ids still ascending per thread
    const float4* P4 = reinterpret_cast<const float4*>(P + (int64_t)b * V);
    const int V4 = V / 4;
    for (int v0 = tid; v0 < V4; v0 += 1024) {
      float4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (v0 + 256 * u < V4) x[u] = P4[v0 + 256 * u];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v4 = v0 + 256 * u;
        if (v4 >= V4) break;
        if (logits) reinterpret_cast<float4*>(logits + (int64_t)b * V)[v4] = x[u];
        const float e[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (e[k] > best) {
            best = e[k];
            arg = 4 * v4 + k;
          }
      }
    }
  } else {
    for (int v = tid; v < V; v += 256) {
      float x = 0.f;
      for (int s = 0; s < split; ++s) x += P[s * pstride + (int64_t)b * V + v];
      if (logits) logits[(int64_t)b * V + v] = x;
      if (x > best) {
        best = x;
        arg = v;
      }
    }
  }
  bv[tid] = best;
  bi[tid] = arg;
  __syncthreads();
  for (int o = 128; o >= 1; o >>= 1) {
    if (tid < o) {
      const float x = bv[tid + o];
      const int i = bi[tid + o];
      if (x > bv[tid] || (x == bv[tid] && i < bi[tid])) {
        bv[tid] = x;
        bi[tid] = i;
      }
    }
    __syncthreads();
  }
  if (tid == 0 && next) next[b] = bi[0];
}

// Index of this thread among the block's threads with `on` set (thread
// order), and their number in `total`.  256 threads; every thread calls it.
__device__ int block_rank(bool on, int* wtot, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(on);
  const int below = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wtot[wave] = __popcll(m);
  __syncthreads();
  int base = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    base += w < wave ? wtot[w] : 0;
    total += wtot[w];
  }
  __syncthreads();
  return base + below;
}

// Bookkeeping of the online controller for layer l, on the device: one block,
// one thread per packed row (R <= 256).  For l inside the decision window it
// applies the layer's admissions (candidate c with flag[c] set: admit[row] =
// l, the frozen target's bypass bit joins the row's code), writes every row's
// code for layers l..L-1, builds layer l's row lists in `reg` (attention rows,
// row -> slot map, FFN rows, row -> slot map; R ints each, rows in order) with
// their counts at cnt[2 (l & 1)], and for l + 1 inside the window the next
// candidate list (visual rows not admitted yet: cand[i] = row, cand[R + i] =
// its sample) with its count at cnt[4].  l = -1 initialises the row state and
// builds the candidate list of layer 0.
__global__ void __launch_bounds__(256) online_plan_kernel(int l, int L, int Wn, int R, int bit,
                                                          const int32_t* __restrict__ vis,
                                                          const int32_t* __restrict__ flag,
                                                          int32_t* __restrict__ cand, int32_t* __restrict__ admit,
                                                          int32_t* __restrict__ code, uint8_t* __restrict__ codes,
                                                          int32_t* __restrict__ reg, int32_t* __restrict__ cnt) {
  __shared__ int wtot[4];
  __shared__ int s_admit[256], s_code[256];
  const int r = threadIdx.x;
  const bool row = r < R;
  if (row) {
    s_admit[r] = l < 0 ? -1 : admit[r];
    s_code[r] = l < 0 ? 0 : code[r];
  }
  const int nc = (l >= 0 && l < Wn) ? cnt[4] : 0;
  const bool adm = r < nc && flag[r] != 0;
  const int arow = adm ? cand[r] : 0;
  __syncthreads();
  if (adm) {
    s_admit[arow] = l;
    s_code[arow] |= bit;
  }
  __syncthreads();
  const int a_r = row ? s_admit[r] : 0, c_r = row ? s_code[r] : 0;
  if (row) {
    admit[r] = a_r;
    code[r] = c_r;
  }
  if (l >= 0) {
    if (row)
      for (int l2 = l; l2 < L; ++l2) codes[(size_t)l2 * R + r] = (uint8_t)c_r;
    const bool onA = row && !(c_r & 1), onF = row && !(c_r & 2);
    int nA, nF;
    const int iA = block_rank(onA, wtot, nA);
    const int iF = block_rank(onF, wtot, nF);
    if (row) {
      if (onA) reg[iA] = r;
      reg[R + r] = onA ? iA : -1;
      if (onF) reg[2 * R + iF] = r;
      reg[3 * R + r] = onF ? iF : -1;
    }
    if (r == 0) {
      cnt[2 * (l & 1)] = nA;
      cnt[2 * (l & 1) + 1] = nF;
    }
  }
  if (l + 1 < Wn) {
    const bool on = row && vis[r] >= 0 && a_r < 0;
    int n;
    const int i = block_rank(on, wtot, n);
    if (on) {
      cand[i] = r;
      cand[R + i] = vis[r];
    }
    if (r == 0) cnt[4] = n;
  }
}

// ------------------------------------------------------------------ host side
struct LayerTables {
  int nA = 0, nF = 0;
  int offA = -1, offF = -1;         // offsets of the row lists (ints)
  int offSlotA = -1, offSlotF = -1;  // offsets of the row -> slot maps
  // >= 0: the live counts (attention rows, FFN rows) are the two ints at this
  // offset on the device, and nA, nF are the bounds the launches are sized for
  int offCnt = -1;
};

// Pinned host buffer for the row tables of one thread's prefill calls.  It is
// reused once the previous upload has completed (event), and is deliberately
// not released at thread exit (the HIP runtime may already be shut down
// then); the OS reclaims it with the process.
struct Staging {
  void* host = nullptr;
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};
thread_local Staging g_stage;

// Pinned host buffer for the admission flags read back by the online controller.
struct Readback {
  void* host = nullptr;
  size_t cap = 0;
};
thread_local Readback g_back;

#define SPIDER_TRY(expr)                 \
  do {                                   \
    spider_status s_ = (expr);           \
    if (s_ != SPIDER_OK) return s_;      \
  } while (0)

// Copies n ints from host memory to dst (device) on st through the pinned
// staging buffer; returns once the copy is enqueued.
spider_status upload_ints(const int32_t* src, size_t n, int32_t* dst, hipStream_t st) {
  const size_t bytes = n * sizeof(int32_t);
  if (bytes == 0) return SPIDER_OK;
  if (g_stage.pending) {
    SPIDER_HIP(hipEventSynchronize(g_stage.ev));
    g_stage.pending = false;
  }
  if (g_stage.cap < bytes) {
    if (g_stage.host) SPIDER_HIP(hipHostFree(g_stage.host));
    g_stage.host = nullptr;
    g_stage.cap = 0;
    SPIDER_HIP(hipHostMalloc(&g_stage.host, bytes));
    g_stage.cap = bytes;
  }
  if (!g_stage.ev) SPIDER_HIP(hipEventCreateWithFlags(&g_stage.ev, hipEventDisableTiming));
  std::memcpy(g_stage.host, src, bytes);
  SPIDER_HIP(hipMemcpyAsync(dst, g_stage.host, bytes, hipMemcpyHostToDevice, st));
  SPIDER_HIP(hipEventRecord(g_stage.ev, st));
  g_stage.pending = true;
  return SPIDER_OK;
}

// Row lists of layers appended to `tab`: for each sub-layer the rows whose
// code lacks its bypass bit, then the row -> slot map (-1 for bypassing rows).
// Layers with identical sets share one list.  Offsets are relative to the
// device table base; tab[0] sits at offset `base`.
struct TableBuilder {
  std::vector<int32_t>& tab;
  int base;
  std::map<std::string, std::pair<int, int>> seen[2];
  // whole code columns already added (hash -> column, its tables): a layer
  // whose column repeats an earlier one reuses its tables without rebuilding
  // the per-sub-layer keys (R bytes each)
  std::multimap<uint64_t, std::pair<const uint8_t*, LayerTables>> cols;

  static uint64_t hash_col(const uint8_t* p, int n) {
    uint64_t h = 1469598103934665603ull;  // FNV-1a offset basis
    int i = 0;
    for (; i + 8 <= n; i += 8) {
      uint64_t w;
      std::memcpy(&w, p + i, 8);
      h = (h ^ w) * 1099511628211ull;
    }
    for (; i < n; ++i) h = (h ^ p[i]) * 1099511628211ull;
    return h;
  }

  LayerTables add(const uint8_t* col, int R) {
    const uint64_t hc = hash_col(col, R);
    for (auto [it, end] = cols.equal_range(hc); it != end; ++it)
      if (std::memcmp(it->second.first, col, (size_t)R) == 0) return it->second.second;
    const LayerTables t = add_new(col, R);
    cols.emplace(hc, std::make_pair(col, t));
    return t;
  }

  LayerTables add_new(const uint8_t* col, int R) {
    LayerTables t;
    for (int which = 0; which < 2; ++which) {
      const uint8_t bit = which == 0 ? 1 : 2;
      std::string key(R, '\0');
      int cnt = 0;
      for (int r = 0; r < R; ++r) {
        const bool active = !(col[r] & bit);
        key[r] = active ? 1 : 0;
        cnt += active;
      }
      auto it = seen[which].find(key);
      std::pair<int, int> offs;
      if (it != seen[which].end()) {
        offs = it->second;
      } else {
        const int off_list = base + (int)tab.size();
        for (int r = 0; r < R; ++r)
          if (key[r]) tab.push_back(r);
        const int off_slot = base + (int)tab.size();
        int s = 0;
        for (int r = 0; r < R; ++r) tab.push_back(key[r] ? s++ : -1);
        offs = {off_list, off_slot};
        seen[which][key] = offs;
      }
      if (which == 0) {
        t.nA = cnt;
        t.offA = offs.first;
        t.offSlotA = offs.second;
      } else {
        t.nF = cnt;
        t.offF = offs.first;
        t.offSlotF = offs.second;
      }
    }
    return t;
  }
};

int split_max_for_rows(int R) { return std::max(1, std::min(8, 4096 / std::max(1, R))); }

struct PrefillWs {
  int32_t* tables;
  float2* rope;
  void *xn, *q, *k, *v, *o, *act;
  float *Pq, *Pk, *Pv, *Pres;
  size_t bytes;
};

// Rows of the transposed V buffer: R rounded up to the 32-key blocks of attention.
int vt_rows(int R) { return (R + 31) / 32 * 32; }

size_t table_ints_bound(int L, int R) { return (size_t)R * 3 + (size_t)L * 4 * R + 64; }

struct Carver {
  char* base;
  size_t off = 0;
  void* take(size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return base ? base + o : nullptr;
  }
};

PrefillWs prefill_layout(const spider_decoder_cfg& c, int R, Carver& cv) {
  PrefillWs w{};
  const size_t es = c.dtype == SPIDER_BF16 ? 2 : 4;
  const int dh = c.d / c.H;
  const int sm = split_max_for_rows(R);
  w.tables = reinterpret_cast<int32_t*>(cv.take(table_ints_bound(c.L, R) * 4));
  w.rope = reinterpret_cast<float2*>(cv.take((size_t)R * (dh / 2) * sizeof(float2)));
  w.xn = cv.take((size_t)R * c.d * es);
  w.q = cv.take((size_t)R * c.d * es);
  w.k = cv.take((size_t)R * c.d * es);
  w.v = cv.take((size_t)vt_rows(R) * c.d * es);  // bf16: V^T [d][vt_rows(R)]
  w.o = cv.take((size_t)R * c.d * es);
  w.act = cv.take((size_t)R * c.d_ff * es);
  w.Pq = reinterpret_cast<float*>(cv.take((size_t)sm * R * c.d * 4));
  w.Pk = reinterpret_cast<float*>(cv.take((size_t)sm * R * c.d * 4));
  w.Pv = reinterpret_cast<float*>(cv.take((size_t)sm * R * c.d * 4));
  w.Pres = reinterpret_cast<float*>(cv.take((size_t)sm * R * c.d * 4));
  w.bytes = cv.off;
  return w;
}

PrefillWs prefill_layout(const spider_decoder_cfg& c, int R, char* base) {
  Carver cv{base};
  return prefill_layout(c, R, cv);
}

// Integer tables of the online prefill (offsets in ints from the table base):
// positions, sample starts, cu_seqlens, the sample of every visual row (-1
// for text rows), two regions for the row lists of the current layer
// (alternating, so the slot map of the previous layer's pending residual stays
// intact until it is consumed), the candidate list and the sample of each
// candidate; then the row state kept on the device when the bookkeeping runs
// there: admission layer and code per row, the list counts (attention and FFN
// rows of the two regions, candidates) and the codes [L][R] as bytes.
struct OnlineTabs {
  int pos, start, cu, vis, reg[2], cand, admit, code, cnt, codes, total;
};

OnlineTabs online_tabs(int R, int B, int L) {
  OnlineTabs t;
  t.pos = 0;
  t.start = R;
  t.cu = 2 * R;
  t.vis = 2 * R + B + 1;
  t.reg[0] = (3 * R + B + 1 + 63) / 64 * 64;
  t.reg[1] = t.reg[0] + 4 * R;
  t.cand = t.reg[1] + 4 * R;
  t.admit = t.cand + 2 * R;
  t.code = t.admit + R;
  t.cnt = t.code + R;
  t.codes = t.cnt + 8;
  t.total = t.codes + (int)(((int64_t)L * R + 3) / 4);
  return t;
}

struct OnlineWs {
  PrefillWs p;
  int32_t* tab;   // OnlineTabs
  void* hc;       // [R, d] candidate rows in the activation dtype
  float* tmean;   // [B, d] text mean per sample
  double* F;      // [R] F_itc per candidate
  float* logits;  // [R, V] logit lens of the candidates (unfused path), else null
  float* stats;   // [R, V/128, 4] per-tile softmax statistics (fused bf16 path), else null
  double* acc;    // [R] accumulated skip score per packed row
  int32_t* flag;  // [R] admission flag per candidate
  size_t bytes;
};

// bf16 with V a multiple of 128: the lens GEMM's epilogue reduces each row's
// 128-column tiles to softmax statistics (no logits in memory); otherwise
// the GEMM writes fp32 logits and a separate kernel reduces them.
bool lens_fused(const spider_decoder_cfg& c, int V) { return c.dtype == SPIDER_BF16 && V % 128 == 0; }

OnlineWs online_layout(const spider_decoder_cfg& c, int B, int R, int V, char* base) {
  Carver cv{base};
  OnlineWs w{};
  w.p = prefill_layout(c, R, cv);
  const size_t es = c.dtype == SPIDER_BF16 ? 2 : 4;
  w.tab = reinterpret_cast<int32_t*>(cv.take((size_t)online_tabs(R, B, c.L).total * 4));
  w.hc = cv.take((size_t)R * c.d * es);
  w.tmean = reinterpret_cast<float*>(cv.take((size_t)B * c.d * 4));
  w.F = reinterpret_cast<double*>(cv.take((size_t)R * 8));
  if (lens_fused(c, V))
    w.stats = reinterpret_cast<float*>(cv.take((size_t)R * (V / 128) * 16));
  else
    w.logits = reinterpret_cast<float*>(cv.take((size_t)R * V * 4));
  w.acc = reinterpret_cast<double*>(cv.take((size_t)R * 8));
  w.flag = reinterpret_cast<int32_t*>(cv.take((size_t)R * 4));
  w.bytes = cv.off;
  return w;
}

spider_status validate_cfg(const spider_decoder_cfg* cfg) {
  SPIDER_REQUIRE(cfg, SPIDER_ERR_INVALID_ARG, "spider_prefill: cfg is null");
  SPIDER_REQUIRE(cfg->L >= 1 && cfg->d >= 1 && cfg->H >= 1 && cfg->d_ff >= 1,
                 SPIDER_ERR_INVALID_ARG, "spider_prefill: L, d, H, d_ff must be >= 1");
  SPIDER_REQUIRE(cfg->d % cfg->H == 0, SPIDER_ERR_SHAPE, "spider_prefill: d must be divisible by H");
  const int dh = cfg->d / cfg->H;
  SPIDER_REQUIRE(dh % 2 == 0, SPIDER_ERR_SHAPE, "spider_prefill: dh must be even");
  SPIDER_REQUIRE(cfg->dtype == SPIDER_F32 || cfg->dtype == SPIDER_BF16, SPIDER_ERR_INVALID_ARG,
                 "spider_prefill: bad dtype");
  SPIDER_REQUIRE(cfg->d % 4 == 0 && cfg->d <= 8192, SPIDER_ERR_UNSUPPORTED,
                 "spider_prefill: d must be a multiple of 4 and at most 8192");
  SPIDER_REQUIRE(std::isfinite(cfg->eps) && cfg->eps >= 0.f && std::isfinite(cfg->theta) &&
                     cfg->theta > 0.f,
                 SPIDER_ERR_INVALID_ARG, "spider_prefill: eps must be >= 0 and theta > 0");
  if (cfg->dtype == SPIDER_BF16) {
    SPIDER_REQUIRE(dh == 128, SPIDER_ERR_UNSUPPORTED, "spider_prefill: bf16 path needs dh == 128");
    SPIDER_REQUIRE(cfg->d % 64 == 0 && cfg->d_ff % 64 == 0, SPIDER_ERR_UNSUPPORTED,
                   "spider_prefill: bf16 path needs d and d_ff multiples of 64");
  } else {
    SPIDER_REQUIRE(dh <= 256, SPIDER_ERR_UNSUPPORTED, "spider_prefill: fp32 path needs dh <= 256");
  }
  return SPIDER_OK;
}

// Argument checks shared by both prefill entry points (rows = cu_seqlens[B] > 0).
spider_status validate_prefill_args(const spider_decoder_cfg* cfg, const spider_layer_weights* layers,
                                    const void* x, const float* h_out) {
  SPIDER_REQUIRE(x && h_out, SPIDER_ERR_INVALID_ARG, "spider_prefill: x and h_out must be non-null");
  for (int l = 0; l < cfg->L; ++l) {
    const spider_layer_weights& w = layers[l];
    SPIDER_REQUIRE(w.attn_norm && w.wq && w.wk && w.wv && w.wo && w.ffn_norm && w.wg && w.wu && w.wd,
                   SPIDER_ERR_INVALID_ARG, "spider_prefill: null weight pointer in layer %d", l);
  }
  SPIDER_REQUIRE(((uintptr_t)h_out % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                 "spider_prefill: h_out must be 16-byte aligned");
  for (int l = 0; l < cfg->L; ++l)
    SPIDER_REQUIRE(((uintptr_t)layers[l].attn_norm % 16) == 0 &&
                       ((uintptr_t)layers[l].ffn_norm % 16) == 0,
                   SPIDER_ERR_UNSUPPORTED, "spider_prefill: norm weights must be 16-byte aligned");
  if (cfg->dtype == SPIDER_BF16) {
    SPIDER_REQUIRE(((uintptr_t)x % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                   "spider_prefill: x must be 16-byte aligned");
    for (int l = 0; l < cfg->L; ++l) {
      const spider_layer_weights& w = layers[l];
      const void* m[7] = {w.wq, w.wk, w.wv, w.wo, w.wg, w.wu, w.wd};
      for (int i = 0; i < 7; ++i)
        SPIDER_REQUIRE(((uintptr_t)m[i] % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                       "spider_prefill: weight matrices must be 16-byte aligned (layer %d)", l);
    }
  }
  return SPIDER_OK;
}

spider_status validate_cu(int B, const int32_t* cu_seqlens, const spider_layer_weights* layers) {
  SPIDER_REQUIRE(B >= 1, SPIDER_ERR_INVALID_ARG, "spider_prefill: B must be >= 1");
  SPIDER_REQUIRE(cu_seqlens && layers, SPIDER_ERR_INVALID_ARG,
                 "spider_prefill: cu_seqlens and layers must be non-null");
  SPIDER_REQUIRE(cu_seqlens[0] == 0, SPIDER_ERR_SHAPE, "spider_prefill: cu_seqlens[0] must be 0");
  for (int b = 0; b < B; ++b)
    SPIDER_REQUIRE(cu_seqlens[b + 1] >= cu_seqlens[b], SPIDER_ERR_SHAPE,
                   "spider_prefill: cu_seqlens must be non-decreasing");
  return SPIDER_OK;
}

// The layer forward of one prefill call.  Row tables live in device memory
// at `tab` (LayerTables offsets are relative to it); the residual partials of
// the last O or down GEMM stay pending until the next norm (or flush) adds
// them to h.
template <typename AT>
struct PrefillRun {
  const spider_decoder_cfg& c;
  const spider_layer_weights* W;
  float* h;
  const PrefillWs& ws;
  const int32_t* tab;
  const int32_t* dpos;    // [R] position of each row within its sample
  const int32_t* dstart;  // [R] first row of the sample that owns each row
  int R, max_s;
  hipStream_t st;
  int pend_split = 0;
  int64_t pend_stride = 0;  // elements between the pending partial slabs
  const int32_t* pend_slot = nullptr;
  // optional KV cache output ([L][B][cap][d]) and the sample of every row
  AT* ck = nullptr;
  AT* cv = nullptr;
  int kv_cap = 0, kv_B = 0;
  const int32_t* row_sample = nullptr;

  bool bf16() const { return c.dtype == SPIDER_BF16; }
  int64_t pstride() const { return (int64_t)R * c.d; }

  int split_cap(int cap) const { return std::min(split_max_for_rows(R), cap); }
  // Split-K cap of a residual launch (O, down) over `rows` rows whose partial
  // slabs are packed at rows * d: the residual buffer holds
  // split_max_for_rows(R) * R rows of partials, so a layer with few active
  // rows (e.g. only the text rows) may split as far as the streaming kernel
  // wants even when R is large.
  int split_cap_rows(int cap, int rows) const {
    const int64_t slots = (int64_t)split_max_for_rows(R) * R;
    return (int)std::max<int64_t>(1, std::min<int64_t>(std::min(cap, 8), slots / std::max(1, rows)));
  }
  hipError_t gemm(GemmArgs& ga, int cap) {
    const int sm = split_cap(cap);
    return bf16() ? launch_gemm_bf16(ga, sm, st) : launch_gemm_f32(ga, sm, st);
  }

  // RoPE table and h = x
  spider_status begin(const void* x) {
    const int half = c.d / c.H / 2, dh = c.d / c.H;
    {
      const int64_t n = (int64_t)max_s * half;
      rope_table_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(ws.rope, max_s, half, dh,
                                                                    std::log2((double)c.theta));
      SPIDER_LAUNCHED("rope_table");
    }
    {
      ProfScope ps(KC_EMBED, st);
      const int64_t n = (int64_t)R * c.d;
      embed_kernel<AT><<<(unsigned)((n + 255) / 256), 256, 0, st>>>(reinterpret_cast<const AT*>(x), h, n);
      SPIDER_LAUNCHED("embed");
    }
    return SPIDER_OK;
  }

  // adds the pending residual partials to h
  spider_status flush() {
    if (pend_split == 0) return SPIDER_OK;
    ProfScope ps(KC_RESIDUAL, st);
    launch_norm<AT>(R, h, c.d, ws.Pres, pend_split, pend_stride, pend_slot, nullptr, 0.f, nullptr, 0,
                    static_cast<AT*>(nullptr), st);
    SPIDER_LAUNCHED("residual_add");
    pend_split = 0;
    pend_slot = nullptr;
    return SPIDER_OK;
  }

  spider_status layer(int l, const LayerTables& T) {
    const spider_layer_weights& w = W[l];
    const int d = c.d, dh = d / c.H;
    const int32_t* cntA = T.offCnt >= 0 ? tab + T.offCnt : nullptr;
    const int32_t* cntF = T.offCnt >= 0 ? tab + T.offCnt + 1 : nullptr;
    const int64_t ps_ = pstride();
    AT* xn = reinterpret_cast<AT*>(ws.xn);
    AT* qb = reinterpret_cast<AT*>(ws.q);
    AT* kb = reinterpret_cast<AT*>(ws.k);
    AT* vb = reinterpret_cast<AT*>(ws.v);
    AT* ob = reinterpret_cast<AT*>(ws.o);
    AT* act = reinterpret_cast<AT*>(ws.act);
    // split-K caps: the QKV partials are re-read by the finalize kernel and the
    // O/down partials by the next norm, so splitting is kept modest.  With a KV
    // cache the keys and values are produced in every layer, also where no row
    // is a query.
    if (T.nA > 0 || ck) {
      {
        ProfScope ps(KC_RMSNORM, st);
        launch_norm<AT>(R, h, d, ws.Pres, pend_split, pend_stride, pend_slot, w.attn_norm, c.eps, nullptr, 1,
                        xn, st);
        SPIDER_LAUNCHED("rmsnorm(attn)");
        pend_split = 0;
        pend_slot = nullptr;
      }
      GemmArgs ga{};
      ga.K = d;
      ga.lda = d;
      ga.epilogue = EPI_PARTIAL_F32;
      const GemmGroup gk{xn, nullptr, R, w.wk, nullptr, d, ws.Pk, d, ps_, 0, 0, 0};
      const GemmGroup gv{xn, nullptr, R, w.wv, nullptr, d, ws.Pv, d, ps_, 0, 0, 0};
      if (T.nA > 0) {
        ga.ngroups = 3;
        ga.g[0] = GemmGroup{xn, tab + T.offA, T.nA, w.wq, nullptr, d, ws.Pq, d, ps_, 0, 0, 0};
        ga.g[0].m_dev = cntA;
        ga.g[1] = gk;
        ga.g[2] = gv;
      } else {
        ga.ngroups = 2;
        ga.g[0] = gk;
        ga.g[1] = gv;
      }
      // Without a cache and with the tile kernel unsplit (many rows), the
      // GEMM's epilogue applies RoPE and writes bf16 Q, K and V^T itself:
      // no fp32 round trip and no finalize launch.
      const bool fused = bf16() && !ck && dh == 128 && gemm_tile_unsplit_blocks(ga, split_cap(2)) > 0;
      if (fused) {
        ga.epilogue = EPI_QKV_BF16;
        ga.rope = ws.rope;
        ga.pos = dpos;
        ga.ldvt = vt_rows(R);
        void* outs[3] = {qb, kb, vb};
        const int kinds[3] = {1, 1, 2};
        const int first = ga.ngroups == 3 ? 0 : 1;
        for (int i = 0; i < ga.ngroups; ++i) {
          ga.g[i].out = outs[first + i];
          ga.g[i].kind = kinds[first + i];
        }
      }
      {
        ProfScope ps(KC_GEMM_QKV, st);
        hipError_t e = gemm(ga, 2);
        SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "gemm_qkv: %s", hipGetErrorString(e));
      }
      if (!fused) {
        ProfScope ps(KC_QKV_FINALIZE, st);
        const int64_t ldvt = bf16() ? vt_rows(R) : 0;
        const int vblocks = bf16() ? (vt_rows(R) / 32) * (d / 64) : R;
        qkv_finalize_kernel<AT><<<T.nA + R + vblocks, 256, 0, st>>>(
            ws.Pq, ws.Pk, ws.Pv, ga.split, ps_, T.nA, R, d, dh, tab + T.offA, dpos, ws.rope, qb, kb, vb,
            ldvt, cntA);
        SPIDER_LAUNCHED("qkv_finalize");
        if (ck) {
          kv_store_kernel<AT><<<R, 256, 0, st>>>(kb, ws.Pv, ga.split, ps_, d, row_sample, dpos, ck, cv,
                                                 (int64_t)l * kv_B * kv_cap * d, kv_cap);
          SPIDER_LAUNCHED("kv_store");
        }
      }
    }
    if (T.nA > 0) {
      {
        ProfScope ps(KC_ATTENTION, st);
        AttnArgs aa{qb, tab + T.offA, kb, vb, bf16() ? (int64_t)vt_rows(R) : 0, dstart, ob, T.nA, R,
                    c.H, dh, d, (float)(1.0 / std::sqrt((double)dh)), cntA};
        hipError_t e = bf16() ? launch_attention_bf16(aa, st) : launch_attention_f32(aa, max_s, st);
        SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "attention: %s", hipGetErrorString(e));
      }
      GemmArgs go{};
      go.ngroups = 1;
      go.K = d;
      go.lda = d;
      go.epilogue = EPI_PARTIAL_F32;
      go.g[0] = GemmGroup{ob, nullptr, T.nA, w.wo, nullptr, d, ws.Pres, d, (int64_t)T.nA * d, 0, 0, 0};
      go.g[0].m_dev = cntA;
      {
        ProfScope ps(KC_GEMM_O, st);
        hipError_t e = bf16() ? launch_gemm_bf16(go, split_cap_rows(8, T.nA), st)
                              : launch_gemm_f32(go, split_cap_rows(8, T.nA), st);
        SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "gemm_o: %s", hipGetErrorString(e));
      }
      pend_split = go.split;
      pend_stride = go.g[0].split_stride;
      pend_slot = tab + T.offSlotA;
    }
    if (T.nF > 0) {
      {
        ProfScope ps(KC_RMSNORM, st);
        launch_norm<AT>(R, h, d, ws.Pres, pend_split, pend_stride, pend_slot, w.ffn_norm, c.eps,
                        tab + T.offSlotF, 0, xn, st);
        SPIDER_LAUNCHED("rmsnorm(ffn)");
        pend_split = 0;
        pend_slot = nullptr;
      }
      GemmArgs gu{};
      gu.ngroups = 1;
      gu.K = d;
      gu.lda = d;
      gu.epilogue = EPI_SWIGLU;
      gu.g[0] = GemmGroup{xn, nullptr, T.nF, w.wg, w.wu, c.d_ff, act, c.d_ff, 0, 0, 0, 0};
      gu.g[0].m_dev = cntF;
      // the QKV partials are consumed before attention: free scratch for the
      // GEMM's split tail tiles until the next layer's QKV GEMM
      gu.scratch = ws.Pq;
      gu.scratch_bytes = (size_t)split_max_for_rows(R) * R * c.d * 4;
      {
        ProfScope ps(KC_GEMM_GATEUP, st);
        hipError_t e = gemm(gu, 1);
        SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "gemm_gateup: %s", hipGetErrorString(e));
      }
      GemmArgs gd{};
      gd.ngroups = 1;
      gd.K = c.d_ff;
      gd.lda = c.d_ff;
      gd.epilogue = EPI_PARTIAL_F32;
      gd.g[0] = GemmGroup{act, nullptr, T.nF, w.wd, nullptr, d, ws.Pres, d, (int64_t)T.nF * d, 0, 0, 0};
      gd.g[0].m_dev = cntF;
      {
        ProfScope ps(KC_GEMM_DOWN, st);
        hipError_t e = bf16() ? launch_gemm_bf16(gd, split_cap_rows(8, T.nF), st)
                              : launch_gemm_f32(gd, split_cap_rows(8, T.nF), st);
        SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "gemm_down: %s", hipGetErrorString(e));
      }
      pend_split = gd.split;
      pend_stride = gd.g[0].split_stride;
      pend_slot = tab + T.offSlotF;
    }
    return SPIDER_OK;
  }
};

// positions within the sample and sample starts of every row; returns the
// longest sample
int fill_positions(int B, const int32_t* cu, int32_t* pos, int32_t* start) {
  int max_s = 1;
  for (int b = 0; b < B; ++b) {
    max_s = std::max(max_s, cu[b + 1] - cu[b]);
    for (int r = cu[b]; r < cu[b + 1]; ++r) {
      pos[r] = r - cu[b];
      start[r] = cu[b];
    }
  }
  return max_s;
}

template <typename AT>
spider_status run_prefill(const spider_decoder_cfg& c, const spider_layer_weights* W, int B,
                          const int32_t* cu, const void* x, const uint8_t* codes, float* h,
                          const PrefillWs& ws, hipStream_t st, const spider_kv_cache* kv = nullptr) {
  const int R = cu[B];
  // tables: positions [R], sample starts [R], with a KV cache the sample of
  // every row [R], then the row lists of every layer
  std::vector<int32_t> tab;
  tab.reserve(table_ints_bound(c.L, R));
  tab.resize(kv ? 3 * R : 2 * R);
  const int max_s = fill_positions(B, cu, tab.data(), tab.data() + R);
  if (kv)
    for (int b = 0; b < B; ++b)
      for (int r = cu[b]; r < cu[b + 1]; ++r) tab[2 * R + r] = b;
  std::vector<LayerTables> lt(c.L);
  TableBuilder tb{tab, 0};
  for (int l = 0; l < c.L; ++l) lt[l] = tb.add(codes + (size_t)l * R, R);
  SPIDER_TRY(upload_ints(tab.data(), tab.size(), ws.tables, st));

  PrefillRun<AT> run{c, W, h, ws, ws.tables, ws.tables, ws.tables + R, R, max_s, st};
  if (kv) {
    run.ck = reinterpret_cast<AT*>(kv->k);
    run.cv = reinterpret_cast<AT*>(kv->v);
    run.kv_cap = kv->cap;
    run.kv_B = B;
    run.row_sample = ws.tables + 2 * R;
  }
  SPIDER_TRY(run.begin(x));
  for (int l = 0; l < c.L; ++l) SPIDER_TRY(run.layer(l, lt[l]));
  return run.flush();
}

struct OnlineParams {
  int n_text;
  const void* wu;
  int V;
  const double* slc_sel;
  const uint8_t* target;
  double w1, w2, t_skip;
  uint32_t ablation;  // SPIDER_ONLINE_* bits
  // code bits an admission at window layer l sets: the layer's SLC target, or
  // both sub-layers without SLC
  int bypass_bits(int l) const {
    return (ablation & SPIDER_ONLINE_WHOLE_LAYER) ? 3 : (target[l] == 1 ? 2 : 1);
  }
};

// Whether the online prefill keeps its bookkeeping on the device.  Needs at
// most 256 rows (one thread per row in online_plan_kernel); every GEMM of the
// call is then a streaming, LDS-staged or fp32 kernel whose split-K factor and
// per-element summation order do not depend on the row count, so launches
// sized for the bound and reading the live count on the device give the bits
// of launches sized for the live rows.  Text rows never bypass, so each
// sub-layer keeps at least B * n_text rows: five or more keep the static
// prefill off the decode-row kernel, which is also what the bf16 logits lens
// needs of its candidates.  The bf16 attention has to take its per-32-query
// kernel at the bound as it does at the live count.
bool online_on_device(const spider_decoder_cfg& c, int B, int R, int n_text, int nvis, int V) {
  if (R > 256 || (int64_t)B * n_text < 5) return false;
  if (c.dtype == SPIDER_BF16) {
    if ((int64_t)ceil_div(R, 128) * c.H >= 128) return false;
    if (!lens_fused(c, V) && nvis > 0 && nvis < 5) return false;
  }
  return true;
}

// Prefill with the online controller: at every layer l < floor(L/2) the
// visual rows not yet in skip mode are scored on the hidden state entering
// layer l, admitted rows get their frozen target bypassed from layer l on,
// and layer l runs with the updated row lists.
//
// Up to 256 rows (online_on_device) the admissions, codes, candidate lists and
// row lists stay on the device (online_plan_kernel after each window layer's
// lens); every launch of a window layer is sized for its bound and reads the
// live count, and the codes and admission layers come back once, at the end.
// Otherwise the admission flags come back to the host once per window layer
// (the stream is synchronised there) and the row lists are built there.
template <typename AT>
spider_status run_prefill_online(const spider_decoder_cfg& c, const spider_layer_weights* W, int B,
                                 const int32_t* cu, const void* x, const OnlineParams& op,
                                 uint8_t* codes, int32_t* admit_out, float* s_sa_out, float* h,
                                 const OnlineWs& ows, hipStream_t st) {
  const bool bf16 = c.dtype == SPIDER_BF16;
  const int R = cu[B], L = c.L, Wn = c.L / 2, d = c.d;
  const OnlineTabs ot = online_tabs(R, B, L);
  std::memset(codes, 0, (size_t)L * R);
  std::vector<int32_t> admit(R, -1);

  std::vector<int32_t> fixed(ot.reg[0], 0);
  const int max_s = fill_positions(B, cu, fixed.data() + ot.pos, fixed.data() + ot.start);
  std::copy(cu, cu + B + 1, fixed.begin() + ot.cu);
  int nvis = 0;
  for (int b = 0; b < B; ++b)
    for (int r = cu[b]; r < cu[b + 1]; ++r) {
      const bool visual = r < cu[b + 1] - op.n_text;
      fixed[ot.vis + r] = visual ? b : -1;
      nvis += visual;
    }
  const bool on_dev = online_on_device(c, B, R, op.n_text, nvis, op.V);
  SPIDER_TRY(upload_ints(fixed.data(), fixed.size(), ows.tab, st));

  PrefillRun<AT> run{c, W, h, ows.p, ows.tab, ows.tab + ot.pos, ows.tab + ot.start, R, max_s, st};
  SPIDER_TRY(run.begin(x));
  SPIDER_HIP(launch_fill_zero(ows.acc, (size_t)R * sizeof(double), st));
  if (s_sa_out && Wn > 0) SPIDER_HIP(launch_fill_zero(s_sa_out, (size_t)Wn * R * sizeof(float), st));

  int32_t* dcand = ows.tab + ot.cand;
  uint8_t* dcodes = reinterpret_cast<uint8_t*>(ows.tab + ot.codes);
  // Logit lens and admission test of layer l over `nc` candidates (with
  // nc_dev: a launch bound, the live count on the device); sets ows.flag.
  auto lens = [&](int l, int nc, const int32_t* nc_dev) -> spider_status {
    SPIDER_TRY(run.flush());
    {
      ProfScope ps(KC_LENS_PREP, st);
      hipError_t e = launch_text_mean(h, d, ows.tab + ot.cu, B, op.n_text, ows.tmean, st);
      if (e == hipSuccess)
        e = launch_lens_prep(bf16, h, d, dcand, dcand + (nc_dev ? R : nc), nc, nc_dev, ows.tmean, ows.hc,
                             ows.F, st);
      SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "lens_prep: %s", hipGetErrorString(e));
    }
    const bool fused = lens_fused(c, op.V);
    const int ntiles = op.V / 128;
    {
      ProfScope ps(KC_GEMM_LENS, st);
      GemmArgs gl{};
      gl.ngroups = 1;
      gl.K = d;
      gl.lda = d;
      hipError_t e = hipSuccess;
      if (fused) {
        // up to 256 candidates per launch (one pass over the unembedding each)
        const int nchunk = (nc + 255) / 256;
        const int per = (nc + nchunk - 1) / nchunk;
        gl.epilogue = EPI_LENS_STATS;
        for (int c0 = 0; c0 < nc && e == hipSuccess; c0 += per) {
          const int mc = std::min(per, nc - c0);
          GemmArgs gc = gl;
          gc.g[0] = GemmGroup{reinterpret_cast<const uint16_t*>(ows.hc) + (size_t)c0 * d, nullptr, mc,
                              op.wu, nullptr, op.V, ows.stats + (size_t)c0 * ntiles * 4, ntiles, 0,
                              0, 0, 0};
          gc.g[0].m_dev = nc_dev;  // one launch then (nc <= 256)
          e = launch_gemm_bf16(gc, 1, st);
        }
      } else {
        gl.epilogue = EPI_PARTIAL_F32;
        gl.g[0] = GemmGroup{ows.hc, nullptr, nc, op.wu, nullptr, op.V, ows.logits, op.V,
                            (int64_t)nc * op.V, 0, 0, 0};
        gl.g[0].m_dev = nc_dev;
        e = bf16 ? launch_gemm_bf16(gl, 1, st) : launch_gemm_f32(gl, 1, st);
      }
      SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "gemm_lens: %s", hipGetErrorString(e));
    }
    {
      ProfScope ps(KC_LENS_ADMIT, st);
      const double w2_sel = (op.ablation & SPIDER_ONLINE_WHOLE_LAYER) ? 0.0 : op.w2 * op.slc_sel[l];
      LensAdmitArgs p{std::log((double)op.V), op.w1, w2_sel, op.t_skip, ows.acc, ows.flag,
                      s_sa_out ? s_sa_out + (size_t)l * R : nullptr, op.ablation};
      hipError_t e = fused ? launch_lens_admit_stats(ows.stats, ntiles, dcand, nc, nc_dev, ows.F, p, st)
                           : launch_lens_admit(ows.logits, op.V, dcand, nc, nc_dev, ows.F, p, st);
      SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "lens_admit: %s", hipGetErrorString(e));
    }
    return SPIDER_OK;
  };
  auto grow_back = [&](size_t bytes) -> spider_status {
    if (g_back.cap < bytes) {
      if (g_back.host) SPIDER_HIP(hipHostFree(g_back.host));
      g_back.host = nullptr;
      g_back.cap = 0;
      SPIDER_HIP(hipHostMalloc(&g_back.host, bytes));
      g_back.cap = bytes;
    }
    return SPIDER_OK;
  };

  if (on_dev) {
    auto plan = [&](int l) -> spider_status {
      const int bit = (l >= 0 && l < Wn) ? op.bypass_bits(l) : 0;
      online_plan_kernel<<<1, 256, 0, st>>>(l, L, Wn, R, bit, ows.tab + ot.vis, ows.flag, dcand,
                                            ows.tab + ot.admit, ows.tab + ot.code, dcodes,
                                            ows.tab + ot.reg[l > 0 ? (l & 1) : 0], ows.tab + ot.cnt);
      SPIDER_LAUNCHED("online_plan");
      return SPIDER_OK;
    };
    SPIDER_TRY(plan(-1));
    LayerTables T;
    for (int l = 0; l < L; ++l) {
      if (l < Wn && nvis > 0) SPIDER_TRY(lens(l, nvis, ows.tab + ot.cnt + 4));
      if (l <= Wn) {
        SPIDER_TRY(plan(l));
        const int rg = ot.reg[l & 1];
        T.nA = T.nF = R;
        T.offA = rg;
        T.offSlotA = rg + R;
        T.offF = rg + 2 * R;
        T.offSlotF = rg + 3 * R;
        T.offCnt = ot.cnt + 2 * (l & 1);
      }
      SPIDER_TRY(run.layer(l, T));
    }
    SPIDER_TRY(run.flush());
    const size_t cbytes = (size_t)L * R, abytes = (size_t)R * sizeof(int32_t);
    SPIDER_TRY(grow_back(abytes + cbytes));
    uint8_t* back = reinterpret_cast<uint8_t*>(g_back.host);
    SPIDER_HIP(hipMemcpyAsync(back, ows.tab + ot.admit, abytes, hipMemcpyDeviceToHost, st));
    SPIDER_HIP(hipMemcpyAsync(back + abytes, dcodes, cbytes, hipMemcpyDeviceToHost, st));
    SPIDER_HIP(hipStreamSynchronize(st));
    std::memcpy(codes, back + abytes, cbytes);
    if (admit_out) std::memcpy(admit_out, back, abytes);
    return SPIDER_OK;
  }

  std::vector<int32_t> cand, lists;
  LayerTables T;
  for (int l = 0; l < L; ++l) {
    if (l < Wn) {
      cand.clear();
      for (int b = 0; b < B; ++b)
        for (int r = cu[b]; r < cu[b + 1] - op.n_text; ++r)
          if (admit[r] < 0) cand.push_back(r);
      const int nc = (int)cand.size();
      if (nc > 0) {
        for (int b = 0; b < B; ++b)
          for (int r = cu[b]; r < cu[b + 1] - op.n_text; ++r)
            if (admit[r] < 0) cand.push_back(b);
        SPIDER_TRY(upload_ints(cand.data(), cand.size(), dcand, st));
        SPIDER_TRY(lens(l, nc, nullptr));
        const size_t fbytes = (size_t)nc * sizeof(int32_t);
        SPIDER_TRY(grow_back(fbytes));
        SPIDER_HIP(hipMemcpyAsync(g_back.host, ows.flag, fbytes, hipMemcpyDeviceToHost, st));
        SPIDER_HIP(hipStreamSynchronize(st));
        const int32_t* flag = reinterpret_cast<const int32_t*>(g_back.host);
        const uint8_t bit = (uint8_t)op.bypass_bits(l);
        for (int i = 0; i < nc; ++i) {
          if (!flag[i]) continue;
          const int r = cand[i];
          admit[r] = l;
          for (int l2 = l; l2 < L; ++l2) codes[(size_t)l2 * R + r] |= bit;
        }
      }
    }
    if (l <= Wn) {  // row lists change only inside the window
      lists.clear();
      TableBuilder tb{lists, ot.reg[l & 1]};
      T = tb.add(codes + (size_t)l * R, R);
      SPIDER_TRY(upload_ints(lists.data(), lists.size(), ows.tab + ot.reg[l & 1], st));
    }
    SPIDER_TRY(run.layer(l, T));
  }
  SPIDER_TRY(run.flush());
  if (admit_out) std::copy(admit.begin(), admit.end(), admit_out);
  return SPIDER_OK;
}

// ------------------------------------------------------------------ decode
constexpr int kHeadSplit = 8;

struct DecodeWs {
  PrefillWs p;     // activations and partials for B rows
  float2* rope;    // [cap][dh/2]
  int32_t* tab;    // identity row map [B], positions of the new tokens [B]
  float* Plog;     // LM head partials [kHeadSplit][B][V]
  size_t bytes;
};

DecodeWs decode_layout(const spider_decoder_cfg& c, int B, int cap, int V, char* base) {
  Carver cv{base};
  DecodeWs w{};
  w.p = prefill_layout(c, B, cv);
  const int half = c.d / c.H / 2;
  w.rope = reinterpret_cast<float2*>(cv.take((size_t)cap * half * sizeof(float2)));
  w.tab = reinterpret_cast<int32_t*>(cv.take((size_t)2 * B * sizeof(int32_t)));
  w.Plog = V > 0 ? reinterpret_cast<float*>(cv.take((size_t)kHeadSplit * B * V * sizeof(float))) : nullptr;
  w.bytes = cv.off;
  return w;
}

// One decode step: every sample's new token (input row x[b], position lens[b])
// runs through all layers with nothing bypassed, its key and value appended to
// the cache; then the final norm, the LM head and the greedy choice.
template <typename AT>
spider_status run_decode(const spider_decoder_cfg& c, const spider_layer_weights* W, int B, const int32_t* lens,
                         const void* x, const spider_kv_cache& kv, const float* final_norm, const void* wu, int V,
                         float* h, float* logits, int32_t* next, const DecodeWs& ws, hipStream_t st) {
  const bool bf16 = c.dtype == SPIDER_BF16;
  const int d = c.d, dh = d / c.H, half = dh / 2;
  const PrefillWs& p = ws.p;
  std::vector<int32_t> tab(2 * B);
  int max_pos = 0;
  for (int b = 0; b < B; ++b) {
    tab[b] = b;
    tab[B + b] = lens[b];
    max_pos = std::max(max_pos, lens[b]);
  }
  SPIDER_TRY(upload_ints(tab.data(), tab.size(), ws.tab, st));
  const int32_t* ident = ws.tab;
  const int32_t* dlens = ws.tab + B;
  {
    const int64_t n = (int64_t)(max_pos + 1) * half;
    rope_table_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(ws.rope, max_pos + 1, half, dh,
                                                                  std::log2((double)c.theta));
    SPIDER_LAUNCHED("rope_table");
  }
  {
    ProfScope ps(KC_EMBED, st);
    const int64_t n = (int64_t)B * d;
    embed_kernel<AT><<<(unsigned)((n + 255) / 256), 256, 0, st>>>(reinterpret_cast<const AT*>(x), h, n);
    SPIDER_LAUNCHED("embed");
  }
  AT* xn = reinterpret_cast<AT*>(p.xn);
  AT* qb = reinterpret_cast<AT*>(p.q);
  AT* ob = reinterpret_cast<AT*>(p.o);
  AT* act = reinterpret_cast<AT*>(p.act);
  AT* ck = reinterpret_cast<AT*>(kv.k);
  AT* cv = reinterpret_cast<AT*>(kv.v);
  const int64_t ps_ = (int64_t)B * d;
  const int sm = split_max_for_rows(B);
  auto gemm = [&](GemmArgs& ga, int cap) {
    const int s2 = std::min(sm, cap);
    return bf16 ? launch_gemm_bf16(ga, s2, st) : launch_gemm_f32(ga, s2, st);
  };
  const float scale = (float)(1.0 / std::sqrt((double)dh));
  // At most 4 bf16 rows the GEMMs run as GEMVs that normalise their own input
  // rows (RMSNorm fused) and add O and down results straight into h: five
  // launches per layer instead of eight, no split partials.
  const bool fused = bf16 && B <= 4 && d <= 8192;
  int pend = 0;
  for (int l = 0; l < c.L; ++l) {
    const spider_layer_weights& w = W[l];
    const int64_t loff = (int64_t)l * B * kv.cap * d;
    if (!fused) {
      ProfScope ps(KC_RMSNORM, st);
      launch_norm<AT>(B, h, d, p.Pres, pend, ps_, pend ? ident : nullptr, w.attn_norm, c.eps, nullptr, 1, xn, st);
      SPIDER_LAUNCHED("rmsnorm(attn)");
      pend = 0;
    }
    GemmArgs ga{};
    ga.ngroups = 3;
    ga.K = d;
    ga.lda = d;
    ga.epilogue = EPI_PARTIAL_F32;
    ga.g[0] = GemmGroup{xn, nullptr, B, w.wq, nullptr, d, p.Pq, d, ps_, 0, 0, 0};
    ga.g[1] = GemmGroup{xn, nullptr, B, w.wk, nullptr, d, p.Pk, d, ps_, 0, 0, 0};
    ga.g[2] = GemmGroup{xn, nullptr, B, w.wv, nullptr, d, p.Pv, d, ps_, 0, 0, 0};
    if (fused) {
      ga.norm_h = h;
      ga.norm_w = w.attn_norm;
      ga.norm_eps = c.eps;
      // the GEMV itself applies RoPE, stores Q and appends K and V to the cache
      ga.epilogue = EPI_DECODE_QKV;
      ga.rope = ws.rope;
      ga.pos = dlens;
      ga.kv_cap = kv.cap;
      ga.g[0].out = qb;
      ga.g[0].kind = 1;
      ga.g[1].out = ck + loff;
      ga.g[1].kind = 3;
      ga.g[2].out = cv + loff;
      ga.g[2].kind = 2;
    }
    {
      ProfScope ps(KC_GEMM_QKV, st);
      hipError_t e = gemm(ga, 2);
      SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "decode gemm_qkv: %s", hipGetErrorString(e));
    }
    if (!fused) {
      ProfScope ps(KC_QKV_FINALIZE, st);
      decode_qkv_kernel<AT><<<dim3((unsigned)B, 3), 256, 0, st>>>(p.Pq, p.Pk, p.Pv, ga.split, ps_, d, dh, dlens,
                                                                   ws.rope, qb, ck, cv, loff, kv.cap);
      SPIDER_LAUNCHED("decode_qkv");
    }
    {
      ProfScope ps(KC_ATTENTION, st);
      decode_attention_kernel<AT><<<dim3((unsigned)c.H, (unsigned)B), 256, 0, st>>>(qb, ck, cv, loff, kv.cap,
                                                                                     dlens, d, dh, scale, ob);
      SPIDER_LAUNCHED("decode_attention");
    }
    GemmArgs go{};
    go.ngroups = 1;
    go.K = d;
    go.lda = d;
    go.epilogue = fused ? EPI_RESIDUAL_F32 : EPI_PARTIAL_F32;
    go.g[0] = GemmGroup{ob, nullptr, B, w.wo, nullptr, d, fused ? (void*)h : (void*)p.Pres, d, ps_, 0, 0, 0};
    {
      ProfScope ps(KC_GEMM_O, st);
      hipError_t e = gemm(go, 8);
      SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "decode gemm_o: %s", hipGetErrorString(e));
    }
    if (!fused) {
      pend = go.split;
      ProfScope ps(KC_RMSNORM, st);
      launch_norm<AT>(B, h, d, p.Pres, pend, ps_, ident, w.ffn_norm, c.eps, nullptr, 1, xn, st);
      SPIDER_LAUNCHED("rmsnorm(ffn)");
      pend = 0;
    }
    GemmArgs gu{};
    gu.ngroups = 1;
    gu.K = d;
    gu.lda = d;
    gu.epilogue = EPI_SWIGLU;
    gu.g[0] = GemmGroup{xn, nullptr, B, w.wg, w.wu, c.d_ff, act, c.d_ff, 0, 0, 0, 0};
    if (fused) {
      gu.norm_h = h;
      gu.norm_w = w.ffn_norm;
      gu.norm_eps = c.eps;
    }
    {
      ProfScope ps(KC_GEMM_GATEUP, st);
      hipError_t e = gemm(gu, 1);
      SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "decode gemm_gateup: %s", hipGetErrorString(e));
    }
    GemmArgs gd{};
    gd.ngroups = 1;
    gd.K = c.d_ff;
    gd.lda = c.d_ff;
    gd.epilogue = fused ? EPI_RESIDUAL_F32 : EPI_PARTIAL_F32;
    gd.g[0] = GemmGroup{act, nullptr, B, w.wd, nullptr, d, fused ? (void*)h : (void*)p.Pres, d, ps_, 0, 0, 0};
    {
      ProfScope ps(KC_GEMM_DOWN, st);
      hipError_t e = gemm(gd, 8);
      SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "decode gemm_down: %s", hipGetErrorString(e));
    }
    pend = fused ? 0 : gd.split;
  }
  if (pend) {
    ProfScope ps(KC_RESIDUAL, st);
    launch_norm<AT>(B, h, d, p.Pres, pend, ps_, ident, nullptr, 0.f, nullptr, 0, static_cast<AT*>(nullptr), st);
    SPIDER_LAUNCHED("residual_add");
  }
  if (wu) {
    ProfScope ps(KC_LM_HEAD, st);
    GemmArgs gh{};
    gh.ngroups = 1;
    gh.K = d;
    gh.lda = d;
    gh.epilogue = EPI_PARTIAL_F32;
    gh.g[0] = GemmGroup{xn, nullptr, B, wu, nullptr, V, ws.Plog, V, (int64_t)B * V, 0, 0, 0};
    if (fused) {
      gh.norm_h = h;
      gh.norm_w = final_norm;
      gh.norm_eps = c.eps;
    } else {
      launch_norm<AT>(B, h, d, nullptr, 0, 0, nullptr, final_norm, c.eps, nullptr, 1, xn, st);
      SPIDER_LAUNCHED("final_norm");
    }
    hipError_t e = bf16 ? launch_gemm_bf16(gh, kHeadSplit, st) : launch_gemm_f32(gh, kHeadSplit, st);
    SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "lm head: %s", hipGetErrorString(e));
    logits_argmax_kernel<<<B, 256, 0, st>>>(ws.Plog, gh.split, (int64_t)B * V, V, logits, next);
    SPIDER_LAUNCHED("logits_argmax");
  }
  return SPIDER_OK;
}

}  // namespace
}  // namespace spider

using namespace spider;

extern "C" size_t spider_prefill_workspace_size(const spider_decoder_cfg* cfg, int B, int rows) {
  if (!cfg || cfg->L < 1 || cfg->d < 1 || cfg->H < 1 || cfg->d % cfg->H || B < 1 || rows < 0)
    return 0;
  return prefill_layout(*cfg, std::max(rows, 1), nullptr).bytes;
}

extern "C" spider_status spider_prefill(const spider_decoder_cfg* cfg,
                                        const spider_layer_weights* layers, int B,
                                        const int32_t* cu_seqlens, const void* x,
                                        const uint8_t* codes, float* h_out, void* workspace,
                                        size_t workspace_bytes, spider_stream stream) {
  clear_error();
  SPIDER_TRY(validate_cfg(cfg));
  SPIDER_TRY(validate_cu(B, cu_seqlens, layers));
  const int R = cu_seqlens[B];
  if (R == 0) return SPIDER_OK;
  SPIDER_REQUIRE(codes, SPIDER_ERR_INVALID_ARG, "spider_prefill: codes must be non-null");
  SPIDER_TRY(validate_prefill_args(cfg, layers, x, h_out));
  for (size_t i = 0; i < (size_t)cfg->L * R; ++i)
    SPIDER_REQUIRE(codes[i] <= 3, SPIDER_ERR_INVALID_ARG,
                   "spider_prefill: code %u at %zu is not in [0, 3]", (unsigned)codes[i], i);
  const PrefillWs need = prefill_layout(*cfg, R, nullptr);
  SPIDER_REQUIRE(workspace && workspace_bytes >= need.bytes, SPIDER_ERR_WORKSPACE,
                 "spider_prefill: workspace of %zu bytes needed, %zu given", need.bytes,
                 workspace_bytes);
  SPIDER_REQUIRE(((uintptr_t)workspace % 256) == 0, SPIDER_ERR_WORKSPACE,
                 "spider_prefill: workspace must be 256-byte aligned");
  const PrefillWs ws = prefill_layout(*cfg, R, reinterpret_cast<char*>(workspace));
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (cfg->dtype == SPIDER_BF16)
    return run_prefill<uint16_t>(*cfg, layers, B, cu_seqlens, x, codes, h_out, ws, st);
  return run_prefill<float>(*cfg, layers, B, cu_seqlens, x, codes, h_out, ws, st);
}

extern "C" size_t spider_prefill_online_workspace_size(const spider_decoder_cfg* cfg, int B, int rows,
                                                       int V) {
  if (!cfg || cfg->L < 1 || cfg->d < 1 || cfg->H < 1 || cfg->d % cfg->H || B < 1 || rows < 0 || V < 1)
    return 0;
  return online_layout(*cfg, B, std::max(rows, 1), V, nullptr).bytes;
}

namespace spider {
namespace {
spider_status prefill_online_entry(const spider_decoder_cfg* cfg, const spider_layer_weights* layers, int B,
                                   const int32_t* cu_seqlens, const void* x, int n_text, const void* w_unembed,
                                   int V, const double* slc_sel, const uint8_t* target, double w1, double w2,
                                   double T_skip, uint32_t ablation, uint8_t* codes_out, int32_t* admit_out,
                                   float* s_sa_out, float* h_out, void* workspace, size_t workspace_bytes,
                                   spider_stream stream) {
  SPIDER_TRY(validate_cfg(cfg));
  SPIDER_TRY(validate_cu(B, cu_seqlens, layers));
  SPIDER_REQUIRE(n_text >= 1, SPIDER_ERR_INVALID_ARG, "spider_prefill_online: n_text must be >= 1");
  for (int b = 0; b < B; ++b)
    SPIDER_REQUIRE(cu_seqlens[b + 1] - cu_seqlens[b] >= n_text, SPIDER_ERR_SHAPE,
                   "spider_prefill_online: sample %d has fewer than n_text rows", b);
  SPIDER_REQUIRE(V >= 2 && w_unembed, SPIDER_ERR_INVALID_ARG,
                 "spider_prefill_online: w_unembed must be non-null with V >= 2");
  SPIDER_REQUIRE(((uintptr_t)w_unembed % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                 "spider_prefill_online: w_unembed must be 16-byte aligned");
  SPIDER_REQUIRE(cfg->dtype != SPIDER_BF16 || V % 64 == 0, SPIDER_ERR_UNSUPPORTED,
                 "spider_prefill_online: bf16 path needs V a multiple of 64");
  SPIDER_REQUIRE(std::isfinite(w1) && std::isfinite(w2) && std::isfinite(T_skip), SPIDER_ERR_INVALID_ARG,
                 "spider_prefill_online: w1, w2 and T_skip must be finite");
  const int Wn = cfg->L / 2;
  if (Wn > 0) {
    SPIDER_REQUIRE(slc_sel && target, SPIDER_ERR_INVALID_ARG,
                   "spider_prefill_online: slc_sel and target must be non-null");
    for (int l = 0; l < Wn; ++l) {
      SPIDER_REQUIRE(std::isfinite(slc_sel[l]), SPIDER_ERR_INVALID_ARG,
                     "spider_prefill_online: slc_sel[%d] is not finite", l);
      SPIDER_REQUIRE(target[l] <= 1, SPIDER_ERR_INVALID_ARG,
                     "spider_prefill_online: target[%d] must be 0 or 1", l);
    }
  }
  const int R = cu_seqlens[B];
  if (R == 0) return SPIDER_OK;
  SPIDER_REQUIRE(codes_out, SPIDER_ERR_INVALID_ARG, "spider_prefill_online: codes_out must be non-null");
  SPIDER_TRY(validate_prefill_args(cfg, layers, x, h_out));
  const OnlineWs need = online_layout(*cfg, B, R, V, nullptr);
  SPIDER_REQUIRE(workspace && workspace_bytes >= need.bytes, SPIDER_ERR_WORKSPACE,
                 "spider_prefill_online: workspace of %zu bytes needed, %zu given", need.bytes,
                 workspace_bytes);
  SPIDER_REQUIRE(((uintptr_t)workspace % 256) == 0, SPIDER_ERR_WORKSPACE,
                 "spider_prefill_online: workspace must be 256-byte aligned");
  const OnlineWs ows = online_layout(*cfg, B, R, V, reinterpret_cast<char*>(workspace));
  const OnlineParams op{n_text, w_unembed, V, slc_sel, target, w1, w2, T_skip, ablation};
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (cfg->dtype == SPIDER_BF16)
    return run_prefill_online<uint16_t>(*cfg, layers, B, cu_seqlens, x, op, codes_out, admit_out, s_sa_out,
                                        h_out, ows, st);
  return run_prefill_online<float>(*cfg, layers, B, cu_seqlens, x, op, codes_out, admit_out, s_sa_out,
                                   h_out, ows, st);
}
}  // namespace
}  // namespace spider

extern "C" spider_status spider_prefill_online(
    const spider_decoder_cfg* cfg, const spider_layer_weights* layers, int B, const int32_t* cu_seqlens,
    const void* x, int n_text, const void* w_unembed, int V, const double* slc_sel, const uint8_t* target,
    double w1, double w2, double T_skip, uint8_t* codes_out, int32_t* admit_out, float* s_sa_out,
    float* h_out, void* workspace, size_t workspace_bytes, spider_stream stream) {
  clear_error();
  return prefill_online_entry(cfg, layers, B, cu_seqlens, x, n_text, w_unembed, V, slc_sel, target, w1, w2,
                              T_skip, 0u, codes_out, admit_out, s_sa_out, h_out, workspace, workspace_bytes,
                              stream);
}

extern "C" spider_status spider_prefill_online_ablation(
    const spider_decoder_cfg* cfg, const spider_layer_weights* layers, int B, const int32_t* cu_seqlens,
    const void* x, int n_text, const void* w_unembed, int V, const double* slc_sel, const uint8_t* target,
    double w1, double w2, double T_skip, uint32_t ablation, uint8_t* codes_out, int32_t* admit_out,
    float* s_sa_out, float* h_out, void* workspace, size_t workspace_bytes, spider_stream stream) {
  clear_error();
  SPIDER_REQUIRE((ablation & ~15u) == 0, SPIDER_ERR_INVALID_ARG,
                 "spider_prefill_online_ablation: unknown ablation bits 0x%x", ablation & ~15u);
  return prefill_online_entry(cfg, layers, B, cu_seqlens, x, n_text, w_unembed, V, slc_sel, target, w1, w2,
                              T_skip, ablation, codes_out, admit_out, s_sa_out, h_out, workspace,
                              workspace_bytes, stream);
}

extern "C" spider_status spider_prefill_kv(const spider_decoder_cfg* cfg, const spider_layer_weights* layers, int B,
                                           const int32_t* cu_seqlens, const void* x, const uint8_t* codes,
                                           float* h_out, const spider_kv_cache* kv, void* workspace,
                                           size_t workspace_bytes, spider_stream stream) {
  clear_error();
  SPIDER_TRY(validate_cfg(cfg));
  SPIDER_TRY(validate_cu(B, cu_seqlens, layers));
  SPIDER_REQUIRE(kv && kv->k && kv->v && kv->cap >= 1, SPIDER_ERR_INVALID_ARG,
                 "spider_prefill_kv: kv cache with k, v and cap >= 1 required");
  for (int b = 0; b < B; ++b)
    SPIDER_REQUIRE(cu_seqlens[b + 1] - cu_seqlens[b] <= kv->cap, SPIDER_ERR_SHAPE,
                   "spider_prefill_kv: sample %d has more rows than the cache holds", b);
  if (cfg->dtype == SPIDER_BF16)
    SPIDER_REQUIRE(((uintptr_t)kv->k % 16) == 0 && ((uintptr_t)kv->v % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                   "spider_prefill_kv: cache must be 16-byte aligned");
  const int R = cu_seqlens[B];
  if (R == 0) return SPIDER_OK;
  SPIDER_REQUIRE(codes, SPIDER_ERR_INVALID_ARG, "spider_prefill_kv: codes must be non-null");
  SPIDER_TRY(validate_prefill_args(cfg, layers, x, h_out));
  for (size_t i = 0; i < (size_t)cfg->L * R; ++i)
    SPIDER_REQUIRE(codes[i] <= 3, SPIDER_ERR_INVALID_ARG,
                   "spider_prefill_kv: code %u at %zu is not in [0, 3]", (unsigned)codes[i], i);
  const PrefillWs need = prefill_layout(*cfg, R, nullptr);
  SPIDER_REQUIRE(workspace && workspace_bytes >= need.bytes, SPIDER_ERR_WORKSPACE,
                 "spider_prefill_kv: workspace of %zu bytes needed, %zu given", need.bytes, workspace_bytes);
  SPIDER_REQUIRE(((uintptr_t)workspace % 256) == 0, SPIDER_ERR_WORKSPACE,
                 "spider_prefill_kv: workspace must be 256-byte aligned");
  const PrefillWs ws = prefill_layout(*cfg, R, reinterpret_cast<char*>(workspace));
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (cfg->dtype == SPIDER_BF16)
    return run_prefill<uint16_t>(*cfg, layers, B, cu_seqlens, x, codes, h_out, ws, st, kv);
  return run_prefill<float>(*cfg, layers, B, cu_seqlens, x, codes, h_out, ws, st, kv);
}

extern "C" size_t spider_decode_workspace_size(const spider_decoder_cfg* cfg, int B, int cap, int V) {
  if (!cfg || cfg->L < 1 || cfg->d < 1 || cfg->H < 1 || cfg->d % cfg->H || B < 1 || cap < 1 || V < 0) return 0;
  return decode_layout(*cfg, B, cap, V, nullptr).bytes;
}

extern "C" spider_status spider_decode_step(const spider_decoder_cfg* cfg, const spider_layer_weights* layers,
                                            int B, const int32_t* lens, const void* x, const spider_kv_cache* kv,
                                            const float* final_norm, const void* w_unembed, int V, float* h_out,
                                            float* logits_out, int32_t* next_out, void* workspace,
                                            size_t workspace_bytes, spider_stream stream) {
  clear_error();
  SPIDER_TRY(validate_cfg(cfg));
  SPIDER_REQUIRE(B >= 1 && layers && lens, SPIDER_ERR_INVALID_ARG,
                 "spider_decode_step: B >= 1, layers and lens required");
  SPIDER_REQUIRE(kv && kv->k && kv->v && kv->cap >= 1, SPIDER_ERR_INVALID_ARG,
                 "spider_decode_step: kv cache with k, v and cap >= 1 required");
  SPIDER_REQUIRE(cfg->d / cfg->H <= kDecodeMaxDh, SPIDER_ERR_UNSUPPORTED, "spider_decode_step: dh must be <= 256");
  // decode attention reads cached rows as 16-byte vectors
  SPIDER_REQUIRE((cfg->d / cfg->H) % (cfg->dtype == SPIDER_BF16 ? 8 : 4) == 0, SPIDER_ERR_UNSUPPORTED,
                 "spider_decode_step: dh must be a multiple of 16 bytes");
  SPIDER_REQUIRE(((uintptr_t)kv->k % 16) == 0 && ((uintptr_t)kv->v % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                 "spider_decode_step: cache must be 16-byte aligned");
  for (int b = 0; b < B; ++b)
    SPIDER_REQUIRE(lens[b] >= 0 && lens[b] < kv->cap && lens[b] + 1 <= kDecodeMaxKeys, SPIDER_ERR_SHAPE,
                   "spider_decode_step: lens[%d] = %d outside [0, min(cap, 8192) - 1]", b, lens[b]);
  if (w_unembed) {
    SPIDER_REQUIRE(V >= 1 && final_norm, SPIDER_ERR_INVALID_ARG,
                   "spider_decode_step: the LM head needs V >= 1 and final_norm");
    SPIDER_REQUIRE(cfg->dtype != SPIDER_BF16 || V % 64 == 0, SPIDER_ERR_UNSUPPORTED,
                   "spider_decode_step: bf16 LM head needs V a multiple of 64");
    SPIDER_REQUIRE(((uintptr_t)w_unembed % 16) == 0 && ((uintptr_t)final_norm % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                   "spider_decode_step: w_unembed and final_norm must be 16-byte aligned");
  }
  SPIDER_TRY(validate_prefill_args(cfg, layers, x, h_out));
  if (cfg->dtype == SPIDER_BF16)
    SPIDER_REQUIRE(((uintptr_t)kv->k % 16) == 0 && ((uintptr_t)kv->v % 16) == 0, SPIDER_ERR_UNSUPPORTED,
                   "spider_decode_step: cache must be 16-byte aligned");
  const int Vh = w_unembed ? V : 0;
  const DecodeWs need = decode_layout(*cfg, B, kv->cap, Vh, nullptr);
  SPIDER_REQUIRE(workspace && workspace_bytes >= need.bytes, SPIDER_ERR_WORKSPACE,
                 "spider_decode_step: workspace of %zu bytes needed, %zu given", need.bytes, workspace_bytes);
  SPIDER_REQUIRE(((uintptr_t)workspace % 256) == 0, SPIDER_ERR_WORKSPACE,
                 "spider_decode_step: workspace must be 256-byte aligned");
  const DecodeWs ws = decode_layout(*cfg, B, kv->cap, Vh, reinterpret_cast<char*>(workspace));
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (cfg->dtype == SPIDER_BF16)
    return run_decode<uint16_t>(*cfg, layers, B, lens, x, *kv, final_norm, w_unembed, Vh, h_out, logits_out,
                                next_out, ws, st);
  return run_decode<float>(*cfg, layers, B, lens, x, *kv, final_norm, w_unembed, Vh, h_out, logits_out, next_out,
                           ws, st);
}
