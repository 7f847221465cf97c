// Online skip controller of ASL-Skip (Sec. 4.2.1, Eq. 4; accumulation and
// admission of Eq. 6 / Algorithm 1), evaluated on the device at every layer
// of the decision window for the visual rows not yet in skip mode.
//
//   text_mean   q_b = mean of sample b's text rows of h (double sums)
//   lens_prep   per candidate row i of sample b: a copy of h_i in the
//               activation dtype (the logit-lens GEMM operand) and
//               F_itc = (1 + cos(h_i, q_b)) / 2 (double)
//   [GEMM]      z = copy x W_unembed^T (the decoder GEMMs, fp32 accumulation):
//               bf16 with V % 128 == 0 reduces each row's 128-column tiles
//               to (max, S, T) in the GEMM epilogue, else writes the logits
//   lens_admit  E_ii = H(softmax(z)) / ln V with H = ln S - T / S,
//               S = sum e^(z - max), T = sum e^(z - max) (z - max) (tile
//               statistics merged in double in a fixed order);
//               S_sa = max(0, 1 - (E_ii + F_itc)); acc_i += w1 S_sa + w2 sel_l;
//               flag_i = acc_i >= T_skip
//
// Every reduction runs in a fixed order (per-thread strided sums, then a
// fixed tree), so identical inputs give identical flags.
#include "kernels.h"

namespace spider {
namespace {

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum over the 256 threads of a block (4 waves); every thread gets the result.
template <int N>
__device__ __forceinline__ void block_sum_d(double (&v)[N], double (*red)[4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = wave_sum_d(v[i]);
  if (lane == 0)
#pragma unroll
    for (int i = 0; i < N; ++i) red[i][wave] = v[i];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = (red[i][0] + red[i][1]) + (red[i][2] + red[i][3]);
}

// grid (ceil(d / 64), B): 64 columns x 4 row slices per block; slice j sums
// the text rows j, j+4, ... in order (double), then (s0 + s1) + (s2 + s3).
// Text rows of sample b are cu[b+1]-n_text .. cu[b+1]-1.
__global__ void __launch_bounds__(256) text_mean_kernel(const float* __restrict__ h, int d,
                                                        const int32_t* __restrict__ cu, int n_text,
                                                        float* __restrict__ tmean) {
  __shared__ double part[4][64];
  const int b = blockIdx.y;
  const int cl = threadIdx.x & 63, j = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + cl;
  const int r1 = cu[b + 1];
  double s = 0.0;
  if (c < d) {
#pragma unroll 4
    for (int r = r1 - n_text + j; r < r1; r += 4) s += (double)h[(int64_t)r * d + c];
  }
  part[j][cl] = s;
  __syncthreads();
  if (j == 0 && c < d)
    tmean[(int64_t)b * d + c] = (float)(((part[0][cl] + part[1][cl]) + (part[2][cl] + part[3][cl])) / n_text);
}

// one block per candidate; d % 4 == 0
template <typename AT>
__global__ void __launch_bounds__(256) lens_prep_kernel(const float* __restrict__ h, int d,
                                                        const int32_t* __restrict__ cand,
                                                        const int32_t* __restrict__ cand_sample,
                                                        const float* __restrict__ tmean,
                                                        AT* __restrict__ hc, double* __restrict__ F,
                                                        const int32_t* __restrict__ nc_dev) {
  __shared__ double red[3][4];
  const int c = blockIdx.x;
  if (nc_dev && c >= *nc_dev) return;
  const float* hr = h + (int64_t)cand[c] * d;
  const float* tq = tmean + (int64_t)cand_sample[c] * d;
  AT* out = hc + (int64_t)c * d;
  double acc[3] = {0.0, 0.0, 0.0};  // h.q, h.h, q.q
  for (int i = threadIdx.x * 4; i < d; i += 1024) {
    const floatx4 x = *reinterpret_cast<const floatx4*>(hr + i);
    const floatx4 q = *reinterpret_cast<const floatx4*>(tq + i);
    if constexpr (std::is_same<AT, uint16_t>::value) {
      const uint32_t lo = (uint32_t)f32_to_bf16_bits(x[0]) | ((uint32_t)f32_to_bf16_bits(x[1]) << 16);
      const uint32_t hi = (uint32_t)f32_to_bf16_bits(x[2]) | ((uint32_t)f32_to_bf16_bits(x[3]) << 16);
      *reinterpret_cast<uint2*>(out + i) = make_uint2(lo, hi);
    } else {
      *reinterpret_cast<floatx4*>(out + i) = x;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[0] += (double)x[e] * (double)q[e];
      acc[1] += (double)x[e] * (double)x[e];
      acc[2] += (double)q[e] * (double)q[e];
    }
  }
  block_sum_d<3>(acc, red);
  if (threadIdx.x == 0) {
    const double den = sqrt(acc[1]) * sqrt(acc[2]);
    const double cosv = den > 0.0 ? acc[0] / den : 0.0;
    F[c] = (1.0 + cosv) / 2.0;
  }
}

// Shared tail of the two admission kernels (thread 0 of the candidate's block).
__device__ __forceinline__ void admit_row(double S, double T, int c, const int32_t* __restrict__ cand,
                                          const double* __restrict__ F, const LensAdmitArgs& p) {
  const double H = log(S) - T / S;
  const double E = (p.ablation & SPIDER_ONLINE_NO_EII) ? 0.0 : H / p.log_v;
  const double Fc = (p.ablation & SPIDER_ONLINE_NO_FITC) ? 0.0 : F[c];
  const double ssa = fmax(0.0, 1.0 - (E + Fc));
  const int r = cand[c];
  const double fuse = p.w1 * ssa + p.w2_sel;
  const double a = (p.ablation & SPIDER_ONLINE_NO_ACCUM) ? fuse : p.acc[r] + fuse;
  p.acc[r] = a;
  p.flag[c] = a >= p.t_skip ? 1 : 0;
  if (p.s_out) p.s_out[r] = (float)ssa;
}

// one block per candidate: normalised entropy of softmax(logits row), Eq. 4,
// accumulation and admission test
__global__ void __launch_bounds__(256) lens_admit_kernel(const float* __restrict__ logits, int V,
                                                         const int32_t* __restrict__ cand,
                                                         const double* __restrict__ F,
                                                         LensAdmitArgs p, const int32_t* __restrict__ nc_dev) {
  __shared__ float redf[4];
  __shared__ double redd[2][4];
  const int c = blockIdx.x;
  if (nc_dev && c >= *nc_dev) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* z = logits + (int64_t)c * V;
  float m = -INFINITY;
  for (int j = threadIdx.x; j < V; j += 256) m = fmaxf(m, z[j]);
  m = wave_max(m);
  if (lane == 0) redf[wave] = m;
  __syncthreads();
  m = fmaxf(fmaxf(redf[0], redf[1]), fmaxf(redf[2], redf[3]));
  float s = 0.f, t = 0.f;
  for (int j = threadIdx.x; j < V; j += 256) {
    const float u = z[j] - m;
    const float e = expf(u);
    s += e;
    t = fmaf(e, u, t);
  }
  double st[2] = {(double)s, (double)t};
  block_sum_d<2>(st, redd);
  if (threadIdx.x == 0) admit_row(st[0], st[1], c, cand, F, p);
}

struct StatD {
  double m, s, t;
};

__device__ __forceinline__ StatD stat_merge(StatD a, StatD b) {
  const double m = fmax(a.m, b.m);
  const double da = a.m - m, db = b.m - m;
  const double ea = exp(da), eb = exp(db);
  return {m, ea * a.s + eb * b.s, ea * (a.t + a.s * da) + eb * (b.t + b.s * db)};
}

// one wave per candidate: merges the row's per-tile statistics (tile j =
// lane, lane + 64, ... in order, then a fixed butterfly over the lanes)
__global__ void __launch_bounds__(64) lens_admit_stats_kernel(const float* __restrict__ stats, int ntiles,
                                                              const int32_t* __restrict__ cand,
                                                              const double* __restrict__ F,
                                                              LensAdmitArgs p,
                                                              const int32_t* __restrict__ nc_dev) {
  const int c = blockIdx.x, lane = threadIdx.x;
  if (nc_dev && c >= *nc_dev) return;
  const floatx4* row = reinterpret_cast<const floatx4*>(stats) + (int64_t)c * ntiles;
  StatD st{0.0, 0.0, 0.0};
  bool have = false;
  for (int j = lane; j < ntiles; j += 64) {
    const floatx4 v = row[j];
    const StatD x{(double)v[0], (double)v[1], (double)v[2]};
    st = have ? stat_merge(st, x) : x;
    have = true;
  }
  // lanes without a tile (ntiles < 64) take the neutral piece of their partner
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const StatD other{__shfl_xor(st.m, o, 64), __shfl_xor(st.s, o, 64), __shfl_xor(st.t, o, 64)};
    const bool other_have = __shfl_xor((int)have, o, 64) != 0;
    if (have && other_have) st = (lane & o) ? stat_merge(other, st) : stat_merge(st, other);
    else if (other_have) st = other;
    have = have || other_have;
  }
  if (lane == 0) admit_row(st.s, st.t, c, cand, F, p);
}

__global__ void __launch_bounds__(256) fill_zero_kernel(uint32_t* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0u;
}

}  // namespace

hipError_t launch_text_mean(const float* h, int d, const int32_t* cu, int B, int n_text, float* tmean,
                            hipStream_t st) {
  if (B <= 0) return hipSuccess;
  text_mean_kernel<<<dim3((unsigned)ceil_div(d, 64), (unsigned)B), 256, 0, st>>>(h, d, cu, n_text, tmean);
  return hipGetLastError();
}

hipError_t launch_lens_prep(bool bf16, const float* h, int d, const int32_t* cand,
                            const int32_t* cand_sample, int nc, const int32_t* nc_dev, const float* tmean,
                            void* hc, double* F, hipStream_t st) {
  if (nc <= 0) return hipSuccess;
  if (d % 4) return hipErrorInvalidValue;
  if (bf16)
    lens_prep_kernel<uint16_t><<<nc, 256, 0, st>>>(h, d, cand, cand_sample, tmean,
                                                    reinterpret_cast<uint16_t*>(hc), F, nc_dev);
  else
    lens_prep_kernel<float><<<nc, 256, 0, st>>>(h, d, cand, cand_sample, tmean,
                                                 reinterpret_cast<float*>(hc), F, nc_dev);
  return hipGetLastError();
}

hipError_t launch_lens_admit(const float* logits, int V, const int32_t* cand, int nc, const int32_t* nc_dev,
                             const double* F, const LensAdmitArgs& p, hipStream_t st) {
  if (nc <= 0) return hipSuccess;
  lens_admit_kernel<<<nc, 256, 0, st>>>(logits, V, cand, F, p, nc_dev);
  return hipGetLastError();
}

hipError_t launch_lens_admit_stats(const float* stats, int ntiles, const int32_t* cand, int nc,
                                   const int32_t* nc_dev, const double* F, const LensAdmitArgs& p,
                                   hipStream_t st) {
  if (nc <= 0) return hipSuccess;
  if (ntiles <= 0) return hipErrorInvalidValue;
  lens_admit_stats_kernel<<<nc, 64, 0, st>>>(stats, ntiles, cand, F, p, nc_dev);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st) {
  if (bytes % 4) return hipErrorInvalidValue;
  const int64_t n = (int64_t)(bytes / 4);
  if (n == 0) return hipSuccess;
  fill_zero_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(reinterpret_cast<uint32_t*>(p), n);
  return hipGetLastError();
}

}  // namespace spider
