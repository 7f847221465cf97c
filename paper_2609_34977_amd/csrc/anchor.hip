// Anchor-score inputs computed on the device (Sec. 4.1.1).
//
// Encoders without [CLS]: the attention each
// patch receives, averaged over heads and over the patches attending to it,
//   a[g, j] = (1 / (H n)) sum_h sum_i attn[g, h, i, j].
//
// A streaming reduction of H n^2 fp32 values per tile (21 MB for a 16-head
// 576-patch map), bound by HBM.  Two launches, fixed summation order:
//   colmean_partial  grid (ceil(n/256), H * ceil(n/128), G), 256 threads: one
//                    block per (head, 128-row chunk, 256 columns); wave w adds
//                    rows w, w+4, ... of the chunk in ascending order (16-byte
//                    non-temporal loads, the maps are read once; lane l owns
//                    columns 4l..4l+3, all 32 rows of a wave in flight before
//                    the adds); the four waves are added as (w0 + w1) + (w2 + w3).
//   colmean_final    grid (ceil(n/64), G): per column, four interleaved sets of
//                    the H * ceil(n/128) chunk sums (set s: b = s, s+4, ... with
//                    b = head * chunks + chunk) each added in ascending order,
//                    the sets added as (s0 + s1) + (s2 + s3), then one IEEE
//                    division by H n.
//
// Encoders that never store attention maps: the [CLS] row of a layer rebuilt
// from its CLS query and keys, softmax_j(scale * q . k_j) per head
// (cls_attention_kernel below); spider_score then averages it over heads.
#include <cmath>

#include "kernels.h"

namespace spider {
namespace {

constexpr int kChunkRows = 128;
constexpr int kRowsPerWave = kChunkRows / 4;

__global__ void __launch_bounds__(256) colmean_partial_kernel(int H, int n, const float* __restrict__ attn,
                                                              int64_t sg, int64_t sh, int64_t sr,
                                                              float* __restrict__ part) {
  __shared__ floatx4 red[4][64];
  const int g = blockIdx.z;
  const int nrc = (n + kChunkRows - 1) / kChunkRows;
  const int h = blockIdx.y / nrc, rc = blockIdx.y - h * nrc;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = blockIdx.x * 256 + 4 * lane;
  const bool active = c < n;  // n % 4 == 0: the whole float4 is in range
  const int r0 = rc * kChunkRows, r1 = min(n, r0 + kChunkRows);
  const float* base = attn + (int64_t)g * sg + (int64_t)h * sh + c;
  floatx4 v[kRowsPerWave];
#pragma unroll
  for (int t = 0; t < kRowsPerWave; ++t) {
    const int i = r0 + wave + 4 * t;
    v[t] = (active && i < r1) ? __builtin_nontemporal_load(reinterpret_cast<const floatx4*>(base + (int64_t)i * sr))
                              : floatx4{};
  }
  floatx4 acc = v[0];
#pragma unroll
  for (int t = 1; t < kRowsPerWave; ++t) acc += v[t];
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0 && active) {
    const floatx4 s = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
    *reinterpret_cast<floatx4*>(part + ((int64_t)g * H * nrc + blockIdx.y) * n + c) = s;
  }
}

// grid (ceil(n / 64), G), 256 threads: lane l owns column 64 blockIdx.x + l,
// wave s adds the chunk sums b = s, s+4, ... (b = head * chunks + chunk) in
// ascending order; the four waves are added as (s0 + s1) + (s2 + s3).
__global__ void __launch_bounds__(256) colmean_final_kernel(int H, int n, const float* __restrict__ part,
                                                            float* __restrict__ a_out) {
  __shared__ float red[4][64];
  const int g = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j = blockIdx.x * 64 + lane;
  const int nb = H * ((n + kChunkRows - 1) / kChunkRows);
  float s = 0.f;
  if (j < n) {
    const float* p = part + (int64_t)g * nb * n + j;
#pragma unroll 8
    for (int b = wave; b < nb; b += 4) s = __fadd_rn(s, p[(int64_t)b * n]);
  }
  red[wave][lane] = s;
  __syncthreads();
  if (wave == 0 && j < n)
    a_out[(int64_t)g * n + j] =
        __fdiv_rn(__fadd_rn(__fadd_rn(red[0][lane], red[1][lane]), __fadd_rn(red[2][lane], red[3][lane])),
                  (float)H * (float)n);
}

// ---------------------------------------------------------------- CLS row from q, K
// One block per (head, tile): thread t takes tokens t, t+256, ...; logit =
// scale * sum_c q[c] k[c] (fmaf over c ascending), softmax with the block's max,
// the exponentials summed per thread in token order then over the block in a
// fixed tree, one IEEE division per token.
template <typename FT>
__device__ __forceinline__ void load4f(const FT* p, float* x) {
  if constexpr (std::is_same<FT, float>::value) {
    const floatx4 v = *reinterpret_cast<const floatx4*>(p);
    x[0] = v[0]; x[1] = v[1]; x[2] = v[2]; x[3] = v[3];
  } else {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    x[0] = bf16_bits_to_f32((uint16_t)(v.x & 0xFFFFu));
    x[1] = bf16_bits_to_f32((uint16_t)(v.x >> 16));
    x[2] = bf16_bits_to_f32((uint16_t)(v.y & 0xFFFFu));
    x[3] = bf16_bits_to_f32((uint16_t)(v.y >> 16));
  }
}

constexpr int kMaxDh = 256;
constexpr int kMaxTokens = 4097;

template <typename FT>
__global__ void __launch_bounds__(256) cls_attention_kernel(int H, int dh, int T, const FT* __restrict__ q,
                                                            int64_t sqg, const FT* __restrict__ k, int64_t skg,
                                                            int64_t skr, float scale, float* __restrict__ out) {
  __shared__ float qs[kMaxDh];
  __shared__ float z[kMaxTokens];
  __shared__ float red[4];
  const int h = blockIdx.x, g = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const FT* qh = q + (int64_t)g * sqg + (int64_t)h * dh;
  for (int c = 4 * tid; c < dh; c += 1024) load4f<FT>(qh + c, qs + c);
  __syncthreads();
  const FT* kg = k + (int64_t)g * skg + (int64_t)h * dh;
  float mx = -INFINITY;
  for (int j = tid; j < T; j += 256) {
    const FT* kr = kg + (int64_t)j * skr;
    float acc = 0.f;
    for (int c = 0; c < dh; c += 4) {
      float x[4];
      load4f<FT>(kr + c, x);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc = fmaf(qs[c + e], x[e], acc);
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
  for (int j = tid; j < T; j += 256) {
    const float e = expf(z[j] - mx);
    z[j] = e;
    s += e;
  }
  s = wave_sum(s);
  if (lane == 0) red[wave] = s;
  __syncthreads();
  s = (red[0] + red[1]) + (red[2] + red[3]);
  float* o = out + ((int64_t)g * H + h) * T;
  for (int j = tid; j < T; j += 256) o[j] = __fdiv_rn(z[j], s);
}

size_t colmean_ws_bytes(int G, int H, int n) {
  return (size_t)G * H * ((n + kChunkRows - 1) / kChunkRows) * n * sizeof(float);
}

}  // namespace
}  // namespace spider

using namespace spider;

extern "C" size_t spider_anchor_colmean_workspace_size(int G, int H, int n) {
  if (G <= 0 || H <= 0 || n <= 0) return 0;
  return colmean_ws_bytes(G, H, n);
}

extern "C" spider_status spider_anchor_colmean(int G, int H, int n, const float* attn, int64_t stride_g,
                                               int64_t stride_h, int64_t stride_row, float* a_out,
                                               void* workspace, size_t workspace_bytes,
                                               spider_stream stream) {
  clear_error();
  SPIDER_REQUIRE(G >= 1 && H >= 1 && n >= 1, SPIDER_ERR_INVALID_ARG,
                 "spider_anchor_colmean: G, H and n must be >= 1");
  SPIDER_REQUIRE(n <= 4096 && H <= 1024 && G <= 65535, SPIDER_ERR_UNSUPPORTED,
                 "spider_anchor_colmean: needs n <= 4096, H <= 1024 and G <= 65535");
  SPIDER_REQUIRE(attn && a_out, SPIDER_ERR_INVALID_ARG, "spider_anchor_colmean: null pointer argument");
  SPIDER_REQUIRE(stride_row >= n && stride_h >= (int64_t)(n - 1) * stride_row + n &&
                     stride_g >= (int64_t)(H - 1) * stride_h + (int64_t)(n - 1) * stride_row + n,
                 SPIDER_ERR_SHAPE, "spider_anchor_colmean: strides do not cover [H, n, n]");
  SPIDER_REQUIRE(n % 4 == 0 && stride_row % 4 == 0 && stride_h % 4 == 0 && stride_g % 4 == 0 &&
                     ((uintptr_t)attn % 16) == 0,
                 SPIDER_ERR_UNSUPPORTED,
                 "spider_anchor_colmean: n and the strides must be multiples of 4 and attn 16-byte aligned");
  const size_t need = colmean_ws_bytes(G, H, n);
  SPIDER_REQUIRE(workspace && workspace_bytes >= need, SPIDER_ERR_WORKSPACE,
                 "spider_anchor_colmean: workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  SPIDER_REQUIRE(((uintptr_t)workspace % 256) == 0, SPIDER_ERR_WORKSPACE,
                 "spider_anchor_colmean: workspace must be 256-byte aligned");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  float* part = reinterpret_cast<float*>(workspace);
  const int nrc = (n + kChunkRows - 1) / kChunkRows;
  {
    ProfScope ps(KC_COLMEAN, st);
    colmean_partial_kernel<<<dim3((unsigned)ceil_div(n, 256), (unsigned)(H * nrc), (unsigned)G), 256, 0, st>>>(
        H, n, attn, stride_g, stride_h, stride_row, part);
    SPIDER_LAUNCHED("colmean_partial");
    colmean_final_kernel<<<dim3((unsigned)ceil_div(n, 64), (unsigned)G), 256, 0, st>>>(H, n, part, a_out);
    SPIDER_LAUNCHED("colmean_final");
  }
  return SPIDER_OK;
}

extern "C" spider_status spider_cls_attention(int G, int H, int dh, int n_tok, const void* q,
                                              int64_t q_stride_g, const void* k, int64_t k_stride_g,
                                              int64_t k_stride_row, spider_dtype dtype, float scale,
                                              float* attn_out, spider_stream stream) {
  clear_error();
  SPIDER_REQUIRE(G >= 1 && H >= 1 && dh >= 1 && n_tok >= 1, SPIDER_ERR_INVALID_ARG,
                 "spider_cls_attention: G, H, dh and n_tok must be >= 1");
  SPIDER_REQUIRE(q && k && attn_out, SPIDER_ERR_INVALID_ARG, "spider_cls_attention: null pointer argument");
  SPIDER_REQUIRE(dtype == SPIDER_F32 || dtype == SPIDER_BF16, SPIDER_ERR_INVALID_ARG,
                 "spider_cls_attention: bad dtype");
  SPIDER_REQUIRE(std::isfinite(scale), SPIDER_ERR_INVALID_ARG, "spider_cls_attention: scale must be finite");
  SPIDER_REQUIRE(dh <= kMaxDh && n_tok <= kMaxTokens && G <= 65535 && H <= 65535, SPIDER_ERR_UNSUPPORTED,
                 "spider_cls_attention: needs dh <= 256, n_tok <= 4097, G and H <= 65535");
  SPIDER_REQUIRE(q_stride_g >= (int64_t)H * dh && k_stride_row >= (int64_t)H * dh &&
                     k_stride_g >= (int64_t)(n_tok - 1) * k_stride_row + (int64_t)H * dh,
                 SPIDER_ERR_SHAPE, "spider_cls_attention: strides do not cover [H, dh] / [n_tok, H, dh]");
  constexpr int vec = 4;  // elements per load: 16 B of fp32, 8 B of bf16
  const int align = dtype == SPIDER_F32 ? 16 : 8;
  SPIDER_REQUIRE(dh % vec == 0 && q_stride_g % vec == 0 && k_stride_g % vec == 0 && k_stride_row % vec == 0 &&
                     ((uintptr_t)q % align) == 0 && ((uintptr_t)k % align) == 0,
                 SPIDER_ERR_UNSUPPORTED,
                 "spider_cls_attention: dh and strides must be multiples of 4, q and k aligned to 4 elements");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  {
    ProfScope ps(KC_CLS_ATTN, st);
    const dim3 grid((unsigned)H, (unsigned)G);
    if (dtype == SPIDER_BF16)
      cls_attention_kernel<uint16_t><<<grid, 256, 0, st>>>(H, dh, n_tok, reinterpret_cast<const uint16_t*>(q),
                                                            q_stride_g, reinterpret_cast<const uint16_t*>(k),
                                                            k_stride_g, k_stride_row, scale, attn_out);
    else
      cls_attention_kernel<float><<<grid, 256, 0, st>>>(H, dh, n_tok, reinterpret_cast<const float*>(q),
                                                         q_stride_g, reinterpret_cast<const float*>(k), k_stride_g,
                                                         k_stride_row, scale, attn_out);
    SPIDER_LAUNCHED("cls_attention");
  }
  return SPIDER_OK;
}
