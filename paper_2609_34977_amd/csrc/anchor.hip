// Anchor scores of encoders without [CLS] (Sec. 4.1.1): the attention each
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
