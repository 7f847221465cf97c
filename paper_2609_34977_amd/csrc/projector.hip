// Multimodal projector on the kept rows only (pruning happens in the ViT
// feature space, before the projector: the appendix's reading for LLaVA and
// its AnyRes tiles).  y = W2 GELU(W1 x + b1) + b2, exact GELU.
//
//   proj_rows     per (tile g, slot r < cap): the feature row of kept patch
//                 idx[g, r] and its row in the packed decoder input (kept rows
//                 of a sample's tiles in tile order, then the sample's text rows,
//                 as spider_select assembles them); slots r >= count[g] read a
//                 valid row and are never stored
//   GEMM1         gathered feature rows x W1^T -> fp32 split-K partials
//   proj_hidden   h = act(sum of partials (split order) + b1): GELU, rounded to
//                 the activation dtype
//   GEMM2         h x W2^T -> fp32 split-K partials
//   proj_out      x_out[dst] = act(sum of partials + b2)
#include <cmath>

#include "kernels.h"

namespace spider {
namespace {

template <typename AT>
struct ProjAct;
template <>
struct ProjAct<float> {
  __device__ static inline void store(float* p, float v) { *p = v; }
};
template <>
struct ProjAct<uint16_t> {
  __device__ static inline void store(uint16_t* p, float v) { *p = f32_to_bf16_bits(v); }
};

__device__ __forceinline__ float gelu_erf(float t) { return 0.5f * t * (1.0f + erff(t * 0.70710678118654752440f)); }

// one thread per (tile, slot)
__global__ void __launch_bounds__(256) proj_rows_kernel(int G, int tps, int cap, const int32_t* __restrict__ idx,
                                                        const int32_t* __restrict__ count, int64_t rows_per_tile,
                                                        int row0, int n_text, int32_t* __restrict__ src,
                                                        int32_t* __restrict__ dst) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)G * cap) return;
  const int g = (int)(t / cap), r = (int)(t - (int64_t)g * cap);
  const int cnt = count[g];
  int64_t base = (int64_t)(g / tps) * n_text;  // rows before tile g in the packed input
  for (int u = 0; u < g; ++u) base += count[u];
  const int64_t tile_row = (int64_t)g * rows_per_tile + row0;
  if (r < cnt) {
    src[t] = (int32_t)(tile_row + idx[t]);
    dst[t] = (int32_t)(base + r);
  } else {
    src[t] = (int32_t)tile_row;
    dst[t] = -1;
  }
}

template <typename AT>
__global__ void __launch_bounds__(256) proj_hidden_kernel(int d, const float* __restrict__ P, int split,
                                                          int64_t pstride, const float* __restrict__ b,
                                                          AT* __restrict__ h) {
  const int64_t m = blockIdx.x;
  for (int c = threadIdx.x; c < d; c += 256) {
    float v = 0.f;
    for (int s = 0; s < split; ++s) v += P[s * pstride + m * d + c];
    if (b) v += b[c];
    ProjAct<AT>::store(h + m * d + c, gelu_erf(v));
  }
}

template <typename AT>
__global__ void __launch_bounds__(256) proj_out_kernel(int d, const float* __restrict__ P, int split,
                                                       int64_t pstride, const float* __restrict__ b,
                                                       const int32_t* __restrict__ dst, AT* __restrict__ y) {
  const int64_t m = blockIdx.x;
  const int r = dst[m];
  if (r < 0) return;
  for (int c = threadIdx.x; c < d; c += 256) {
    float v = 0.f;
    for (int s = 0; s < split; ++s) v += P[s * pstride + m * d + c];
    if (b) v += b[c];
    ProjAct<AT>::store(y + (int64_t)r * d + c, v);
  }
}

constexpr int kProjSplitMax = 4;

struct ProjWs {
  int32_t *src, *dst;
  void* h;
  float *P1, *P2;
  size_t bytes;
};

ProjWs proj_layout(int G, int cap, int d_hid, int d_out, spider_dtype dt, char* base) {
  ProjWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return base ? base + o : nullptr;
  };
  const size_t M = (size_t)G * cap, es = dt == SPIDER_BF16 ? 2 : 4;
  w.src = reinterpret_cast<int32_t*>(take(M * 4));
  w.dst = reinterpret_cast<int32_t*>(take(M * 4));
  w.h = take(M * d_hid * es);
  w.P1 = reinterpret_cast<float*>(take((size_t)kProjSplitMax * M * d_hid * 4));
  w.P2 = reinterpret_cast<float*>(take((size_t)kProjSplitMax * M * d_out * 4));
  w.bytes = off;
  return w;
}

template <typename AT>
spider_status run_projector(int G, int tps, int cap, const int32_t* idx, const int32_t* count, const void* feats,
                            int64_t rows_per_tile, int64_t ld_feat, int row0, int d_in, const void* w1,
                            const float* b1, int d_hid, const void* w2, const float* b2, int d_out, int n_text,
                            void* x_out, const ProjWs& ws, hipStream_t st) {
  const bool bf16 = std::is_same<AT, uint16_t>::value;
  const int M = G * cap;
  ProfScope ps(KC_PROJECTOR, st);
  proj_rows_kernel<<<(unsigned)((M + 255) / 256), 256, 0, st>>>(G, tps, cap, idx, count, rows_per_tile, row0,
                                                                 n_text, ws.src, ws.dst);
  SPIDER_LAUNCHED("proj_rows");
  GemmArgs g1{};
  g1.ngroups = 1;
  g1.K = d_in;
  g1.lda = ld_feat;
  g1.epilogue = EPI_PARTIAL_F32;
  g1.g[0] = GemmGroup{feats, ws.src, M, w1, nullptr, d_hid, ws.P1, d_hid, (int64_t)M * d_hid, 0, 0, 0};
  hipError_t e = bf16 ? launch_gemm_bf16(g1, kProjSplitMax, st) : launch_gemm_f32(g1, kProjSplitMax, st);
  SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "projector gemm 1: %s", hipGetErrorString(e));
  proj_hidden_kernel<AT><<<M, 256, 0, st>>>(d_hid, ws.P1, g1.split, (int64_t)M * d_hid, b1,
                                            reinterpret_cast<AT*>(ws.h));
  SPIDER_LAUNCHED("proj_hidden");
  GemmArgs g2{};
  g2.ngroups = 1;
  g2.K = d_hid;
  g2.lda = d_hid;
  g2.epilogue = EPI_PARTIAL_F32;
  g2.g[0] = GemmGroup{ws.h, nullptr, M, w2, nullptr, d_out, ws.P2, d_out, (int64_t)M * d_out, 0, 0, 0};
  e = bf16 ? launch_gemm_bf16(g2, kProjSplitMax, st) : launch_gemm_f32(g2, kProjSplitMax, st);
  SPIDER_REQUIRE(e == hipSuccess, SPIDER_ERR_HIP, "projector gemm 2: %s", hipGetErrorString(e));
  proj_out_kernel<AT><<<M, 256, 0, st>>>(d_out, ws.P2, g2.split, (int64_t)M * d_out, b2, ws.dst,
                                         reinterpret_cast<AT*>(x_out));
  SPIDER_LAUNCHED("proj_out");
  return SPIDER_OK;
}

}  // namespace
}  // namespace spider

using namespace spider;

extern "C" size_t spider_project_kept_workspace_size(int G, int cap, int d_hid, int d_out, spider_dtype dtype) {
  if (G <= 0 || cap <= 0 || d_hid <= 0 || d_out <= 0 || (dtype != SPIDER_F32 && dtype != SPIDER_BF16)) return 0;
  return proj_layout(G, cap, d_hid, d_out, dtype, nullptr).bytes;
}

extern "C" spider_status spider_project_kept(int G, int tiles_per_sample, int cap, const int32_t* idx,
                                             const int32_t* count, const void* feats, int64_t feat_stride_g,
                                             int64_t feat_stride_row, int feat_row0, int d_in, const void* w1,
                                             const float* b1, int d_hid, const void* w2, const float* b2,
                                             int d_out, int n_text, spider_dtype dtype, void* x_out,
                                             void* workspace, size_t workspace_bytes, spider_stream stream) {
  clear_error();
  SPIDER_REQUIRE(G >= 1 && cap >= 1 && d_in >= 1 && d_hid >= 1 && d_out >= 1 && n_text >= 0,
                 SPIDER_ERR_INVALID_ARG, "spider_project_kept: G, cap, d_in, d_hid, d_out >= 1, n_text >= 0");
  SPIDER_REQUIRE(tiles_per_sample >= 1 && G % tiles_per_sample == 0, SPIDER_ERR_SHAPE,
                 "spider_project_kept: tiles_per_sample must divide G");
  SPIDER_REQUIRE(idx && count && feats && w1 && w2 && x_out, SPIDER_ERR_INVALID_ARG,
                 "spider_project_kept: null pointer argument");
  SPIDER_REQUIRE(dtype == SPIDER_F32 || dtype == SPIDER_BF16, SPIDER_ERR_INVALID_ARG,
                 "spider_project_kept: bad dtype");
  SPIDER_REQUIRE(feat_row0 >= 0 && feat_stride_row >= d_in && feat_stride_g >= feat_stride_row &&
                     feat_stride_g % feat_stride_row == 0,
                 SPIDER_ERR_SHAPE,
                 "spider_project_kept: need feat_stride_row >= d_in and feat_stride_g a multiple of it");
  const int64_t rows_per_tile = feat_stride_g / feat_stride_row;
  SPIDER_REQUIRE((int64_t)G * rows_per_tile < INT32_MAX && (int64_t)G * cap < INT32_MAX, SPIDER_ERR_UNSUPPORTED,
                 "spider_project_kept: feature rows exceed 32-bit indices");
  if (dtype == SPIDER_BF16) {
    SPIDER_REQUIRE(d_in % 64 == 0 && d_hid % 64 == 0 && d_out % 64 == 0 && feat_stride_row % 8 == 0,
                   SPIDER_ERR_UNSUPPORTED,
                   "spider_project_kept: bf16 needs d_in, d_hid, d_out multiples of 64 and the row stride of 8");
    SPIDER_REQUIRE(((uintptr_t)feats % 16) == 0 && ((uintptr_t)w1 % 16) == 0 && ((uintptr_t)w2 % 16) == 0,
                   SPIDER_ERR_UNSUPPORTED, "spider_project_kept: feats, w1 and w2 must be 16-byte aligned");
  }
  const ProjWs need = proj_layout(G, cap, d_hid, d_out, dtype, nullptr);
  SPIDER_REQUIRE(workspace && workspace_bytes >= need.bytes, SPIDER_ERR_WORKSPACE,
                 "spider_project_kept: workspace of %zu bytes needed, %zu given", need.bytes, workspace_bytes);
  SPIDER_REQUIRE(((uintptr_t)workspace % 256) == 0, SPIDER_ERR_WORKSPACE,
                 "spider_project_kept: workspace must be 256-byte aligned");
  const ProjWs ws = proj_layout(G, cap, d_hid, d_out, dtype, reinterpret_cast<char*>(workspace));
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (dtype == SPIDER_BF16)
    return run_projector<uint16_t>(G, tiles_per_sample, cap, idx, count, feats, rows_per_tile, feat_stride_row,
                                   feat_row0, d_in, w1, b1, d_hid, w2, b2, d_out, n_text, x_out, ws, st);
  return run_projector<float>(G, tiles_per_sample, cap, idx, count, feats, rows_per_tile, feat_stride_row,
                              feat_row0, d_in, w1, b1, d_hid, w2, b2, d_out, n_text, x_out, ws, st);
}
