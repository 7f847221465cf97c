// Complementary-token selection and decoder-input assembly (Sec. 4.1.2,
// Eq. 2; Sec. 4.1 spatial-order union; Sec. 5 AnyRes per-tile budgets).
//
// select_kernel   grid G x 1024.  Per tile: cluster sizes (LDS integer
//                 counters), quotas N_k computed exactly in integers by one
//                 thread, an LDS bitonic sort of 64-bit keys
//                 (cluster, order(s), index) that puts every cluster's
//                 members in ascending score order (ties to the lower index),
//                 membership flags for anchors and each cluster's first N_k,
//                 and a block scan that writes the kept indices ascending.
// assemble_kernel grid (ceil(cap/8), G + B) x 256.  Blocks y < G copy the
//                 kept rows of tile y (when src is given), blocks y >= G copy the text rows of
//                 sample y - G; every block derives its destination row from
//                 the tile counts (a short serial prefix over at most G
//                 values), block (0,0) writes cu_seqlens.  16-byte copies.
#include "common.h"

namespace spider {
namespace {

constexpr int kMaxN = 4096;
constexpr int kMaxK = 8;

__device__ inline void bitonic_sort(uint64_t* keys, int N) {
  for (int k = 2; k <= N; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int t = threadIdx.x; t < N / 2; t += blockDim.x) {
        const int i = (t / j) * 2 * j + (t % j);
        const int p = i + j;
        const bool up = (i & k) == 0;
        const uint64_t x = keys[i], y = keys[p];
        if ((x > y) == up) {
          keys[i] = y;
          keys[p] = x;
        }
      }
      __syncthreads();
    }
  }
}

// round(p / q) with halves to even; p >= 0, q > 0.
__device__ inline long long rne_div(long long p, long long q) {
  long long t = p / q, r = p - t * q;
  if (2 * r > q || (2 * r == q && (t & 1))) ++t;
  return t;
}

__global__ void __launch_bounds__(1024) select_kernel(int n, const int32_t* __restrict__ cluster,
                                                      const float* __restrict__ s, int n_cmp, int K,
                                                      int quota_mode, int32_t* __restrict__ idx_out,
                                                      int32_t* __restrict__ count_out, int cap) {
  __shared__ uint64_t keys[kMaxN];
  __shared__ uint16_t keep[kMaxN];
  __shared__ int size[kMaxK], quota[kMaxK], start[kMaxK];
  __shared__ int scratch[17];
  const int g = blockIdx.x;
  const int32_t* cl = cluster + (int64_t)g * n;
  const float* sg = s + (int64_t)g * n;
  if (threadIdx.x < kMaxK) size[threadIdx.x] = 0;
  __syncthreads();
  int N = 1;
  while (N < n) N <<= 1;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    uint64_t key = ~0ull;
    if (i < n) {
      const int c = cl[i];
      if (c >= 0 && c < K) {
        atomicAdd(&size[c], 1);
        key = ((uint64_t)c << 56) | ((uint64_t)float_order_key(sg[i]) << 24) | (uint64_t)i;
        keep[i] = 0;
      } else {
        keep[i] = 1;  // anchor
        key = (0xFFull << 56) | (uint64_t)i;
      }
    }
    keys[i] = key;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    long long D = 0;
    for (int k = 0; k < K; ++k) D += size[k];
    if (n_cmp <= 0 || D == 0) {
      for (int k = 0; k < K; ++k) quota[k] = 0;
    } else if (quota_mode == 0) {
      for (int k = 0; k < K; ++k) {
        const int sz = size[k];
        long long q = sz == 0 ? 0 : rne_div((long long)n_cmp * sz, D);
        if (sz > 0 && q < 1) q = 1;
        if (q > sz) q = sz;
        quota[k] = (int)q;
      }
    } else {
      const long long budget = n_cmp < D ? n_cmp : D;
      long long used = 0;
      long long rem[kMaxK];
      for (int k = 0; k < K; ++k) {
        quota[k] = (int)((budget * size[k]) / D);
        rem[k] = (budget * size[k]) % D;
        used += quota[k];
      }
      long long left = budget - used;
      bool taken[kMaxK] = {};
      for (; left > 0; --left) {
        int best = -1;
        for (int k = 0; k < K; ++k)
          if (!taken[k] && (best < 0 || rem[k] > rem[best])) best = k;
        taken[best] = true;
        quota[best] += 1;
      }
      for (int k = 0; k < K; ++k)
        if (quota[k] > size[k]) quota[k] = size[k];
    }
    int run = 0;
    for (int k = 0; k < K; ++k) {
      start[k] = run;
      run += size[k];
    }
  }
  __syncthreads();
  bitonic_sort(keys, N);
  for (int p = threadIdx.x; p < n; p += blockDim.x) {
    const uint64_t key = keys[p];
    const int c = (int)(key >> 56);
    if (c < K) {
      const int rank = p - start[c];
      if (rank < quota[c]) keep[(int)(key & 0xFFFFFFu)] = 1;
    }
  }
  __syncthreads();
  // block scan of keep flags -> ascending indices
  const int T = blockDim.x;
  const int per = (n + T - 1) / T;
  const int beg = threadIdx.x * per;
  const int end = min(n, beg + per);
  int local = 0;
  for (int i = beg; i < end; ++i) local += keep[i];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int v = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  if (lane == 63) scratch[wave] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < T / 64; ++w) {
      const int t = scratch[w];
      scratch[w] = run;
      run += t;
    }
    scratch[16] = run;
  }
  __syncthreads();
  int run = scratch[wave] + v - local;
  int32_t* out = idx_out + (int64_t)g * cap;
  for (int i = beg; i < end; ++i) {
    if (keep[i]) {
      if (run < cap) out[run] = i;
      ++run;
    }
  }
  const int total = scratch[16];
  const int cnt = total < cap ? total : cap;
  for (int t = cnt + threadIdx.x; t < cap; t += blockDim.x) out[t] = -1;
  if (threadIdx.x == 0) count_out[g] = cnt;
}

// Destination row of the first kept row of tile g, and of the text rows of
// sample b (g = b*tps + tps), in the packed layout.
__device__ inline int64_t packed_row(const int32_t* count, int g_end, int tps, int n_text) {
  int64_t r = 0;
  for (int t = 0; t < g_end; ++t) r += count[t];
  return r + (int64_t)(g_end / tps) * n_text;
}

__global__ void __launch_bounds__(256) assemble_kernel(
    int G, int tps, int cap, const int32_t* __restrict__ idx, const int32_t* __restrict__ count,
    const uint8_t* __restrict__ src, int64_t src_stride_g_bytes, int row_bytes,
    const uint8_t* __restrict__ text, int n_text, uint8_t* __restrict__ x,
    int32_t* __restrict__ cu_seqlens) {
  const int y = blockIdx.y;
  const int B = G / tps;
  if (blockIdx.x == 0 && y == 0 && threadIdx.x <= B)
    cu_seqlens[threadIdx.x] = (int32_t)packed_row(count, threadIdx.x * tps, tps, n_text);
  const int chunks = row_bytes / 16;
  if (y < G) {
    if (!src) return;
    const int cnt = count[y];
    const int64_t base = packed_row(count, y, tps, n_text);
    for (int r = blockIdx.x * 8; r < min(cnt, blockIdx.x * 8 + 8); ++r) {
      const int i = idx[(int64_t)y * cap + r];
      const uint4* sp = reinterpret_cast<const uint4*>(src + y * src_stride_g_bytes + (int64_t)i * row_bytes);
      uint4* dp = reinterpret_cast<uint4*>(x + (base + r) * row_bytes);
      for (int c = threadIdx.x; c < chunks; c += blockDim.x) dp[c] = sp[c];
    }
  } else {
    const int b = y - G;
    const int64_t base = packed_row(count, (b + 1) * tps, tps, n_text) - n_text;
    for (int r = blockIdx.x * 8; r < min(n_text, blockIdx.x * 8 + 8); ++r) {
      const uint4* sp = reinterpret_cast<const uint4*>(text + ((int64_t)b * n_text + r) * row_bytes);
      uint4* dp = reinterpret_cast<uint4*>(x + (base + r) * row_bytes);
      for (int c = threadIdx.x; c < chunks; c += blockDim.x) dp[c] = sp[c];
    }
  }
}

}  // namespace
}  // namespace spider

using namespace spider;

extern "C" spider_status spider_select(int G, int n, const int32_t* cluster, const float* s,
                                       int n_anchor, int n_cmp, int K, int quota_mode,
                                       int32_t* idx_out, int32_t* count_out, int cap,
                                       int tiles_per_sample, const void* src, int64_t src_stride_g,
                                       int d_model, spider_dtype act_dtype, const void* text,
                                       int n_text, void* x_out, int32_t* cu_seqlens_out,
                                       spider_stream stream) {
  clear_error();
  SPIDER_REQUIRE(G >= 1 && n >= 1, SPIDER_ERR_INVALID_ARG, "spider_select: G and n must be >= 1");
  SPIDER_REQUIRE(n <= kMaxN, SPIDER_ERR_UNSUPPORTED, "spider_select: n = %d exceeds 4096", n);
  SPIDER_REQUIRE(K >= 1 && K <= kMaxK, SPIDER_ERR_UNSUPPORTED, "spider_select: K must be in [1, 8]");
  SPIDER_REQUIRE(quota_mode == 0 || quota_mode == 1, SPIDER_ERR_INVALID_ARG,
                 "spider_select: quota_mode must be 0 (literal) or 1 (exact)");
  SPIDER_REQUIRE(n_anchor >= 0 && n_anchor <= n && n_cmp >= 0, SPIDER_ERR_SHAPE,
                 "spider_select: need 0 <= n_anchor <= n and n_cmp >= 0");
  SPIDER_REQUIRE(cluster && s && idx_out && count_out, SPIDER_ERR_INVALID_ARG,
                 "spider_select: null pointer argument");
  const long long need_cap = std::min<long long>(n, (long long)n_anchor + n_cmp + K);
  SPIDER_REQUIRE(cap >= need_cap, SPIDER_ERR_SHAPE,
                 "spider_select: cap = %d is below min(n, n_anchor + n_cmp + K) = %lld", cap, need_cap);
  SPIDER_REQUIRE(tiles_per_sample >= 1 && G % tiles_per_sample == 0, SPIDER_ERR_SHAPE,
                 "spider_select: tiles_per_sample must divide G");
  // assembly: with src, kept rows and text rows; with x_out but no src, the
  // text rows and boundaries only (the kept rows come from spider_project_kept)
  const bool assemble = src != nullptr || x_out != nullptr;
  size_t esz = 0;
  if (assemble) {
    SPIDER_REQUIRE(act_dtype == SPIDER_F32 || act_dtype == SPIDER_BF16, SPIDER_ERR_INVALID_ARG,
                   "spider_select: bad activation dtype");
    esz = act_dtype == SPIDER_BF16 ? 2 : 4;
    SPIDER_REQUIRE(d_model >= 8 && d_model % 8 == 0, SPIDER_ERR_UNSUPPORTED,
                   "spider_select: d_model must be a positive multiple of 8");
    SPIDER_REQUIRE(!src || (src_stride_g >= (int64_t)n * d_model && src_stride_g % 8 == 0), SPIDER_ERR_SHAPE,
                   "spider_select: src_stride_g must be >= n*d_model and a multiple of 8");
    SPIDER_REQUIRE(x_out && cu_seqlens_out, SPIDER_ERR_INVALID_ARG,
                   "spider_select: assembly needs x_out and cu_seqlens_out");
    SPIDER_REQUIRE(n_text >= 0 && (n_text == 0 || text), SPIDER_ERR_INVALID_ARG,
                   "spider_select: n_text > 0 needs text rows");
    SPIDER_REQUIRE(((uintptr_t)src % 16) == 0 && ((uintptr_t)x_out % 16) == 0 &&
                       (!text || ((uintptr_t)text % 16) == 0),
                   SPIDER_ERR_UNSUPPORTED, "spider_select: src, text and x_out must be 16-byte aligned");
    SPIDER_REQUIRE(G / tiles_per_sample <= 255, SPIDER_ERR_UNSUPPORTED,
                   "spider_select: at most 255 samples per call");
  }
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  {
    ProfScope ps(KC_SELECT, st);
    select_kernel<<<G, 1024, 0, st>>>(n, cluster, s, n_cmp, K, quota_mode, idx_out, count_out, cap);
    SPIDER_LAUNCHED("select");
  }
  if (assemble) {
    ProfScope ps(KC_ASSEMBLE, st);
    const int B = G / tiles_per_sample;
    const int rows_per_y = std::max(cap, n_text);
    dim3 grid(std::max(1, ceil_div(rows_per_y, 8)), G + B);
    assemble_kernel<<<grid, 256, 0, st>>>(
        G, tiles_per_sample, cap, idx_out, count_out, reinterpret_cast<const uint8_t*>(src),
        src_stride_g * (int64_t)esz, (int)(d_model * esz), reinterpret_cast<const uint8_t*>(text),
        n_text, reinterpret_cast<uint8_t*>(x_out), cu_seqlens_out);
    SPIDER_LAUNCHED("assemble");
  }
  return SPIDER_OK;
}
