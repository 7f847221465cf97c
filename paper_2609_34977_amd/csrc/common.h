// Internal helpers shared by the HIP sources of libspider (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdarg>
#include <cstdio>
#include <string>
#include <type_traits>

#include "../../include/spider.h"

namespace spider {

// ----------------------------------------------------------------- errors
void set_error(const char* fmt, ...);
void clear_error();

#define SPIDER_REQUIRE(cond, code, ...)        \
  do {                                         \
    if (!(cond)) {                             \
      ::spider::set_error(__VA_ARGS__);        \
      return code;                             \
    }                                          \
  } while (0)

#define SPIDER_HIP(call)                                                          \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess) {                                                       \
      ::spider::set_error("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_),  \
                          __FILE__, __LINE__);                                    \
      return SPIDER_ERR_HIP;                                                      \
    }                                                                             \
  } while (0)

#define SPIDER_LAUNCHED(what)                                                       \
  do {                                                                              \
    hipError_t e_ = hipGetLastError();                                              \
    if (e_ != hipSuccess) {                                                         \
      ::spider::set_error("launch of %s failed: %s", what, hipGetErrorString(e_));  \
      return SPIDER_ERR_HIP;                                                        \
    }                                                                               \
  } while (0)

// ----------------------------------------------------------------- profiler
enum KernelClass {
  KC_SCORE_PREP = 0,
  KC_ANCHOR_TOPK,
  KC_KMEANS,
  KC_MAXSIM,
  KC_SCORE_FINAL,
  KC_SELECT,
  KC_ASSEMBLE,
  KC_EMBED,
  KC_RMSNORM,
  KC_GEMM_QKV,
  KC_QKV_FINALIZE,
  KC_ATTENTION,
  KC_GEMM_O,
  KC_GEMM_GATEUP,
  KC_GEMM_DOWN,
  KC_RESIDUAL,
  KC_LENS_PREP,
  KC_GEMM_LENS,
  KC_LENS_ADMIT,
  KC_COLMEAN,
  KC_CLS_ATTN,
  KC_PROJECTOR,
  KC_LM_HEAD,
  KC_COUNT
};

// Records a start event when profiling is enabled; the matching prof_end()
// records the stop event.  Both are no-ops otherwise.
void prof_begin(int cls, hipStream_t s);
void prof_end(int cls, hipStream_t s);

struct ProfScope {
  int cls;
  hipStream_t s;
  ProfScope(int c, hipStream_t st) : cls(c), s(st) { prof_begin(c, st); }
  ~ProfScope() { prof_end(cls, s); }
};

// ----------------------------------------------------------------- math helpers
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
// Native 16-byte vector (HIP's uint4 is a struct whose copies can be lowered
// through private memory).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Order-preserving map of a float to uint32 (-0.0 is mapped like +0.0).
__device__ __forceinline__ uint32_t float_order_key(float f) {
  if (f == 0.0f) f = 0.0f;
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace spider
