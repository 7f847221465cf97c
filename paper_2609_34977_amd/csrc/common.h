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

// ----------------------------------------------------------------- LDS DMA
// 16-byte-per-lane DMA from global memory into LDS at byte offset `lds` (+16
// per lane), issued as inline assembly: the compiler does not track an LDS
// DMA it cannot see, so its own LDS-read waits stay exact counts (with the
// builtin, any DMA in flight turns every fragment wait into a wait for all
// LDS reads).  Completion is the caller's business: dma_wait_barrier().
// `lds` must be the same in every lane.  NT: non-temporal (data read once).
// (m0 is declared clobbered on purpose: the compiler sets it before each of its
// own LDS DMAs, and clang warns about clobbering a reserved register)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
template <bool NT = false>
__device__ __forceinline__ void dma16(const uint16_t* g, uint32_t lds) {
  lds = __builtin_amdgcn_readfirstlane(lds);  // wave-uniform by construction
  if constexpr (NT)
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(g), "s"(lds) : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}

#pragma clang diagnostic pop

// At most N of this wave's DMAs still in flight, then the block barrier: the
// older DMAs of every wave have landed and every wave is done reading what
// the next DMAs overwrite.  One assembly statement with a memory clobber, so
// no LDS access moves across it.
template <int N = 0>
__device__ __forceinline__ void dma_wait_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}

// Every DMA of this wave complete (no barrier), as a compiler fence.
__device__ __forceinline__ void dma_wait_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// LDS byte offset of a __shared__ address (the DMA's M0 operand).
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint8_t*)p;
}

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace spider
