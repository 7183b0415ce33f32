// Internal helpers shared by the HIP translation units of libdvs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dvs.h"

namespace dvs {

// Per-thread error message for dvs_last_error().
void set_error(const char* fmt, ...);
void clear_error();

#define DVS_CHECK_ARG(cond, ...)                  \
  do {                                            \
    if (!(cond)) {                                \
      ::dvs::set_error(__VA_ARGS__);              \
      return DVS_EINVAL;                          \
    }                                             \
  } while (0)

#define DVS_CHECK_SUPPORTED(cond, ...)            \
  do {                                            \
    if (!(cond)) {                                \
      ::dvs::set_error(__VA_ARGS__);              \
      return DVS_EUNSUPPORTED;                    \
    }                                             \
  } while (0)

// Launch status after hipLaunchKernelGGL.
int launch_status(const char* what);

// Sampled two-forward round (sample.hip).
int launch_row_stats(const float* logits, int rows, int V, float invT, float2* stats,
                     int32_t* err, hipStream_t st);
int launch_sample_rows(const float* logits, const float2* stats, int V, float invT,
                       const float* u, int u_stride, int S, int R, int32_t* tok, hipStream_t st);
int launch_accept_final(int S, int B, int V, float invT, const float* zv, const float2* sv,
                        const float* zd, const float2* sd, const int32_t* draft, int draft_width,
                        const float* u, int u_stride, int32_t* accept_len, int32_t* am,
                        hipStream_t st);

// Bytes at the start of an attention workspace that hold the split-merge
// counters (zero between calls) for the given call shape.
size_t attn_counter_bytes(int S, int R, int Hq, int Hkv, int D, int max_pages, int chunk_keys,
                          int dtype);

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b16) {
  return __uint_as_float(b16 << 16);
}

// The value of lane ^ 32 and this lane's, in lane order: (v[l & 31], v[l | 32]).
// gfx950's v_permlane32_swap exchanges the upper half of its first operand
// with the lower half of its second; with both equal to v, lane l ends up
// holding v[l & 31] in the first result and v[l | 32] in the second (a VALU
// exchange, not the LDS round trip of a general shuffle).  Both halves see the
// pair in the same order, so a sum of the two is identical on all 64 lanes.
__device__ __forceinline__ f32x2 halves_pair(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return f32x2{__uint_as_float(r[0]), __uint_as_float(r[1])};
}

__device__ __forceinline__ void set_err(int32_t* err, int32_t bit) {
  if (err) atomicOr(err, bit);
}

// Compile-time loop: f(IC<I>{}) for I = B .. E-1, so that an index can select
// registers (ring slots, fragment arrays) without dynamic indexing.
template <int N>
struct IC {
  static constexpr int value = N;
};

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(IC<I>{});
    static_for<I + 1, N>(f);
  }
}

// Compute units of the current device (queried once; 256 if the query fails).
inline int device_cus() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      cus = v;
    else
      cus = 256;
  }
  return cus;
}

}  // namespace dvs
