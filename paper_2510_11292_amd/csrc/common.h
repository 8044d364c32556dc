// Shared device helpers and host-side error plumbing for libLouisKV.
#pragma once

#include <hip/hip_runtime.h>
#include <algorithm>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "louiskv.h"

namespace louiskv {

constexpr int kHeadDim = 128;   // head dimension supported by every kernel
constexpr int kWave = 64;       // CDNA wavefront width

// ---------------------------------------------------------------- host side

void set_error(const char* fmt, ...);
const char* g_err_text();
int fail(int status, const char* fmt, ...);   // records the message, returns status
// Device address of a pinned, device-mapped host allocation (NULL stays NULL);
// LOUISKV_ERR_UNSUPPORTED for any other pointer.
int device_view_of_host_pool(const void* p, void** dev);

#define LKV_CHECK_HIP(expr)                                                        \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess)                                                          \
      return ::louiskv::fail(LOUISKV_ERR_HIP, "%s failed: %s (%s:%d)", #expr,      \
                             hipGetErrorString(e_), __FILE__, __LINE__);           \
  } while (0)

#define LKV_CHECK_LAUNCH() LKV_CHECK_HIP(hipGetLastError())

// LOUISKV_OK when a launch of `kernel` with `dynamic_lds` bytes of dynamic
// LDS fits the current device's LDS per workgroup (its static LDS counted),
// else LOUISKV_ERR_UNSUPPORTED: such a launch is refused, never attempted.
int check_lds(const void* kernel, size_t dynamic_lds);

// Compute units of the current device (looked up once per device), or 0 if
// the runtime cannot tell.
int device_cu_count();

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Carves aligned sub-buffers out of a caller-owned workspace.
struct Carver {
  char* base;
  size_t used = 0;
  explicit Carver(void* p) : base(static_cast<char*>(p)) {}
  template <class T>
  T* take(size_t n) {
    used = align_up(used, 256);
    T* p = reinterpret_cast<T*>(base ? base + used : nullptr);
    used += n * sizeof(T);
    return p;
  }
};

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ---------------------------------------------------------------- device side

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float32 -> bfloat16, round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <class T>
__device__ __forceinline__ float load_as_f32(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_as_f32<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_as_f32<uint16_t>(const uint16_t* p, int64_t i) {
  return bf16_to_f32(p[i]);
}

template <class T>
__device__ __forceinline__ void store_from_f32(T* p, int64_t i, float v);
template <>
__device__ __forceinline__ void store_from_f32<float>(float* p, int64_t i, float v) { p[i] = v; }
template <>
__device__ __forceinline__ void store_from_f32<uint16_t>(uint16_t* p, int64_t i, float v) {
  p[i] = f32_to_bf16(v);
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ double wave_max(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, kWave));
  return v;
}
__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

}  // namespace louiskv
