// Shared device helpers of libmoe (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/moe.h"

namespace moe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Compute units of the current device (cached per device; 256 if unknown).
inline int num_cus() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

// bf16 bit pattern -> float (exact)
__device__ __forceinline__ float bf2f(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// float -> bf16 bit pattern, round to nearest even (hardware v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint16_t f2bf(float f) {
  __bf16 b = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, b);
}

// two floats -> packed bf16x2 (lo in bits 0..15)
__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
  bf16x2 v;
  v.x = static_cast<__bf16>(lo);
  v.y = static_cast<__bf16>(hi);
  return __builtin_bit_cast(uint32_t, v);
}

// 16 bytes = 8 bf16 <-> 8 floats
__device__ __forceinline__ void unpack8(const uint4& v, float* f) {
  f[0] = __uint_as_float(v.x << 16); f[1] = __uint_as_float(v.x & 0xFFFF0000u);
  f[2] = __uint_as_float(v.y << 16); f[3] = __uint_as_float(v.y & 0xFFFF0000u);
  f[4] = __uint_as_float(v.z << 16); f[5] = __uint_as_float(v.z & 0xFFFF0000u);
  f[6] = __uint_as_float(v.w << 16); f[7] = __uint_as_float(v.w & 0xFFFF0000u);
}
__device__ __forceinline__ uint4 pack8(const float* f) {
  uint4 v;
  v.x = pack2bf(f[0], f[1]); v.y = pack2bf(f[2], f[3]);
  v.z = pack2bf(f[4], f[5]); v.w = pack2bf(f[6], f[7]);
  return v;
}

// Element traits: the kernels move 16-byte vectors, 8 bf16 or 4 fp32 values.
template <typename T> struct Elem;
template <> struct Elem<uint16_t> {
  static constexpr int kVec = 8;  // elements per 16 bytes
  __device__ static __forceinline__ void load(const uint4& v, float* f) { unpack8(v, f); }
  __device__ static __forceinline__ uint4 store(const float* f) { return pack8(f); }
  __device__ static __forceinline__ float to_f(uint16_t h) { return bf2f(h); }
  __device__ static __forceinline__ uint16_t from_f(float x) { return f2bf(x); }
};
template <> struct Elem<float> {
  static constexpr int kVec = 4;
  __device__ static __forceinline__ void load(const uint4& v, float* f) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
  __device__ static __forceinline__ uint4 store(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]),
                      __float_as_uint(f[2]), __float_as_uint(f[3]));
  }
  __device__ static __forceinline__ float to_f(float x) { return x; }
  __device__ static __forceinline__ float from_f(float x) { return x; }
};

// Wave-wide sums (64 lanes) via cross-lane shuffles.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ int ceil_div_i(int a, int b) { return (a + b - 1) / b; }

// ---- opt-in kernel timing (moe_timing_enable / moe_timing_report) ---------
// While enabled, each library kernel launch is bracketed by two HIP events
// recorded on the launch stream; the report aggregates them by kernel name.
bool timing_enabled();
void timing_record(const char* name, hipStream_t s, bool start);

struct TimedLaunch {
  const char* name;
  hipStream_t s;
  bool on;
  TimedLaunch(const char* n, hipStream_t st) : name(n), s(st), on(timing_enabled()) {
    if (on) timing_record(name, s, true);
  }
  ~TimedLaunch() {
    if (on) timing_record(name, s, false);
  }
};

}  // namespace moe

#define MOE_TIMED(name, stream) ::moe::TimedLaunch moe_timed_scope_(name, stream)

// Host-side launch check: returns MOE_EHIP from the calling entry point.
#define MOE_LAUNCH_CHECK()                                   \
  do {                                                       \
    if (hipGetLastError() != hipSuccess) return MOE_EHIP;    \
  } while (0)
