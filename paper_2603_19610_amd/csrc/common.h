// Internal helpers shared by the pvlm HIP sources (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cmath>
#include <cstddef>

#include "pvlm.h"

namespace pvlm {

// ------------------------------------------------------------------ host --
void set_hip_error(hipError_t e);
pvlm_status hip_check(hipError_t e);
#define PVLM_HIP(call)                               \
  do {                                               \
    hipError_t e_ = (call);                          \
    if (e_ != hipSuccess) return ::pvlm::hip_check(e_); \
  } while (0)
#define PVLM_LAUNCHED()                                        \
  do {                                                         \
    hipError_t e_ = hipGetLastError();                         \
    if (e_ != hipSuccess) return ::pvlm::hip_check(e_);        \
  } while (0)

struct DeviceInfo {
  int cus = 0;
  int xcds = 8;
};
// Compute-unit count of the current device (queried once per device).
pvlm_status device_info(DeviceInfo* out);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------- device --
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ void dev_flag(int32_t* status, int bit) {
  if (status) __hip_atomic_fetch_or(status, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Coherent (agent-scope) scalar loads/stores for data exchanged between
// workgroups that may sit on different XCDs.
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_agent(const double* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(double* p, double v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_agent(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Upper bound on polls of an inter-workgroup wait (each poll sleeps ~64
// clocks); a wait that exceeds it flags PVLM_DEV_TIMEOUT and gives up, so every
// wave always exits.
constexpr int kSpinLimit = 1 << 20;

// Arrive at a counter and wait until it reaches `target`.  Must be called by
// every thread of the workgroup (thread 0 does the atomics).  All global
// writes made by the workgroup before the call are visible (agent scope) to
// every workgroup that returns from a wait on the same counter.
__device__ __forceinline__ void wg_arrive_wait(int* counter, int target, int32_t* status,
                                               bool wait = true) {
  // every thread publishes its own prior writes before the workgroup arrives
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    if (wait) {
      int spins = 0;
      while (__hip_atomic_load(counter, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSpinLimit) {
          dev_flag(status, PVLM_DEV_TIMEOUT);
          break;
        }
      }
    }
  }
  __syncthreads();
  if (wait) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double warp_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace pvlm
