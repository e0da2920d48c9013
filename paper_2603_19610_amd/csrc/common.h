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
  int cus = 0;   // compute units a call may plan for: the device's, or the stream's budget
  int xcds = 0;  // accelerator complex dies (workgroup i runs on die i % xcds); 0 = unknown
  bool budgeted = false;  // the stream has a compute-unit budget (pvlm_set_stream_cu_budget)
};
// Compute-unit and XCD counts of the current device (queried once per
// device); with a stream, its compute-unit budget when it has one.
pvlm_status device_info(DeviceInfo* out);
pvlm_status device_info(DeviceInfo* out, hipStream_t stream);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Every workspace starts with a fixed-size region that holds all counters of
// the inter-workgroup waits, so a zero-filled workspace can be reused by calls
// of any shape: their data areas (after the region) may overlap earlier data,
// their counters never do.  Calls whose counters return to zero use the low
// part of the region; monotonic counters (each call leaves them consistent,
// never resets them) use the rest: verify's from kSyncMonoOff, top-k's from
// kSyncTopkOff (one line per batch row), accept's at kSyncAcceptOff.
constexpr size_t kSyncRegion = 1024 * 1024;
constexpr size_t kSyncMonoOff = 256 * 1024;
constexpr size_t kSyncTopkOff = 768 * 1024;
constexpr size_t kSyncAcceptOff = 896 * 1024;
// Counters that many workgroups update or poll get a 128-byte line each, so
// the memory-side atomics and polls of different counters never contend.
constexpr size_t kSyncLine = 128;

// Raise a kernel's dynamic-LDS limit to `bytes` (done once per kernel and size).
hipError_t allow_dynamic_lds(const void* kernel, int bytes);

// PVLM_OK when `grid` workgroups of `kernel` (with `block` threads and `lds`
// dynamic LDS bytes) fit on the current device at once: the occupancy the
// runtime reports per compute unit times the compute units (the stream's
// budget when it has one).  Every launch whose workgroups wait on each other
// checks this before launching.
pvlm_status check_coresident(const void* kernel, int grid, int block, int lds,
                             hipStream_t stream);

// Launch a kernel whose workgroups wait on each other: cooperatively (the
// runtime guarantees co-residency), or as an ordinary launch while the stream
// is being captured into a graph or has a compute-unit budget (then
// co-residency rests on check_coresident and on the caller's contract: the
// device not shared, or the budgets of overlapping streams within its compute
// units).  Grids are at most one workgroup per CU.
hipError_t launch_coresident(const void* kernel, dim3 grid, dim3 block, void** args, int lds,
                             hipStream_t stream);

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

// Coherent (agent-scope) loads/stores for data exchanged between workgroups
// that may sit on different XCDs.  Each XCD has its own L2; a plain load can
// hit a stale line in the reader's L2 even after an acquire, so every read of
// another workgroup's data goes through these (they are independent loads and
// pipeline when issued back to back).
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
__device__ __forceinline__ void st_agent(float2* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), __builtin_bit_cast(uint64_t, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_agent(const float2* p) {
  const uint64_t u = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return __builtin_bit_cast(float2, u);
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

// Inter-workgroup exchange protocol.  Data another workgroup will read is
// written with st_agent (device-coherent stores) and read with ld_agent
// (device-coherent loads).  A workgroup signals with wg_signal*: every wave
// first waits for its own memory operations to complete (s_waitcnt 0, after
// which its coherent stores are visible device-wide), then thread 0 bumps the
// counter with a relaxed atomic.  Waiters poll with relaxed atomic loads.  No
// cache-wide fence is needed because no exchanged datum ever lives only in a
// non-coherent cache.
// `writer_wave0` limits the completion wait to wave 0 when only wave 0 wrote
// data other workgroups will read (the other waves may keep loads in flight).
__device__ __forceinline__ void wg_signal_wait(int* counter, int target, int32_t* status,
                                               bool wait, bool writer_wave0 = false) {
  // wave-uniform (scalar) branch: an exec-masked one would still run the wait
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (!writer_wave0 || wave == 0) __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (wait) {
      int spins = 0;
      while (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSpinLimit) {
          dev_flag(status, PVLM_DEV_TIMEOUT);
          break;
        }
      }
    }
  }
  __syncthreads();
}

// Signal without waiting; true in every thread of the workgroup whose signal
// brought the counter to `target` (the last arriver).  `s_flag` is a
// __shared__ int.
__device__ __forceinline__ bool wg_signal_last(int* counter, int target, int* s_flag) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0)
    *s_flag = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              target - 1;
  __syncthreads();
  const bool last = *s_flag != 0;
  __syncthreads();
  return last;
}

// Workgroup barrier that orders LDS only: global loads and stores stay in
// flight across it (a full __syncthreads waits for every outstanding memory
// operation of the wave first).
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ uint64_t pack_bf16x4(float x, float y, float z, float w) {
  return (uint64_t)f32_to_bf16(x) | ((uint64_t)f32_to_bf16(y) << 16) | ((uint64_t)f32_to_bf16(z) << 32) |
         ((uint64_t)f32_to_bf16(w) << 48);
}

// Monotonic group counters.  Every launch adds one arrival per workgroup of a
// group to that group's counter and never resets it; the count the counter
// had when the launch began ("base") is kept beside it.  Every workgroup reads
// the base at kernel start, waits for base + (workgroups in the group) with
// wrapping arithmetic, and the launch's last arrival at the group's final
// counter advances the base.  No end-of-kernel reset round trip is needed.
__device__ __forceinline__ unsigned grp_arrive(unsigned* counter) {
  return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned grp_read(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Bounded poll until *counter has reached `target`; flags PVLM_DEV_TIMEOUT
// and gives up after kSpinLimit polls.
__device__ __forceinline__ void grp_poll(const unsigned* counter, unsigned target, int32_t* status) {
  int spins = 0;
  while ((int)(grp_read(counter) - target) < 0) {
    __builtin_amdgcn_s_sleep(1);
    if (++spins > kSpinLimit) {
      dev_flag(status, PVLM_DEV_TIMEOUT);
      break;
    }
  }
}

// Stores and loads of data exchanged between workgroups.  LOCAL: every
// workgroup of the exchange runs on one XCD and so shares one L2; data is
// written and read once per launch at addresses the reader has not touched
// before in the launch (its L1 holds no copy), so plain accesses through that
// L2 are coherent.  Otherwise device-coherent accesses are used.
template <bool LOCAL>
__device__ __forceinline__ void x_store(float* p, float v) {
  if constexpr (LOCAL) *p = v; else st_agent(p, v);
}
template <bool LOCAL>
__device__ __forceinline__ void x_store(uint64_t* p, uint64_t v) {
  if constexpr (LOCAL) *p = v;
  else __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <bool LOCAL>
__device__ __forceinline__ void x_store(float2* p, float2 v) {
  if constexpr (LOCAL) *p = v; else st_agent(p, v);
}
template <bool LOCAL>
__device__ __forceinline__ float2 x_load(const float2* p) {
  if constexpr (LOCAL) return *p; else return ld_agent(p);
}
template <bool LOCAL>
__device__ __forceinline__ uint64_t x_load(const uint64_t* p) {
  if constexpr (LOCAL) return *p;
  else return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The cache rows of one (batch, KV head): contiguous (base = the head's row
// 0, rows of D elements), or paged: pages of 2^shift rows (a multiple of the
// 32-row block) in a pool [n_pages][Hkv][2^shift][D]; base = the pool plus
// the head's offset inside a page, page_elems = elements of one page (all
// heads), table = the sequence's page-table row (logical page -> pool page).
// A kernel may stage the entries it will use in LDS (staged, from logical
// page page0), which takes the table load off each block's address path.
struct KvRows {
  const uint16_t* base;
  const int32_t* table;  // read only when paged
  const int32_t* staged; // LDS copy of the entries from logical page page0 (used when in_lds)
  int64_t page_elems;
  int64_t n_pages;
  int shift, page0;
  bool paged, in_lds;
};

// LDS byte address of a generic pointer into LDS: the shared aperture starts
// at a multiple of 2^32, so the address is the pointer's low 32 bits.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}

// log2 of a page size that is a power of two in [32, 2^20], else -1.
inline int page_shift_of(int page_size) {
  if (page_size < 32 || page_size > (1 << 20) || (page_size & (page_size - 1))) return -1;
  int s = 0;
  while ((1 << s) < page_size) ++s;
  return s;
}

// The address of row te, where te is the 32-row block start tb, or for a
// block past the chunk end c1 the start of the block holding row c1 - 1;
// rows te .. te + 31 are contiguous from it.  A page-table entry outside the
// pool is clamped into it (the kernel flags it separately).
template <int D>
__device__ __forceinline__ const uint16_t* kv_block(const KvRows& kv, int tb, int c1, int& te) {
  te = tb < c1 ? tb : ((c1 - 1) & ~31);
  if (!kv.paged) return kv.base + (size_t)te * D;
  int page;
  if (kv.in_lds) {
    page = kv.staged[(te >> kv.shift) - kv.page0];  // already clamped
  } else {
    page = kv.table[te >> kv.shift];
    page = page < 0 ? 0 : (page >= kv.n_pages ? (int)(kv.n_pages - 1) : page);
  }
  return kv.base + (size_t)page * kv.page_elems + (size_t)(te & ((1 << kv.shift) - 1)) * D;
}

// Cross-lane exchanges that stay in the VALU (no LDS crossbar round trip):
// DPP row operations and the gfx950 permlane swaps.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xf,
                                                               0xf, false));
}
__device__ __forceinline__ float lane_xor1(float x) { return dpp_mov<0xB1>(x); }   // quad_perm 1,0,3,2
__device__ __forceinline__ float lane_xor2(float x) { return dpp_mov<0x4E>(x); }   // quad_perm 2,3,0,1
__device__ __forceinline__ float lane_xor8(float x) { return dpp_mov<0x128>(x); }  // row_ror:8
// lane i of every 8 receives lane 7 - i (row_half_mirror): partners differ in bit 2
__device__ __forceinline__ float lane_mirror8(float x) { return dpp_mov<0x141>(x); }
// Sum / max over the four lanes l, l^16, l^32, l^48 (every lane gets the result).
__device__ __forceinline__ float rows4_sum(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);  // lower row + upper row
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);            // lower half + upper half
}
__device__ __forceinline__ float rows4_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
// The value of lane l ^ 16 and of lane l ^ 32.
__device__ __forceinline__ float lane_xor16(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float((threadIdx.x & 16) ? a[0] : a[1]);
}
__device__ __forceinline__ float lane_xor32(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float((threadIdx.x & 32) ? a[0] : a[1]);
}

__device__ __forceinline__ void reset_counter(int* counter) {
  __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
