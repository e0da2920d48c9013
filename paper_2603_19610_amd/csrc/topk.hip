// Top-K keep (gfx950): Eq. (topk_selection) of ParallelVLM Sec. 4.1, keeping
// the top 1 - alpha fraction of visual tokens (Sec. 4.2).
//
// Ranking: larger score first, lower index first among equal scores, -0.0
// equal to +0.0, NaN below every number.  Each score maps to a 32-bit key
// whose unsigned order is that ranking (ties aside); the K-th largest key is
// found by an MSB-first radix select (four 8-bit digits, LDS histograms), and
// one ordered pass then emits, in ascending index order, every index whose key
// is above the threshold plus the lowest-indexed ones equal to it.
// One 1024-thread workgroup per batch row; the whole selection is integer
// work, so the result is bit-exact.
#include "common.h"

namespace pvlm {
namespace {

constexpr int kTopkThreads = 1024;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kPerThread = 16;  // consecutive elements per thread in the ordered pass

__device__ __forceinline__ uint32_t rank_key(float f) {
  if (f != f) return 0u;                 // NaN: lowest
  uint32_t u = __float_as_uint(f);
  if (f == 0.f) u = 0u;                  // -0.0 ranks as +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the workgroup; returns the exclusive prefix of
// this thread and writes the total to *total.
__device__ __forceinline__ int block_exclusive_scan(int v, int* s_warp, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_warp[w] = x;
  __syncthreads();
  if (w == 0) {
    int t = lane < kTopkWaves ? s_warp[lane] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(t, o, 64);
      if (lane >= o) t += y;
    }
    if (lane < kTopkWaves) s_warp[lane] = t;  // inclusive over waves
  }
  __syncthreads();
  const int before = w > 0 ? s_warp[w - 1] : 0;
  *total = s_warp[kTopkWaves - 1];
  __syncthreads();
  return before + x - v;
}

__global__ void __launch_bounds__(kTopkThreads) topk_kernel(const float* score, const int32_t* m,
                                                            const int32_t* k, int64_t m_cap,
                                                            int k_cap, int32_t* idx,
                                                            int32_t* status) {
  __shared__ int hist[256];
  __shared__ int s_warp[kTopkWaves];
  __shared__ int s_digit, s_above;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const float* sc = score + (size_t)b * m_cap;
  int32_t* out = idx + (size_t)b * k_cap;

  int mb = m[b], kb = k[b];
  bool bad = false;
  if (mb < 0 || mb > m_cap) {
    bad = true;
    mb = mb < 0 ? 0 : (int)m_cap;
  }
  const int kmax = mb < k_cap ? mb : k_cap;
  if (kb < 0 || kb > kmax) {
    bad = true;
    kb = kb < 0 ? 0 : kmax;
  }
  if (bad && tid == 0) dev_flag(status, PVLM_DEV_RANGE);
  for (int r = kb + tid; r < k_cap; r += kTopkThreads) out[r] = -1;
  if (kb == 0) return;

  // ---- radix select of the kb-th largest key
  uint32_t prefix = 0, mask = 0;
  int above = 0;  // keys strictly above the current prefix range
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = tid; i < 256; i += kTopkThreads) hist[i] = 0;
    __syncthreads();
    for (int i = tid; i < mb; i += kTopkThreads) {
      const uint32_t key = rank_key(sc[i]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1);
    }
    __syncthreads();
    if (tid < 64) {
      // lane l owns digits 255-4l .. 252-4l (descending); scan from the top
      int c[4], own = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[q] = hist[255 - 4 * tid - q];
        own += c[q];
      }
      int incl = own;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (tid >= o) incl += y;
      }
      const int excl = incl - own;
      const int need = kb - above;
      if (excl < need && need <= incl) {
        int acc = excl;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (acc + c[q] >= need) {
            s_digit = 255 - 4 * tid - q;
            s_above = above + acc;
            break;
          }
          acc += c[q];
        }
      }
    }
    __syncthreads();
    prefix |= (uint32_t)s_digit << shift;
    mask |= 255u << shift;
    above = s_above;
    __syncthreads();
  }
  const uint32_t tau = prefix;
  const int need_eq = kb - above;  // >= 1 keys equal to tau, lowest indices first

  // ---- ordered emission in ascending index order
  int carry_eq = 0, carry_out = 0;
  for (int base = 0; base < mb; base += kTopkThreads * kPerThread) {
    const int i0 = base + tid * kPerThread;
    uint32_t keys[kPerThread];
    int n_gt = 0, n_eq = 0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int i = i0 + e;
      keys[e] = i < mb ? rank_key(sc[i]) : 0u;
      const bool valid = i < mb;
      n_gt += valid && keys[e] > tau;
      n_eq += valid && keys[e] == tau;
    }
    int tot_eq;
    const int eq_before = carry_eq + block_exclusive_scan(n_eq, s_warp, &tot_eq);
    int take_eq = need_eq - eq_before;
    take_eq = take_eq < 0 ? 0 : (take_eq > n_eq ? n_eq : take_eq);
    int tot_sel;
    int pos = carry_out + block_exclusive_scan(n_gt + take_eq, s_warp, &tot_sel);
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int i = i0 + e;
      if (i < mb) {
        bool sel = keys[e] > tau;
        if (keys[e] == tau && take_eq > 0) {
          sel = true;
          --take_eq;
        }
        if (sel && pos < kb) out[pos++] = i;
      }
    }
    carry_eq += tot_eq;
    carry_out += tot_sel;
  }
}

}  // namespace
}  // namespace pvlm

using namespace pvlm;

extern "C" size_t pvlm_topk_workspace_size(int B, int64_t m_cap) {
  (void)B;
  (void)m_cap;
  return 0;
}

extern "C" pvlm_status pvlm_topk_select(int B, int64_t m_cap, const int32_t* m, const int32_t* k,
                                        int32_t k_cap, const float* score, int32_t* idx, void* ws,
                                        size_t ws_bytes, int32_t* status, hipStream_t stream) {
  (void)ws;
  (void)ws_bytes;
  if (!m || !k || !score || !idx) return PVLM_ERR_NULL;
  if (B < 1 || m_cap < 1 || k_cap < 0 || m_cap > ((int64_t)1 << 30)) return PVLM_ERR_SHAPE;
  if (k_cap == 0) return PVLM_OK;
  hipLaunchKernelGGL(topk_kernel, dim3(B), dim3(kTopkThreads), 0, stream, score, m, k, m_cap,
                     k_cap, idx, status);
  PVLM_LAUNCHED();
  return PVLM_OK;
}
