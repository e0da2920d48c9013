// Top-K keep (gfx950): Eq. (topk_selection) of ParallelVLM Sec. 4.1, keeping
// the top 1 - alpha fraction of visual tokens (Sec. 4.2).
//
// Ranking: larger score first, lower index first among equal scores, -0.0
// equal to +0.0, NaN below every number.  Each score maps to a 32-bit key
// whose unsigned order is that ranking (ties aside); the K-th largest key is
// found by an MSB-first radix select (four 8-bit digits), and one ordered
// pass then emits, in ascending index order, every index whose key is above
// the threshold plus the lowest-indexed ones equal to it.  The whole
// selection is integer work, so the result is bit-exact.
//
// Rows of up to 16384 scores take one 1024-thread workgroup each, the keys in
// registers.  Longer rows are split over NW workgroups (one launch, grid
// co-resident):
// per digit, every workgroup histograms its slice in LDS and publishes it;
// the last to arrive sums the NW histograms, picks the digit and publishes
// it; the others wait for it.  The emission step exchanges per-slice counts
// the same way so every workgroup knows where its slice's output starts.
#include "common.h"

namespace pvlm {
namespace {

constexpr int kTopkThreads = 256;
constexpr int kTopkWaves = kTopkThreads / 64;
constexpr int kPerThread = 16;   // consecutive scores per thread (register slice, ordered pass)
constexpr int kSlice = kTopkThreads * kPerThread;  // scores per workgroup unless B*NW would exceed the CUs
constexpr int kBarriers = 5;     // four digits and the emission counts
static_assert(kTopkThreads == 256, "one histogram bin per thread");

__device__ __forceinline__ uint32_t rank_key(float f) {
  if (f != f) return 0u;                 // NaN: lowest
  uint32_t u = __float_as_uint(f);
  if (f == 0.f) u = 0u;                  // -0.0 ranks as +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over a workgroup of WAVES waves; returns the exclusive
// prefix of this thread and writes the total to *total.
template <int WAVES = kTopkWaves>
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
  int before = 0;
#pragma unroll
  for (int ww = 0; ww < WAVES; ++ww) before += ww < w ? s_warp[ww] : 0;
  int tot = 0;
#pragma unroll
  for (int ww = 0; ww < WAVES; ++ww) tot += s_warp[ww];
  *total = tot;
  __syncthreads();
  return before + x - v;
}

// One wave (lanes 0-63): the digit of a 256-bin histogram (counts of the
// keys in the current prefix range, by next digit) that holds the need-th
// largest key, scanning digits from the top.  Lane l owns digits 255 - 4l ..
// 252 - 4l.  The lane that finds it calls found(digit, keys above the digit).
template <typename F>
__device__ __forceinline__ void find_digit(const int* hist, int need, F found) {
  const int lane = threadIdx.x & 63;
  int c[4], own = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    c[q] = hist[255 - 4 * lane - q];
    own += c[q];
  }
  int incl = own;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  const int excl = incl - own;
  if (excl < need && need <= incl) {
    int acc = excl;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (acc + c[q] >= need) {
        found(255 - 4 * lane - q, acc);
        break;
      }
      acc += c[q];
    }
  }
}

struct TArgs {
  const float* score;    // scores, or (fused MASS form) crit^L
  const float* sub;      // fused MASS form: crit^0, subtracted from crit^L; else NULL
  float* score_out;      // fused MASS form: the scores written out (nullable)
  const int32_t* m;
  const int32_t* k;
  int32_t* idx;
  int32_t* status;
  int* hist;       // [B][NW][256] per-slice digit histograms
  int* res;        // [B][4]: digit, keys above the prefix range
  int* cnt;        // [B][NW][2]: keys above the threshold, keys equal to it
  int* arrive;     // [B] arrivals (128 B apart), back to zero after each call
  unsigned* gen;   // [B] generation words (128 B apart), advanced per barrier
  int64_t m_cap;
  int k_cap, NW, slice;
};

constexpr int kLine = (int)(kSyncLine / sizeof(int));

// Entry i of a row (row offset `off`): the score, or in the fused MASS form
// the UV-Prune variation crit^L - crit^0 of Eq. (average_similarity),
// rounded exactly as pvlm_uvprune_score(MASS) rounds it (one fp32 subtraction).
template <bool FUSED>
__device__ __forceinline__ float score_at(const TArgs& a, size_t off, int64_t i) {
  if constexpr (FUSED) return a.score[off + i] - a.sub[off + i];
  else return a.score[off + i];
}

// A pair of ints exchanged between workgroups as one device-coherent 64-bit
// access (8-byte aligned): one round trip for both, and a consistent pair.
__device__ __forceinline__ void st_pair(int* p, int lo, int hi) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), (uint64_t)(uint32_t)lo | ((uint64_t)(uint32_t)hi << 32),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int2 ld_pair(const int* p) {
  const uint64_t v =
      __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_int2((int)(uint32_t)v, (int)(uint32_t)(v >> 32));
}

// Barrier `p` (0-based) of row b.  Thread 0 arrives; the launch's last arrival
// runs `last` (with the whole workgroup) and then releases the others, which
// wait for the generation word to reach g0 + p + 1.  Returns in every thread.
template <typename F>
__device__ __forceinline__ void row_barrier(const TArgs& a, int b, int p, unsigned g0, int* s_flag,
                                            F last) {
  __builtin_amdgcn_s_waitcnt(0);  // this workgroup's published data is visible
  __syncthreads();
  if (threadIdx.x == 0) {
    const int old = __hip_atomic_fetch_add(a.arrive + b * kLine, 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
    *s_flag = old == a.NW * (p + 1) - 1;
  }
  __syncthreads();
  if (*s_flag) {
    last();
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
      if (p == kBarriers - 1)  // every workgroup has arrived for the last time
        __hip_atomic_store(a.arrive + b * kLine, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.gen + b * kLine, g0 + (unsigned)p + 1u, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
  } else if (threadIdx.x == 0) {
    grp_poll(a.gen + b * kLine, g0 + (unsigned)p + 1u, a.status);
  }
  __syncthreads();
}

// REG: the slice (at most kTopkThreads * kPerThread scores) is read once into
// registers, thread t holding the scores s0 + kPerThread*t + e; otherwise it
// is read again from memory for every pass, in chunks of that size.
template <bool REG, bool FUSED>
__global__ void __launch_bounds__(kTopkThreads) topk_kernel(TArgs a) {
  constexpr int kChunk = kTopkThreads * kPerThread;
  __shared__ int hist[256];
  __shared__ int s_warp[kTopkWaves];
  __shared__ int s_flag, s_res[2];
  const int b = blockIdx.x / a.NW, j = blockIdx.x % a.NW;
  const int tid = threadIdx.x;
  const size_t roff = (size_t)b * a.m_cap;
  int32_t* out = a.idx + (size_t)b * a.k_cap;
  // the generation at launch start, read before this workgroup first arrives
  // (only thread 0 arrives and waits)
  const unsigned g0 = tid == 0 ? grp_read(a.gen + b * kLine) : 0u;

  int mb = a.m[b], kb = a.k[b];
  bool bad = false;
  if (mb < 0 || mb > a.m_cap) {
    bad = true;
    mb = mb < 0 ? 0 : (int)a.m_cap;
  }
  const int kmax = mb < a.k_cap ? mb : a.k_cap;
  if (kb < 0 || kb > kmax) {
    bad = true;
    kb = kb < 0 ? 0 : kmax;
  }
  if (bad && j == 0 && tid == 0) dev_flag(a.status, PVLM_DEV_RANGE);
  if (j == 0)
    for (int r = kb + tid; r < a.k_cap; r += kTopkThreads) out[r] = -1;
  const int s0 = min(mb, j * a.slice), s1 = min(mb, s0 + a.slice);
  int* hrow = a.hist + (size_t)b * a.NW * 256;
  if constexpr (FUSED) {  // the scores of this workgroup's share of the row (0 past m[b])
    if (a.score_out && !REG) {
      const int64_t e1 = min((int64_t)(j + 1) * a.slice, a.m_cap);
      for (int64_t i = (int64_t)j * a.slice + tid; i < e1; i += kTopkThreads)
        a.score_out[roff + i] = i < mb ? score_at<true>(a, roff, i) : 0.f;
    } else if (a.score_out) {  // past m[b] only; the kept slice is written with its keys
      const int64_t e0 = max((int64_t)j * a.slice, (int64_t)mb);
      const int64_t e1 = min((int64_t)(j + 1) * a.slice, a.m_cap);
      for (int64_t i = e0 + tid; i < e1; i += kTopkThreads) a.score_out[roff + i] = 0.f;
    }
  }

  uint32_t kr[kPerThread];
  if constexpr (REG) {
    const int i0 = s0 + tid * kPerThread;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e)
      kr[e] = __float_as_uint(score_at<FUSED>(a, roff, min(i0 + e, s1 > 0 ? s1 - 1 : 0)));
    if constexpr (FUSED) {
      if (a.score_out)
#pragma unroll
        for (int e = 0; e < kPerThread; ++e)
          if (i0 + e < s1) a.score_out[roff + i0 + e] = __uint_as_float(kr[e]);
    }
#pragma unroll  // (clamped loads, all in flight together, then the keys)
    for (int e = 0; e < kPerThread; ++e) kr[e] = i0 + e < s1 ? rank_key(__uint_as_float(kr[e])) : 0u;
  }
  // f(key) over this thread's scores of the slice
  auto visit = [&](auto f) {
    if constexpr (REG) {
      const int nv = s1 - (s0 + tid * kPerThread);
#pragma unroll
      for (int e = 0; e < kPerThread; ++e)
        if (e < nv) f(kr[e]);
    } else {
      for (int i = s0 + tid; i < s1; i += kTopkThreads) f(rank_key(score_at<FUSED>(a, roff, i)));
    }
  };

  // ---- radix select of the kb-th largest key.  With kb == 0 nothing is
  //      counted, but every barrier is still passed.
  uint32_t prefix = 0, mask = 0;
  int above = 0;  // keys strictly above the current prefix range
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    hist[tid] = 0;
    __syncthreads();
    if (kb > 0)
      visit([&](uint32_t key) {
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1);
      });
    __syncthreads();
    st_agent(hrow + j * 256 + tid, hist[tid]);
    row_barrier(a, b, pass, g0, &s_flag, [&]() {
      // the last workgroup: total histogram, then the digit holding the
      // kb-th largest key (scanning digits from the top)
      int t = 0;
      for (int j0 = 0; j0 < a.NW; j0 += 8) {
        int v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {  // clamped loads, all in flight together
          const int x = ld_agent(hrow + min(j0 + q, a.NW - 1) * 256 + tid);
          v[q] = j0 + q < a.NW ? x : 0;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) t += v[q];
      }
      hist[tid] = t;
      __syncthreads();
      if (tid < 64)
        find_digit(hist, kb - above, [&](int digit, int acc) {
          st_pair(a.res + b * 4, digit, above + acc);
        });
    });
    if (tid == 0) {
      const int2 r = ld_pair(a.res + b * 4);
      s_res[0] = r.x;
      s_res[1] = r.y;
    }
    __syncthreads();
    if (kb > 0) {
      prefix |= (uint32_t)s_res[0] << shift;
      mask |= 255u << shift;
      above = s_res[1];
    }
    __syncthreads();
  }
  const uint32_t tau = prefix;
  const int need_eq = kb - above;  // keys equal to tau to keep, lowest indices first

  // ---- this slice's counts, exchanged: where its output starts
  int n_gt = 0, n_eq = 0;
  if (kb > 0)
    visit([&](uint32_t key) {
      n_gt += key > tau;
      n_eq += key == tau;
    });
  int slice_gt, slice_eq;
  block_exclusive_scan(n_gt, s_warp, &slice_gt);
  block_exclusive_scan(n_eq, s_warp, &slice_eq);
  if (tid == 0) {
    st_pair(a.cnt + ((size_t)b * a.NW + j) * 2, slice_gt, slice_eq);
  }
  row_barrier(a, b, 4, g0, &s_flag, []() {});
  if (kb == 0) return;
  if (tid < 64) {  // counts of the slices before this one
    int gt = 0, eq = 0;
    for (int q = tid; q < j; q += 64) {
      const int2 c = ld_pair(a.cnt + ((size_t)b * a.NW + q) * 2);
      gt += c.x;
      eq += c.y;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      gt += __shfl_xor(gt, o, 64);
      eq += __shfl_xor(eq, o, 64);
    }
    if (tid == 0) {
      s_res[0] = gt;
      s_res[1] = eq;
    }
  }
  __syncthreads();
  int carry_out = s_res[0] + min(s_res[1], need_eq);
  int carry_eq = s_res[1];

  // ---- ordered emission of the slice in ascending index order
  for (int base = s0; base < s1; base += kChunk) {
    const int i0 = base + tid * kPerThread;
    uint32_t keys[kPerThread];
    int g = 0, e_ = 0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const bool valid = i0 + e < s1;
      if constexpr (REG) keys[e] = kr[e];
      else {
        const float x = score_at<FUSED>(a, roff, min(i0 + e, s1 - 1));  // clamped (s1 > base >= 0)
        keys[e] = valid ? rank_key(x) : 0u;
      }
      g += valid && keys[e] > tau;
      e_ += valid && keys[e] == tau;
    }
    int tot_eq;
    const int eq_before = carry_eq + block_exclusive_scan(e_, s_warp, &tot_eq);
    int take_eq = need_eq - eq_before;
    take_eq = take_eq < 0 ? 0 : (take_eq > e_ ? e_ : take_eq);
    int tot_sel;
    int pos = carry_out + block_exclusive_scan(g + take_eq, s_warp, &tot_sel);
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      if (i0 + e < s1) {
        bool sel = keys[e] > tau;
        if (keys[e] == tau && take_eq > 0) {
          sel = true;
          --take_eq;
        }
        if (sel && pos < kb) out[pos++] = i0 + e;
      }
    }
    carry_eq += tot_eq;
    carry_out += tot_sel;
  }
}

// Rows of at most kSmallMax scores: one 1024-thread workgroup per row, no
// inter-workgroup exchange.  Thread t holds the keys of entries e * 1024 + t
// (coalesced loads) in registers.  The radix select takes three digits of
// 12, 10 and 10 bits: float keys of real data share few values of their top
// 8 bits (sign and exponent), and a first digit that wide spreads them over
// enough histogram bins that the LDS atomics rarely collide.  The ordered
// emission computes every selected entry's output position directly from
// per-(entry round, wave) counts, so no thread needs a contiguous range.
constexpr int kSmallThreads = 1024;
constexpr int kSmallWaves = kSmallThreads / 64;
constexpr int kSmallMaxPer = 16;  // beyond 16384 scores, several workgroups per row are faster
constexpr int kSmallMax = kSmallThreads * kSmallMaxPer;
constexpr int kSmallBins = 4096;
// Every histogram bin has kHistCopies counters, lane l adding to copy l % 8:
// scores concentrate in few top digits (the UV-Prune scores of a 72B layer
// fill 29 of the 4096 first-pass bins), and LDS atomics of one instruction to
// one address serialise.
constexpr int kHistCopies = 8;
constexpr int kSmallLds = kSmallBins * (kHistCopies + 1) * 4;  // the copies, then the bin totals

template <int PER, bool FUSED>
__global__ void __launch_bounds__(kSmallThreads) topk_small_kernel(TArgs a) {
  extern __shared__ __align__(16) int hist[];  // [kSmallBins][kHistCopies], then [kSmallBins] totals
  int* bins = hist + kSmallBins * kHistCopies;
  __shared__ int s_warp[kSmallWaves];
  __shared__ int s_res[2];
  __shared__ int s_cnt[2][PER][kSmallWaves];  // per (round e, wave): keys above tau, equal to tau
  const int b = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const size_t roff = (size_t)b * a.m_cap;
  int32_t* out = a.idx + (size_t)b * a.k_cap;
  int mb = a.m[b], kb = a.k[b];
  bool bad = false;
  if (mb < 0 || mb > a.m_cap) {
    bad = true;
    mb = mb < 0 ? 0 : (int)a.m_cap;
  }
  const int kmax = mb < a.k_cap ? mb : a.k_cap;
  if (kb < 0 || kb > kmax) {
    bad = true;
    kb = kb < 0 ? 0 : kmax;
  }
  if (bad && tid == 0) dev_flag(a.status, PVLM_DEV_RANGE);
  for (int r = kb + tid; r < a.k_cap; r += kSmallThreads) out[r] = -1;
  if (!FUSED && kb == 0) return;  // uniform across the workgroup
  // unconditional loads (indices clamped into the row, or to entry 0 of an
  // empty row) so that all PER are in flight together, then the entries past
  // the row are zeroed
  float v[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) v[e] = score_at<FUSED>(a, roff, min(e * kSmallThreads + tid, max(mb - 1, 0)));
  // the first digit's histogram (every copy) is cleared while the keys load
  __builtin_amdgcn_sched_barrier(0);
  for (int i = tid; i < kSmallBins * kHistCopies / 4; i += kSmallThreads)
    reinterpret_cast<int4*>(hist)[i] = make_int4(0, 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (FUSED) {  // the scores written out (0 past m[b]), then the selection
    if (a.score_out)
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const int i = e * kSmallThreads + tid;
        if (i < a.m_cap) a.score_out[roff + i] = i < mb ? v[e] : 0.f;
      }
    if (kb == 0) return;
  }
  uint32_t kr[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) kr[e] = e * kSmallThreads + tid < mb ? rank_key(v[e]) : 0u;

  // ---- radix select of the kb-th largest key: digits [31:20], [19:10], [9:0].
  // The first digit's keys crowd into few bins (the sign and exponent of
  // real scores), so its histogram has kHistCopies counters per bin; the later
  // digits count only the keys left in the chosen bin, one counter per bin.
  uint32_t prefix = 0, mask = 0;
  int above = 0;
#pragma unroll 1
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 20 : (pass == 1 ? 10 : 0);
    const int nb = pass == 0 ? 4096 : 1024;
    const int copies = pass == 0 ? kHistCopies : 1;
    if (pass > 0)
      for (int i = tid; i < nb / 4; i += kSmallThreads) reinterpret_cast<int4*>(hist)[i] = make_int4(0, 0, 0, 0);
    __syncthreads();
    const int copy = pass == 0 ? (lane & (kHistCopies - 1)) : 0;
#pragma unroll
    for (int e = 0; e < PER; ++e)
      if (e * kSmallThreads + tid < mb && (kr[e] & mask) == prefix)
        atomicAdd(&hist[((kr[e] >> shift) & (uint32_t)(nb - 1)) * copies + copy], 1);
    __syncthreads();
    if (pass == 0) {
      // each bin's copies summed, consecutive threads on consecutive bins
      for (int i = tid; i < nb; i += kSmallThreads) {
        const int4* h = reinterpret_cast<const int4*>(hist + i * kHistCopies);
        const int4 x = h[0], y = h[1];
        bins[i] = x.x + x.y + x.z + x.w + y.x + y.y + y.z + y.w;
      }
      __syncthreads();
    }
    const int* totals = pass == 0 ? bins : hist;
    // bins in descending order: thread t owns q = nb / 1024 consecutive ones
    const int q = nb / kSmallThreads;
    const int top = nb - 1 - tid * q;
    int cnt[kSmallBins / kSmallThreads];
    int own = 0;
#pragma unroll
    for (int j = 0; j < kSmallBins / kSmallThreads; ++j) {
      cnt[j] = j < q ? totals[top - j] : 0;
      own += cnt[j];
    }
    int tot;
    const int excl = block_exclusive_scan<kSmallWaves>(own, s_warp, &tot);
    const int need = kb - above;
    if (excl < need && need <= excl + own) {
      int acc = excl;
#pragma unroll
      for (int j = 0; j < kSmallBins / kSmallThreads; ++j) {
        if (j < q) {
          if (acc + cnt[j] >= need) {
            s_res[0] = top - j;
            s_res[1] = above + acc;
            break;
          }
          acc += cnt[j];
        }
      }
    }
    __syncthreads();
    prefix |= (uint32_t)s_res[0] << shift;
    mask |= (uint32_t)(nb - 1) << shift;
    above = s_res[1];
  }
  const uint32_t tau = prefix;
  const int need_eq = kb - above;  // keys equal to tau to keep, lowest indices first

  // ---- emission: output position of entry (e, w, lane) = keys above tau
  //      before it + min(keys equal to tau before it, need_eq)
  uint64_t bg[PER], be[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const bool valid = e * kSmallThreads + tid < mb;
    bg[e] = __ballot(valid && kr[e] > tau);
    be[e] = __ballot(valid && kr[e] == tau);
    if (lane == 0) {
      s_cnt[0][e][w] = __popcll(bg[e]);
      s_cnt[1][e][w] = __popcll(be[e]);
    }
  }
  __syncthreads();
  // exclusive prefix over (e, w) in that order, by one wave: lane l takes
  // PER * kSmallWaves / 64 consecutive slots
  if (w == 0) {
    constexpr int kSlots = PER * kSmallWaves;
    constexpr int kPerLane = (kSlots + 63) / 64;
    int* cg = &s_cnt[0][0][0];
    int* ce = &s_cnt[1][0][0];
    int sg = 0, se = 0;
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) {
      const int sl = lane * kPerLane + j;
      if (sl < kSlots) {
        sg += cg[sl];
        se += ce[sl];
      }
    }
    int ig = sg, ie = se;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int yg = __shfl_up(ig, o, 64), ye = __shfl_up(ie, o, 64);
      if (lane >= o) {
        ig += yg;
        ie += ye;
      }
    }
    int rg = ig - sg, re = ie - se;
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) {
      const int sl = lane * kPerLane + j;
      if (sl < kSlots) {
        const int g = cg[sl], q = ce[sl];
        cg[sl] = rg;
        ce[sl] = re;
        rg += g;
        re += q;
      }
    }
  }
  __syncthreads();
  const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const bool gt = (bg[e] >> lane) & 1ull, eq = (be[e] >> lane) & 1ull;
    if (gt || eq) {
      const int gt_before = s_cnt[0][e][w] + __popcll(bg[e] & below);
      const int eq_before = s_cnt[1][e][w] + __popcll(be[e] & below);
      if (gt || eq_before < need_eq) {
        const int pos = gt_before + min(eq_before, need_eq);
        if (pos < kb) out[pos] = e * kSmallThreads + tid;
      }
    }
  }
}

struct TPlan {
  int NW, slice;
  size_t off_arrive, off_gen, off_hist, off_res, off_cnt, bytes;
};

// stream / with_stream: as for verify's plan (the stream's compute-unit budget).
pvlm_status plan_topk(int B, int64_t m_cap, TPlan* p, hipStream_t stream, bool with_stream) {
  if (B < 1 || m_cap < 1 || m_cap > ((int64_t)1 << 30)) return PVLM_ERR_SHAPE;
  if (m_cap <= kSmallMax) {  // one workgroup per row, no workspace
    p->NW = 1;
    p->slice = (int)m_cap;
    p->bytes = 0;
    return PVLM_OK;
  }
  DeviceInfo di;
  pvlm_status st = with_stream ? device_info(&di, stream) : device_info(&di);
  if (st != PVLM_OK) return st;
  if (B > di.cus) return PVLM_ERR_UNSUPPORTED;
  const int nw_max = di.cus / B;  // co-resident: at most one workgroup per CU
  int64_t nw = (m_cap + kSlice - 1) / kSlice;
  if (nw > nw_max) nw = nw_max;
  if (nw < 1) nw = 1;
  p->NW = (int)nw;
  p->slice = (int)((m_cap + nw - 1) / nw);
  // counters: arrivals return to zero (low part), generations are monotonic
  // (their own part of the monotonic region)
  if (kSyncLine * (size_t)B > kSyncAcceptOff - kSyncTopkOff) return PVLM_ERR_UNSUPPORTED;
  p->off_arrive = 0;
  p->off_gen = kSyncTopkOff;
  size_t off = kSyncRegion;
  p->off_hist = off;
  off = align_up(off + sizeof(int) * (size_t)B * p->NW * 256, 256);
  p->off_res = off;
  off = align_up(off + sizeof(int) * (size_t)B * 4, 256);
  p->off_cnt = off;
  off = align_up(off + sizeof(int) * (size_t)B * p->NW * 2, 256);
  p->bytes = off;
  return PVLM_OK;
}

}  // namespace
}  // namespace pvlm

using namespace pvlm;

extern "C" size_t pvlm_topk_workspace_size(int B, int64_t m_cap) {
  TPlan p;
  if (plan_topk(B, m_cap, &p, nullptr, false) != PVLM_OK) return 0;
  return p.bytes;
}

namespace {
// score: the scores, or with sub the fused MASS form (score = crit^L,
// sub = crit^0, optional score_out).
pvlm_status topk_run(int B, int64_t m_cap, const int32_t* m, const int32_t* k, int32_t k_cap,
                     const float* score, const float* sub, float* score_out, int32_t* idx,
                     void* ws, size_t ws_bytes, int32_t* status, hipStream_t stream) {
  if (!m || !k || !score || (k_cap > 0 && !idx)) return PVLM_ERR_NULL;
  if (B < 1 || m_cap < 1 || k_cap < 0 || m_cap > ((int64_t)1 << 30)) return PVLM_ERR_SHAPE;
  if (k_cap == 0 && !score_out) return PVLM_OK;
  TPlan p;
  pvlm_status st = plan_topk(B, m_cap, &p, stream, true);
  if (st != PVLM_OK) return st;
  if (p.bytes > 0 && (!ws || ws_bytes < p.bytes)) return PVLM_ERR_WORKSPACE;
  TArgs a = {};
  a.score = score;
  a.sub = sub;
  a.score_out = score_out;
  a.m = m;
  a.k = k;
  a.idx = idx;
  a.status = status;
  a.m_cap = m_cap;
  a.k_cap = k_cap;
  a.NW = p.NW;
  a.slice = p.slice;
  void* args[] = {&a};
  const bool fused = sub != nullptr;
  if (m_cap <= kSmallMax) {
    const int per = m_cap <= kSmallThreads * 4 ? 4 : (m_cap <= kSmallThreads * 8 ? 8 : kSmallMaxPer);
    const void* kern =
        per == 4 ? (fused ? reinterpret_cast<const void*>(topk_small_kernel<4, true>)
                          : reinterpret_cast<const void*>(topk_small_kernel<4, false>))
        : per == 8 ? (fused ? reinterpret_cast<const void*>(topk_small_kernel<8, true>)
                            : reinterpret_cast<const void*>(topk_small_kernel<8, false>))
                   : (fused ? reinterpret_cast<const void*>(topk_small_kernel<kSmallMaxPer, true>)
                            : reinterpret_cast<const void*>(topk_small_kernel<kSmallMaxPer, false>));
    PVLM_HIP(allow_dynamic_lds(kern, kSmallLds));
    PVLM_HIP(hipLaunchKernel(kern, dim3(B), dim3(kSmallThreads), args, kSmallLds, stream));
    return PVLM_OK;
  }
  char* wsb = static_cast<char*>(ws);
  a.hist = reinterpret_cast<int*>(wsb + p.off_hist);
  a.res = reinterpret_cast<int*>(wsb + p.off_res);
  a.cnt = reinterpret_cast<int*>(wsb + p.off_cnt);
  a.arrive = reinterpret_cast<int*>(wsb + p.off_arrive);
  a.gen = reinterpret_cast<unsigned*>(wsb + p.off_gen);
  const bool reg = p.slice <= kTopkThreads * kPerThread;
  const void* kern = reg ? (fused ? reinterpret_cast<const void*>(topk_kernel<true, true>)
                                  : reinterpret_cast<const void*>(topk_kernel<true, false>))
                         : (fused ? reinterpret_cast<const void*>(topk_kernel<false, true>)
                                  : reinterpret_cast<const void*>(topk_kernel<false, false>));
  {
    const pvlm_status cs = check_coresident(kern, B * p.NW, kTopkThreads, 0, stream);
    if (cs != PVLM_OK) return cs;
  }
  PVLM_HIP(launch_coresident(kern, dim3(B * p.NW), dim3(kTopkThreads), args, 0, stream));
  return PVLM_OK;
}
}  // namespace

extern "C" pvlm_status pvlm_topk_select(int B, int64_t m_cap, const int32_t* m, const int32_t* k,
                                        int32_t k_cap, const float* score, int32_t* idx, void* ws,
                                        size_t ws_bytes, int32_t* status, hipStream_t stream) {
  return topk_run(B, m_cap, m, k, k_cap, score, nullptr, nullptr, idx, ws, ws_bytes, status,
                  stream);
}

extern "C" pvlm_status pvlm_uvprune_topk_mass(int B, int L, int64_t m_cap, const int32_t* m,
                                              const float* crit_stack, const int32_t* k,
                                              int32_t k_cap, float* score, int32_t* idx, void* ws,
                                              size_t ws_bytes, int32_t* status,
                                              hipStream_t stream) {
  if (!crit_stack) return PVLM_ERR_NULL;
  if (B < 1 || L < 1 || m_cap < 1 || m_cap > ((int64_t)1 << 30)) return PVLM_ERR_SHAPE;
  return topk_run(B, m_cap, m, k, k_cap, crit_stack + (size_t)L * B * m_cap, crit_stack, score, idx,
                  ws, ws_bytes, status, stream);
}
