// Speculative-sampling accept/reject (gfx950): ParallelVLM Sec. 2.2 (accept
// with probability min(1, p/q); on rejection draw from norm(max(0, p - q)))
// and the bonus token after full acceptance (Suppl. B).
//
// One cooperative launch of 512-thread workgroups, three phases separated by
// two grid-wide waits:
//  1. every (batch, row, vocabulary chunk) item: the chunk's max (lowest
//     argmax) and sum of exp((z - max) / temperature) in float64, from one
//     coalesced read of the chunk held in registers;
//  2. every workgroup with draw work combines the chunk results of its batch
//     into each row's max and normaliser, evaluates the accept test of every
//     drafted position in parallel (float64) and takes the first rejection a,
//     then computes the mass of its small chunk of the draw distribution (the
//     residual max(0, p_a - q_a), or p_gamma for the bonus), keeping the
//     values; the draw chunks are spread over the whole grid;
//  3. after the second wait every such workgroup scans the chunk masses to
//     locate the chunk where the cumulative mass first exceeds u' * total;
//     that chunk's workgroup scans its kept values and writes the outputs.
// temperature == 0 stops after the first wait (greedy argmax).
//
// The waits: see grid_wait (no end-of-kernel round trip returns anything to
// zero).
#include "common.h"

namespace pvlm {
namespace {

constexpr int kAccThreads = 512;
constexpr int kAccWaves = kAccThreads / 64;
constexpr int kAccPer = 24;
constexpr int kChunk = kAccThreads * kAccPer;  // vocabulary entries per item
constexpr int kAccMaxB = 256;
// Entries per thread in the draw phases: 2, or 8 when the batch would
// otherwise have more draw chunks than the grid has workgroups.
constexpr int kDrawPerMin = 2;
constexpr int kDrawPerMax = 8;
constexpr int kMaxDraw = 1024;  // draw chunks per batch row: V <= kMaxDraw * kAccThreads * kDrawPerMin
constexpr int kSumPer = kMaxDraw / kAccThreads;  // draw-chunk sums per thread in the crossing search
constexpr int kMaxRows = 65;                    // 2 * gamma + 1, gamma <= 32
constexpr double kNearTie = 1e-9;
constexpr double kNegInfD = -__builtin_huge_val();

// Inputs, then sizes, then outputs and workspace: the argument loads merge
// adjacent fields into wide scalar loads allocated (and spilled) as one
// unit, so fields used at different times sit in separate runs.
struct AArgs {
  const float* dl;
  const float* tl;
  const int32_t* tok;
  const double* ua;
  const double* us;
  int B, gamma, V, NC;  // NC: phase-1 chunks per row
  int ND;               // draw chunks per batch row
  double tau;
  int greedy;
  int32_t* nacc;
  int32_t* next;
  int32_t* near;
  int32_t* status;
  double* pm;       // [B][RW][NC] chunk max
  double* ps;       // [B][RW][NC] chunk exp-sum (relative to the chunk max)
  int* pi;          // [B][RW][NC] chunk argmax (lowest index)
  double* rs;       // [B][ND] residual mass of each draw chunk
  double* qs;       // [B][ND] p mass of each draw chunk (used when the residual is empty)
  int* arrive;      // [2][kArriveSets + 1] arrival counters of the two waits (128 bytes apart), zero at rest
  unsigned* gen;    // [kArriveSets] generation words (128 bytes apart), advanced once per wait
};

__device__ __forceinline__ const float* row_ptr(const AArgs& a, int b, int rho) {
  if (rho <= a.gamma) return a.tl + ((size_t)b * (a.gamma + 1) + rho) * a.V;
  return a.dl + ((size_t)b * a.gamma + (rho - a.gamma - 1)) * a.V;
}

// Grid-wide wait `p` (0 or 1): arrive, and (if `wait`) wait for every
// workgroup's arrival.  The workgroups form eight sets (by index mod 8).
// Arrivals go to their set's counter, so no counter line takes more than an
// eighth of the grid's atomics (same-line atomics serialise); the last
// arrival of each set counts it at a second counter, and the last of those
// advances the generation word, one copy per set, which the set's others
// poll (polling a counter itself would slow the arrivals down).  Every
// counter returns to zero when its last arrival has seen it.  The generation
// is never reset: every workgroup reads its set's copy at its start, before
// its first arrival, so wait p releases at that value + p + 1.
constexpr int kArriveSets = 8;
__device__ __forceinline__ unsigned* gen_word(const AArgs& a) {
  return a.gen + (blockIdx.x % kArriveSets) * (kSyncLine / sizeof(unsigned));
}
__device__ void grid_wait(const AArgs& a, int p, unsigned g0, bool wait) {
  __builtin_amdgcn_s_waitcnt(0);  // this workgroup's published data is visible
  __syncthreads();
  if (threadIdx.x == 0) {
    constexpr int kLineI = (int)(kSyncLine / sizeof(int));
    int* base = a.arrive + p * (kArriveSets + 1) * kLineI;
    const int set = (int)(blockIdx.x % kArriveSets);
    const int members = ((int)gridDim.x - set + kArriveSets - 1) / kArriveSets;
    const int sets = (int)gridDim.x < kArriveSets ? (int)gridDim.x : kArriveSets;
    bool released = false;
    int* c1 = base + set * kLineI;
    if (__hip_atomic_fetch_add(c1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == members - 1) {
      reset_counter(c1);
      int* c2 = base + kArriveSets * kLineI;
      if (__hip_atomic_fetch_add(c2, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == sets - 1) {
        reset_counter(c2);
        for (int k = 0; k < kArriveSets; ++k)
          __hip_atomic_store(a.gen + k * kLineI, g0 + (unsigned)p + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        released = true;
      }
    }
    if (!released && wait) grp_poll(a.gen + set * kLineI, g0 + (unsigned)p + 1u, a.status);
  }
  __syncthreads();
}

// Exclusive scans of two doubles per thread over the workgroup (fixed order,
// the same as block_scan_f64's), sharing the barriers.
__device__ void block_scan2_f64(double v0, double v1, double* s_w, double& e0, double& e1, double& t0,
                                double& t1) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double x0 = v0, x1 = v1;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y0 = __shfl_up(x0, o, 64), y1 = __shfl_up(x1, o, 64);
    if (lane >= o) {
      x0 += y0;
      x1 += y1;
    }
  }
  if (lane == 63) {
    s_w[w] = x0;
    s_w[kAccWaves + w] = x1;
  }
  __syncthreads();
  double b0 = 0.0, b1 = 0.0, a0 = 0.0, a1 = 0.0;
#pragma unroll
  for (int k = 0; k < kAccWaves; ++k) {
    if (k == w) {
      b0 = a0;
      b1 = a1;
    }
    a0 += s_w[k];
    a1 += s_w[kAccWaves + k];
  }
  t0 = a0;
  t1 = a1;
  e0 = b0 + (x0 - v0);
  e1 = b1 + (x1 - v1);
  __syncthreads();
}

// Exclusive scan of one double per thread over the workgroup (fixed order).
__device__ double block_scan_f64(double v, double* s_w, double* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_w[w] = x;
  __syncthreads();
  double before = 0.0, tot = 0.0;
#pragma unroll
  for (int k = 0; k < kAccWaves; ++k) {
    if (k == w) before = tot;
    tot += s_w[k];
  }
  *total = tot;
  __syncthreads();
  return before + (x - v);
}

// Workgroup-wide max with lowest-index tie-break (value, index).
__device__ void block_argmax(float& v, int& i, float* s_v, int* s_i) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(v, o, 64);
    const int i2 = __shfl_xor(i, o, 64);
    if (v2 > v || (v2 == v && i2 < i)) {
      v = v2;
      i = i2;
    }
  }
  if (lane == 0) {
    s_v[w] = v;
    s_i[w] = i;
  }
  __syncthreads();
  v = s_v[0];
  i = s_i[0];
#pragma unroll
  for (int k = 1; k < kAccWaves; ++k)
    if (s_v[k] > v || (s_v[k] == v && s_i[k] < i)) {
      v = s_v[k];
      i = s_i[k];
    }
  __syncthreads();
}

// Workgroup-wide minimum of lo and maximum of hi (butterflies within each
// wave, then the waves' results through LDS; no atomics, whose per-lane
// serialisation is slow when many lanes take part).
__device__ void block_minmax(int& lo, int& hi, int* s_w) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    lo = min(lo, __shfl_xor(lo, o, 64));
    hi = max(hi, __shfl_xor(hi, o, 64));
  }
  if (lane == 0) {
    s_w[w] = lo;
    s_w[kAccWaves + w] = hi;
  }
  __syncthreads();
  lo = s_w[0];
  hi = s_w[kAccWaves];
#pragma unroll
  for (int k = 1; k < kAccWaves; ++k) {
    lo = min(lo, s_w[k]);
    hi = max(hi, s_w[kAccWaves + k]);
  }
  __syncthreads();
}

__device__ double block_sum(double x, double* s_v) {
  x = warp_sum(x);
  if ((threadIdx.x & 63) == 0) s_v[threadIdx.x >> 6] = x;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int k = 0; k < kAccWaves; ++k) t += s_v[k];
  __syncthreads();
  return t;
}

// The kAccPer entries of chunk [y0, y1) this thread reads in phase 1 (coalesced:
// entry 4 * (k * kAccThreads + tid) + e of the chunk), -inf past y1.
template <bool VEC>
__device__ __forceinline__ void load_strided(const float* z, int y0, int y1, float (&v)[kAccPer]) {
#pragma unroll
  for (int k = 0; k < kAccPer / 4; ++k) {
    const int y = y0 + 4 * (k * kAccThreads + (int)threadIdx.x);
    // clamped loads, all in flight together (VEC: rows and chunk ends are
    // multiples of 4, so y1 - 4 is an aligned entry of the chunk)
    if constexpr (VEC) {
      const float4 f = *reinterpret_cast<const float4*>(z + (y < y1 ? y : y1 - 4));
      const bool in = y < y1;
      v[4 * k] = in ? f.x : -INFINITY;
      v[4 * k + 1] = in ? f.y : -INFINITY;
      v[4 * k + 2] = in ? f.z : -INFINITY;
      v[4 * k + 3] = in ? f.w : -INFINITY;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x = z[min(y + e, y1 - 1)];
        v[4 * k + e] = y + e < y1 ? x : -INFINITY;
      }
    }
  }
}
__device__ __forceinline__ int strided_index(int y0, int j) {
  return y0 + 4 * ((j / 4) * kAccThreads + (int)threadIdx.x) + (j % 4);
}

// Per-batch state every draw workgroup derives after the first wait.
struct Decision {
  int acc, tie;
  double pM, pZ, qM, qZ;
};

template <bool VEC, int kDrawPer>
__global__ void __launch_bounds__(kAccThreads) accept_kernel(AArgs a) {
  constexpr int kDrawChunk = kAccThreads * kDrawPer;
  __shared__ float s_fv[kAccWaves];
  __shared__ int s_fi[kAccWaves];
  __shared__ double s_d[2 * kAccWaves];
  __shared__ double s_M[kMaxRows], s_Z[kMaxRows];
  __shared__ int s_arg[kMaxRows], s_rej[32], s_tie[32];
  __shared__ Decision s_dec;
  __shared__ double s_pre;
  __shared__ int s_mm[2 * kAccWaves];
  const int tid = threadIdx.x;
  const int RW = 2 * a.gamma + 1;
  const int W = gridDim.x;
  const double inv_tau = a.greedy ? 0.0 : 1.0 / a.tau;
  const unsigned g0 = tid == 0 ? grp_read(gen_word(a)) : 0u;
  // the inputs of the decisions and the draw for this workgroup's first
  // batch, loaded up front (drafted position t on thread kAccThreads - 32 + t)
  const int nd_items = a.greedy ? 1 : a.B * a.ND;
  const int pb = (int)blockIdx.x < nd_items ? (a.greedy ? 0 : (int)blockIdx.x % a.B) : -1;
  const int t_d = tid - (kAccThreads - 32);
  const bool drafter = t_d >= 0 && t_d < a.gamma;
  int pf_x = -1;
  float pf_px = 0.f, pf_qx = 0.f;
  double pf_ua = 0.0;
  auto load_draft = [&](int b, int& x, float& px, float& qx, double& ua) {
    const int xt = a.tok[(size_t)b * a.gamma + t_d];
    x = xt >= 0 && xt < a.V ? xt : -1;
    if (!a.greedy) {  // clamped loads, all in flight; the values count only when x >= 0
      const int xc = x >= 0 ? x : 0;
      px = row_ptr(a, b, t_d)[xc];
      qx = row_ptr(a, b, a.gamma + 1 + t_d)[xc];
      ua = a.ua[(size_t)b * a.gamma + t_d];
    }
  };
  if (pb >= 0 && drafter) load_draft(pb, pf_x, pf_px, pf_qx, pf_ua);
  const double pf_us = pb >= 0 && !a.greedy ? a.us[pb] : 0.0;

  // ---- phase 1: chunk max / argmax / exp-sum (greedy: target rows only)
  const int rows1 = a.greedy ? a.gamma + 1 : RW;
  const int items1 = a.B * rows1 * a.NC;
  for (int it = blockIdx.x; it < items1; it += W) {
    const int c = it % a.NC, rho = (it / a.NC) % rows1, b = it / (a.NC * rows1);
    const size_t slot = ((size_t)b * RW + rho) * a.NC + c;
    const float* z = row_ptr(a, b, rho);
    const int y0 = c * kChunk, y1 = min(a.V, y0 + kChunk);
    float v[kAccPer];
    load_strided<VEC>(z, y0, y1, v);
    float mx = -INFINITY;
    int am = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < kAccPer; ++j)
      if (v[j] > mx) {  // ascending index order within the thread: first max kept
        mx = v[j];
        am = strided_index(y0, j);
      }
    block_argmax(mx, am, s_fv, s_fi);
    double sum = 0.0;
    if (!a.greedy && mx != -INFINITY) {
      // no branches around the exponentials (entries past the chunk are -inf
      // and contribute exp(-inf) = 0), so their evaluations interleave
      const double M = mx;
      double e[kAccPer];
#pragma unroll
      for (int j = 0; j < kAccPer; ++j) e[j] = exp(((double)v[j] - M) * inv_tau);
#pragma unroll
      for (int j = 0; j < kAccPer; ++j) sum += e[j];
    }
    sum = block_sum(sum, s_d);
    if (tid == 0) {
      st_agent(a.pm + slot, mx == -INFINITY ? kNegInfD : (double)mx);
      st_agent(a.ps + slot, sum);
      st_agent(a.pi + slot, am);
    }
  }
  const int items3 = a.B * a.ND;
  const bool draws = !a.greedy && (int)blockIdx.x < items3;
  const bool greedy_out = a.greedy && blockIdx.x == 0;
  grid_wait(a, 0, g0, draws || greedy_out);

  // every row's max, argmax and normaliser of batch b, the accept test of
  // every drafted position (in parallel), and the first rejection, into
  // s_dec (greedy: the outputs)
  auto decide = [&](int b) {
    const int rows = a.greedy ? a.gamma + 1 : RW;
    // the drafted tokens and their logits (threads of the last wave), loaded
    // up front for the first batch
    const int t = t_d;
    int x = pf_x;
    float px = pf_px, qx = pf_qx;
    double ua = pf_ua;
    if (drafter && b != pb) load_draft(b, x, px, qx, ua);
    // row r's NC chunk results are combined by an aligned group of NCp lanes
    // (NCp = NC rounded up to a power of two, at most 64), lane k taking
    // chunks k, k + NCp, ...; max and lowest argmax, then the normaliser, by
    // butterflies within the group
    const int NCp = a.NC <= 1 ? 1 : min(64, 1 << (32 - __clz(a.NC - 1)));
    const int rpp = (kAccThreads - 64) / NCp;  // the last wave holds the drafted tokens
    for (int r0 = 0; r0 < rows; r0 += rpp) {
      const int r = r0 + tid / NCp, k0 = tid % NCp;
      const bool act = r < rows && tid < rpp * NCp;
      const size_t base = ((size_t)b * RW + r) * a.NC;
      double M = kNegInfD, m0 = kNegInfD, s0 = 0.0;
      int A = 0x7fffffff;
      if (act) {
        // the lane's first chunk: its three results loaded together (clamped)
        const int kc = min(k0, a.NC - 1);
        const double m2 = ld_agent(a.pm + base + kc);
        const int i2 = ld_agent(a.pi + base + kc);
        const double sv = a.greedy ? 0.0 : ld_agent(a.ps + base + kc);
        if (k0 < a.NC) {
          m0 = M = m2;
          s0 = sv;
          A = i2;
        }
        for (int k = k0 + NCp; k < a.NC; k += NCp) {
          const double m3 = ld_agent(a.pm + base + k);
          const int i3 = ld_agent(a.pi + base + k);
          if (m3 > M || (m3 == M && i3 < A)) {
            M = m3;
            A = i3;
          }
        }
      }
      for (int o = NCp / 2; o > 0; o >>= 1) {
        const double m2 = __shfl_xor(M, o, 64);
        const int i2 = __shfl_xor(A, o, 64);
        if (m2 > M || (m2 == M && i2 < A)) {
          M = m2;
          A = i2;
        }
      }
      double Z = 0.0;
      if (act && !a.greedy && M != kNegInfD)
        for (int k = k0; k < a.NC; k += NCp) {
          const double m2 = k == k0 ? m0 : ld_agent(a.pm + base + k);
          const double s2 = k == k0 ? s0 : ld_agent(a.ps + base + k);
          if (m2 != kNegInfD) Z += s2 * exp((m2 - M) * inv_tau);
        }
      for (int o = NCp / 2; o > 0; o >>= 1) Z += __shfl_xor(Z, o, 64);
      if (act && k0 == 0) {
        s_M[r] = M;
        s_Z[r] = Z;
        s_arg[r] = A == 0x7fffffff ? 0 : A;
      }
    }
    __syncthreads();
    if (drafter) {
      int rej, tie = 0;
      if (x < 0) {
        rej = 2;  // invalid drafted token
      } else if (a.greedy) {
        rej = x != s_arg[t];
      } else {
        const int qr = a.gamma + 1 + t;
        const double p = exp((px - s_M[t]) * inv_tau) / s_Z[t];
        const double q = exp((qx - s_M[qr]) * inv_tau) / s_Z[qr];
        const double lhs = ua * q;
        tie = fabs(lhs - p) <= kNearTie * fmax(lhs, p);
        rej = !(lhs < p);
      }
      s_rej[t] = rej;
      s_tie[t] = tie;
    }
    __syncthreads();
    if (tid == 0) {
      int acc = a.gamma, tie = 0;
      for (int u = 0; u < a.gamma; ++u) {
        tie |= s_tie[u];
        if (s_rej[u]) {
          if (s_rej[u] == 2) dev_flag(a.status, PVLM_DEV_RANGE);
          acc = u;
          break;
        }
      }
      Decision d;
      d.acc = acc;
      d.tie = tie;
      d.pM = s_M[acc];
      d.pZ = s_Z[acc];
      d.qM = acc < a.gamma ? s_M[a.gamma + 1 + acc] : 0.0;
      d.qZ = acc < a.gamma ? s_Z[a.gamma + 1 + acc] : 1.0;
      s_dec = d;
      if (a.greedy) {
        a.nacc[b] = acc;
        a.next[b] = s_arg[acc];
        if (a.near) a.near[b] = 0;
      }
    }
    __syncthreads();
  };

  if (greedy_out)
    for (int b = 0; b < a.B; ++b) decide(b);
  if (a.greedy) return;

  // Entries y = c * kDrawChunk + kDrawPer * tid + j of draw chunk c: r(y) of
  // the draw distribution (the residual max(0, p - q), or p for the bonus)
  // or, with want_p, p(y); returns this thread's sum of p(y) as well.
  auto draw_values = [&](int b, int c, bool want_p, double (&r)[kDrawPer]) -> double {
    const Decision d = s_dec;
    const bool resid = !want_p && d.acc < a.gamma;
    const double ipz = 1.0 / d.pZ, iqz = 1.0 / d.qZ;
    const float* zpr = row_ptr(a, b, d.acc);
    const float* zqr = row_ptr(a, b, a.gamma + 1 + min(d.acc, a.gamma - 1));
    const int y = c * kDrawChunk + kDrawPer * tid;
    float zp[kDrawPer], zq[kDrawPer];
#pragma unroll
    for (int j = 0; j < kDrawPer; ++j) {
      // clamped loads, all in flight together; past V: p = 0, q = 0
      const float xp = zpr[min(y + j, a.V - 1)], xq = zqr[min(y + j, a.V - 1)];
      zp[j] = y + j < a.V ? xp : -INFINITY;
      zq[j] = y + j < a.V && resid ? xq : -INFINITY;
    }
    double psum = 0.0;
#pragma unroll
    for (int j = 0; j < kDrawPer; ++j) {
      const double p = exp(((double)zp[j] - d.pM) * inv_tau) * ipz;
      const double q = exp(((double)zq[j] - d.qM) * inv_tau) * iqz;
      psum += p;
      r[j] = !resid ? p : (p > q ? p - q : 0.0);
    }
    return psum;
  };

  // ---- phase 2: masses of the draw chunks (the values of the workgroup's
  //      last item are kept)
  double rr[kDrawPer];
  double rr_excl = 0.0;  // exclusive prefix of the kept values' thread sums (residual)
  int kept = -1, dec_b = -1;
  for (int it = blockIdx.x; it < items3; it += W) {
    const int b = it % a.B, c = it / a.B;
    if (b != dec_b) {
      decide(b);
      dec_b = b;
    }
    const double sp = draw_values(b, c, false, rr);
    kept = it;
    double sr = 0.0;
#pragma unroll
    for (int j = 0; j < kDrawPer; ++j) sr += rr[j];
    double tr, tp, ep;
    block_scan2_f64(sr, sp, s_d, rr_excl, ep, tr, tp);
    if (tid == 0) {
      st_agent(a.rs + (size_t)b * a.ND + c, tr);
      st_agent(a.qs + (size_t)b * a.ND + c, tp);
    }
  }
  grid_wait(a, 1, g0, draws);
  if (!draws) return;

  // ---- phase 3: the chunk where the cumulative mass first exceeds u' * Z
  //      scans its values and writes the outputs
  for (int it = blockIdx.x; it < items3; it += W) {
    const int b = it % a.B, c = it / a.B;
    // chunk sums of batch b in order: thread t owns chunks kSumPer * t + i
    double cr[kSumPer], cq[kSumPer];
    double own_r = 0.0, own_q = 0.0;
#pragma unroll
    for (int i = 0; i < kSumPer; ++i) {
      const int k = kSumPer * tid + i;
      const double xr = ld_agent(a.rs + (size_t)b * a.ND + min(k, a.ND - 1));  // clamped loads
      const double xq = ld_agent(a.qs + (size_t)b * a.ND + min(k, a.ND - 1));
      cr[i] = k < a.ND ? xr : 0.0;
      cq[i] = k < a.ND ? xq : 0.0;
      own_r += cr[i];
      own_q += cq[i];
    }
    double Zr, Zq, ex_r, ex_q;
    block_scan2_f64(own_r, own_q, s_d, ex_r, ex_q, Zr, Zq);
    const bool use_r = Zr > 0.0;  // else the residual is empty: draw from p
    const double Z = use_r ? Zr : Zq;
    const double thr = (b == pb ? pf_us : a.us[b]) * Z;
    // the first chunk whose cumulative mass passes u' * Z, and the last
    // chunk with positive mass
    double run = use_r ? ex_r : ex_q;
    double pre_of[kSumPer];
    int first = 0x7fffffff, last = -1;
#pragma unroll
    for (int i = 0; i < kSumPer; ++i) {
      const int k = kSumPer * tid + i;
      const double sk = use_r ? cr[i] : cq[i];
      pre_of[i] = run;
      if (k < a.ND) {
        if (first == 0x7fffffff && run + sk > thr) first = k;
        if (sk > 0.0) last = k;
      }
      run += sk;
    }
    block_minmax(first, last, s_mm);
    const bool fallback = first == 0x7fffffff;  // rounding: no chunk passes u' * Z
    const int cross = fallback ? max(last, 0) : first;
#pragma unroll
    for (int i = 0; i < kSumPer; ++i)
      if (kSumPer * tid + i == cross) s_pre = last < 0 ? 0.0 : pre_of[i];
    __syncthreads();
    const double pre = s_pre;
    __syncthreads();
    if (cross != c) continue;  // uniform across the workgroup
    if (b != dec_b) {
      decide(b);
      dec_b = b;
    }
    // the kept values, unless they belong to another item or the draw
    // falls back to p
    double excl = rr_excl;
    if (it != kept || !use_r) {
      draw_values(b, c, !use_r, rr);
      kept = use_r ? it : -1;
      double own = 0.0;
#pragma unroll
      for (int j = 0; j < kDrawPer; ++j) own += rr[j];
      double tot;
      excl = block_scan_f64(own, s_d, &tot);
    }
    // this thread's first entry passing u' * Z and last positive entry; the
    // workgroup's first crossing wins, else (rounding, or the fallback
    // chunk) its last positive entry
    const int ybase = c * kDrawChunk + kDrawPer * tid;
    double cum = pre + excl;
    int cross_y = 0x7fffffff, last_y = -1;
    double below = cum, at = cum;
#pragma unroll
    for (int j = 0; j < kDrawPer; ++j) {
      const double prev = cum;
      cum += rr[j];
      if (!fallback && cross_y == 0x7fffffff && cum > thr) {
        cross_y = ybase + j;
        below = prev;
        at = cum;
      }
      if (rr[j] > 0.0) last_y = ybase + j;
    }
    int lo = cross_y, hi = last_y;
    block_minmax(lo, hi, s_mm);
    const bool edge = fallback || lo == 0x7fffffff;
    const int win = edge ? hi : lo;
    const int mine = edge ? last_y : cross_y;
    const Decision d = s_dec;
    if (win < 0 && tid == 0) {  // no positive mass anywhere: degenerate input
      dev_flag(a.status, PVLM_DEV_RANGE);
      a.nacc[b] = d.acc;
      a.next[b] = 0;
      if (a.near) a.near[b] = 1;
    }
    if (mine == win && win >= 0) {
      int tie = d.tie;
      if (!edge) {
        if (fabs(at - thr) <= kNearTie * Z) tie = 1;
        if (win > 0 && fabs(below - thr) <= kNearTie * Z) tie = 1;
      } else {
        tie = 1;
      }
      a.nacc[b] = d.acc;
      a.next[b] = win;
      if (a.near) a.near[b] = tie;
    }
    __syncthreads();
  }
}

struct APlan {
  int NC, ND;
  size_t off_arrive, off_gen, off_pm, off_ps, off_pi, off_rs, off_qs, bytes;
};

pvlm_status plan_accept(int B, int gamma, int V, APlan* p) {
  if (B < 1 || gamma < 1 || V < 1) return PVLM_ERR_SHAPE;
  if (B > kAccMaxB || gamma > 32 || V > kMaxDraw * kAccThreads * kDrawPerMin)
    return PVLM_ERR_UNSUPPORTED;
  p->NC = (V + kChunk - 1) / kChunk;
  p->ND = (V + kAccThreads * kDrawPerMin - 1) / (kAccThreads * kDrawPerMin);  // at most
  const size_t rows = (size_t)B * (2 * gamma + 1);
  const size_t parts = rows * p->NC;
  // counters inside the fixed synchronisation region, data after it
  p->off_arrive = 0;
  p->off_gen = kSyncAcceptOff;
  size_t off = kSyncRegion;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  p->off_pm = take(parts * sizeof(double));
  p->off_ps = take(parts * sizeof(double));
  p->off_pi = take(parts * sizeof(int));
  p->off_rs = take((size_t)B * p->ND * sizeof(double));
  p->off_qs = take((size_t)B * p->ND * sizeof(double));
  p->bytes = off;
  return PVLM_OK;
}

}  // namespace
}  // namespace pvlm

using namespace pvlm;

extern "C" size_t pvlm_spec_accept_workspace_size(int B, int gamma, int V) {
  APlan p;
  if (plan_accept(B, gamma, V, &p) != PVLM_OK) return 0;
  return p.bytes;
}

extern "C" pvlm_status pvlm_spec_accept(int B, int gamma, int V, float temperature,
                                        const float* draft_logits, const float* target_logits,
                                        const int32_t* draft_tokens, const double* u_accept,
                                        const double* u_sample, int32_t* n_accepted,
                                        int32_t* next_token, int32_t* near_tie, void* ws,
                                        size_t ws_bytes, int32_t* status, hipStream_t stream) {
  if (!draft_logits || !target_logits || !draft_tokens || !u_accept || !u_sample || !n_accepted ||
      !next_token)
    return PVLM_ERR_NULL;
  if (!(temperature >= 0.f) || !std::isfinite(temperature)) return PVLM_ERR_SHAPE;
  APlan p;
  pvlm_status st = plan_accept(B, gamma, V, &p);
  if (st != PVLM_OK) return st;
  if (!ws || ws_bytes < p.bytes) return PVLM_ERR_WORKSPACE;
  DeviceInfo di;
  st = device_info(&di, stream);
  if (st != PVLM_OK) return st;
  char* wsb = static_cast<char*>(ws);
  AArgs a;
  a.dl = draft_logits;
  a.tl = target_logits;
  a.tok = draft_tokens;
  a.ua = u_accept;
  a.us = u_sample;
  a.nacc = n_accepted;
  a.next = next_token;
  a.near = near_tie;
  a.status = status;
  a.pm = reinterpret_cast<double*>(wsb + p.off_pm);
  a.ps = reinterpret_cast<double*>(wsb + p.off_ps);
  a.pi = reinterpret_cast<int*>(wsb + p.off_pi);
  a.rs = reinterpret_cast<double*>(wsb + p.off_rs);
  a.qs = reinterpret_cast<double*>(wsb + p.off_qs);
  a.arrive = reinterpret_cast<int*>(wsb + p.off_arrive);
  a.gen = reinterpret_cast<unsigned*>(wsb + p.off_gen);
  a.B = B;
  a.gamma = gamma;
  a.V = V;
  a.NC = p.NC;
  // draw chunks: 2 entries per thread unless that gives more items than CUs
  const int dp = B * p.ND <= di.cus ? kDrawPerMin : kDrawPerMax;
  a.ND = (V + kAccThreads * dp - 1) / (kAccThreads * dp);
  a.tau = (double)temperature;
  a.greedy = temperature == 0.f;
  const int items = max(B * (a.greedy ? gamma + 1 : 2 * gamma + 1) * p.NC, a.greedy ? 1 : B * a.ND);
  // a multiple of 8 workgroups (the XCD count) keeps the cooperative queue's
  // round-robin XCD placement aligned for the launches that follow
  int grid = (items + 7) / 8 * 8;
  if (grid > di.cus) grid = di.cus;
  if (grid < 1) grid = 1;
  // float4 loads when every row starts on a 16-byte boundary
  const bool vec = V % 4 == 0 && reinterpret_cast<uintptr_t>(draft_logits) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(target_logits) % 16 == 0;
  void* args[] = {&a};
  const void* kern =
      vec ? (dp == kDrawPerMin ? reinterpret_cast<const void*>(accept_kernel<true, kDrawPerMin>)
                               : reinterpret_cast<const void*>(accept_kernel<true, kDrawPerMax>))
          : (dp == kDrawPerMin ? reinterpret_cast<const void*>(accept_kernel<false, kDrawPerMin>)
                               : reinterpret_cast<const void*>(accept_kernel<false, kDrawPerMax>));
  {
    const pvlm_status cs = check_coresident(kern, grid, kAccThreads, 0, stream);
    if (cs != PVLM_OK) return cs;
  }
  PVLM_HIP(launch_coresident(kern, dim3(grid), dim3(kAccThreads), args, 0, stream));
  return PVLM_OK;
}
