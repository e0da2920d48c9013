// Speculative-sampling accept/reject (gfx950): ParallelVLM Sec. 2.2 (accept
// with probability min(1, p/q); on rejection draw from norm(max(0, p - q)))
// and the bonus token after full acceptance (Suppl. B).
//
// One cooperative launch, four phases separated by grid-wide waits:
//  1. every (batch, row, vocab chunk) item: chunk max (and lowest argmax) and
//     sum of exp((z - max) / temperature) in float64;
//  2. every workgroup with later work combines those into each row's max and
//     normaliser and replays the sequential accept decisions (float64) to find
//     the first rejection a -- redundantly, so no extra wait is needed;
//  3. every (batch, chunk) item: the chunk's mass of the draw distribution
//     (the residual max(0, p_a - q_a), or p_gamma for the bonus), summed with
//     the same blocked scan phase 4 uses;
//  4. the chunk where the cumulative mass first exceeds u' * total scans its
//     elements and writes the outputs.
// temperature == 0 stops after phase 2 (greedy argmax).
#include "common.h"

namespace pvlm {
namespace {

constexpr int kAccThreads = 256;
constexpr int kAccPer = 16;
constexpr int kChunk = kAccThreads * kAccPer;  // vocabulary entries per item
constexpr int kAccMaxB = 256;
constexpr double kNearTie = 1e-9;

struct AArgs {
  const float* dl;
  const float* tl;
  const int32_t* tok;
  const double* ua;
  const double* us;
  int32_t* nacc;
  int32_t* next;
  int32_t* near;
  int32_t* status;
  double* pm;   // [B][RW][NC] chunk max
  double* ps;   // [B][RW][NC] chunk exp-sum
  int* pi;      // [B][RW][NC] chunk argmax (lowest index)
  double* rs;   // [B][NC] residual chunk mass
  double* qs;   // [B][NC] p chunk mass (fallback when the residual is empty)
  int* bar;     // [0] arrivals, [1] finished workgroups
  int B, gamma, V, NC;
  double tau;
  int greedy;
};

__device__ __forceinline__ const float* row_ptr(const AArgs& a, int b, int rho) {
  if (rho <= a.gamma) return a.tl + ((size_t)b * (a.gamma + 1) + rho) * a.V;
  return a.dl + ((size_t)b * a.gamma + (rho - a.gamma - 1)) * a.V;
}

__device__ __forceinline__ void grid_wait(const AArgs& a, int target) {
  wg_arrive_wait(a.bar, target, a.status, true);
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
  for (int k = 0; k < kAccThreads / 64; ++k) {
    if (k == w) before = tot;
    tot += s_w[k];
  }
  *total = tot;
  __syncthreads();
  return before + (x - v);
}

__global__ void __launch_bounds__(kAccThreads) accept_kernel(AArgs a) {
  __shared__ double s_red[kAccThreads / 64];
  __shared__ int s_ired[kAccThreads / 64];
  __shared__ double s_M[65], s_Z[65];
  __shared__ int s_arg[65];
  __shared__ int s_a[kAccMaxB], s_tie[kAccMaxB];
  __shared__ double s_pM[kAccMaxB], s_pZ[kAccMaxB], s_qM[kAccMaxB], s_qZ[kAccMaxB];
  __shared__ int s_win;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int RW = 2 * a.gamma + 1;
  const int W = gridDim.x;
  const double tau = a.tau;

  // ---- phase 1: per-chunk max / argmax / exp-sum
  const int items1 = a.B * RW * a.NC;
  for (int it = blockIdx.x; it < items1; it += W) {
    const int c = it % a.NC, rho = (it / a.NC) % RW, b = it / (a.NC * RW);
    if (a.greedy && rho > a.gamma) continue;
    const float* z = row_ptr(a, b, rho);
    const int y0 = c * kChunk, y1 = min(a.V, y0 + kChunk);
    float mx = -__builtin_huge_valf();
    int am = 0x7fffffff;
    for (int y = y0 + tid; y < y1; y += kAccThreads) {
      const float v = z[y];
      if (v > mx) {
        mx = v;
        am = y;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float m2 = __shfl_xor(mx, o, 64);
      const int a2 = __shfl_xor(am, o, 64);
      if (m2 > mx || (m2 == mx && a2 < am)) {
        mx = m2;
        am = a2;
      }
    }
    if (lane == 0) {
      s_red[w] = mx;
      s_ired[w] = am;
    }
    __syncthreads();
    double M = s_red[0];
    int AM = s_ired[0];
    for (int k = 1; k < kAccThreads / 64; ++k)
      if (s_red[k] > M || (s_red[k] == M && s_ired[k] < AM)) {
        M = s_red[k];
        AM = s_ired[k];
      }
    __syncthreads();
    double s = 0.0;
    if (!a.greedy && M != -__builtin_huge_val()) {
      for (int y = y0 + tid; y < y1; y += kAccThreads) s += exp(((double)z[y] - M) / tau);
    }
    s = warp_sum(s);
    if (lane == 0) s_red[w] = s;
    __syncthreads();
    if (tid == 0) {
      double S = 0.0;
      for (int k = 0; k < kAccThreads / 64; ++k) S += s_red[k];
      st_agent(&a.pm[it], M);
      st_agent(&a.ps[it], S);
      st_agent(&a.pi[it], AM);
    }
    __syncthreads();
  }
  grid_wait(a, W);

  // ---- phase 2: row normalisers and the sequential accept decisions
  const bool has_late = a.greedy ? blockIdx.x == 0 : blockIdx.x < a.B * a.NC;
  if (has_late) {
    for (int b = 0; b < a.B; ++b) {
      if (tid < RW && (!a.greedy || tid <= a.gamma)) {
        const size_t base = ((size_t)b * RW + tid) * a.NC;
        double M = -__builtin_huge_val(), Z = 0.0;
        int AM = 0;
        for (int c = 0; c < a.NC; ++c) {
          const double m2 = ld_agent(&a.pm[base + c]);
          if (m2 > M) {
            M = m2;
            AM = ld_agent(&a.pi[base + c]);
          }
        }
        if (!a.greedy && M != -__builtin_huge_val()) {
          for (int c = 0; c < a.NC; ++c) {
            const double m2 = ld_agent(&a.pm[base + c]);
            if (m2 != -__builtin_huge_val()) Z += ld_agent(&a.ps[base + c]) * exp((m2 - M) / tau);
          }
        }
        s_M[tid] = M;
        s_Z[tid] = Z;
        s_arg[tid] = AM;
      }
      __syncthreads();
      if (tid == 0) {
        int acc = a.gamma, tie = 0;
        for (int t = 0; t < a.gamma; ++t) {
          int x = a.tok[(size_t)b * a.gamma + t];
          if (x < 0 || x >= a.V) {
            dev_flag(a.status, PVLM_DEV_RANGE);
            acc = t;
            break;
          }
          bool ok;
          if (a.greedy) {
            ok = x == s_arg[t];
          } else {
            const double p = exp(((double)row_ptr(a, b, t)[x] - s_M[t]) / tau) / s_Z[t];
            const int qr = a.gamma + 1 + t;
            const double q = exp(((double)row_ptr(a, b, qr)[x] - s_M[qr]) / tau) / s_Z[qr];
            const double lhs = a.ua[(size_t)b * a.gamma + t] * q;
            if (fabs(lhs - p) <= kNearTie * fmax(lhs, p)) tie = 1;
            ok = lhs < p;
          }
          if (!ok) {
            acc = t;
            break;
          }
        }
        s_a[b] = acc;
        s_tie[b] = tie;
        s_pM[b] = s_M[acc];
        s_pZ[b] = s_Z[acc];
        if (acc < a.gamma) {
          s_qM[b] = s_M[a.gamma + 1 + acc];
          s_qZ[b] = s_Z[a.gamma + 1 + acc];
        }
        if (a.greedy) {
          a.nacc[b] = acc;
          a.next[b] = s_arg[acc];
          if (a.near) a.near[b] = 0;
        }
      }
      __syncthreads();
    }
  }
  if (a.greedy) {
    __syncthreads();
    if (tid == 0) {
      const int done = __hip_atomic_fetch_add(a.bar + 1, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      if (done == W - 1) {
        __hip_atomic_store(a.bar, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(a.bar + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    return;
  }

  // r(y) of the draw distribution at row a of batch b; also p(y)
  auto draw_mass = [&](int b, int y, double& p_out) -> double {
    const int acc = s_a[b];
    const double p = exp(((double)row_ptr(a, b, acc)[y] - s_pM[b]) / tau) / s_pZ[b];
    p_out = p;
    if (acc == a.gamma) return p;
    const double q = exp(((double)row_ptr(a, b, a.gamma + 1 + acc)[y] - s_qM[b]) / tau) / s_qZ[b];
    return p > q ? p - q : 0.0;
  };

  // ---- phase 3: chunk masses of the draw distribution
  const int items3 = a.B * a.NC;
  for (int it = blockIdx.x; it < items3; it += W) {
    const int b = it / a.NC, c = it % a.NC;
    const int y0 = c * kChunk + tid * kAccPer;
    double sr = 0.0, sp = 0.0;
    for (int e = 0; e < kAccPer; ++e) {
      const int y = y0 + e;
      if (y < a.V) {
        double p;
        sr += draw_mass(b, y, p);
        sp += p;
      }
    }
    double tr, tp;
    block_scan_f64(sr, s_red, &tr);
    block_scan_f64(sp, s_red, &tp);
    if (tid == 0) {
      st_agent(&a.rs[it], tr);
      st_agent(&a.qs[it], tp);
    }
    __syncthreads();
  }
  grid_wait(a, 2 * W);

  // ---- phase 4: locate the crossing chunk, scan it, write the outputs
  for (int it = blockIdx.x; it < items3; it += W) {
    const int b = it / a.NC, c = it % a.NC;
    double Zr = 0.0, Zp = 0.0;
    for (int k = 0; k < a.NC; ++k) {
      Zr += ld_agent(&a.rs[(size_t)b * a.NC + k]);
      Zp += ld_agent(&a.qs[(size_t)b * a.NC + k]);
    }
    const bool use_r = Zr > 0.0;
    const double* sums = use_r ? a.rs : a.qs;
    const double Z = use_r ? Zr : Zp;
    const double thr = a.us[b] * Z;
    double run = 0.0, pre = 0.0;
    int cross = -1, last_pos = -1;
    for (int k = 0; k < a.NC; ++k) {
      const double sk = ld_agent(&sums[(size_t)b * a.NC + k]);
      if (k == c) pre = run;
      if (sk > 0.0) last_pos = k;
      run += sk;
      if (cross < 0 && run > thr) cross = k;
    }
    const bool fallback = cross < 0;
    if (fallback) cross = last_pos < 0 ? 0 : last_pos;
    if (c != cross) continue;  // uniform across the workgroup
    const int y0 = c * kChunk + tid * kAccPer;
    double r[kAccPer];
    double own = 0.0;
    for (int e = 0; e < kAccPer; ++e) {
      const int y = y0 + e;
      r[e] = 0.0;
      if (y < a.V) {
        double p;
        const double rv = draw_mass(b, y, p);
        r[e] = use_r ? rv : p;
      }
      own += r[e];
    }
    double tot;
    const double excl = block_scan_f64(own, s_red, &tot);
    if (tid == 0) s_win = fallback ? -1 : 0x7fffffff;
    __syncthreads();
    double cum = pre + excl;
    int mine = -1;
    double below = cum, at = cum;
    for (int e = 0; e < kAccPer; ++e) {
      const double prev = cum;
      cum += r[e];
      if (fallback) {
        if (r[e] > 0.0) mine = y0 + e;
      } else if (mine < 0 && cum > thr) {
        mine = y0 + e;
        below = prev;
        at = cum;
      }
    }
    if (mine >= 0) {
      if (fallback)
        atomicMax(&s_win, mine);
      else
        atomicMin(&s_win, mine);
    }
    __syncthreads();
    int win = s_win;
    bool edge = fallback;
    if (!fallback && win == 0x7fffffff) {  // rounding left no crossing: last positive
      __syncthreads();
      if (tid == 0) s_win = -1;
      __syncthreads();
      mine = -1;
      for (int e = 0; e < kAccPer; ++e)
        if (r[e] > 0.0) mine = y0 + e;
      if (mine >= 0) atomicMax(&s_win, mine);
      __syncthreads();
      win = s_win;
      edge = true;
    }
    if (win < 0 && tid == 0) {  // no positive mass anywhere: degenerate input
      dev_flag(a.status, PVLM_DEV_RANGE);
      a.nacc[b] = s_a[b];
      a.next[b] = 0;
      if (a.near) a.near[b] = 1;
    }
    if (mine == win && win >= 0) {
      int tie = s_tie[b];
      if (!edge) {
        if (fabs(at - thr) <= kNearTie * Z) tie = 1;
        if (win > 0 && fabs(below - thr) <= kNearTie * Z) tie = 1;
      } else {
        tie = 1;
      }
      a.nacc[b] = s_a[b];
      a.next[b] = win;
      if (a.near) a.near[b] = tie;
    }
    __syncthreads();
  }
  __syncthreads();
  if (tid == 0) {
    const int done = __hip_atomic_fetch_add(a.bar + 1, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (done == W - 1) {
      __hip_atomic_store(a.bar, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.bar + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

struct APlan {
  int NC;
  size_t off_bar, off_pm, off_ps, off_pi, off_rs, off_qs, bytes;
};

pvlm_status plan_accept(int B, int gamma, int V, APlan* p) {
  if (B < 1 || gamma < 1 || V < 1) return PVLM_ERR_SHAPE;
  if (B > kAccMaxB || gamma > 32 || V > (1 << 30)) return PVLM_ERR_UNSUPPORTED;
  p->NC = (V + kChunk - 1) / kChunk;
  const size_t rows = (size_t)B * (2 * gamma + 1) * p->NC;
  size_t off = 0;
  p->off_bar = off;
  off = align_up(off + 2 * sizeof(int), 256);
  p->off_pm = off;
  off = align_up(off + rows * sizeof(double), 256);
  p->off_ps = off;
  off = align_up(off + rows * sizeof(double), 256);
  p->off_pi = off;
  off = align_up(off + rows * sizeof(int), 256);
  p->off_rs = off;
  off = align_up(off + (size_t)B * p->NC * sizeof(double), 256);
  p->off_qs = off;
  off = align_up(off + (size_t)B * p->NC * sizeof(double), 256);
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
  st = device_info(&di);
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
  a.bar = reinterpret_cast<int*>(wsb + p.off_bar);
  a.B = B;
  a.gamma = gamma;
  a.V = V;
  a.NC = p.NC;
  a.tau = (double)temperature;
  a.greedy = temperature == 0.f;
  const int items = B * (2 * gamma + 1) * p.NC;
  int grid = di.cus < items ? di.cus : items;
  if (grid < 1) grid = 1;
  void* args[] = {&a};
  PVLM_HIP(hipLaunchCooperativeKernel(reinterpret_cast<const void*>(accept_kernel), dim3(grid),
                                      dim3(kAccThreads), args, 0, stream));
  return PVLM_OK;
}
