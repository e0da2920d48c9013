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
constexpr int kMaxChunks = 1024;                // V <= kMaxChunks * kChunk
constexpr double kNearTie = 1e-9;
constexpr double kNegInfD = -__builtin_huge_val();

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
  double* pm;     // [B][RW][NC] chunk max
  double* ps;     // [B][RW][NC] chunk exp-sum (relative to the chunk max)
  int* pi;        // [B][RW][NC] chunk argmax (lowest index)
  double* rowM;   // [B][RW] row max
  double* rowZ;   // [B][RW] row normaliser
  int* rowA;      // [B][RW] row argmax
  int* rowcnt;    // [B][RW] chunks finished (last one combines the row)
  double* rs;     // [B][NC] residual chunk mass
  double* qs;     // [B][NC] p chunk mass (used when the residual is empty)
  int* bcnt;      // [B] chunks finished in phase 3
  double* bZ;     // [B] total mass of the draw distribution
  double* bPre;   // [B] mass before the crossing chunk
  int* bCross;    // [B] crossing chunk
  int* bMode;     // [B] bit 0: draw from the residual; bit 1: rounding fallback
  int* bar;       // [0] arrivals, [1] finished workgroups
  int B, gamma, V, NC;
  double tau;
  int greedy;
};

__device__ __forceinline__ const float* row_ptr(const AArgs& a, int b, int rho) {
  if (rho <= a.gamma) return a.tl + ((size_t)b * (a.gamma + 1) + rho) * a.V;
  return a.dl + ((size_t)b * a.gamma + (rho - a.gamma - 1)) * a.V;
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

// Workgroup-wide max with lowest-index tie-break (value, index), fixed order.
__device__ void block_argmax(double& v, int& i, double* s_v, int* s_i) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double v2 = __shfl_xor(v, o, 64);
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
  for (int k = 1; k < kAccThreads / 64; ++k)
    if (s_v[k] > v || (s_v[k] == v && s_i[k] < i)) {
      v = s_v[k];
      i = s_i[k];
    }
  __syncthreads();
}

__device__ double block_sum(double x, double* s_v) {
  x = warp_sum(x);
  if ((threadIdx.x & 63) == 0) s_v[threadIdx.x >> 6] = x;
  __syncthreads();
  double t = 0.0;
  for (int k = 0; k < kAccThreads / 64; ++k) t += s_v[k];
  __syncthreads();
  return t;
}

__device__ __forceinline__ void finish(const AArgs& a, int* s_flag) {
  if (wg_signal_last(a.bar + 1, gridDim.x, s_flag) && threadIdx.x == 0) {
    reset_counter(a.bar);
    reset_counter(a.bar + 1);
  }
}

__global__ void __launch_bounds__(kAccThreads) accept_kernel(AArgs a) {
  __shared__ double s_v[kAccThreads / 64];
  __shared__ int s_i[kAccThreads / 64];
  __shared__ double s_M[65], s_Z[65], s_px[32], s_qx[32];
  __shared__ int s_arg[65], s_xok[32];
  __shared__ int s_a[kAccMaxB], s_tie[kAccMaxB];
  __shared__ double s_pM[kAccMaxB], s_pZ[kAccMaxB], s_qM[kAccMaxB], s_qZ[kAccMaxB];
  __shared__ double s_cr[kMaxChunks], s_cq[kMaxChunks];
  __shared__ int s_win, s_flag;
  const int tid = threadIdx.x;
  const int RW = 2 * a.gamma + 1;
  const int W = gridDim.x;
  const double tau = a.tau;

  // ---- phase 1: chunk max / argmax / exp-sum; the last chunk of a row
  //      combines the row's totals
  const int items1 = a.B * RW * a.NC;
  for (int it = blockIdx.x; it < items1; it += W) {
    const int c = it % a.NC, rho = (it / a.NC) % RW, b = it / (a.NC * RW);
    if (a.greedy && rho > a.gamma) continue;
    const float* z = row_ptr(a, b, rho);
    const int y0 = c * kChunk, y1 = min(a.V, y0 + kChunk);
    double mx = kNegInfD;
    int am = 0x7fffffff;
    for (int y = y0 + tid; y < y1; y += kAccThreads) {
      const double v = z[y];
      if (v > mx) {
        mx = v;
        am = y;
      }
    }
    block_argmax(mx, am, s_v, s_i);
    double sum = 0.0;
    if (!a.greedy && mx != kNegInfD)
      for (int y = y0 + tid; y < y1; y += kAccThreads) sum += exp(((double)z[y] - mx) / tau);
    sum = block_sum(sum, s_v);
    if (tid == 0) {
      st_agent(a.pm + it, mx);
      st_agent(a.ps + it, sum);
      st_agent(a.pi + it, am);
    }
    const int r = b * RW + rho;
    if (wg_signal_last(a.rowcnt + r, a.NC, &s_flag)) {
      const size_t base = (size_t)r * a.NC;
      double M = kNegInfD;
      int A = 0x7fffffff;
      for (int k = tid; k < a.NC; k += kAccThreads) {
        const double m2 = ld_agent(a.pm + base + k);
        const int i2 = ld_agent(a.pi + base + k);
        if (m2 > M || (m2 == M && i2 < A)) {
          M = m2;
          A = i2;
        }
      }
      block_argmax(M, A, s_v, s_i);
      double Z = 0.0;
      if (!a.greedy && M != kNegInfD)
        for (int k = tid; k < a.NC; k += kAccThreads) {
          const double m2 = ld_agent(a.pm + base + k);
          if (m2 != kNegInfD) Z += ld_agent(a.ps + base + k) * exp((m2 - M) / tau);
        }
      Z = block_sum(Z, s_v);
      if (tid == 0) {
        st_agent(a.rowM + r, M);
        st_agent(a.rowZ + r, Z);
        st_agent(a.rowA + r, A);
        reset_counter(a.rowcnt + r);
      }
    }
    __syncthreads();
  }
  wg_signal_wait(a.bar, W, a.status, true);

  // ---- phase 2: the sequential accept decisions (every workgroup with later
  //      work replays them from the row totals)
  const bool has_late = a.greedy ? blockIdx.x == 0 : blockIdx.x < a.B * a.NC;
  if (has_late) {
    for (int b = 0; b < a.B; ++b) {
      if (tid < RW && (!a.greedy || tid <= a.gamma)) {
        s_M[tid] = ld_agent(a.rowM + b * RW + tid);
        s_Z[tid] = ld_agent(a.rowZ + b * RW + tid);
        s_arg[tid] = ld_agent(a.rowA + b * RW + tid);
      }
      if (tid >= 64 && tid < 64 + a.gamma) {
        const int t = tid - 64;
        const int x = a.tok[(size_t)b * a.gamma + t];
        const int ok = x >= 0 && x < a.V;
        s_xok[t] = ok ? x : -1;
        if (ok && !a.greedy) {
          s_px[t] = row_ptr(a, b, t)[x];
          s_qx[t] = row_ptr(a, b, a.gamma + 1 + t)[x];
        }
      }
      __syncthreads();
      if (tid == 0) {
        int acc = a.gamma, tie = 0;
        for (int t = 0; t < a.gamma; ++t) {
          const int x = s_xok[t];
          if (x < 0) {
            dev_flag(a.status, PVLM_DEV_RANGE);
            acc = t;
            break;
          }
          bool ok;
          if (a.greedy) {
            ok = x == s_arg[t];
          } else {
            const int qr = a.gamma + 1 + t;
            const double p = exp((s_px[t] - s_M[t]) / tau) / s_Z[t];
            const double q = exp((s_qx[t] - s_M[qr]) / tau) / s_Z[qr];
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
    finish(a, &s_flag);
    return;
  }

  // r(y) of the draw distribution of batch b; also p(y)
  auto draw_mass = [&](int b, int y, double& p_out) -> double {
    const int acc = s_a[b];
    const double p = exp(((double)row_ptr(a, b, acc)[y] - s_pM[b]) / tau) / s_pZ[b];
    p_out = p;
    if (acc == a.gamma) return p;
    const double q = exp(((double)row_ptr(a, b, a.gamma + 1 + acc)[y] - s_qM[b]) / tau) / s_qZ[b];
    return p > q ? p - q : 0.0;
  };

  // ---- phase 3: chunk masses of the draw distribution; the last chunk of a
  //      batch row locates the crossing chunk
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
    block_scan_f64(sr, s_v, &tr);
    block_scan_f64(sp, s_v, &tp);
    if (tid == 0) {
      st_agent(a.rs + it, tr);
      st_agent(a.qs + it, tp);
    }
    if (wg_signal_last(a.bcnt + b, a.NC, &s_flag)) {
      for (int k = tid; k < a.NC; k += kAccThreads) {
        s_cr[k] = ld_agent(a.rs + (size_t)b * a.NC + k);
        s_cq[k] = ld_agent(a.qs + (size_t)b * a.NC + k);
      }
      __syncthreads();
      if (tid == 0) {
        double Zr = 0.0, Zp = 0.0;
        for (int k = 0; k < a.NC; ++k) {
          Zr += s_cr[k];
          Zp += s_cq[k];
        }
        const bool use_r = Zr > 0.0;
        const double* sums = use_r ? s_cr : s_cq;
        const double Z = use_r ? Zr : Zp;
        const double thr = a.us[b] * Z;
        double run = 0.0, pre = 0.0, pre_last = 0.0;
        int cross = -1, last_pos = -1;
        for (int k = 0; k < a.NC; ++k) {
          const double sk = sums[k];
          if (sk > 0.0) {
            last_pos = k;
            pre_last = run;
          }
          if (cross < 0 && run + sk > thr) {
            cross = k;
            pre = run;
          }
          run += sk;
        }
        int mode = use_r ? 1 : 0;
        if (cross < 0) {
          mode |= 2;
          cross = last_pos < 0 ? 0 : last_pos;
          pre = pre_last;
        }
        st_agent(a.bZ + b, Z);
        st_agent(a.bPre + b, pre);
        st_agent(a.bCross + b, cross);
        st_agent(a.bMode + b, mode);
        reset_counter(a.bcnt + b);
      }
    }
    __syncthreads();
  }
  wg_signal_wait(a.bar, 2 * W, a.status, true);

  // ---- phase 4: the crossing chunk scans its elements and writes the outputs
  for (int it = blockIdx.x; it < items3; it += W) {
    const int b = it / a.NC, c = it % a.NC;
    if (c != ld_agent(a.bCross + b)) continue;  // uniform across the workgroup
    const int mode = ld_agent(a.bMode + b);
    const bool use_r = mode & 1, fallback = mode & 2;
    const double Z = ld_agent(a.bZ + b), pre = ld_agent(a.bPre + b);
    const double thr = a.us[b] * Z;
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
    const double excl = block_scan_f64(own, s_v, &tot);
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
  finish(a, &s_flag);
}

struct APlan {
  int NC;
  size_t off_bar, off_pm, off_ps, off_pi, off_rowM, off_rowZ, off_rowA, off_rowcnt, off_rs, off_qs,
      off_bcnt, off_bZ, off_bPre, off_bCross, off_bMode, bytes;
};

pvlm_status plan_accept(int B, int gamma, int V, APlan* p) {
  if (B < 1 || gamma < 1 || V < 1) return PVLM_ERR_SHAPE;
  if (B > kAccMaxB || gamma > 32 || V > kMaxChunks * kChunk) return PVLM_ERR_UNSUPPORTED;
  p->NC = (V + kChunk - 1) / kChunk;
  const size_t rows = (size_t)B * (2 * gamma + 1);
  const size_t parts = rows * p->NC;
  // counters first (inside the fixed synchronisation region), data after it
  size_t sync = 0;
  auto take_sync = [&](size_t bytes) {
    const size_t at = sync;
    sync += bytes;
    return at;
  };
  p->off_bar = take_sync(2 * sizeof(int));
  p->off_rowcnt = take_sync(rows * sizeof(int));
  p->off_bcnt = take_sync(B * sizeof(int));
  if (sync > kSyncMonoOff) return PVLM_ERR_UNSUPPORTED;
  size_t off = kSyncRegion;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  p->off_pm = take(parts * sizeof(double));
  p->off_ps = take(parts * sizeof(double));
  p->off_pi = take(parts * sizeof(int));
  p->off_rowM = take(rows * sizeof(double));
  p->off_rowZ = take(rows * sizeof(double));
  p->off_rowA = take(rows * sizeof(int));
  p->off_rs = take((size_t)B * p->NC * sizeof(double));
  p->off_qs = take((size_t)B * p->NC * sizeof(double));
  p->off_bZ = take(B * sizeof(double));
  p->off_bPre = take(B * sizeof(double));
  p->off_bCross = take(B * sizeof(int));
  p->off_bMode = take(B * sizeof(int));
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
  a.rowM = reinterpret_cast<double*>(wsb + p.off_rowM);
  a.rowZ = reinterpret_cast<double*>(wsb + p.off_rowZ);
  a.rowA = reinterpret_cast<int*>(wsb + p.off_rowA);
  a.rowcnt = reinterpret_cast<int*>(wsb + p.off_rowcnt);
  a.rs = reinterpret_cast<double*>(wsb + p.off_rs);
  a.qs = reinterpret_cast<double*>(wsb + p.off_qs);
  a.bcnt = reinterpret_cast<int*>(wsb + p.off_bcnt);
  a.bZ = reinterpret_cast<double*>(wsb + p.off_bZ);
  a.bPre = reinterpret_cast<double*>(wsb + p.off_bPre);
  a.bCross = reinterpret_cast<int*>(wsb + p.off_bCross);
  a.bMode = reinterpret_cast<int*>(wsb + p.off_bMode);
  a.bar = reinterpret_cast<int*>(wsb + p.off_bar);
  a.B = B;
  a.gamma = gamma;
  a.V = V;
  a.NC = p.NC;
  a.tau = (double)temperature;
  a.greedy = temperature == 0.f;
  const int items = B * (2 * gamma + 1) * p.NC;
  // a multiple of 8 workgroups (the XCD count) keeps the cooperative queue's
  // round-robin XCD placement aligned for the launches that follow
  int grid = (items + 7) / 8 * 8;
  if (grid > di.cus) grid = di.cus;
  if (grid < 1) grid = 1;
  void* args[] = {&a};
  PVLM_HIP(launch_coresident(reinterpret_cast<const void*>(accept_kernel), dim3(grid),
                             dim3(kAccThreads), args, 0, stream));
  return PVLM_OK;
}
