// Verify attention with fused per-token attention mass (gfx950).
//
// Computes the target's verification forward over the video KV cache
// (ParallelVLM Sec. 2.2; Sec. 4.2 Parallel Decoding) for the gamma + 1 verify
// rows, fused with the per-token attention mass that attention-guided pruning
// ranks visual tokens by (Sec. 3, Challenge 2; Suppl. D, attention criterion).
// The paper notes that pruning by attention needs explicit scores, which
// block-wise attention kernels never materialise (Sec. 3; Sec. 5.3,
// FlashAttention compatibility): here the mass is produced inside the
// block-wise kernel, with no score matrix in memory.
//
// Design (one launch, grid co-resident: one workgroup per CU):
//  * Work unit = (batch b, KV head g, row group rg, token chunk).  All
//    (Hq/Hkv) * T query rows of a KV head are packed as the N side of
//    v_mfma_f32_16x16x32_bf16 tiles (16 rows per tile, at most 5 tiles per
//    workgroup); tokens are the M side, so each lane owns one query row and
//    four tokens of every score tile.  The workgroups of one (b, g, rg) are
//    placed on one XCD.
//  * "Resident" variant (chunks up to 512 tokens): every wave puts its K
//    blocks in flight straight into MFMA operand registers, waves 1-3 stream
//    the chunk's V into LDS behind them (global_load_lds), and the scores stay
//    in registers as probabilities relative to the workgroup's row maxima.
//    The row statistics are published and, by the time V has landed, the
//    group's other chunks have published theirs: one wait, then every row's
//    global log-sum-exp makes the resident probabilities exact (one multiply
//    per score), and P.V runs fused with the mass of the chunk's tokens, so
//    the scores die block by block.  The four waves' O fragments are
//    reduce-scattered through LDS and the normalised chunk partial (bf16) is
//    published; after a second wait each workgroup writes one slice of O as
//    the plain sum of the group's chunk partials.
//  * "Stream" variant (longer chunks): statistics are exchanged after pass 1,
//    pass 2 recomputes the scores from K (K is read twice) with the exact
//    global log-sum-exp, and a second wait precedes the O sum.
//  * The mass is summed over KV heads and row groups by whichever workgroup
//    of a chunk arrives last.  Every sum runs in a fixed order, so results
//    are bit-reproducible.
//  * Workgroups exchange data through stores the writer waits for, a relaxed
//    counter increment and a polling wait (no cache flush).  Within a group
//    the stores and loads are plain when every workgroup of the group runs
//    on one XCD (one L2; each address is written once per launch), else
//    device-coherent; across groups (the mass sum) always device-coherent.
//  * fp32 inputs take a VALU path with the two-wait structure.
#include <mutex>

#include "common.h"

namespace pvlm {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kMaxRT = 5;        // 16-row tiles per workgroup
constexpr int kPageSlots = 512;  // page-table entries a workgroup stages in LDS
constexpr int kOSets = 8;        // max thread sets splitting the O-partial sum
constexpr int kNB = 4;           // 32-token blocks per wave (resident variant)
constexpr int kResTokens = kWaves * kNB * 32;
constexpr int kF32Tile = 64;     // tokens per step of the fp32 path
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_huge_valf();

// Field order matters for the kernels' scalar registers: the argument loads
// merge adjacent fields into wide scalar loads whose registers are then
// allocated (and, under pressure, spilled and restored) as one unit.  The
// inputs read at the start, the sizes used throughout, and the workspace and
// output pointers used late therefore sit in three separate runs.
struct VArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* ctx_len;
  const int32_t* table;  // paged caches: [B][max_pages] pool page of each logical page; NULL: padded
  int64_t n_pages;       // pool pages
  int max_pages, page_shift;
  int64_t n_cap;
  int B, T, Hq, Hkv, G, R, RG, RT, D;
  int max_ctx;
  int splits, chunk, grp_base, ngrp, grid;
  int xmap;         // workgroup i runs on XCD i % xmap (1: no XCD-aware mapping)
  int local;        // every group's workgroups share one XCD
  float sl2;        // scale * log2(e)
  int f32;
  float* stats;     // [groups][splits] records of ROWS + 1 float2 (padded to 128 B):
                    // (log2-domain max, exp-sum) per row, then the launch tag
  float* opart;     // [groups][splits][ROWS][D] (bf16 pairs, or fp32)
  float* mpart;     // [B][Hkv*RG][n_cap]
  unsigned* slots;  // [groups][3] monotonic, one 128-byte line each: arrivals
                    // with published statistics, arrivals with published O
                    // partials, and the counters' value when the launch began
  int* mcnt;        // [B][splits] arrivals per chunk for the mass sum (128 B apart)
  void* out;
  float* lse;
  float* mass;
  int32_t* status;
};

struct Unit {
  int grp, split, b, g, rg, ctx, N, c0, c1;
};

__device__ __forceinline__ bool decode_unit(const VArgs& a, Unit& u) {
  const int i = blockIdx.x;
  const int per_xcd = a.grid / a.xmap;
  // Consecutive logical units share an XCD.  Workgroup i runs on XCD
  // (i + s) % xmap for a launch-wide offset s (s = 0 on an idle queue), so in
  // the same-XCD exchange mode the logical index is built from the XCD the
  // workgroup actually runs on, which keeps every group on one XCD for any s.
  int x = i % a.xmap;
  if (a.local) {
    int xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    xcc &= 0xf;
    if (xcc < a.xmap) x = xcc;
    else if (threadIdx.x == 0) dev_flag(a.status, PVLM_DEV_PLACEMENT);
  }
  const int lg = x * per_xcd + i / a.xmap;
  if (lg >= a.ngrp * a.splits) return false;
  u.grp = a.grp_base + lg / a.splits;
  u.split = lg % a.splits;
  u.rg = u.grp % a.RG;
  const int bg = u.grp / a.RG;
  u.g = bg % a.Hkv;
  u.b = bg / a.Hkv;
  int ctx = a.ctx_len[u.b];
  if (ctx < 0 || ctx > a.max_ctx) {
    if (u.split == 0 && threadIdx.x == 0) dev_flag(a.status, PVLM_DEV_RANGE);
    ctx = ctx < 0 ? 0 : a.max_ctx;
  }
  u.ctx = ctx;
  u.N = ctx + a.T;
  u.c0 = u.split * a.chunk;
  u.c1 = min(u.c0 + a.chunk, u.N);
  return true;
}

// exp2 on the hardware transcendental unit (v_exp_f32).  It flushes results
// below 2^-126 to zero, which only drops probabilities under the mass
// tolerance's absolute floor.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ void lse_combine(float& m, float& z, float m2, float z2) {
  const float M = fmaxf(m, m2);
  if (M == kNegInf) {
    m = kNegInf;
    z = 0.f;
    return;
  }
  z = z * fast_exp2(m - M) + z2 * fast_exp2(m2 - M);
  m = M;
}

// ---------------------------------------------------- group exchanges --
// The workgroups of one (b, g, rg) group meet at two monotonic counters
// (common.h): cnt_s once their row statistics are published, cnt_o once their
// O partials are.  Every workgroup arrives at cnt_s before cnt_o, and the
// launch's last arrival at cnt_o advances the group's base.

constexpr int kLineU = (int)(kSyncLine / sizeof(unsigned));  // counters per 128-byte line
__device__ __forceinline__ unsigned* cnt_s(const VArgs& a, const Unit& u) {
  return a.slots + (3 * u.grp) * kLineU;
}
__device__ __forceinline__ unsigned* cnt_o(const VArgs& a, const Unit& u) {
  return a.slots + (3 * u.grp + 1) * kLineU;
}
__device__ __forceinline__ unsigned* cnt_base(const VArgs& a, const Unit& u) {
  return a.slots + (3 * u.grp + 2) * kLineU;
}

// The group's counter base for this launch (every thread reads it).
__device__ __forceinline__ unsigned read_base(const VArgs& a, const Unit& u) {
  return grp_read(cnt_base(a, u));
}

// Release word of the statistics exchange, on the base's line: the last
// arrival at cnt_s stores the count every workgroup waits for, and the others
// poll that word instead of the counter, so that their polls do not contend
// with the arrivals' atomics on the counter's line.  Like the counters it
// only grows, and at rest it equals the base.  (The O exchange polls cnt_o
// itself: there the release's extra hop after the last arrival cost more
// than the contention it saves.)
__device__ __forceinline__ unsigned* rel_s(const VArgs& a, const Unit& u) { return cnt_base(a, u) + 8; }

// Thread 0: arrive at cnt_s (statistics published) and, if asked, wait for
// the whole group.
__device__ __forceinline__ void stats_arrive(const VArgs& a, const Unit& u, unsigned base, bool wait) {
  const unsigned target = base + (unsigned)a.splits;
  if (grp_arrive(cnt_s(a, u)) == target - 1u)
    __hip_atomic_store(rel_s(a, u), target, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else if (wait)
    grp_poll(rel_s(a, u), target, a.status);
}

// Each workgroup's statistics record holds ROWS (max, exp-sum) pairs and a
// header stamped with the launch's tag (base + 1, different in every launch
// of the group), which readers check: a record missing from this launch
// (misplaced workgroup, stale data) raises PVLM_DEV_PLACEMENT.
// Records are padded to whole 128-byte lines so no two workgroups' records
// share a cache line.
template <int ROWS>
constexpr int rec_stride() { return (ROWS + 1 + 15) / 16 * 16; }  // float2 units
template <int ROWS>
__device__ __forceinline__ float2* stats_rec(const VArgs& a, const Unit& u, int split) {
  return reinterpret_cast<float2*>(a.stats) + ((size_t)u.grp * a.splits + split) * rec_stride<ROWS>();
}

// Wave 0 publishes this workgroup's per-row (max, exp-sum) and the tag.
template <int ROWS, bool LOCAL>
__device__ __forceinline__ void stats_store(const VArgs& a, const Unit& u, const float* s_m,
                                            const float* s_z, unsigned base) {
  if (threadIdx.x < 64) {
    float2* st = stats_rec<ROWS>(a, u, u.split);
    for (int r = threadIdx.x; r < ROWS; r += 64) x_store<LOCAL>(st + r, make_float2(s_m[r], s_z[r]));
    if (threadIdx.x == 0) x_store<LOCAL>(st + ROWS, make_float2(__uint_as_float(base + 1u), 0.f));
  }
}

// Thread 0, after its O-partial arrival returned `old`: the launch's last
// arrival advances the base, every other workgroup waits (if asked) for all.
__device__ __forceinline__ void o_finish(const VArgs& a, const Unit& u, unsigned base, unsigned old,
                                         bool wait) {
  if (old - base == (unsigned)a.splits - 1u)
    __hip_atomic_store(cnt_base(a, u), base + (unsigned)a.splits, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  else if (wait)
    grp_poll(cnt_o(a, u), base + (unsigned)a.splits, a.status);
}

// Every row's statistics over the group's nsp chunks, combined in parallel
// (P thread sets per row): leaves the row's log2-sum-exp in s_lse (+inf for
// padding rows, whose probabilities are then 0), its global max in s_pm[0]
// and 1/sum in s_pz[0] (0 for padding rows).
template <int ROWS, bool LOCAL>
__device__ void stats_combine(const VArgs& a, const Unit& u, int nsp, float* s_lse,
                              float (*s_pm)[ROWS], float (*s_pz)[ROWS], unsigned base) {
  constexpr int kU = 16;
  constexpr int P = kThreads / ROWS < kWaves ? kThreads / ROWS : kWaves;
  const int tid = threadIdx.x;
  const float2* st0 = stats_rec<ROWS>(a, u, 0);
  // every chunk's record is from this launch (its tag word); the first
  // kThreads tags load together with the statistics and are checked after
  const float2 tag = x_load<LOCAL>(st0 + (size_t)min(tid, nsp - 1) * rec_stride<ROWS>() + ROWS);
  if (tid < P * ROWS) {
    const int r = tid % ROWS, part = tid / ROWS;
    float M = kNegInf, Z = 0.f;
    for (int s0 = part; s0 < nsp; s0 += P * kU) {
      float2 v[kU];
#pragma unroll
      for (int j = 0; j < kU; ++j)  // unconditional (clamped) loads: fine-grained waits
        v[j] = x_load<LOCAL>(st0 + (size_t)min(s0 + j * P, nsp - 1) * rec_stride<ROWS>() + r);
      // the batch's maximum (exact in any order), then its exp-sum relative
      // to it: independent exp2s instead of a chain of pairwise combines.
      // Branch-free, so both halves of every record load together (a record
      // with no visible token is (-inf, 0) and adds 0).
      float bm = kNegInf;
#pragma unroll
      for (int j = 0; j < kU; ++j) bm = fmaxf(bm, s0 + j * P < nsp ? v[j].x : kNegInf);
      const float bref = bm == kNegInf ? 0.f : bm;
      float bz = 0.f;
#pragma unroll
      for (int j = 0; j < kU; ++j) bz += s0 + j * P < nsp ? v[j].y * fast_exp2(v[j].x - bref) : 0.f;
      lse_combine(M, Z, bm, bz);
    }
    s_pm[part][r] = M;
    s_pz[part][r] = Z;
  }
  if (__float_as_uint(tag.x) != base + 1u) dev_flag(a.status, PVLM_DEV_PLACEMENT);
  for (int sp = tid + kThreads; sp < nsp; sp += kThreads) {
    const float2 h = x_load<LOCAL>(st0 + (size_t)sp * rec_stride<ROWS>() + ROWS);
    if (__float_as_uint(h.x) != base + 1u) dev_flag(a.status, PVLM_DEV_PLACEMENT);
  }
  lds_sync();
  if (tid < ROWS) {
    const int r = tid;
    float M = s_pm[0][r], Z = s_pz[0][r];
#pragma unroll
    for (int p = 1; p < P; ++p) lse_combine(M, Z, s_pm[p][r], s_pz[p][r]);
    const bool ok = u.rg * a.RT * 16 + r < a.R && Z > 0.f;
    s_lse[r] = ok ? M + __log2f(Z) : __builtin_huge_valf();
    s_pm[0][r] = M;
    s_pz[0][r] = ok ? 1.f / Z : 0.f;
  }
  lds_sync();
}

// Statistics exchange of the two-pass variants: publish, arrive, and (unless
// the chunk is empty) wait for the whole group and combine into s_lse.
template <int ROWS, bool LOCAL>
__device__ void exchange_stats(const VArgs& a, const Unit& u, const float* s_m, const float* s_z,
                               float* s_lse, float (*s_pm)[ROWS], float (*s_pz)[ROWS],
                               unsigned base, bool wait) {
  __syncthreads();
  stats_store<ROWS, LOCAL>(a, u, s_m, s_z, base);
  // wave-uniform branch: only wave 0 wrote, only it waits for its stores
  if (__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) == 0) __builtin_amdgcn_s_waitcnt(0);
  if (threadIdx.x == 0) stats_arrive(a, u, base, wait);
  __syncthreads();
  if (wait)
    stats_combine<ROWS, LOCAL>(a, u, (u.N + a.chunk - 1) / a.chunk, s_lse, s_pm, s_pz, base);
}

// Per-token mass summed over the KV heads and row groups by the last
// workgroup of each chunk to arrive (the chunk's workgroups sit on different
// XCDs, so these exchanges are device-coherent).
__device__ __forceinline__ int* mass_counter(const VArgs& a, const Unit& u) {
  return a.mcnt + ((size_t)u.b * a.splits + u.split) * (kSyncLine / sizeof(int));
}
// The chunk's mass sum, by its last arrival (every partial is published).
__device__ void mass_sum(const VArgs& a, const Unit& u) {
  const int tid = threadIdx.x;
  const int P = a.Hkv * a.RG;
  const int64_t lo = u.c0;
  const int64_t hi_sum = u.c1 > u.c0 ? u.c1 : u.c0;
  const int64_t chunk_end = (int64_t)u.c0 + a.chunk;
  const int64_t hi = u.split == a.splits - 1 ? a.n_cap : (chunk_end < a.n_cap ? chunk_end : a.n_cap);
  const float* mp = a.mpart + (size_t)u.b * P * a.n_cap;
  float* ms = a.mass + (size_t)u.b * a.n_cap;
  // two tokens per thread and pass, all their loads in flight together
  // (clamped indices; the sums run over p in order, so results do not depend
  // on the batching)
  for (int64_t i0 = lo + tid; i0 < hi; i0 += 2 * kThreads) {
    const int64_t i1 = i0 + kThreads;
    float acc0 = 0.f, acc1 = 0.f;
    if (hi_sum > lo) {
      const int64_t t0 = i0 < hi_sum ? i0 : hi_sum - 1, t1 = i1 < hi_sum ? i1 : hi_sum - 1;
      for (int p0 = 0; p0 < P; p0 += 8) {
        float v0[8], v1[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float* row = mp + (size_t)min(p0 + j, P - 1) * a.n_cap;
          v0[j] = ld_agent(row + t0);
          v1[j] = ld_agent(row + t1);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          if (p0 + j < P) {
            acc0 += v0[j];
            acc1 += v1[j];
          }
        }
      }
      if (i0 >= hi_sum) acc0 = 0.f;
      if (i1 >= hi_sum) acc1 = 0.f;
    }
    ms[i0] = acc0;
    if (i1 < hi) ms[i1] = acc1;
  }
  if (tid == 0) reset_counter(mass_counter(a, u));
}
__device__ void mass_combine(const VArgs& a, const Unit& u, int* s_flag) {
  if (!a.mass) return;
  if (wg_signal_last(mass_counter(a, u), a.Hkv * a.RG, s_flag)) mass_sum(a, u);
}

// End of the two-pass variants: the O partials are published (every wave's
// stores complete), arrive at cnt_o and wait; O = sum of the chunk partials
// (one slice per workgroup), lse; then the mass sum.
template <int ROWS, int D, bool LOCAL>
__device__ void verify_epilogue(const VArgs& a, const Unit& u, const float* s_lse, bool empty,
                                int* s_flag, unsigned base) {
  const int tid = threadIdx.x;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0) o_finish(a, u, base, grp_arrive(cnt_o(a, u)), !empty);
  __syncthreads();
  if (!empty) {
    const int row0 = u.rg * a.RT * 16;
    const int nsp = (u.N + a.chunk - 1) / a.chunk;
    const int rows = min(ROWS, a.R - row0);
    const int E4 = rows * D / 4;  // groups of four consecutive values
    const int per = (E4 + nsp - 1) / nsp;
    const int e0 = u.split * per, e1 = min(E4, e0 + per);
    for (int e = e0 + tid; e < e1; e += kThreads) {
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      if (a.f32) {  // fp32 partials, two float pairs per group
        const float2* op = reinterpret_cast<const float2*>(a.opart + (size_t)u.grp * a.splits * ROWS * D);
        for (int s0 = 0; s0 < nsp; s0 += 8) {
          float2 v[8][2];
#pragma unroll
          for (int j = 0; j < 8; ++j)
#pragma unroll
            for (int h = 0; h < 2; ++h)
              v[j][h] = x_load<LOCAL>(op + ((size_t)min(s0 + j, nsp - 1) * ROWS * D) / 2 + 2 * e + h);
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            if (s0 + j < nsp) {
              acc[0] += v[j][0].x;
              acc[1] += v[j][0].y;
              acc[2] += v[j][1].x;
              acc[3] += v[j][1].y;
            }
          }
        }
      } else {  // bf16 partials, one 64-bit load per group
        const uint64_t* op = reinterpret_cast<const uint64_t*>(a.opart) + (size_t)u.grp * a.splits * ROWS * D / 4;
        for (int s0 = 0; s0 < nsp; s0 += 16) {
          uint64_t v[16];
#pragma unroll
          for (int j = 0; j < 16; ++j)
            v[j] = x_load<LOCAL>(op + (size_t)min(s0 + j, nsp - 1) * ROWS * D / 4 + e);
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if (s0 + j < nsp) {
#pragma unroll
              for (int h = 0; h < 4; ++h) acc[h] += bf16_to_f32((uint16_t)(v[j] >> (16 * h)));
            }
        }
      }
      const int row = row0 + (4 * e) / D, d = (4 * e) % D;
      const int t = row / a.G, h = u.g * a.G + row % a.G;
      const size_t oi = (((size_t)u.b * a.T + t) * a.Hq + h) * D + d;
      if (a.f32)
        *reinterpret_cast<float4*>(static_cast<float*>(a.out) + oi) = make_float4(acc[0], acc[1], acc[2], acc[3]);
      else
        *reinterpret_cast<uint64_t*>(static_cast<uint16_t*>(a.out) + oi) =
            pack_bf16x4(acc[0], acc[1], acc[2], acc[3]);
    }
    if (a.lse && u.split == 0) {
      for (int r = tid; r < rows; r += kThreads) {
        const int row = row0 + r, t = row / a.G, h = u.g * a.G + row % a.G;
        a.lse[((size_t)u.b * a.Hq + h) * a.T + t] = s_lse[r] * kLn2;
      }
    }
  }
  mass_combine(a, u, s_flag);
}

// ------------------------------------------------------------ MFMA path --
template <int D>
struct VVec;
template <>
struct VVec<128> {
  typedef uint4 T;
};
template <>
struct VVec<64> {
  typedef uint2 T;
};

__device__ __forceinline__ uint32_t word_of(const uint4& v, int w) {
  return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
}
__device__ __forceinline__ uint32_t word_of(const uint2& v, int w) { return w == 0 ? v.x : v.y; }

// B operand of P.V for output column group jd: element s is V[token(s)][DPL*n + jd].
template <typename VT>
__device__ __forceinline__ bf16x8 pack_v(const VT (&vr)[8], int jd) {
  const uint32_t sel = (jd & 1) ? 0x07060302u : 0x05040100u;
  uint32_t w[4];
#pragma unroll
  for (int p = 0; p < 4; ++p)
    w[p] = __builtin_amdgcn_perm(word_of(vr[2 * p + 1], jd >> 1), word_of(vr[2 * p], jd >> 1), sel);
  uint4 u = make_uint4(w[0], w[1], w[2], w[3]);
  return __builtin_bit_cast(bf16x8, u);
}

// K operand of one 32-token block: lane (n, gq) loads token tb + 16*tt + n,
// d in [32*ks + 8*gq, +8).  Tokens past the chunk load the chunk's last row
// (their scores are masked), keeping the loads unconditional so the
// compiler can wait for one block while the later ones stay in flight.
// NT: non-temporal loads (cache rows read once, so they need not displace the
// exchange data in L2).
template <int D, bool NT = false>
__device__ __forceinline__ void load_k_block(const KvRows& kv, int tb, int c1, int n, int gq,
                                             uint4 (&Kr)[2][D / 32]) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  int te;
  const uint16_t* r0 = kv_block<D>(kv, tb, c1, te);
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    const int tok = min(tb + 16 * tt + n, c1 - 1);
    const uint16_t* kp = r0 + (size_t)(tok - te) * D + 8 * gq;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      if constexpr (NT)
        Kr[tt][ks] = __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kp + 32 * ks)));
      else
        Kr[tt][ks] = *reinterpret_cast<const uint4*>(kp + 32 * ks);
    }
  }
}

// V operand rows of one 32-token block: lane (n, gq) loads tokens
// tb + {4gq..4gq+3, 16+4gq..16+4gq+3}, d in [DPL*n, DPL*n + DPL).  Tokens past
// the chunk load its last row (their probabilities are 0).
template <int D, bool NT = false>
__device__ __forceinline__ void load_v_block(const KvRows& kv, int tb, int c1, int n, int gq,
                                             typename VVec<D>::T (&Vr)[8]) {
  typedef typename VVec<D>::T VT;
  typedef uint32_t vec_t __attribute__((ext_vector_type(sizeof(VT) / 4)));
  constexpr int DPL = D / 16;
  int te;
  const uint16_t* r0 = kv_block<D>(kv, tb, c1, te);
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const int tok = min(tb + (s < 4 ? 4 * gq + s : 16 + 4 * gq + (s - 4)), c1 - 1);
    const uint16_t* p = r0 + (size_t)(tok - te) * D + DPL * n;
    if constexpr (NT)
      Vr[s] = __builtin_bit_cast(VT, __builtin_nontemporal_load(reinterpret_cast<const vec_t*>(p)));
    else
      Vr[s] = *reinterpret_cast<const VT*>(p);
  }
}

// Stream one 32-token block of V into LDS with coalesced global->LDS loads:
// instruction k of the wave covers cache rows tb + k*RPI .. +RPI (RPI = 512/D),
// lane l writes the 16 bytes at column (l % (D/8)) of row (l / (D/8)).  Rows
// past the chunk re-read its last row (their probabilities are 0).
// The loads are issued through inline asm so the compiler's wait insertion
// does not track them (it would otherwise wait for them before any later LDS
// access); untracked loads can only lengthen the compiler's own vmcnt waits.
// The consumer waits explicitly (s_waitcnt vmcnt(0) + workgroup barrier).
template <int D, bool NT = false>
__device__ __forceinline__ void issue_v_lds(const KvRows& kv, int tb, int c1, uint16_t* lds_blk,
                                            int lane) {
  constexpr int CPR = D / 8;    // 16-byte columns per row
  constexpr int RPI = 64 / CPR; // rows per instruction
  int te;
  const uint16_t* r0 = kv_block<D>(kv, tb, c1, te);
#pragma unroll
  for (int k = 0; k < 32 / RPI; ++k) {
    const int row = k * RPI + lane / CPR;
    const int tok = min(tb + row, c1 - 1);
    const uint16_t* src = r0 + (size_t)(tok - te) * D + 8 * (lane % CPR);
    const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_addr(lds_blk + k * RPI * D));
    if constexpr (NT)
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt"
                   :
                   : "s"(lds), "v"(src)
                   : "memory", "m0");
    else
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                   :
                   : "s"(lds), "v"(src)
                   : "memory", "m0");
  }
}

// V operand rows of one block from LDS (row-major [32][D] bf16).
template <int D>
__device__ __forceinline__ void read_v_lds(const uint16_t* lds_blk, int n, int gq,
                                           typename VVec<D>::T (&Vr)[8]) {
  typedef typename VVec<D>::T VT;
  constexpr int DPL = D / 16;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const int row = s < 4 ? 4 * gq + s : 16 + 4 * gq + (s - 4);
    Vr[s] = *reinterpret_cast<const VT*>(lds_blk + row * D + DPL * n);
  }
}

// Stream one 32-token block of K into LDS in the Q tile's layout (16-byte
// chunks XOR-swizzled by row, so the MFMA operand reads hit distinct banks),
// through untracked global->LDS loads like issue_v_lds.  Rows past the chunk
// re-read its last row.
template <int D, bool NT = false>
__device__ __forceinline__ void issue_k_lds(const KvRows& kv, int tb, int c1, uint16_t* lds_blk,
                                            int lane) {
  constexpr int CH = D / 8;
  constexpr int NI = 32 * CH / 64;
  int te;
  const uint16_t* r0 = kv_block<D>(kv, tb, c1, te);
#pragma unroll
  for (int ins = 0; ins < NI; ++ins) {
    const int slot = ins * 64 + lane, r = slot / CH, c = (slot % CH) ^ (r % CH);
    const uint16_t* src = r0 + (size_t)(min(tb + r, c1 - 1) - te) * D + 8 * c;
    const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_addr(lds_blk + ins * 64 * 8));
    if constexpr (NT)
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt"
                   :
                   : "s"(lds), "v"(src)
                   : "memory", "m0");
    else
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                   :
                   : "s"(lds), "v"(src)
                   : "memory", "m0");
  }
}

// K operand of one block from its swizzled LDS copy: the registers
// load_k_block would fill.
template <int D>
__device__ __forceinline__ void read_k_lds(const uint16_t* lds_blk, int n, int gq, uint4 (&Kr)[2][D / 32]) {
  constexpr int CH = D / 8;
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    const int r = 16 * tt + n;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const int c = 4 * ks + gq;
      Kr[tt][ks] = *reinterpret_cast<const uint4*>(lds_blk + (r * CH + (c ^ (r % CH))) * 8);
    }
  }
}

// Global->LDS loads of one 32-token block of K and V (issue_k_lds, issue_v_lds).
template <int D>
constexpr int kBlockDma = 32 * (D / 8) / 64 + 32 / (64 / (D / 8));

// Wait until at most `younger` vector memory operations are outstanding, for
// younger in {0, 1, kBlockDma, kBlockDma + 1} (wave-uniform): every older
// one, in particular an untracked global->LDS load, has then completed.  The
// asm's memory clobber keeps the LDS reads that follow after it.
template <int D>
__device__ __forceinline__ void wait_vm_younger(int younger) {
  constexpr int N = kBlockDma<D>;
  static_assert(N + 1 < 64, "vmcnt holds 6 bits");
  if (younger == 0)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if (younger == 1)
    asm volatile("s_waitcnt vmcnt(1)" ::: "memory");
  else if (younger == N)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
  else
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N + 1) : "memory");
}

// Scores of one block in the log2 domain, masked to -inf outside the chunk,
// past the causal limit of each verify row, and on padding rows.
template <int D, int RT>
__device__ __forceinline__ void scores_block(const VArgs& a, const Unit& u, const uint4 (&Kr)[2][D / 32],
                                             const uint16_t* s_q, int tb, int n, int gq,
                                             const int (&lim)[RT], float (&S)[2][RT][4]);

template <int RT>
__device__ __forceinline__ void running_stats(const float (&S)[2][RT][4], float (&m)[RT], float (&z)[RT]) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float mx = kNegInf;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, S[tt][rt][i]);
    const float M = fmaxf(m[rt], mx);
    if (M != kNegInf) {
      float acc = z[rt] * fast_exp2(m[rt] - M);
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc += fast_exp2(S[tt][rt][i] - M);
      z[rt] = acc;
      m[rt] = M;
    }
  }
}

// Reduce a per-lane value of each row over the four lane groups (max or sum)
// and the four waves into s_out[row] (scaled by `scale`); LDS barriers only.
template <int RT, bool MAX>
__device__ __forceinline__ void reduce_rows(float (&v)[RT], int n, int gq, int w, float (*s_w)[RT * 16],
                                            float* s_out, float scale) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    v[rt] = MAX ? rows4_max(v[rt]) : rows4_sum(v[rt]);
    if (gq == 0) s_w[w][rt * 16 + n] = v[rt];
  }
  lds_sync();
  for (int r = threadIdx.x; r < RT * 16; r += kThreads) {
    float acc = s_w[0][r];
#pragma unroll
    for (int ww = 1; ww < kWaves; ++ww) acc = MAX ? fmaxf(acc, s_w[ww][r]) : acc + s_w[ww][r];
    s_out[r] = acc == kNegInf ? kNegInf : acc * scale;
  }
  lds_sync();
}

// Reduce the per-lane (m, z) of each row over the four lane groups and the
// four waves into s_m / s_z.
template <int RT>
__device__ __forceinline__ void reduce_stats(float (&m)[RT], float (&z)[RT], int n, int gq, int w,
                                             float (*s_wm)[RT * 16], float (*s_wz)[RT * 16], float* s_m,
                                             float* s_z) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float m2 = off == 16 ? lane_xor16(m[rt]) : lane_xor32(m[rt]);
      const float z2 = off == 16 ? lane_xor16(z[rt]) : lane_xor32(z[rt]);
      lse_combine(m[rt], z[rt], m2, z2);
    }
    if (gq == 0) {
      s_wm[w][rt * 16 + n] = m[rt];
      s_wz[w][rt * 16 + n] = z[rt];
    }
  }
  lds_sync();
  for (int r = threadIdx.x; r < RT * 16; r += kThreads) {
    float M = s_wm[0][r], Z = s_wz[0][r];
#pragma unroll
    for (int ww = 1; ww < kWaves; ++ww) lse_combine(M, Z, s_wm[ww][r], s_wz[ww][r]);
    s_m[r] = M;
    s_z[r] = Z;
  }
  lds_sync();
}

// Probabilities of one block relative to a per-row reference (the
// workgroup's local row maximum), accumulated into O on MFMA.
template <int D, int RT>
__device__ __forceinline__ void pv_local(const float (&S)[2][RT][4], const float (&ref)[RT],
                                         const typename VVec<D>::T (&Vr)[8],
                                         floatx4 (&O)[RT][D / 16]) {
  constexpr int DPL = D / 16;
  bf16x8 Pa[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) Pa[rt][4 * tt + i] = static_cast<__bf16>(fast_exp2(S[tt][rt][i] - ref[rt]));
#pragma unroll
  for (int jd = 0; jd < DPL; ++jd) {
    const bf16x8 vb = pack_v(Vr, jd);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
      O[rt][jd] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Pa[rt], vb, O[rt][jd], 0, 0, 0);
  }
}

// Sum each lane's 8 token values over the 16 lanes (rows) of its lane group
// and store the per-token sums (lanes with even n hold one token each).
__device__ __forceinline__ void mass_reduce_store(const float (&pm)[8], float* mp, int tb, int c1, int n,
                                                  int gq) {
  // transpose-reduce: each step a lane keeps half of its values (chosen by
  // one bit of n) and adds the partner's copy of that half; partners differ
  // in that bit (n^8, then n^7 within each 8, n^2, n^1)
  const bool h8 = n & 8, h4 = n & 4, h2 = n & 2;
  float a8[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float send = h8 ? pm[k] : pm[4 + k];
    a8[k] = (h8 ? pm[4 + k] : pm[k]) + lane_xor8(send);
  }
  float a4[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const float send = h4 ? a8[k] : a8[2 + k];
    a4[k] = (h4 ? a8[2 + k] : a8[k]) + lane_mirror8(send);
  }
  const float send2 = h2 ? a4[0] : a4[1];
  float a2 = (h2 ? a4[1] : a4[0]) + lane_xor2(send2);
  a2 += lane_xor1(a2);
  const int v = (h8 ? 4 : 0) + (h4 ? 2 : 0) + (h2 ? 1 : 0);
  const int tok = tb + 16 * (v >> 2) + 4 * gq + (v & 3);
  if (!(n & 1) && tok < c1) st_agent(mp + tok, a2);
}

// The same per-token sums of one block written to LDS (dst[token - tb] for
// the block's 32 tokens).  Kept apart from mass_reduce_store: sharing one
// helper changed the register allocation of the kernels that use that one.
__device__ __forceinline__ void mass_reduce_lds(const float (&pm)[8], float* dst, int n, int gq) {
  const bool h8 = n & 8, h4 = n & 4, h2 = n & 2;
  float a8[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float send = h8 ? pm[k] : pm[4 + k];
    a8[k] = (h8 ? pm[4 + k] : pm[k]) + lane_xor8(send);
  }
  float a4[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const float send = h4 ? a8[k] : a8[2 + k];
    a4[k] = (h4 ? a8[2 + k] : a8[k]) + lane_mirror8(send);
  }
  const float send2 = h2 ? a4[0] : a4[1];
  float a2 = (h2 ? a4[1] : a4[0]) + lane_xor2(send2);
  a2 += lane_xor1(a2);
  const int v = (h8 ? 4 : 0) + (h4 ? 2 : 0) + (h2 ? 1 : 0);
  if (!(n & 1)) dst[16 * (v >> 2) + 4 * gq + (v & 3)] = a2;
}

// ---- resident variant: the raw score accumulators stay exactly as the MFMA
// produced them (unscaled, unmasked), which lets the compiler keep them in
// accumulation registers; the scale and the causal / chunk-end mask are
// applied where the scores are used.  vis[rt] is the last token visible to
// the lane's row of tile rt (-1 for padding rows); element (tt, i) of a block
// starting at token tb is token tb + 16 tt + 4 gq + i.
// The workgroup's Q tile in LDS for the resident variant: ROWS rows of D/8
// 16-byte chunks, chunk c of row r stored at position c ^ (r mod D/8) of the
// row (an XOR swizzle: the 16 rows a B-operand read touches then fall on
// distinct banks).  It is loaded straight into LDS (global_load_lds, no
// registers), one 64-chunk run per instruction; padding rows repeat the last
// real row (their scores are masked).
template <int D, int RT>
__device__ __forceinline__ void issue_q_lds(const VArgs& a, const Unit& u, uint16_t* s_q, int w,
                                            int lane) {
  constexpr int CH = D / 8;
  constexpr int NI = RT * 16 * CH / 64;  // instructions per workgroup
  const uint16_t* q = static_cast<const uint16_t*>(a.q);
#pragma unroll
  for (int k = 0; k < (NI + kWaves - 1) / kWaves; ++k) {
    const int ins = w + kWaves * k;
    if (ins < NI) {
      const int slot = ins * 64 + lane, r = slot / CH, c = (slot % CH) ^ (r % CH);
      const int row = min(u.rg * a.RT * 16 + r, a.R - 1);
      const int t = row / a.G, h = u.g * a.G + row % a.G;
      const uint16_t* src = q + (((size_t)u.b * a.T + t) * a.Hq + h) * D + 8 * c;
      const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_addr(s_q + ins * 64 * 8));
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                   :
                   : "s"(lds), "v"(src)
                   : "memory", "m0");
    }
  }
}

template <int D, int RT>
__device__ __forceinline__ bf16x8 q_operand(const uint16_t* s_q, int rt, int ks, int n, int gq) {
  constexpr int CH = D / 8;
  const int r = rt * 16 + n, c = 4 * ks + gq;
  return __builtin_bit_cast(
      bf16x8, *reinterpret_cast<const uint4*>(s_q + (r * CH + (c ^ (r % CH))) * 8));
}

// Scaled (log2 domain; unscaled with SCALED false), masked scores of one
// block for the two-pass variants (qop(rt, ks): the Q operand of tile rt,
// k-step ks): -inf past the chunk,
// past the causal limit of each verify row (lim: the last token the lane's
// row of each tile sees, -1 on padding rows), and on padding rows.  A block
// every real row sees whole is only scaled: its padding rows keep finite
// scores, whose log-sum-exp the statistics set to +inf, so their
// probabilities are 0.
template <int D, int RT, bool SCALED = true, typename QOp>
__device__ __forceinline__ void scores_from(const VArgs& a, const Unit& u, const uint4 (&Kr)[2][D / 32],
                                            QOp qop, int tb, int gq, const int (&lim)[RT],
                                            float (&S)[2][RT][4]) {
  const float sc = SCALED ? a.sl2 : 1.f;
  const bool full = tb + 31 <= min(u.c1 - 1, u.ctx);  // row 0 sees the least
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
    floatx4 acc[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[rt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const bf16x8 kk = __builtin_bit_cast(bf16x8, Kr[tt][ks]);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qop(rt, ks), acc[rt], 0, 0, 0);
    }
    if (full) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) S[tt][rt][i] = SCALED ? acc[rt][i] * sc : acc[rt][i];
    } else {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = tb + 16 * tt + 4 * gq + i;
          S[tt][rt][i] = tok <= lim[rt] ? (SCALED ? acc[rt][i] * sc : acc[rt][i]) : kNegInf;
        }
    }
  }
}

// ... with the Q operands read from the workgroup's LDS tile (stream variant).
template <int D, int RT>
__device__ __forceinline__ void scores_block(const VArgs& a, const Unit& u, const uint4 (&Kr)[2][D / 32],
                                             const uint16_t* s_q, int tb, int n, int gq,
                                             const int (&lim)[RT], float (&S)[2][RT][4]) {
  scores_from<D, RT>(a, u, Kr, [&](int rt, int ks) { return q_operand<D, RT>(s_q, rt, ks, n, gq); }, tb,
                     gq, lim, S);
}

template <int D, int RT>
__device__ __forceinline__ void scores_raw(const uint4 (&Kr)[2][D / 32], const uint16_t* s_q, int n,
                                           int gq, floatx4 (&S)[2][RT]) {
#pragma unroll
  for (int tt = 0; tt < 2; ++tt) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) S[tt][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const bf16x8 kk = __builtin_bit_cast(bf16x8, Kr[tt][ks]);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        S[tt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, q_operand<D, RT>(s_q, rt, ks, n, gq),
                                                            S[tt][rt], 0, 0, 0);
    }
  }
}

// Masks a block's raw scores in place: -inf past the chunk, past the causal
// limit of each verify row, and on padding rows (vis = -1).  Only blocks
// that some real row does not see whole need it; every other block skips it,
// which keeps the per-score work of the maximum and the probabilities free of
// compares.  Padding rows of unmasked blocks keep finite values, which only
// reach their own statistics (their factor c is 0 wherever it is used).
template <int RT>
__device__ __forceinline__ void mask_block(floatx4 (&S)[2][RT], const int (&vis)[RT], int tb, int gq) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int off = vis[rt] - tb - 4 * gq;  // element (tt, i) visible iff 16 tt + i <= off
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (16 * tt + i > off) S[tt][rt][i] = kNegInf;
  }
}

// Per-lane maximum of one block's (masked) raw scores, per row tile.
template <int RT>
__device__ __forceinline__ void block_max_raw(const floatx4 (&S)[2][RT], float (&mx)[RT]) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
      mx[rt] = fmaxf(fmaxf(mx[rt], fmaxf(S[tt][rt][0], S[tt][rt][1])), fmaxf(S[tt][rt][2], S[tt][rt][3]));
}

// Raw scores -> probabilities relative to the workgroup's row maxima,
// P = exp2(scale * s - ref), in place (masked scores are -inf and the scale
// is positive, so they give 0); per-lane row sums.
template <int RT>
__device__ __forceinline__ void block_probs(floatx4 (&S)[2][RT], float sl2, const float (&ref)[RT],
                                            float (&z)[RT]) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = fast_exp2(fmaf(S[tt][rt][i], sl2, -ref[rt]));
        S[tt][rt][i] = p;
        z[rt] += p;
      }
}

// One resident block with the global statistics known: exact probabilities
// p = P * c (P relative to the workgroup's row maximum ref, c = exp2(ref -
// lse) per row), their sum over the block's rows (the workgroup's share of
// each token's mass, written to mp when mp is set) and O += p.V on MFMA (p
// converted to bf16).
template <int D, int RT>
__device__ __forceinline__ void pv_exact_resident(const floatx4 (&P)[2][RT], const float (&c)[RT],
                                                  const typename VVec<D>::T (&Vr)[8],
                                                  floatx4 (&O)[RT][D / 16], float* mp, int tb, int c1,
                                                  int n, int gq) {
  constexpr int DPL = D / 16;
  float pm[8];
#pragma unroll
  for (int v = 0; v < 8; ++v) pm[v] = 0.f;
  bf16x8 Pa[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = P[tt][rt][i] * c[rt];
        pm[4 * tt + i] += p;
        Pa[rt][4 * tt + i] = static_cast<__bf16>(p);
      }
  if (mp) mass_reduce_store(pm, mp, tb, c1, n, gq);
#pragma unroll
  for (int jd = 0; jd < DPL; ++jd) {
    const bf16x8 vb = pack_v(Vr, jd);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
      O[rt][jd] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Pa[rt], vb, O[rt][jd], 0, 0, 0);
  }
}

// P = exp2(S - lse2) of one block: the MFMA A operands (bf16) and each
// lane's per-token sums over its rows.
template <int RT>
__device__ __forceinline__ void probs_block(const float (&S)[2][RT][4], const float (&lse)[RT],
                                            bf16x8 (&Pa)[RT], float (&pm)[8]) {
#pragma unroll
  for (int v = 0; v < 8; ++v) pm[v] = 0.f;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = fast_exp2(S[tt][rt][i] - lse[rt]);
        pm[4 * tt + i] += p;
        Pa[rt][4 * tt + i] = static_cast<__bf16>(p);
      }
  }
}

// O += P.V of one block on MFMA.
template <int D, int RT>
__device__ __forceinline__ void pv_mfma(const bf16x8 (&Pa)[RT], const typename VVec<D>::T (&Vr)[8],
                                        floatx4 (&O)[RT][D / 16]) {
  constexpr int DPL = D / 16;
#pragma unroll
  for (int jd = 0; jd < DPL; ++jd) {
    const bf16x8 vb = pack_v(Vr, jd);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
      O[rt][jd] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Pa[rt], vb, O[rt][jd], 0, 0, 0);
  }
}

// P = exp2(S - lse2): per-token mass (sum over the block's rows, written to
// mp) and O += P.V on MFMA.
template <int D, int RT>
__device__ __forceinline__ void pv_block(const float (&S)[2][RT][4], const float (&lse)[RT],
                                         const typename VVec<D>::T (&Vr)[8], floatx4 (&O)[RT][D / 16],
                                         float* mp, int tb, int c1, int n, int gq) {
  bf16x8 Pa[RT];
  float pm[8];
  probs_block<RT>(S, lse, Pa, pm);
  mass_reduce_store(pm, mp, tb, c1, n, gq);
  pv_mfma<D, RT>(Pa, Vr, O);
}

// Sum the four waves' O fragments and write the chunk partial (row-major
// [ROWS][D], bf16) to the workspace.  Reduce-scatter through LDS: the MFMA
// tiles of O form units of four tiles (one 16-row tile, four consecutive d per
// lane); unit k belongs to wave k % 4.  Every wave parks the units it does not
// own, one barrier, then each owner adds the three parked copies to its own
// and stores the sum (8 bytes per lane and row) straight from registers.
template <int D, int RT, bool LOCAL>
__device__ __forceinline__ void write_opart(const VArgs& a, const Unit& u, floatx4 (&O)[RT][D / 16],
                                            float* s_o, int lane, int w, int n, int gq) {
  constexpr int DPL = D / 16;
  constexpr int FU = 4;          // tiles per unit
  constexpr int HU = DPL / FU;   // units per 16-row tile
  constexpr int U = RT * HU;
  static_assert(DPL % FU == 0, "head dim must be a multiple of 64");
  floatx4* buf = reinterpret_cast<floatx4*>(s_o);
  const int wu = __builtin_amdgcn_readfirstlane(w);
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int own = k % kWaves;
    if (own != wu) {
      const int s = (wu - own + kWaves) % kWaves - 1;  // 0..2
      floatx4* dst = buf + (k * 3 + s) * FU * 64 + lane;
#pragma unroll
      for (int j = 0; j < FU; ++j) dst[j * 64] = O[k / HU][(k % HU) * FU + j];
    }
  }
  lds_sync();
  uint64_t* op = reinterpret_cast<uint64_t*>(a.opart) + ((size_t)u.grp * a.splits + u.split) * RT * 16 * D / 4;
#pragma unroll
  for (int k = 0; k < U; ++k) {
    if (k % kWaves == wu) {
      const int rt = k / HU, h = k % HU;
      floatx4 t[3][FU];
#pragma unroll
      for (int s = 0; s < 3; ++s)
#pragma unroll
        for (int j = 0; j < FU; ++j) t[s][j] = buf[(k * 3 + s) * FU * 64 + j * 64 + lane];
      floatx4 acc[FU];
#pragma unroll
      for (int j = 0; j < FU; ++j) acc[j] = O[rt][h * FU + j] + t[0][j] + t[1][j] + t[2][j];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = rt * 16 + 4 * gq + i;
        x_store<LOCAL>(op + (row * D + DPL * n + FU * h) / 4,
                       pack_bf16x4(acc[0][i], acc[1][i], acc[2][i], acc[3][i]));
      }
    }
  }
}

// Resident variant, after the chunk partial of O (already normalised by the
// rows' global statistics) and the mass partials are published and the
// workgroup has arrived at cnt_o (thread 0 holds the value the arrival
// returned): arrive at the chunk's mass counter (the chunk's last arrival
// sums the mass over KV heads while its group's O partials land), wait for
// the group's O partials, and write this workgroup's slice of O (the plain
// sum over chunks) and the lse.
template <int D, int RT, bool LOCAL>
__device__ void verify_epilogue_resident(const VArgs& a, const Unit& u, const float* s_lse, float* s_acc,
                                         int* s_flag, unsigned base, unsigned old) {
  constexpr int ROWS = RT * 16;
  constexpr int kU = 16;
  const int tid = threadIdx.x;
  const int nsp = (u.N + a.chunk - 1) / a.chunk;
  if (tid == 0) {
    const int mold =
        a.mass ? __hip_atomic_fetch_add(mass_counter(a, u), 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0;
    *s_flag = a.mass && mold == a.Hkv * a.RG - 1;
  }
  __syncthreads();
  if (*s_flag) mass_sum(a, u);
  if (tid == 0) o_finish(a, u, base, old, true);
  __syncthreads();
  // This workgroup's slice of O is the sum over chunks of the partials.  With
  // few elements per workgroup the chunks are split over Q thread sets whose
  // sums meet in LDS.
  const int row0 = u.rg * a.RT * 16;
  const int rows = min(ROWS, a.R - row0);
  const int E4 = rows * D / 4;
  const int per = (E4 + nsp - 1) / nsp;
  const int e0 = min(E4, u.split * per), e1 = min(E4, e0 + per);
  const int cnt = e1 - e0;
  const int Q = cnt <= 0 ? 1 : min(kOSets, max(1, kThreads / cnt));
  const int q = cnt <= 0 ? 0 : tid / cnt, el = cnt <= 0 ? 0 : tid % cnt;
  const bool act = cnt > 0 && q < Q;  // first element e0 + el (Q = 1: el = tid)
  const uint64_t* op = reinterpret_cast<const uint64_t*>(a.opart) + (size_t)u.grp * a.splits * ROWS * D / 4;
  auto sum_parts = [&](int e, int s0, int Qs, float (&acc)[4]) {
    // unconditional (clamped) loads keep the wait counts fine-grained
    uint64_t v[kU];
#pragma unroll
    for (int j = 0; j < kU; ++j)
      v[j] = x_load<LOCAL>(op + (size_t)min(s0 + j * Qs, nsp - 1) * ROWS * D / 4 + e);
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const float f = s0 + j * Qs < nsp ? 1.f : 0.f;
#pragma unroll
      for (int h = 0; h < 4; ++h) acc[h] = fmaf(f, bf16_to_f32((uint16_t)(v[j] >> (16 * h))), acc[h]);
    }
  };
  auto emit = [&](int e, const float (&acc)[4]) {
    const int r = (4 * e) / D;
    const int row = row0 + r, d = (4 * e) % D;
    const int t = row / a.G, h = u.g * a.G + row % a.G;
    const size_t oi = (((size_t)u.b * a.T + t) * a.Hq + h) * D + d;
    *reinterpret_cast<uint64_t*>(static_cast<uint16_t*>(a.out) + oi) =
        pack_bf16x4(acc[0], acc[1], acc[2], acc[3]);
  };
  if (act) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = q; s0 < nsp; s0 += Q * kU) sum_parts(e0 + el, s0, Q, acc);
    if (Q == 1)
      emit(e0 + el, acc);
    else
      reinterpret_cast<float4*>(s_acc)[q * cnt + el] = make_float4(acc[0], acc[1], acc[2], acc[3]);
  }
  if (Q == 1) {
    for (int e = e0 + tid + kThreads; e < e1; e += kThreads) {
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      for (int s0 = 0; s0 < nsp; s0 += kU) sum_parts(e, s0, 1, acc);
      emit(e, acc);
    }
  } else {
    lds_sync();
    if (tid < cnt) {
      const float4* sa = reinterpret_cast<const float4*>(s_acc);
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      for (int qq = 0; qq < Q; ++qq) {
        const float4 v = sa[qq * cnt + tid];
        acc[0] += v.x;
        acc[1] += v.y;
        acc[2] += v.z;
        acc[3] += v.w;
      }
      emit(e0 + tid, acc);
    }
  }
  if (a.lse && u.split == 0) {
    for (int r = tid; r < rows; r += kThreads) {
      const int row = row0 + r, t = row / a.G, h = u.g * a.G + row % a.G;
      a.lse[((size_t)u.b * a.Hq + h) * a.T + t] = s_lse[r] * kLn2;
    }
  }
}

// A chunk past this sequence's end: publish empty statistics, arrive at both
// counters without waiting (advancing the base if last), join the mass sum.
template <int ROWS, bool LOCAL>
__device__ void empty_chunk(const VArgs& a, const Unit& u, const float* s_m, const float* s_z,
                            unsigned base, int* s_flag) {
  stats_store<ROWS, LOCAL>(a, u, s_m, s_z, base);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    stats_arrive(a, u, base, false);
    __builtin_amdgcn_s_waitcnt(0);  // the statistics arrival lands before the O arrival
    o_finish(a, u, base, grp_arrive(cnt_o(a, u)), false);
  }
  __syncthreads();
  mass_combine(a, u, s_flag);
}

// This (batch, KV head)'s K and V rows: a padded cache's base, or the pool
// through the page table, the chunk's page entries checked against the pool,
// clamped into it and staged in LDS when they fit (every thread takes part).
template <int D>
__device__ __forceinline__ void kv_rows_setup(const VArgs& a, const Unit& u, int32_t* s_pages, KvRows& kg,
                                              KvRows& vg) {
  if (a.table) {
    const size_t hoff = ((size_t)u.g << a.page_shift) * D;
    const int32_t* tab = a.table + (size_t)u.b * a.max_pages;
    const int64_t pe = ((int64_t)a.Hkv << a.page_shift) * D;
    // The chunk's page entries, checked against the pool, clamped into it
    // and staged in LDS when they fit.
    const int p0 = u.c0 >> a.page_shift, p1 = (u.c1 - 1) >> a.page_shift;
    const bool fit = p1 - p0 < kPageSlots;
    for (int pg = p0 + threadIdx.x; pg <= p1; pg += kThreads) {
      int e = tab[pg];
      if (e < 0 || e >= a.n_pages) {
        dev_flag(a.status, PVLM_DEV_RANGE);
        e = e < 0 ? 0 : (int)(a.n_pages - 1);
      }
      if (fit) s_pages[pg - p0] = e;
    }
    __syncthreads();
    kg = {static_cast<const uint16_t*>(a.k) + hoff, tab, s_pages, pe, a.n_pages, a.page_shift, p0,
          true, fit};
    vg = {static_cast<const uint16_t*>(a.v) + hoff, tab, s_pages, pe, a.n_pages, a.page_shift, p0,
          true, fit};
  } else {
    const size_t kv_off = ((size_t)u.b * a.Hkv + u.g) * a.n_cap * D;
    kg = {static_cast<const uint16_t*>(a.k) + kv_off, a.ctx_len, s_pages, 0, 1, 5, 0, false, false};
    vg = {static_cast<const uint16_t*>(a.v) + kv_off, a.ctx_len, s_pages, 0, 1, 5, 0, false, false};
  }
}

template <int D, int RT, bool RESIDENT, bool LOCAL>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
verify_mfma_kernel(VArgs a) {
  constexpr int ROWS = RT * 16;
  constexpr int KS = D / 32;
  constexpr int DPL = D / 16;
  typedef typename VVec<D>::T VT;
  __shared__ float s_wm[kWaves][ROWS], s_wz[kWaves][ROWS];
  __shared__ float s_m[ROWS], s_z[ROWS], s_lse[ROWS];
  __shared__ int s_flag;
  __shared__ int32_t s_pages[kPageSlots];  // paged caches: the chunk's pool pages
  extern __shared__ __align__(256) float s_o[];  // 16-byte LDS accesses need 16-byte alignment

  Unit u;
  if (!decode_unit(a, u)) return;
  const unsigned base = read_base(a, u);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 15, gq = lane >> 4;
  if (u.c0 >= u.N) {  // chunk past this sequence's end: empty statistics, no wait
    for (int r = threadIdx.x; r < ROWS; r += kThreads) {
      s_m[r] = kNegInf;
      s_z[r] = 0.f;
    }
    __syncthreads();
    empty_chunk<ROWS, LOCAL>(a, u, s_m, s_z, base, &s_flag);
    return;
  }
  KvRows kg, vg;  // this (batch, KV head)'s K and V rows
  kv_rows_setup<D>(a, u, s_pages, kg, vg);
  float* mp = a.mpart + ((size_t)u.b * a.Hkv * a.RG + u.g * a.RG + u.rg) * a.n_cap;

  float m[RT], z[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    m[rt] = kNegInf;
    z[rt] = 0.f;
  }
  floatx4 O[RT][DPL];
  if constexpr (RESIDENT) {
    // ---- pass 1: all K blocks of this wave in flight (registers), then the
    //      whole chunk's V streamed into LDS by waves 1-3 (wave 0 keeps no
    //      loads in flight so it can publish the statistics without waiting
    //      for them); scores kept resident.
    uint16_t* s_v = reinterpret_cast<uint16_t*>(s_o);
    uint16_t* s_q = s_v + kResTokens * D;  // after the V region
    floatx4 S[kNB][2][RT];
    uint4 Kr[kNB][2][KS];
    int vis[RT];  // last token visible to this lane's row of each tile (-1: padding row)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int row = u.rg * a.RT * 16 + rt * 16 + n;
      vis[rt] = row < a.R ? min(u.c1 - 1, u.ctx + row / a.G) : -1;
    }
    // issue order: Q (into LDS), K block 0, 1, ... (the scheduler would
    // otherwise reorder the loads), then, once Q has landed, the chunk's V
    // into LDS from waves 1-3, so HBM streams K and V back to back; wave 0
    // keeps only K in flight so it can publish the statistics without waiting
    // for V.
    issue_q_lds<D, RT>(a, u, s_q, w, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < kNB; ++j) {
      load_k_block<D, true>(kg, u.c0 + 32 * (w + kWaves * j), u.c1, n, gq, Kr[j]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // this wave's Q chunks have landed once at most the 8 * KS K loads issued
    // after them are outstanding; then every wave's (barrier), then V behind K
    static_assert(kNB * 2 * KS == 32 || kNB * 2 * KS == 16, "the wait below counts the K loads");
    if constexpr (kNB * 2 * KS == 32)
      asm volatile("s_waitcnt vmcnt(32)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
    lds_sync();
    __builtin_amdgcn_sched_barrier(0);
    const int nblk = (u.c1 - u.c0 + 31) / 32;
    if (w > 0)
      for (int blk = w - 1; blk < nblk; blk += kWaves - 1)
        issue_v_lds<D, true>(vg, u.c0 + 32 * blk, u.c1, s_v + blk * 32 * D, lane);
    // a block every real row sees whole needs no mask (row 0 sees the least)
    const int vis_all = min(u.c1 - 1, u.ctx);
#pragma unroll
    for (int j = 0; j < kNB; ++j) {
      const int tb = u.c0 + 32 * (w + kWaves * j);
      if (tb < u.c1) {
        scores_raw<D, RT>(Kr[j], s_q, n, gq, S[j]);
        if (tb + 31 > vis_all) mask_block<RT>(S[j], vis, tb, gq);
        block_max_raw<RT>(S[j], m);
      }
    }
    // the workgroup's row maxima (log2 domain), then the resident scores
    // become probabilities relative to them, one exp2 per score
    reduce_rows<RT, true>(m, n, gq, w, s_wm, s_m, a.sl2);
    float ref[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const float mm = s_m[rt * 16 + n];
      ref[rt] = mm == kNegInf ? 0.f : mm;  // rows with no visible token: P = 0 anyway
    }
#pragma unroll
    for (int j = 0; j < kNB; ++j) {
      const int tb = u.c0 + 32 * (w + kWaves * j);
      if (tb < u.c1) block_probs<RT>(S[j], a.sl2, ref, z);
    }
    reduce_rows<RT, false>(z, n, gq, w, s_wz, s_z, 1.f);
    // publish the statistics (wave 0, which loads no V) and arrive as soon
    // as they are stored
    // ---- the group's statistics (published right after each workgroup's
    //      pass 1): every row's global log2-sum-exp, so P becomes exact.
    //      Thread 0 polls while waves 1-3 still wait for their V; their loads
    //      of the records queue behind their V loads (in-order completion).
    stats_store<ROWS, LOCAL>(a, u, s_m, s_z, base);
    if (__builtin_amdgcn_readfirstlane(w) == 0) {
      __builtin_amdgcn_s_waitcnt(0);
      if (lane == 0) stats_arrive(a, u, base, true);
    }
    lds_sync();
    stats_combine<ROWS, LOCAL>(a, u, (u.N + a.chunk - 1) / a.chunk, s_lse, s_wm, s_wz, base);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's V loads are done
    __syncthreads();                // ... and every other wave's
    float c[RT];  // exp2(ref - lse): 0 for padding rows and rows with no visible token here
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const float mm = s_m[rt * 16 + n];
      c[rt] = vis[rt] < 0 || mm == kNegInf ? 0.f : fast_exp2(ref[rt] - s_lse[rt * 16 + n]);
    }
    // ---- pass 2: exact P, the mass partials and P.V on MFMA
    float* mp = a.mass ? a.mpart + ((size_t)u.b * a.Hkv * a.RG + u.g * a.RG + u.rg) * a.n_cap : nullptr;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int jd = 0; jd < DPL; ++jd) O[rt][jd] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < kNB; ++j) {
      const int blk = w + kWaves * j;
      const int tb = u.c0 + 32 * blk;
      if (tb < u.c1) {
        VT Vr[8];
        read_v_lds<D>(s_v + blk * 32 * D, n, gq, Vr);
        pv_exact_resident<D, RT>(S[j], c, Vr, O, mp, tb, u.c1, n, gq);
      }
    }
    __syncthreads();  // V region of LDS is reused below
    write_opart<D, RT, LOCAL>(a, u, O, s_o, lane, w, n, gq);
    __builtin_amdgcn_s_waitcnt(0);  // every wave's O and mass partial stores are complete
    __syncthreads();                // (s_o is reused for the O-slice sums)
    unsigned old = 0;
    if (threadIdx.x == 0) old = grp_arrive(cnt_o(a, u));
    verify_epilogue_resident<D, RT, LOCAL>(a, u, s_lse, s_o, &s_flag, base, old);
    return;
  } else {
    // the Q tile in LDS (the region is reused for the O partials at the end)
    uint16_t* s_q = reinterpret_cast<uint16_t*>(s_o);
    issue_q_lds<D, RT>(a, u, s_q, w, lane);
    __builtin_amdgcn_s_waitcnt(0);
    lds_sync();
    // ---- pass 1: stream K, running statistics only.  Software-pipelined:
    //      the loads of the wave's next two blocks are in flight while the
    //      current two are scored (loads past the chunk are clamped, their
    //      scores masked, so every load is unconditional).
    const int nblk = (u.c1 - u.c0 + 31) / 32;
    int lim[RT];  // last token the lane's row of each tile sees (-1: padding row)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int row = u.rg * a.RT * 16 + rt * 16 + n;
      lim[rt] = row < a.R ? min(u.c1 - 1, u.ctx + row / a.G) : -1;
    }
    auto score_pair = [&](const uint4 (&K2)[2][2][KS], int blk0) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int blk = blk0 + h * kWaves;
        if (blk < nblk) {
          float S[2][RT][4];
          scores_block<D, RT>(a, u, K2[h], s_q, u.c0 + 32 * blk, n, gq, lim, S);
          running_stats<RT>(S, m, z);
        }
      }
    };
    auto load_pair = [&](uint4 (&K2)[2][2][KS], int blk0) {
#pragma unroll
      for (int h = 0; h < 2; ++h) load_k_block<D>(kg, u.c0 + 32 * (blk0 + h * kWaves), u.c1, n, gq, K2[h]);
    };
    {
      uint4 Ka[2][2][KS], Kb[2][2][KS];
      load_pair(Ka, w);
      for (int blk = w; blk < nblk; blk += 4 * kWaves) {
        load_pair(Kb, blk + 2 * kWaves);
        score_pair(Ka, blk);
        if (blk + 2 * kWaves >= nblk) break;
        load_pair(Ka, blk + 4 * kWaves);
        score_pair(Kb, blk + 2 * kWaves);
      }
    }
    reduce_stats<RT>(m, z, n, gq, w, s_wm, s_wz, s_m, s_z);
    exchange_stats<ROWS, LOCAL>(a, u, s_m, s_z, s_lse, s_wm, s_wz, base, true);
    float lse[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) lse[rt] = s_lse[rt * 16 + n];
    // ---- pass 2: recompute scores from K, then P, mass and P.V, the next
    //      block's K and V loading during this one (in registers up to 3 row
    //      tiles; with more, in LDS).  This is the rows' last read, so its
    //      loads are non-temporal; pass 1's are not, because its K stays
    //      cached for this re-read.
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int jd = 0; jd < DPL; ++jd) O[rt][jd] = floatx4{0.f, 0.f, 0.f, 0.f};
    auto step = [&](const uint4 (&Kr)[2][KS], const VT (&Vr)[8], int blk) {
      const int tb = u.c0 + 32 * blk;
      float S[2][RT][4];
      scores_block<D, RT>(a, u, Kr, s_q, tb, n, gq, lim, S);
      pv_block<D, RT>(S, lse, Vr, O, mp, tb, u.c1, n, gq);
    };
    if constexpr (RT <= 3) {
      uint4 Ka[2][KS], Kb[2][KS];
      VT Va[8], Vb[8];
      load_k_block<D, true>(kg, u.c0 + 32 * w, u.c1, n, gq, Ka);
      load_v_block<D, true>(vg, u.c0 + 32 * w, u.c1, n, gq, Va);
      for (int blk = w; blk < nblk; blk += 2 * kWaves) {
        const int b2 = blk + kWaves;
        load_k_block<D, true>(kg, u.c0 + 32 * b2, u.c1, n, gq, Kb);
        load_v_block<D, true>(vg, u.c0 + 32 * b2, u.c1, n, gq, Vb);
        step(Ka, Va, blk);
        if (b2 >= nblk) break;
        load_k_block<D, true>(kg, u.c0 + 32 * (b2 + kWaves), u.c1, n, gq, Ka);
        load_v_block<D, true>(vg, u.c0 + 32 * (b2 + kWaves), u.c1, n, gq, Va);
        step(Kb, Vb, b2);
      }
    } else {
      // No registers for a second block: each wave double-buffers its K and
      // V blocks in LDS (after the Q tile) through untracked global->LDS
      // loads, the next block's in flight while this one is computed.  The
      // waits are counted by hand: younger than a block's loads are the
      // previous block's mass store (one per block, always issued: lane 0
      // holds the block's first token) and the next block's loads.
      uint16_t* kv = s_q + RT * 16 * D + w * 4 * 32 * D;  // [2 buffers][K, V][32][D]
      __builtin_amdgcn_s_waitcnt(0);                       // the counts below start from zero
      if (w < nblk) {
        issue_k_lds<D, true>(kg, u.c0 + 32 * w, u.c1, kv, lane);
        issue_v_lds<D, true>(vg, u.c0 + 32 * w, u.c1, kv + 32 * D, lane);
      }
      int i = 0;
      for (int blk = w; blk < nblk; blk += kWaves, ++i) {
        uint16_t* cur = kv + (i & 1) * 2 * 32 * D;
        const bool next = blk + kWaves < nblk;
        if (next) {
          uint16_t* nxt = kv + ((i + 1) & 1) * 2 * 32 * D;
          issue_k_lds<D, true>(kg, u.c0 + 32 * (blk + kWaves), u.c1, nxt, lane);
          issue_v_lds<D, true>(vg, u.c0 + 32 * (blk + kWaves), u.c1, nxt + 32 * D, lane);
        }
        wait_vm_younger<D>((i > 0 ? 1 : 0) + (next ? kBlockDma<D> : 0));
        uint4 Kr[2][KS];
        read_k_lds<D>(cur, n, gq, Kr);
        VT Vr[8];
        read_v_lds<D>(cur + 32 * D, n, gq, Vr);
        step(Kr, Vr, blk);
      }
    }
  }
  lds_sync();  // every wave is done with the Q tile, whose LDS the partials reuse
  write_opart<D, RT, LOCAL>(a, u, O, s_o, lane, w, n, gq);
  verify_epilogue<ROWS, D, LOCAL>(a, u, s_lse, false, &s_flag, base);
}

// ------------------------------------------------------- wide variant --
// Long chunks with more row tiles than one wave's accumulators hold (6 .. 9
// tiles, e.g. 136 verify rows per KV head).  One workgroup holds every row,
// so each cache row is read once per pass for all of them instead of once
// per row group.  Waves 0-2 own three row tiles each (Q operands in
// registers, O accumulators over the whole head dimension) and score every
// token of the chunk; wave 3 streams the blocks into a ring of LDS slots that
// the three read: K in pass 1, K and V in pass 2.  One workgroup barrier per
// block hands a landed slot to the compute waves and the slot they finished
// back to the loader.  The loader issues no other vector memory operation in
// its loops, so its waits count its own global->LDS loads (which complete in
// issue order).  Scores stay unscaled; the scale goes into the exponent
// (one fused multiply-add per score).
constexpr int kWideRT = 9;      // row tiles per workgroup
constexpr int kWideTW = 3;      // row tiles per compute wave (waves 0 .. 2)
constexpr int kWideSlots1 = 8;  // pass-1 ring: one K block per slot
constexpr int kWideSlots2 = 4;  // pass-2 ring: a K and a V block per slot
// Two workgroups per CU (registers and LDS allow it), so that on every SIMD
// one workgroup's MFMA and exponentials overlap the other's barrier waits
// (one per budgeted CU on a stream with a compute-unit budget).
constexpr int kWidePerCU = 2;
static_assert(kWideRT == kWideTW * (kWaves - 1), "waves 0..2 compute, wave 3 loads");

// Wait until at most `younger` groups of PER loads are outstanding (younger
// in [0, K], wave-uniform; any other value waits for all).
template <int PER, int K>
__device__ __forceinline__ void wait_vm_groups(int younger) {
  static_assert(K * PER < 64, "vmcnt holds 6 bits");
  if constexpr (K == 0) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  } else {
    if (younger == K)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(K * PER) : "memory");
    else
      wait_vm_groups<PER, K - 1>(younger);
  }
}

// running_stats for unscaled scores: the row maximum in the scaled (log2)
// domain, exp2(s * sl2 - M) as one fused multiply-add and an exponential.
template <int RT>
__device__ __forceinline__ void running_stats_raw(const float (&S)[2][RT][4], float sl2, float (&m)[RT],
                                                  float (&z)[RT]) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float mx = kNegInf;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, S[tt][rt][i]);
    const float M = fmaxf(m[rt], mx * sl2);
    if (M != kNegInf) {
      float acc = z[rt] * fast_exp2(m[rt] - M);
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc += fast_exp2(fmaf(S[tt][rt][i], sl2, -M));
      z[rt] = acc;
      m[rt] = M;
    }
  }
}

// probs_block for unscaled scores: p = exp2(s * sl2 - lse2).
template <int RT>
__device__ __forceinline__ void probs_raw(const float (&S)[2][RT][4], float sl2, const float (&lse)[RT],
                                          bf16x8 (&Pa)[RT], float (&pm)[8]) {
#pragma unroll
  for (int v = 0; v < 8; ++v) pm[v] = 0.f;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = fast_exp2(fmaf(S[tt][rt][i], sl2, -lse[rt]));
        pm[4 * tt + i] += p;
        Pa[rt][4 * tt + i] = static_cast<__bf16>(p);
      }
}

// A compute wave's chunk partial of O (its three row tiles, whole head
// dimension; bf16, row-major [ROWS][D]): no reduction across waves.
template <int D, bool LOCAL>
__device__ __forceinline__ void write_opart_wide(const VArgs& a, const Unit& u,
                                                 const floatx4 (&O)[kWideTW][D / 16], int t0, int n, int gq) {
  constexpr int DPL = D / 16, ROWS = kWideRT * 16;
  uint64_t* op = reinterpret_cast<uint64_t*>(a.opart) + ((size_t)u.grp * a.splits + u.split) * ROWS * D / 4;
#pragma unroll
  for (int t = 0; t < kWideTW; ++t)
#pragma unroll
    for (int h = 0; h < DPL / 4; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = (t0 + t) * 16 + 4 * gq + i;
        x_store<LOCAL>(op + (row * D + DPL * n + 4 * h) / 4,
                       pack_bf16x4(O[t][4 * h][i], O[t][4 * h + 1][i], O[t][4 * h + 2][i], O[t][4 * h + 3][i]));
      }
}

template <int D, bool LOCAL>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kWidePerCU, kWidePerCU)))
verify_wide_kernel(VArgs a) {
  constexpr int RT = kWideRT, TW = kWideTW, ROWS = RT * 16, KS = D / 32, DPL = D / 16;
  constexpr int BLK = 32 * D;              // bf16 elements of one 32-token K or V block
  constexpr int KDMA = 32 * (D / 8) / 64;  // global->LDS loads per K (or V) block
  constexpr int S1 = kWideSlots1, S2 = kWideSlots2;
  typedef typename VVec<D>::T VT;
  __shared__ float s_wm[kWaves][ROWS], s_wz[kWaves][ROWS];
  __shared__ float s_m[ROWS], s_z[ROWS], s_lse[ROWS];
  __shared__ float s_mass[2][TW][32];  // per-token sums of a block over each compute wave's rows
  __shared__ int s_flag;
  __shared__ int32_t s_pages[kPageSlots];
  extern __shared__ __align__(256) float s_o[];

  Unit u;
  if (!decode_unit(a, u)) return;
  const unsigned base = read_base(a, u);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = lane & 15, gq = lane >> 4;
  if (u.c0 >= u.N) {  // chunk past this sequence's end: empty statistics, no wait
    for (int r = threadIdx.x; r < ROWS; r += kThreads) {
      s_m[r] = kNegInf;
      s_z[r] = 0.f;
    }
    __syncthreads();
    empty_chunk<ROWS, LOCAL>(a, u, s_m, s_z, base, &s_flag);
    return;
  }
  KvRows kg, vg;
  kv_rows_setup<D>(a, u, s_pages, kg, vg);
  float* mp = a.mpart + ((size_t)u.b * a.Hkv * a.RG + u.g * a.RG + u.rg) * a.n_cap;
  uint16_t* ring = reinterpret_cast<uint16_t*>(s_o);
  const bool loader = __builtin_amdgcn_readfirstlane(w) == kWaves - 1;
  const int nblk = (u.c1 - u.c0 + 31) / 32;
  const float sl2 = a.sl2;

  // The Q tile through LDS into each compute wave's operand registers (the
  // loader's copy is unused); the ring then reuses that LDS.
  issue_q_lds<D, RT>(a, u, ring, w, lane);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  lds_sync();
  const int t0 = loader ? 0 : w * TW;  // first row tile of this wave
  bf16x8 Qr[TW][KS];
  int lim[TW];  // last token the lane's row of each tile sees (-1: padding row)
#pragma unroll
  for (int t = 0; t < TW; ++t) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) Qr[t][ks] = q_operand<D, RT>(ring, t0 + t, ks, n, gq);
    const int row = (t0 + t) * 16 + n;
    lim[t] = row < a.R ? min(u.c1 - 1, u.ctx + row / a.G) : -1;
  }
  lds_sync();
  auto qop = [&](int t, int ks) { return Qr[t][ks]; };

  // ---- pass 1: running row statistics over the chunk
  float m[TW], z[TW];
#pragma unroll
  for (int t = 0; t < TW; ++t) {
    m[t] = kNegInf;
    z[t] = 0.f;
  }
  if (loader) {
    for (int s = 0; s < S1 && s < nblk; ++s) issue_k_lds<D>(kg, u.c0 + 32 * s, u.c1, ring + s * BLK, lane);
    for (int j = 0; j < nblk; ++j) {
      // blocks issued so far: the first S1, then one per barrier after the first
      const int issued = min(nblk, S1 + max(j - 1, 0));
      wait_vm_groups<KDMA, S1 - 1>(issued - j - 1);
      lds_sync();  // block j landed; every compute wave is done with block j - 1
      const int nb = j - 1 + S1;
      if (j >= 1 && nb < nblk) issue_k_lds<D>(kg, u.c0 + 32 * nb, u.c1, ring + (nb % S1) * BLK, lane);
    }
  } else {
    for (int j = 0; j < nblk; ++j) {
      lds_sync();
      uint4 Kr[2][KS];
      read_k_lds<D>(ring + (j % S1) * BLK, n, gq, Kr);
      float S[2][TW][4];
      scores_from<D, TW, false>(a, u, Kr, qop, u.c0 + 32 * j, gq, lim, S);
      running_stats_raw<TW>(S, sl2, m, z);
    }
  }
  lds_sync();  // the ring is free
  if (!loader) {
#pragma unroll
    for (int t = 0; t < TW; ++t) {
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1) {
        const float m2 = off == 16 ? lane_xor16(m[t]) : lane_xor32(m[t]);
        const float z2 = off == 16 ? lane_xor16(z[t]) : lane_xor32(z[t]);
        lse_combine(m[t], z[t], m2, z2);
      }
      if (gq == 0) {
        s_m[(t0 + t) * 16 + n] = m[t];
        s_z[(t0 + t) * 16 + n] = z[t];
      }
    }
  }
  exchange_stats<ROWS, LOCAL>(a, u, s_m, s_z, s_lse, s_wm, s_wz, base, true);
  float lse[TW];
#pragma unroll
  for (int t = 0; t < TW; ++t) lse[t] = s_lse[(t0 + t) * 16 + n];

  // ---- pass 2: scores again from K, exact probabilities, mass and P.V.
  //      Each row's last read, so the loads are non-temporal.
  floatx4 O[TW][DPL];
#pragma unroll
  for (int t = 0; t < TW; ++t)
#pragma unroll
    for (int jd = 0; jd < DPL; ++jd) O[t][jd] = floatx4{0.f, 0.f, 0.f, 0.f};
  // wave 0 adds the three waves' per-token sums of block jj and stores them
  auto store_mass = [&](int jj) {
    const int tok = u.c0 + 32 * jj + lane;
    if (lane < 32 && tok < u.c1)
      st_agent(mp + tok, s_mass[jj & 1][0][lane] + s_mass[jj & 1][1][lane] + s_mass[jj & 1][2][lane]);
  };
  if (loader) {
    for (int s = 0; s < S2 && s < nblk; ++s) {
      issue_k_lds<D, true>(kg, u.c0 + 32 * s, u.c1, ring + s * 2 * BLK, lane);
      issue_v_lds<D, true>(vg, u.c0 + 32 * s, u.c1, ring + s * 2 * BLK + BLK, lane);
    }
    for (int j = 0; j < nblk; ++j) {
      const int issued = min(nblk, S2 + max(j - 1, 0));
      wait_vm_groups<2 * KDMA, S2 - 1>(issued - j - 1);
      lds_sync();
      const int nb = j - 1 + S2;
      if (j >= 1 && nb < nblk) {
        issue_k_lds<D, true>(kg, u.c0 + 32 * nb, u.c1, ring + (nb % S2) * 2 * BLK, lane);
        issue_v_lds<D, true>(vg, u.c0 + 32 * nb, u.c1, ring + (nb % S2) * 2 * BLK + BLK, lane);
      }
    }
    lds_sync();
  } else {
    for (int j = 0; j < nblk; ++j) {
      lds_sync();
      if (w == 0 && j > 0) store_mass(j - 1);
      const uint16_t* slot = ring + (j % S2) * 2 * BLK;
      uint4 Kr[2][KS];
      read_k_lds<D>(slot, n, gq, Kr);
      VT Vr[8];
      read_v_lds<D>(slot + BLK, n, gq, Vr);
      float S[2][TW][4];
      scores_from<D, TW, false>(a, u, Kr, qop, u.c0 + 32 * j, gq, lim, S);
      bf16x8 Pa[TW];
      float pm[8];
      probs_raw<TW>(S, sl2, lse, Pa, pm);
      mass_reduce_lds(pm, s_mass[j & 1][w], n, gq);
      pv_mfma<D, TW>(Pa, Vr, O);
    }
    lds_sync();
    if (w == 0) store_mass(nblk - 1);
    write_opart_wide<D, LOCAL>(a, u, O, t0, n, gq);
  }
  verify_epilogue<ROWS, D, LOCAL>(a, u, s_lse, false, &s_flag, base);
}

// ------------------------------------------------------------ fp32 path --
template <int D, int RT>
__global__ void __launch_bounds__(kThreads) verify_f32_kernel(VArgs a) {
  constexpr int ROWS = RT * 16;
  constexpr int TC = kF32Tile;
  constexpr int OPT = ROWS * D / kThreads;
  // K/V tile rows padded by one word: the score loop's lanes take
  // consecutive tokens, which would otherwise all read one LDS bank
  constexpr int KVS = D + 1;
  extern __shared__ __align__(256) float sm[];
  float* sQ = sm;                // [ROWS][D]
  float* sKV = sQ + ROWS * D;    // [TC][KVS]
  float* sS = sKV + TC * KVS;    // [ROWS][TC]
  __shared__ float s_m[ROWS], s_z[ROWS], s_lse[ROWS];
  __shared__ float s_pm[kWaves][ROWS], s_pz[kWaves][ROWS];
  __shared__ int s_flag;

  Unit u;
  if (!decode_unit(a, u)) return;
  const unsigned base = read_base(a, u);
  const int tid = threadIdx.x;
  for (int r = tid; r < ROWS; r += kThreads) {
    s_m[r] = kNegInf;
    s_z[r] = 0.f;
  }
  if (u.c0 >= u.N) {
    __syncthreads();
    empty_chunk<ROWS, false>(a, u, s_m, s_z, base, &s_flag);
    return;
  }
  const int row0 = u.rg * a.RT * 16;
  const float* q = static_cast<const float*>(a.q);
  for (int e = tid; e < ROWS * D; e += kThreads) {
    const int r = e / D, d = e % D, row = row0 + r;
    float val = 0.f;
    if (row < a.R) {
      const int t = row / a.G, h = u.g * a.G + row % a.G;
      val = q[(((size_t)u.b * a.T + t) * a.Hq + h) * D + d];
    }
    sQ[e] = val;
  }
  const size_t kv_off = ((size_t)u.b * a.Hkv + u.g) * a.n_cap * D;
  const float* kg = static_cast<const float*>(a.k) + kv_off;
  const float* vg = static_cast<const float*>(a.v) + kv_off;
  float* mp = a.mpart + ((size_t)u.b * a.Hkv * a.RG + u.g * a.RG + u.rg) * a.n_cap;

  auto load_rows = [&](const float* src, int base, int nt) {
    for (int e = tid; e < TC * D; e += kThreads) {
      const int tt = e / D, d = e % D;
      sKV[tt * KVS + d] = tt < nt ? src[(size_t)(base + tt) * D + d] : 0.f;
    }
  };
  auto scores = [&](int base, int nt) {  // sS = scaled, masked scores (log2 domain)
    for (int e = tid; e < ROWS * TC; e += kThreads) {
      const int r = e / TC, tt = e % TC, row = row0 + r, tok = base + tt;
      float s = kNegInf;
      if (tt < nt && row < a.R && tok <= u.ctx + row / a.G) {
        float acc = 0.f;
        for (int d = 0; d < D; ++d) acc = fmaf(sQ[r * D + d], sKV[tt * KVS + d], acc);
        s = acc * a.sl2;
      }
      sS[e] = s;
    }
  };

  // ---- pass 1
  for (int base = u.c0; base < u.c1; base += TC) {
    const int nt = min(TC, u.c1 - base);
    __syncthreads();
    load_rows(kg, base, nt);
    __syncthreads();
    scores(base, nt);
    __syncthreads();
    for (int r = tid; r < ROWS; r += kThreads) {
      float M = s_m[r], Z = s_z[r];
      for (int tt = 0; tt < nt; ++tt) lse_combine(M, Z, sS[r * TC + tt], 1.f);
      s_m[r] = M;
      s_z[r] = Z;
    }
  }
  __syncthreads();
  exchange_stats<ROWS, false>(a, u, s_m, s_z, s_lse, s_pm, s_pz, base, true);

  // ---- pass 2
  float O[OPT];
#pragma unroll
  for (int k = 0; k < OPT; ++k) O[k] = 0.f;
  for (int base = u.c0; base < u.c1; base += TC) {
    const int nt = min(TC, u.c1 - base);
    __syncthreads();
    load_rows(kg, base, nt);
    __syncthreads();
    scores(base, nt);
    __syncthreads();
    for (int e = tid; e < ROWS * TC; e += kThreads) sS[e] = fast_exp2(sS[e] - s_lse[e / TC]);
    __syncthreads();
    if (tid < nt) {
      float acc = 0.f;
      for (int r = 0; r < ROWS; ++r) acc += sS[r * TC + tid];
      st_agent(mp + base + tid, acc);
    }
    load_rows(vg, base, nt);
    __syncthreads();
#pragma unroll
    for (int k = 0; k < OPT; ++k) {
      const int e = tid + k * kThreads, r = e / D, d = e % D;
      float acc = O[k];
      for (int tt = 0; tt < nt; ++tt) acc = fmaf(sS[r * TC + tt], sKV[tt * KVS + d], acc);
      O[k] = acc;
    }
  }
  float* op = a.opart + ((size_t)u.grp * a.splits + u.split) * ROWS * D;
#pragma unroll
  for (int k = 0; k < OPT; ++k) st_agent(op + tid + k * kThreads, O[k]);
  verify_epilogue<ROWS, D, false>(a, u, s_lse, false, &s_flag, base);
}

// -------------------------------------------------- allocation-free entry --
// The scratch buffer of pvlm_verify_attn_noalloc: a file-scope device array
// that every call on a device shares (each device holds its own copy for the
// life of the process).  Host code never uses this name as an address: the
// device address comes from hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

__global__ void __launch_bounds__(256) zero_words_kernel(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) p[i] = 0u;
}

// ------------------------------------------------------------------ host --
struct VPlan {
  int G, R, RTT, RG, RT;
  int64_t n_plan;
  int splits, chunk, groups, per_launch, grid;
  bool resident, mfma;
  bool wide;  // one group of kWideRT row tiles (wide variant)
  int lds_dyn;
  int xcds;
  bool budgeted;  // planned for a stream's compute-unit budget
  size_t off_cnt_s, off_mcnt, off_stats, off_opart, off_mpart, bytes;
};

typedef void (*VKernel)(VArgs);

VKernel pick_kernel(int dt, int D, int RT, bool resident, bool local, bool wide) {
  if (wide) {
    if (dt != PVLM_BF16 || RT != kWideRT) return nullptr;
    if (D == 128) return local ? verify_wide_kernel<128, true> : verify_wide_kernel<128, false>;
    if (D == 64) return local ? verify_wide_kernel<64, true> : verify_wide_kernel<64, false>;
    return nullptr;
  }
#define PVLM_VK(DD, R_)                                                                  \
  if (D == DD && RT == R_) {                                                            \
    if (dt == PVLM_F32) return verify_f32_kernel<DD, R_>;                               \
    if (local)                                                                          \
      return resident ? verify_mfma_kernel<DD, R_, true, true>                           \
                      : verify_mfma_kernel<DD, R_, false, true>;                         \
    return resident ? verify_mfma_kernel<DD, R_, true, false>                            \
                    : verify_mfma_kernel<DD, R_, false, false>;                          \
  }
  PVLM_VK(128, 1) PVLM_VK(128, 2) PVLM_VK(128, 3) PVLM_VK(128, 4) PVLM_VK(128, 5)
  PVLM_VK(64, 1) PVLM_VK(64, 2) PVLM_VK(64, 3) PVLM_VK(64, 4) PVLM_VK(64, 5)
#undef PVLM_VK
  return nullptr;
}

int lds_bytes(int dt, int D, int RT, bool resident, bool wide) {
  if (dt == PVLM_F32) return (RT * 16 * D + kF32Tile * (D + 1) + RT * 16 * kF32Tile) * 4;
  if (wide) {  // the Q tile, then the pass-1 and pass-2 rings (bf16)
    int b = kWideRT * 16 * D * 2;
    const int r1 = kWideSlots1 * 32 * D * 2, r2 = kWideSlots2 * 2 * 32 * D * 2;
    b = b > r1 ? b : r1;
    return b > r2 ? b : r2;
  }
  int b = 3 * RT * 16 * D * 4;                                   // O partial reduce-scatter
  if (!resident && RT > 3) {
    const int kv = RT * 16 * D * 2 + kWaves * 4 * 32 * D * 2;     // Q, then two K+V blocks per wave
    b = b > kv ? b : kv;
  }
  if (resident) {
    const int vq = kResTokens * D * 2 + RT * 16 * D * 2;          // the chunk's V, then Q (bf16)
    b = b > vq ? b : vq;
    const int f = kThreads * 16;  // the O-slice sums of the thread sets (at most 256 float4)
    b = b > f ? b : f;
  }
  return b;
}

// stream: the launch's stream, whose compute-unit budget bounds the plan;
// with_stream false plans for the whole device (workspace sizes, an upper
// bound for every budget).
pvlm_status plan_verify(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D, int64_t n_cap,
                        int64_t max_ctx, VPlan* p, hipStream_t stream, bool with_stream) {
  if (dt != PVLM_F32 && dt != PVLM_BF16) return PVLM_ERR_UNSUPPORTED;
  if (B < 1 || T < 1 || Hq < 1 || Hkv < 1 || n_cap < 1) return PVLM_ERR_SHAPE;
  if (T > 32 || Hq % Hkv != 0 || (D != 64 && D != 128)) return PVLM_ERR_UNSUPPORTED;
  if (max_ctx < 0 || max_ctx + T > n_cap || n_cap > (int64_t)1 << 30) return PVLM_ERR_SHAPE;
  p->G = Hq / Hkv;
  p->R = p->G * T;
  if (p->R > 640) return PVLM_ERR_UNSUPPORTED;
  p->RTT = (p->R + 15) / 16;
  p->RG = (p->RTT + kMaxRT - 1) / kMaxRT;
  p->n_plan = max_ctx + T;
  p->mfma = dt == PVLM_BF16;
  DeviceInfo di;
  pvlm_status st = with_stream ? device_info(&di, stream) : device_info(&di);
  if (st != PVLM_OK) return st;
  // Fewer (batch, KV head) groups than XCDs: split the rows into more groups
  // (K/V are then read once per row group) so that every group's workgroups
  // fit one XCD and exchange through its L2.
  if (p->mfma && B * Hkv * p->RG < di.xcds && p->RTT > p->RG) {
    const int want = (di.xcds + B * Hkv - 1) / (B * Hkv);
    p->RG = want < p->RTT ? want : p->RTT;
  }
  p->RT = (p->RTT + p->RG - 1) / p->RG;
  int W = di.cus;  // one workgroup per CU (registers / LDS bound)
  p->xcds = di.xcds;
  p->budgeted = di.budgeted;
  // groups, splits and chunk length for the row grouping in p->RG
  auto layout = [&]() {
    p->groups = B * Hkv * p->RG;
    p->per_launch = p->groups < W ? p->groups : W;
    int splits = W / p->per_launch;
    if (splits < 1) splits = 1;
    if (!p->mfma) {
      const int64_t want = (p->n_plan + kF32Tile - 1) / kF32Tile;
      if (splits > want) splits = (int)want;
    }
    int64_t chunk = (p->n_plan + splits - 1) / splits;
    chunk = (chunk + 31) / 32 * 32;
    p->chunk = (int)chunk;
    p->splits = (int)((p->n_plan + chunk - 1) / chunk);
    p->resident = p->mfma && chunk <= kResTokens;
  };
  layout();
  // Rows that need two row groups, in streamed chunks: one group of the
  // wide variant reads K and V once per pass for all of them instead.
  p->wide = p->mfma && !p->resident && p->RTT > kMaxRT && p->RTT <= kWideRT && B * Hkv >= di.xcds;
  if (p->wide) {
    p->RG = 1;
    p->RT = kWideRT;
    // two workgroups per CU, except on a budgeted stream: there the grid
    // keeps to one workgroup per budgeted CU, so that another stream's
    // waiting calls still find whole CUs free
    if (!di.budgeted) W = kWidePerCU * di.cus;
    layout();
    p->resident = false;
  }
  p->grid = (p->per_launch * p->splits + 7) / 8 * 8;
  p->lds_dyn = lds_bytes(dt, D, p->RT, p->resident, p->wide);
  const int ROWS = p->RT * 16;
  // Monotonic group counters sit at fixed per-group slots (cnt_s, cnt_o, base
  // of group g on lines 3g..3g+2 of the monotonic part), so calls of any shape
  // keep every slot consistent; the mass-sum counters return to zero and live
  // in the low part.
  if (3 * kSyncLine * (size_t)p->groups > kSyncTopkOff - kSyncMonoOff) return PVLM_ERR_UNSUPPORTED;
  if (kSyncLine * (size_t)B * p->splits > kSyncMonoOff) return PVLM_ERR_UNSUPPORTED;
  p->off_cnt_s = kSyncMonoOff;
  p->off_mcnt = 0;
  size_t off = kSyncRegion;
  p->off_stats = off;
  off = align_up(off + sizeof(float) * 2 * (size_t)p->groups * p->splits * ((ROWS + 1 + 15) / 16 * 16),
                 256);
  p->off_opart = off;
  off = align_up(off + sizeof(float) * (size_t)p->groups * p->splits * ROWS * D, 256);
  p->off_mpart = off;
  off = align_up(off + sizeof(float) * (size_t)B * Hkv * p->RG * n_cap, 256);
  p->bytes = off;
  return PVLM_OK;
}

}  // namespace
}  // namespace pvlm

using namespace pvlm;

extern "C" size_t pvlm_verify_attn_workspace_size(pvlm_dtype dt, int B, int T, int Hq, int Hkv,
                                                  int D, int64_t n_cap, int64_t max_ctx) {
  VPlan p;
  if (plan_verify(dt, B, T, Hq, Hkv, D, n_cap, max_ctx, &p, nullptr, false) != PVLM_OK) return 0;
  return p.bytes;
}

namespace {
// The cache rows come from a padded cache (table == NULL) or through a page
// table into a page pool (logical capacity n_cap = max_pages << page_shift).
pvlm_status verify_run(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D, int64_t n_cap,
                       int64_t max_ctx, float scale, const void* q, const void* k_cache,
                       const void* v_cache, const int32_t* table, int64_t n_pages, int max_pages,
                       int page_shift, const int32_t* ctx_len, void* out, float* mass, float* lse,
                       void* ws, size_t ws_bytes, int32_t* status, hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !ctx_len || !out) return PVLM_ERR_NULL;
  if (!(scale > 0.f) || !std::isfinite(scale)) return PVLM_ERR_SHAPE;
  VPlan p;
  pvlm_status st = plan_verify(dt, B, T, Hq, Hkv, D, n_cap, max_ctx, &p, stream, true);
  if (st != PVLM_OK) return st;
  if (!ws) return PVLM_ERR_WORKSPACE;
  if (ws_bytes < p.bytes) return PVLM_ERR_WORKSPACE;
  char* wsb = static_cast<char*>(ws);
  VArgs a;
  a.q = q;
  a.k = k_cache;
  a.v = v_cache;
  a.ctx_len = ctx_len;
  a.table = table;
  a.n_pages = n_pages;
  a.max_pages = max_pages;
  a.page_shift = page_shift;
  a.stats = reinterpret_cast<float*>(wsb + p.off_stats);
  a.opart = reinterpret_cast<float*>(wsb + p.off_opart);
  a.mpart = reinterpret_cast<float*>(wsb + p.off_mpart);
  a.slots = reinterpret_cast<unsigned*>(wsb + p.off_cnt_s);
  a.mcnt = reinterpret_cast<int*>(wsb + p.off_mcnt);
  a.out = out;
  a.lse = lse;
  a.mass = mass;
  a.f32 = dt == PVLM_F32;
  a.status = status;
  a.n_cap = n_cap;
  a.B = B;
  a.T = T;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.G = p.G;
  a.R = p.R;
  a.RG = p.RG;
  a.RT = p.RT;
  a.D = D;
  a.max_ctx = (int)max_ctx;
  a.splits = p.splits;
  a.chunk = p.chunk;
  a.grid = p.grid;
  a.sl2 = scale * kLog2e;
  if (!pick_kernel(dt, D, p.RT, p.resident, false, p.wide)) return PVLM_ERR_UNSUPPORTED;
  // every launch's grid fits the device at once (the first launch's grid is
  // the largest; both exchange variants use the same resources)
  for (int local = 0; local < 2; ++local) {
    const void* k = reinterpret_cast<const void*>(pick_kernel(dt, D, p.RT, p.resident, local != 0, p.wide));
    PVLM_HIP(allow_dynamic_lds(k, p.lds_dyn));
    const pvlm_status cs = check_coresident(k, p.grid, kThreads, p.lds_dyn, stream);
    if (cs != PVLM_OK) return cs;
  }
  for (int g0 = 0; g0 < p.groups; g0 += p.per_launch) {
    a.grp_base = g0;
    a.ngrp = p.groups - g0 < p.per_launch ? p.groups - g0 : p.per_launch;
    a.grid = (a.ngrp * p.splits + 7) / 8 * 8;
    // XCD-aware placement: logical units i*per_xcd.. run on XCD i.  When each
    // group's workgroups then share one XCD (and so one L2), the group's
    // exchanges use plain loads and stores (fp32 path: always device-coherent).
    a.xmap = p.xcds > 0 && a.grid % p.xcds == 0 ? p.xcds : 1;
    // (not on a budgeted stream: another stream's calls then run beside this
    // one, and the same-XCD mode is kept to a device this call has alone)
    a.local = p.mfma && !p.budgeted && p.xcds > 0 && a.xmap == p.xcds &&
              (a.grid / a.xmap) % p.splits == 0;
    VKernel kern = pick_kernel(dt, D, p.RT, p.resident, a.local != 0, p.wide);
    PVLM_HIP(allow_dynamic_lds(reinterpret_cast<const void*>(kern), p.lds_dyn));
    void* args[] = {&a};
    PVLM_HIP(launch_coresident(reinterpret_cast<const void*>(kern), dim3(a.grid), dim3(kThreads),
                               args, p.lds_dyn, stream));
  }
  return PVLM_OK;
}
}  // namespace

extern "C" pvlm_status pvlm_verify_attn(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                        int64_t n_cap, int64_t max_ctx, float scale, const void* q,
                                        const void* k_cache, const void* v_cache,
                                        const int32_t* ctx_len, void* out, float* mass, float* lse,
                                        void* ws, size_t ws_bytes, int32_t* status,
                                        hipStream_t stream) {
  return verify_run(dt, B, T, Hq, Hkv, D, n_cap, max_ctx, scale, q, k_cache, v_cache, nullptr, 0, 0,
                    0, ctx_len, out, mass, lse, ws, ws_bytes, status, stream);
}

extern "C" pvlm_status pvlm_verify_attn_paged(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                              int page_size, int max_pages, int64_t n_pages,
                                              int64_t max_ctx, float scale, const void* q,
                                              const void* k_pool, const void* v_pool,
                                              const int32_t* page_table, const int32_t* ctx_len,
                                              void* out, float* mass, float* lse, void* ws,
                                              size_t ws_bytes, int32_t* status,
                                              hipStream_t stream) {
  if (!page_table) return PVLM_ERR_NULL;
  const int shift = page_shift_of(page_size);
  if (shift < 0 || max_pages < 1 || n_pages < 1 || n_pages > INT32_MAX) return PVLM_ERR_SHAPE;
  if (dt != PVLM_BF16) return PVLM_ERR_UNSUPPORTED;
  return verify_run(dt, B, T, Hq, Hkv, D, (int64_t)max_pages << shift, max_ctx, scale, q, k_pool,
                    v_pool, page_table, n_pages, max_pages, shift, ctx_len, out, mass, lse, ws,
                    ws_bytes, status, stream);
}

namespace {
std::mutex g_scratch_mu;
void* g_scratch[64] = {nullptr};  // device address of `scratch` per device
}  // namespace

extern "C" size_t pvlm_verify_attn_noalloc_max_bytes(void) { return kScratchBytes; }

extern "C" pvlm_status pvlm_verify_attn_noalloc(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                                int64_t n_cap, int64_t max_ctx, float scale,
                                                const void* q, const void* k_cache,
                                                const void* v_cache, const int32_t* ctx_len,
                                                void* out, float* mass, float* lse, int32_t* status,
                                                hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !ctx_len || !out) return PVLM_ERR_NULL;
  if (!(scale > 0.f) || !std::isfinite(scale)) return PVLM_ERR_SHAPE;
  VPlan p;
  pvlm_status st = plan_verify(dt, B, T, Hq, Hkv, D, n_cap, max_ctx, &p, stream, true);
  if (st != PVLM_OK) return st;
  if (p.bytes > kScratchBytes) return PVLM_ERR_WORKSPACE;  // beyond the fixed scratch
  int dev = 0;
  PVLM_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return PVLM_ERR_UNSUPPORTED;
  void* ptr = nullptr;
  bool first = false;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
      void* a = nullptr;
      PVLM_HIP(hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)));
      if (!a) return PVLM_ERR_HIP;
      g_scratch[dev] = a;
      first = true;
    }
    ptr = g_scratch[dev];
  }
  if (first) {  // the synchronisation region starts at zero (a fill kernel, so
                // a capturing caller records no memset node)
    hipLaunchKernelGGL(zero_words_kernel, dim3(256), dim3(256), 0, stream, static_cast<uint32_t*>(ptr),
                       kSyncRegion / sizeof(uint32_t));
    PVLM_LAUNCHED();
  }
  return pvlm_verify_attn(dt, B, T, Hq, Hkv, D, n_cap, max_ctx, scale, q, k_cache, v_cache, ctx_len,
                          out, mass, lse, ptr, kScratchBytes, status, stream);
}
