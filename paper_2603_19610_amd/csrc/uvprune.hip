// UV-Prune score (gfx950): Eq. (average_similarity) of ParallelVLM Sec. 4.1,
// over either the vision-text cosine similarity of Eq. (similarity)
// ("COSSIM") or a precomputed per-layer criterion stack ("MASS", e.g. the
// verifier attention mass; Suppl. D's attention criterion with variation).
//
// The layer sum telescopes exactly, sum_{l=1..L} (S^l - S^{l-1}) = S^L - S^0,
// and the text-token sum is linear in the normalised text vectors,
// sum_j cos(V_i, X_j) = <V_i / |V_i|, sum_j X_j / |X_j|>, so the score needs
// only layers 0 and L and one normalised mat-vec per layer: streaming work
// bound by HBM bandwidth.  Zero-norm vectors contribute cosine 0.
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace pvlm {
namespace {

__device__ __forceinline__ int clampi(int v, int lo, int hi, bool& bad) {
  if (v < lo) {
    bad = true;
    return lo;
  }
  if (v > hi) {
    bad = true;
    return hi;
  }
  return v;
}

// MASS: score[b,i] = crit[L][b][i] - crit[0][b][i] for i < m[b], else 0.
__global__ void __launch_bounds__(256) uv_mass_kernel(const float* crit, const int32_t* m, int B,
                                                      int L, int64_t m_cap, float* score,
                                                      int32_t* status) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (int64_t)B * m_cap) return;
  const int b = gid / m_cap;
  const int64_t i = gid % m_cap;
  // both criteria load together with the row's length (every gid < B * m_cap
  // is inside the stack), which then decides whether the entry counts
  const float cL = crit[(size_t)L * B * m_cap + gid], c0 = crit[gid];
  bool bad = false;
  const int mb = clampi(m[b], 0, (int)m_cap, bad);
  if (bad && i == 0) dev_flag(status, PVLM_DEV_RANGE);
  score[gid] = i < mb ? cL - c0 : 0.f;
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resources (gfx9 descriptor word 3) bound a row segment's
// accesses: loads past the resource's size return zeros and stores there are
// dropped, so partial segments need no per-lane branches or address clamps.
constexpr int kBufWord3 = 0x00020000;
constexpr int kBufNT = 2;  // cache-policy bits: non-temporal (rows streamed once)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufWord3);
}

// Hidden-state element loads: 8 consecutive elements, widened exactly.  NT:
// through the non-temporal cache policy (rows streamed once).  load() only
// issues the load and unpack() widens, so a batch of loads can be in flight
// before the first is used.
template <typename T>
struct HS;
template <>
struct HS<uint16_t> {
  struct Raw {
    u32x4 v;
  };
  template <bool NT = false>
  static __device__ __forceinline__ Raw load(const uint16_t* p) {
    return {NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p))
               : *reinterpret_cast<const u32x4*>(p)};
  }
  static __device__ __forceinline__ void unpack(const Raw& r, float (&f)[8]) {
    const uint32_t w[4] = {r.v.x, r.v.y, r.v.z, r.v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      f[2 * k] = __uint_as_float(w[k] << 16);
      f[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
    }
  }
  template <bool NT = false>
  static __device__ __forceinline__ void load8(const uint16_t* p, float (&f)[8]) {
    unpack(load<NT>(p), f);
  }
  // through a buffer resource: bytes past its size read as zeros
  template <int AUX = kBufNT>
  static __device__ __forceinline__ Raw load_buf(__amdgpu_buffer_rsrc_t rs, int boff) {
    return {__builtin_amdgcn_raw_buffer_load_b128(rs, boff, 0, AUX)};
  }
  // f holds bf16 values (widened exactly), so their high halves are the bf16 words
  template <int AUX = kBufNT>
  static __device__ __forceinline__ void store_buf(const float (&f)[8], __amdgpu_buffer_rsrc_t rs, int boff) {
    uint32_t w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      w[k] = (__float_as_uint(f[2 * k]) >> 16) | (__float_as_uint(f[2 * k + 1]) & 0xFFFF0000u);
    const u32x4 v = {w[0], w[1], w[2], w[3]};
    __builtin_amdgcn_raw_buffer_store_b128(v, rs, boff, 0, AUX);
  }
};
template <>
struct HS<float> {
  struct Raw {
    f32x4 a, b;
  };
  template <bool NT = false>
  static __device__ __forceinline__ Raw load(const float* p) {
    return {NT ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p))
               : *reinterpret_cast<const f32x4*>(p),
            NT ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4))
               : *reinterpret_cast<const f32x4*>(p + 4)};
  }
  static __device__ __forceinline__ void unpack(const Raw& r, float (&f)[8]) {
    f[0] = r.a.x; f[1] = r.a.y; f[2] = r.a.z; f[3] = r.a.w;
    f[4] = r.b.x; f[5] = r.b.y; f[6] = r.b.z; f[7] = r.b.w;
  }
  template <bool NT = false>
  static __device__ __forceinline__ void load8(const float* p, float (&f)[8]) {
    unpack(load<NT>(p), f);
  }
  template <int AUX = kBufNT>
  static __device__ __forceinline__ Raw load_buf(__amdgpu_buffer_rsrc_t rs, int boff) {
    const u32x4 a = __builtin_amdgcn_raw_buffer_load_b128(rs, boff, 0, AUX);
    const u32x4 b = __builtin_amdgcn_raw_buffer_load_b128(rs, boff + 16, 0, AUX);
    return {__builtin_bit_cast(f32x4, a), __builtin_bit_cast(f32x4, b)};
  }
  template <int AUX = kBufNT>
  static __device__ __forceinline__ void store_buf(const float (&f)[8], __amdgpu_buffer_rsrc_t rs, int boff) {
    const f32x4 a = {f[0], f[1], f[2], f[3]}, b = {f[4], f[5], f[6], f[7]};
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, a), rs, boff, 0, AUX);
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, b), rs, boff + 16, 0, AUX);
  }
};

// The prefill epilogue's residual add: prev + delta, the sum taken in fp32
// and rounded once to the storage type.  f (prev) becomes the values that
// are stored, so the criterion uses exactly the stored hidden state.
__device__ __forceinline__ void add_round8(uint16_t, float (&f)[8], const float (&g)[8]) {
#pragma unroll
  for (int k = 0; k < 8; ++k) f[k] = bf16_to_f32(f32_to_bf16(f[k] + g[k]));
}
__device__ __forceinline__ void add_round8(float, float (&f)[8], const float (&g)[8]) {
#pragma unroll
  for (int k = 0; k < 8; ++k) f[k] += g[k];
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Wave totals through DPP lane moves: xor 1 and xor 2 inside each quad,
// then the half-row and row mirrors give every lane its 16-lane row's sum;
// the four row sums are read from lanes 0, 16, 32 and 48 and added in a
// fixed order.  Every lane gets the same total.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, 0xF, 0xF, true);
  return __hiloint2double(hi, lo);
}
__device__ __forceinline__ double lane_f64(double v, int l) {
  return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(v), l),
                          __builtin_amdgcn_readlane(__double2loint(v), l));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;
__device__ __forceinline__ double wave_total_f64(double v) {
  v += dpp_f64<kDppXor1>(v);
  v += dpp_f64<kDppXor2>(v);
  v += dpp_f64<kDppHalfMirror>(v);
  v += dpp_f64<kDppMirror>(v);
  return (lane_f64(v, 0) + lane_f64(v, 16)) + (lane_f64(v, 32) + lane_f64(v, 48));
}
__device__ __forceinline__ float wave_total_f32(float v) {
  v += dpp_f32<kDppXor1>(v);
  v += dpp_f32<kDppXor2>(v);
  v += dpp_f32<kDppHalfMirror>(v);
  v += dpp_f32<kDppMirror>(v);
  auto at = [&](int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l)); };
  return (at(0) + at(16)) + (at(32) + at(48));
}

// The COSSIM criterion is a sum of n cosines that can cancel to far below
// the size of its terms, so it is accumulated in float64: bf16 and fp32
// inputs convert to float64 exactly, every norm, direction sum and dot
// product is formed in float64, and only the final criterion (or the score
// c^L - c^0) is rounded, once, to fp32.

// One wave per text row: inv_norm[slot][b][j] = 1/|ht| (0 for zero norm or j >= n[b]).
template <typename T, bool FUSED>
__global__ void __launch_bounds__(256) txt_norm_kernel(const T* ht, int64_t off0, int64_t off1,
                                                       const int32_t* n_txt,
                                                       int nslots, int B, int64_t n_cap, int Dh,
                                                       double* inv_norm, int32_t* status,
                                                       const T* dt, T* ot) {
  const int64_t wid = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wid >= (int64_t)nslots * B * n_cap) return;
  const int64_t j = wid % n_cap;
  const int b = (wid / n_cap) % B;
  const int slot = wid / (n_cap * B);
  bool bad = false;
  const int nb = clampi(n_txt[b], 0, (int)n_cap, bad);
  if (bad && j == 0 && slot == 0 && lane == 0) dev_flag(status, PVLM_DEV_RANGE);
  double inv = 0.0;
  if (j < nb) {
    const size_t roff = (slot ? off1 : off0) + ((size_t)b * n_cap + j) * Dh;
    double ss = 0.0;
    if constexpr (FUSED) {
      // every piece of the row (prev and delta) in flight before the first
      // store: the stores count in the same wait counter as the loads, so
      // a store between loads would make each later load wait for all
      // (pieces past the row's end read as zeros, add exact zeros, and
      // their stores are dropped); the same order as the plain loop below
      constexpr int NBT = sizeof(T) == 2 ? 16 : 8;
      const int rb = Dh * (int)sizeof(T);
      const auto rs = buf_rsrc(ht + roff, rb), rsd = buf_rsrc(dt + roff, rb), os = buf_rsrc(ot + roff, rb);
      for (int d0 = 0; d0 < Dh; d0 += 512 * NBT) {
        typename HS<T>::Raw r[NBT], rd[NBT];
#pragma unroll
        for (int t = 0; t < NBT; ++t) {
          r[t] = HS<T>::template load_buf<0>(rs, (d0 + lane * 8 + 512 * t) * (int)sizeof(T));
          rd[t] = HS<T>::template load_buf<0>(rsd, (d0 + lane * 8 + 512 * t) * (int)sizeof(T));
        }
#pragma unroll
        for (int t = 0; t < NBT; ++t) {
          float f[8], g[8];
          HS<T>::unpack(r[t], f);
          HS<T>::unpack(rd[t], g);
          add_round8(T(), f, g);
          HS<T>::template store_buf<0>(f, os, (d0 + lane * 8 + 512 * t) * (int)sizeof(T));
#pragma unroll
          for (int k = 0; k < 8; ++k) ss = fma((double)f[k], (double)f[k], ss);
        }
      }
    } else {
#pragma unroll 8  // the row's loads in flight together
      for (int d = lane * 8; d < Dh; d += 512) {
        float f[8];
        HS<T>::load8(ht + roff + d, f);
#pragma unroll
        for (int k = 0; k < 8; ++k) ss = fma((double)f[k], (double)f[k], ss);
      }
    }
    ss = wave_sum_f64(ss);
    inv = ss > 0.0 ? 1.0 / sqrt(ss) : 0.0;
  }
  if (lane == 0) inv_norm[wid] = inv;
}

// u[slot][b][d] in one pass: one 1024-thread workgroup per (512 columns,
// slot, batch row).  Wave w sums rows [w R, (w + 1) R), R = ceil(n / 16), for
// its lanes' 8 columns each, loading kDirRows rows at a time through a buffer
// resource over them; the waves' sums then meet in LDS and are added in wave
// order.
constexpr int kDirWaves = 16;
template <typename T>
__global__ void __launch_bounds__(64 * kDirWaves) txt_dir_kernel(const T* ht, int64_t off0, int64_t off1,
                                                                 const int32_t* n_txt, int B, int64_t n_cap,
                                                                 int Dh, const double* inv_norm, double* u) {
  constexpr int RB = sizeof(T) == 2 ? 16 : 8;  // rows in flight per lane
  __shared__ double s_acc[kDirWaves][512];
  const int sb = blockIdx.y, slot = sb / B, b = sb % B;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: row weights are scalar
  const int d = blockIdx.x * 512 + lane * 8;
  int nb = n_txt[b];
  nb = nb < 0 ? 0 : (nb > n_cap ? (int)n_cap : nb);
  const int R = (nb + kDirWaves - 1) / kDirWaves;
  const int j0 = min(nb, wave * R), rows = min(nb, j0 + R) - j0;
  double acc[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  if (d < Dh) {
    const T* base = ht + (slot ? off1 : off0) + ((size_t)b * n_cap + j0) * Dh;
    const double* inv = inv_norm + ((size_t)slot * B + b) * n_cap + j0;
    for (int jb = 0; jb < rows; jb += RB) {
      const int nr = min(RB, rows - jb);  // rows past nr read as zeros and get weight 0
      const auto rs = buf_rsrc(base + (size_t)jb * Dh, nr * Dh * (int)sizeof(T));
      typename HS<T>::Raw r[RB];
      double w[RB];
#pragma unroll
      for (int i = 0; i < RB; ++i) {
        r[i] = HS<T>::template load_buf<0>(rs, (i * Dh + d) * (int)sizeof(T));
        const double wi = inv[jb + min(i, nr - 1)];
        w[i] = i < nr ? wi : 0.0;
      }
#pragma unroll
      for (int i = 0; i < RB; ++i) {
        float f[8];
        HS<T>::unpack(r[i], f);
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[k] = fma((double)f[k], w[i], acc[k]);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) s_acc[wave][lane * 8 + k] = acc[k];
  __syncthreads();
  if (threadIdx.x < 512) {
    const int dd = blockIdx.x * 512 + threadIdx.x;
    if (dd < Dh) {
      double t = 0.0;
#pragma unroll
      for (int w = 0; w < kDirWaves; ++w) t += s_acc[w][threadIdx.x];
      u[(size_t)sb * Dh + dd] = t;
    }
  }
}

// c_slot = <hv, u_slot> / |hv| (0 for zero norm) for the visual rows.  A
// workgroup of 16 waves first stages the direction vectors of its batch row
// (both slots, float64) in LDS.  It owns a contiguous run of rows, taken in
// rounds of up to kVisRows, and splits each round into units (row, slot,
// segment of 64 * kVisPieces 8-element pieces) that its waves take in turn,
// so every wave carries nearly the same load.  Lane l of a unit handles
// pieces segment * 64 * kVisPieces + l + 64 t, t < kVisPieces (16-byte
// loads).  The plain kernel holds a unit's pieces in registers and, as it
// consumes piece t, issues piece t of its next unit into the same
// registers, so a unit's loads are in flight while the one before is
// reduced.  The fused kernel loads a whole unit (prev and delta) before it
// adds and stores: its stores share the loads' wait counter.
// A unit's dot product and squared norm (wave totals) go to LDS,
// and one thread per row then sums the segments in order.  u is staged as
// s_u[slot][k / 2][d / 8][k % 2]: a lane reads its 8 directions of a piece
// as four 16-byte words, and the lanes of a wave read consecutive words.
// The dot product is float64 (it can cancel); the squared norm sums positive
// terms only, so fp32 keeps its relative error below 1e-5 (fewer than 80
// roundings), far inside the criterion's gate.
// nslots == 2: out = c_1 - c_0 (the score); nslots == 1: out = c_0.
// Largest hidden size whose two float64 direction vectors fit the kernel's
// LDS.
constexpr int kMaxDh = 8192;
constexpr int kVisThreads = 1024;
constexpr int kVisWaves = kVisThreads / 64;
constexpr int kVisRows = 128;
// Pieces per lane and unit: the summation grouping, the same for the fused
// and the plain kernel, so both give the same sums bit for bit.
template <typename T>
constexpr int kVisPieces = sizeof(T) == 2 ? 8 : 4;

// f(integral_constant<int, I>) for I = 0 .. N-1, unrolled at compile time.
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

// One 8-element piece of a visual row against its directions (us points at
// the slot's staged vector, j is the piece's index d / 8, clamped into the
// row).  A piece past the row's end was read as zeros through the buffer
// resource, so it adds exact zeros to both sums, and its store (FUSED, to
// the output resource os) is dropped.
template <typename T, bool FUSED>
__device__ __forceinline__ void vis_piece(const typename HS<T>::Raw& r, const typename HS<T>::Raw& rd,
                                          __amdgpu_buffer_rsrc_t os, int boff, const double* us, int D8,
                                          int j, double& dot, float& ss) {
  float f[8];
  HS<T>::unpack(r, f);
  if constexpr (FUSED) {
    float g[8];
    HS<T>::unpack(rd, g);
    add_round8(T(), f, g);
    HS<T>::template store_buf<kBufNT>(f, os, boff);
  }
  double2 w[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) w[p] = reinterpret_cast<const double2*>(us)[(size_t)p * D8 + j];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    dot = fma((double)f[2 * p], w[p].x, dot);
    dot = fma((double)f[2 * p + 1], w[p].y, dot);
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) ss = fmaf(f[k], f[k], ss);
}

template <typename T, bool FUSED>
__global__ void __launch_bounds__(kVisThreads) vis_kernel(const T* hv, int64_t off0, int64_t off1,
                                                          const int32_t* m, int nslots,
                                                          int B, int64_t m_cap, int Dh, const double* u,
                                                          float* out, int32_t* status, const T* dv,
                                                          T* ov) {
  // [nslots][4][Dh / 8][2] directions, then the units' float64 dot products
  // and fp32 squared norms, [kVisRows][nslots][nseg] each
  extern __shared__ __align__(16) double s_u[];
  constexpr int NP = kVisPieces<T>;
  constexpr int SEG = 64 * NP;  // pieces per segment
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: unit bookkeeping is scalar
  const int D8 = Dh / 8;
  const int nseg = (D8 + SEG - 1) / SEG;
  const int per_row = nslots * nseg;  // units per row
  double* s_pd = s_u + (size_t)nslots * Dh;
  float* s_ps = reinterpret_cast<float*>(s_pd + kVisRows * per_row);
  for (int s = 0; s < nslots; ++s)
    for (int d = threadIdx.x; d < Dh; d += kVisThreads)
      s_u[((size_t)(s * 4 + ((d & 7) >> 1)) * D8 + (d >> 3)) * 2 + (d & 1)] =
          u[((size_t)s * B + b) * Dh + d];
  __syncthreads();
  bool bad = false;
  const int mb = clampi(m[b], 0, (int)m_cap, bad);
  if (bad && blockIdx.x == 0 && threadIdx.x == 0) dev_flag(status, PVLM_DEV_RANGE);
  const int64_t per_wg = (m_cap + gridDim.x - 1) / gridDim.x;
  const int64_t r_begin = (int64_t)blockIdx.x * per_wg;
  const int64_t r_end = min(m_cap, r_begin + per_wg);
  // element offset of unit q's segment start within the hidden-state stacks
  auto unit = [&](int64_t r0, int q, int& seg) -> size_t {
    const int row = q / per_row, rest = q % per_row, s = rest / nseg;
    seg = rest % nseg;
    return (s ? off1 : off0) + ((size_t)b * m_cap + r0 + row) * Dh + (size_t)8 * seg * SEG;
  };
  constexpr int PB = 8 * (int)sizeof(T);  // bytes per piece
  // a resource over the rest of the row from a segment's start
  auto rsrc = [&](const T* base, size_t off, int sg) { return buf_rsrc(base + off, (D8 - sg * SEG) * PB); };
  for (int64_t r0 = r_begin; r0 < r_end; r0 += kVisRows) {
    const int nr = (int)min((int64_t)kVisRows, r_end - r0);
    const int nv = (int)max((int64_t)0, min((int64_t)nr, (int64_t)mb - r0));  // rows with data
    const int U = nv * per_row;
    int q = wave, seg = 0;
    size_t off = 0;
    if constexpr (FUSED) {
      // whole units: every piece's loads (prev and delta), then the adds,
      // stores and sums; the stores count in the same wait counter as the
      // loads, so a store between loads would make each later load wait
      // for all
      for (; q < U; q += kVisWaves) {
        off = unit(r0, q, seg);
        const int s = (q % per_row) / nseg;
        const double* us = s_u + (size_t)s * 8 * D8;
        const auto rs = rsrc(hv, off, seg), rsd = rsrc(dv, off, seg), os = rsrc(ov, off, seg);
        typename HS<T>::Raw r[NP], rd[NP];
#pragma unroll
        for (int t = 0; t < NP; ++t) {
          r[t] = HS<T>::load_buf(rs, (lane + 64 * t) * PB);
          rd[t] = HS<T>::load_buf(rsd, (lane + 64 * t) * PB);
        }
        double dot = 0.0;
        float ss = 0.f;
#pragma unroll
        for (int t = 0; t < NP; ++t) {
          const int j = min(seg * SEG + lane + 64 * t, D8 - 1);
          vis_piece<T, FUSED>(r[t], rd[t], os, (lane + 64 * t) * PB, us, D8, j, dot, ss);
        }
        dot = wave_total_f64(dot);
        ss = wave_total_f32(ss);
        if (lane == 0) {
          s_pd[q] = dot;
          s_ps[q] = ss;
        }
      }
    } else {
      // a unit's NP pieces in registers; consuming piece t frees its
      // registers for piece t of the wave's next unit
      typename HS<T>::Raw r[NP];
      if (q < U) {
        off = unit(r0, q, seg);
        const auto rs = rsrc(hv, off, seg);
#pragma unroll
        for (int t = 0; t < NP; ++t) r[t] = HS<T>::load_buf(rs, (lane + 64 * t) * PB);
      }
      while (q < U) {
        const int qn = q + kVisWaves;
        const int s = (q % per_row) / nseg;
        const double* us = s_u + (size_t)s * 8 * D8;
        double dot = 0.0;
        float ss = 0.f;
        const bool more = qn < U;
        int segn = seg;
        size_t offn = off;
        if (more) offn = unit(r0, qn, segn);
        const auto rsn = rsrc(hv, offn, segn);
        auto step = [&](auto tc, bool next) {
          constexpr int t = decltype(tc)::value;
          const int j = min(seg * SEG + lane + 64 * t, D8 - 1);
          vis_piece<T, FUSED>(r[t], r[t], rsn, (lane + 64 * t) * PB, us, D8, j, dot, ss);
          if (next) r[t] = HS<T>::load_buf(rsn, (lane + 64 * t) * PB);
          // keep the order: a load hoisted above the pieces still to be
          // consumed would hold a second set of registers
          __builtin_amdgcn_sched_barrier(0);
        };
        if (more) {
          static_for<NP>([&](auto tc) { step(tc, true); });
        } else {
          static_for<NP>([&](auto tc) { step(tc, false); });
        }
        seg = segn;
        off = offn;
        dot = wave_total_f64(dot);
        ss = wave_total_f32(ss);
        if (lane == 0) {
          s_pd[q] = dot;
          s_ps[q] = ss;
        }
        q = qn;
      }
    }
    __syncthreads();
    for (int k = threadIdx.x; k < nr; k += kVisThreads) {
      double res = 0.0;
      if (k < nv) {
        double c[2] = {0.0, 0.0};
        for (int s = 0; s < nslots; ++s) {
          double dot = 0.0;
          float ss = 0.f;
          for (int g = 0; g < nseg; ++g) {
            dot += s_pd[k * per_row + s * nseg + g];
            ss += s_ps[k * per_row + s * nseg + g];
          }
          c[s] = ss > 0.f ? dot / sqrt((double)ss) : 0.0;
        }
        res = nslots == 2 ? c[1] - c[0] : c[0];
      }
      out[(size_t)b * m_cap + r0 + k] = (float)res;
    }
    __syncthreads();  // the partials are reused by the next round
  }
}

// The visual kernel's LDS: the staged directions and one round's partials.
template <typename T, bool FUSED>
size_t vis_lds_bytes(int nslots, int Dh) {
  const int seg = 64 * kVisPieces<T>;
  const int nseg = (Dh / 8 + seg - 1) / seg;
  return sizeof(double) * nslots * Dh + (sizeof(double) + sizeof(float)) * kVisRows * nslots * nseg;
}

// inverse norms [2][B][n_cap], u [2][B][Dh], both float64
size_t cossim_ws(int B, int Dh, int64_t n_cap) {
  size_t off = align_up(sizeof(double) * 2 * (size_t)B * n_cap, 256);
  off = align_up(off + sizeof(double) * 2 * (size_t)B * Dh, 256);
  return off;
}

// FUSED (the prefill epilogue, nslots == 1): the rows are prev + delta
// (hv/ht the previous hidden states, dv/dt the deltas), written to ov/ot on
// the first read; the text directions then read ot.
template <typename T, bool FUSED = false>
pvlm_status launch_cossim(int nslots, int64_t voff0, int64_t voff1, int64_t toff0, int64_t toff1,
                          int B, int64_t m_cap, const int32_t* m, int Dh, int64_t n_cap,
                          const int32_t* n_txt, const T* hv, const T* ht, float* outp, double* inv,
                          double* u, int32_t* status, hipStream_t stream,
                          const T* dv = nullptr, T* ov = nullptr, const T* dt = nullptr,
                          T* ot = nullptr) {
  const int lds = (int)vis_lds_bytes<T, FUSED>(nslots, Dh);
  PVLM_HIP(allow_dynamic_lds(reinterpret_cast<const void*>(vis_kernel<T, FUSED>),
                             (int)vis_lds_bytes<T, FUSED>(2, kMaxDh)));
  DeviceInfo di;
  const pvlm_status st = device_info(&di);
  if (st != PVLM_OK) return st;
  // about one workgroup per compute unit over the batch rows
  const int64_t per_b = (di.cus + B - 1) / B;
  const int64_t vis_x = std::max<int64_t>(1, std::min<int64_t>(per_b, (m_cap + 15) / 16));
  const int64_t nw = (int64_t)nslots * B * n_cap;
  hipLaunchKernelGGL((txt_norm_kernel<T, FUSED>), dim3((unsigned)((nw + 3) / 4)), dim3(256), 0, stream,
                     ht, toff0, toff1, n_txt, nslots, B, n_cap, Dh, inv, status, dt, ot);
  PVLM_LAUNCHED();
  hipLaunchKernelGGL(txt_dir_kernel<T>, dim3((Dh + 511) / 512, nslots * B), dim3(64 * kDirWaves), 0, stream,
                     FUSED ? static_cast<const T*>(ot) : ht, toff0, toff1, n_txt, B, n_cap, Dh, inv, u);
  PVLM_LAUNCHED();
  hipLaunchKernelGGL((vis_kernel<T, FUSED>), dim3((unsigned)vis_x, B), dim3(kVisThreads), lds, stream, hv,
                     voff0, voff1, m, nslots, B, m_cap, Dh, u, outp, status, dv, ov);
  PVLM_LAUNCHED();
  return PVLM_OK;
}

// nslots == 2: score from layers 0 and L of [L+1]-layer stacks; nslots == 1:
// the criterion of a single layer (L ignored, stacks hold one layer).
// With the epilogue pointers (dv, ov, dt, ot non-NULL, nslots == 1): the
// rows are hs + delta, stored to the outputs as they are read.
pvlm_status run_cossim(int nslots, int L, int B, int64_t m_cap, const int32_t* m, pvlm_dtype hdt,
                       int Dh, int64_t n_cap, const int32_t* n_txt, const void* hs_vis,
                       const void* hs_txt, float* outp, void* ws, size_t ws_bytes,
                       int32_t* status, hipStream_t stream, const void* dv = nullptr,
                       void* ov = nullptr, const void* dt = nullptr, void* ot = nullptr) {
  if (!m || !n_txt || !hs_vis || !hs_txt || !outp) return PVLM_ERR_NULL;
  if (hdt != PVLM_F32 && hdt != PVLM_BF16) return PVLM_ERR_UNSUPPORTED;
  if (B < 1 || m_cap < 1 || n_cap < 1 || Dh < 8 || Dh % 8 != 0) return PVLM_ERR_SHAPE;
  if (Dh > kMaxDh) return PVLM_ERR_UNSUPPORTED;
  // launch limits: grid y of at most 65535 (the text directions and the
  // visual rows run over 2 * B batch-slots and B batch rows), and one 64-lane
  // wave per text row of both slots, in one launch of at most 2^32 - 256
  // work-items
  if (m_cap > ((int64_t)1 << 30) || 2 * (int64_t)B > 65535 ||
      ((int64_t)2 * B * n_cap + 3) / 4 * 256 > ((int64_t)1 << 32) - 256)
    return PVLM_ERR_SHAPE;
  if (nslots == 2 && L < 1) return PVLM_ERR_SHAPE;
  const size_t need = cossim_ws(B, Dh, n_cap);
  if (!ws || ws_bytes < need) return PVLM_ERR_WORKSPACE;
  char* w = static_cast<char*>(ws);
  double* inv = reinterpret_cast<double*>(w);
  const size_t off_u = align_up(sizeof(double) * 2 * (size_t)B * n_cap, 256);
  double* u = reinterpret_cast<double*>(w + off_u);
  const int64_t vls = (int64_t)B * m_cap * Dh, tls = (int64_t)B * n_cap * Dh;
  const int64_t l1 = nslots == 2 ? L : 0;
  if (dv) {
    typedef uint16_t H;
    if (hdt == PVLM_BF16)
      return launch_cossim<H, true>(1, 0, 0, 0, 0, B, m_cap, m, Dh, n_cap, n_txt,
                                    static_cast<const H*>(hs_vis), static_cast<const H*>(hs_txt),
                                    outp, inv, u, status, stream, static_cast<const H*>(dv),
                                    static_cast<H*>(ov), static_cast<const H*>(dt), static_cast<H*>(ot));
    return launch_cossim<float, true>(1, 0, 0, 0, 0, B, m_cap, m, Dh, n_cap, n_txt,
                                      static_cast<const float*>(hs_vis),
                                      static_cast<const float*>(hs_txt), outp, inv, u, status,
                                      stream, static_cast<const float*>(dv), static_cast<float*>(ov),
                                      static_cast<const float*>(dt), static_cast<float*>(ot));
  }
  if (hdt == PVLM_BF16)
    return launch_cossim<uint16_t>(nslots, 0, l1 * vls, 0, l1 * tls, B, m_cap, m, Dh, n_cap, n_txt,
                                   static_cast<const uint16_t*>(hs_vis),
                                   static_cast<const uint16_t*>(hs_txt), outp, inv, u, status,
                                   stream);
  return launch_cossim<float>(nslots, 0, l1 * vls, 0, l1 * tls, B, m_cap, m, Dh, n_cap, n_txt,
                              static_cast<const float*>(hs_vis), static_cast<const float*>(hs_txt),
                              outp, inv, u, status, stream);
}

}  // namespace
}  // namespace pvlm

using namespace pvlm;

extern "C" size_t pvlm_uvprune_workspace_size(pvlm_crit crit, int B, int Dh, int64_t n_cap) {
  if (crit == PVLM_CRIT_MASS) return 0;
  if (B < 1 || Dh < 1 || n_cap < 1) return 0;
  return cossim_ws(B, Dh, n_cap);
}

extern "C" pvlm_status pvlm_uvprune_score(pvlm_crit crit, int B, int L, int64_t m_cap,
                                          const int32_t* m, const float* crit_stack,
                                          pvlm_dtype hdt, int Dh, int64_t n_cap,
                                          const int32_t* n_txt, const void* hs_vis,
                                          const void* hs_txt, float* score, void* ws,
                                          size_t ws_bytes, int32_t* status, hipStream_t stream) {
  if (crit == PVLM_CRIT_MASS) {
    if (!m || !crit_stack || !score) return PVLM_ERR_NULL;
    if (B < 1 || L < 1 || m_cap < 1 || m_cap > ((int64_t)1 << 30)) return PVLM_ERR_SHAPE;
    const int64_t total = (int64_t)B * m_cap;  // one work-item per score, one launch
    if ((total + 255) / 256 * 256 > ((int64_t)1 << 32) - 256) return PVLM_ERR_SHAPE;
    hipLaunchKernelGGL(uv_mass_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream,
                       crit_stack, m, B, L, m_cap, score, status);
    PVLM_LAUNCHED();
    return PVLM_OK;
  }
  if (crit != PVLM_CRIT_COSSIM) return PVLM_ERR_UNSUPPORTED;
  return run_cossim(2, L, B, m_cap, m, hdt, Dh, n_cap, n_txt, hs_vis, hs_txt, score, ws, ws_bytes,
                    status, stream);
}

extern "C" pvlm_status pvlm_uvprune_criterion_cossim(int B, int64_t m_cap, const int32_t* m,
                                                     pvlm_dtype hdt, int Dh, int64_t n_cap,
                                                     const int32_t* n_txt, const void* hs_vis,
                                                     const void* hs_txt, float* crit_out, void* ws,
                                                     size_t ws_bytes, int32_t* status,
                                                     hipStream_t stream) {
  return run_cossim(1, 0, B, m_cap, m, hdt, Dh, n_cap, n_txt, hs_vis, hs_txt, crit_out, ws,
                    ws_bytes, status, stream);
}

extern "C" pvlm_status pvlm_prefill_epilogue_cossim(int B, int64_t m_cap, const int32_t* m,
                                                    int64_t n_cap, const int32_t* n_txt,
                                                    pvlm_dtype hdt, int Dh, const void* vis_prev,
                                                    const void* vis_delta, void* vis_out,
                                                    const void* txt_prev, const void* txt_delta,
                                                    void* txt_out, float* crit_out, void* ws,
                                                    size_t ws_bytes, int32_t* status,
                                                    hipStream_t stream) {
  if (!vis_delta || !vis_out || !txt_delta || !txt_out) return PVLM_ERR_NULL;
  return run_cossim(1, 0, B, m_cap, m, hdt, Dh, n_cap, n_txt, vis_prev, txt_prev, crit_out, ws,
                    ws_bytes, status, stream, vis_delta, vis_out, txt_delta, txt_out);
}
