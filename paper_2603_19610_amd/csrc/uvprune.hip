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

template <typename T>
struct HS;
template <>
struct HS<uint16_t> {
  // 8 bf16 -> 8 floats
  static __device__ __forceinline__ void load8(const uint16_t* p, float (&f)[8]) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      f[2 * k] = __uint_as_float(w[k] << 16);
      f[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
    }
  }
};
template <>
struct HS<float> {
  static __device__ __forceinline__ void load8(const float* p, float (&f)[8]) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
};

// One wave per text row: inv_norm[slot][b][j] = 1/|ht| (0 for zero norm or j >= n[b]).
template <typename T>
__global__ void __launch_bounds__(256) txt_norm_kernel(const T* ht, int64_t off0, int64_t off1,
                                                       const int32_t* n_txt,
                                                       int nslots, int B, int64_t n_cap, int Dh,
                                                       float* inv_norm, int32_t* status) {
  const int64_t wid = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wid >= (int64_t)nslots * B * n_cap) return;
  const int64_t j = wid % n_cap;
  const int b = (wid / n_cap) % B;
  const int slot = wid / (n_cap * B);
  bool bad = false;
  const int nb = clampi(n_txt[b], 0, (int)n_cap, bad);
  if (bad && j == 0 && slot == 0 && lane == 0) dev_flag(status, PVLM_DEV_RANGE);
  float inv = 0.f;
  if (j < nb) {
    const T* row = ht + (slot ? off1 : off0) + ((size_t)b * n_cap + j) * Dh;
    float ss = 0.f;
#pragma unroll 8  // the row's loads in flight together
    for (int d = lane * 8; d < Dh; d += 512) {
      float f[8];
      HS<T>::load8(row + d, f);
#pragma unroll
      for (int k = 0; k < 8; ++k) ss = fmaf(f[k], f[k], ss);
    }
    ss = warp_sum(ss);
    inv = ss > 0.f ? 1.f / sqrtf(ss) : 0.f;
  }
  if (lane == 0) inv_norm[wid] = inv;
}

// u[slot][b][d] = sum_{j<n[b]} ht[layer][b][j][d] * inv_norm[slot][b][j], in
// two steps so that many workgroups share the rows: partial sums over chunks
// of kTxtChunk text rows (one wave per 512 columns and chunk, each lane 8
// columns), then the chunks' sums in chunk order.
constexpr int kTxtChunk = 32;

template <typename T>
__global__ void __launch_bounds__(64) txt_dir_part_kernel(const T* ht, int64_t off0, int64_t off1,
                                                          const int32_t* n_txt, int B,
                                                          int64_t n_cap, int Dh, int nchunk,
                                                          const float* inv_norm, float* part) {
  const int c = blockIdx.y, sb = blockIdx.z, slot = sb / B, b = sb % B;
  const int d = (blockIdx.x * 64 + threadIdx.x) * 8;
  if (d >= Dh) return;
  int nb = n_txt[b];
  nb = nb < 0 ? 0 : (nb > n_cap ? (int)n_cap : nb);
  const int j0 = c * kTxtChunk, j1 = min(nb, j0 + kTxtChunk);
  const T* base = ht + (slot ? off1 : off0) + (size_t)b * n_cap * Dh + d;
  const float* inv = inv_norm + ((size_t)slot * B + b) * n_cap;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 8  // rows' loads in flight together
  for (int j = j0; j < j1; ++j) {
    const float wj = inv[j];
    float f[8];
    HS<T>::load8(base + (size_t)j * Dh, f);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = fmaf(f[k], wj, acc[k]);
  }
  float* pp = part + ((size_t)sb * nchunk + c) * Dh + d;
  *reinterpret_cast<float4*>(pp) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  *reinterpret_cast<float4*>(pp + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
}

__global__ void __launch_bounds__(256) txt_dir_sum_kernel(const float* part, int Dh, int nchunk,
                                                          float* u) {
  const int sb = blockIdx.y;
  const int d = blockIdx.x * 256 + threadIdx.x;
  if (d >= Dh) return;
  const float* p = part + (size_t)sb * nchunk * Dh + d;
  float acc = 0.f;
  for (int c = 0; c < nchunk; ++c) acc += p[(size_t)c * Dh];
  u[(size_t)sb * Dh + d] = acc;
}

// One wave per visual row: c_slot = <hv, u_slot> / |hv| (0 for zero norm).
// nslots == 2: out = c_1 - c_0 (the score); nslots == 1: out = c_0.
template <typename T>
__global__ void __launch_bounds__(256) vis_kernel(const T* hv, int64_t off0, int64_t off1,
                                                  const int32_t* m, int nslots,
                                                  int B, int64_t m_cap, int Dh, const float* u,
                                                  float* out, int32_t* status) {
  const int64_t wid = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wid >= (int64_t)B * m_cap) return;
  const int b = wid / m_cap;
  const int64_t i = wid % m_cap;
  bool bad = false;
  const int mb = clampi(m[b], 0, (int)m_cap, bad);
  if (bad && i == 0 && lane == 0) dev_flag(status, PVLM_DEV_RANGE);
  float res = 0.f;
  if (i < mb) {
    float c[2] = {0.f, 0.f};
    for (int s = 0; s < nslots; ++s) {
      const T* row = hv + (s ? off1 : off0) + ((size_t)b * m_cap + i) * Dh;
      const float* us = u + ((size_t)s * B + b) * Dh;
      float dot = 0.f, ss = 0.f;
      for (int d = lane * 8; d < Dh; d += 512) {
        float f[8];
        HS<T>::load8(row + d, f);
        const float4 u0 = *reinterpret_cast<const float4*>(us + d);
        const float4 u1 = *reinterpret_cast<const float4*>(us + d + 4);
        const float uu[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          dot = fmaf(f[k], uu[k], dot);
          ss = fmaf(f[k], f[k], ss);
        }
      }
      dot = warp_sum(dot);
      ss = warp_sum(ss);
      c[s] = ss > 0.f ? dot / sqrtf(ss) : 0.f;
    }
    res = nslots == 2 ? c[1] - c[0] : c[0];
  }
  if (lane == 0) out[wid] = res;
}

int txt_chunks(int64_t n_cap) { return (int)((n_cap + kTxtChunk - 1) / kTxtChunk); }

// inverse norms [2][B][n_cap], u [2][B][Dh], chunk partials [2][B][chunks][Dh]
size_t cossim_ws(int B, int Dh, int64_t n_cap) {
  size_t off = align_up(sizeof(float) * 2 * (size_t)B * n_cap, 256);
  off = align_up(off + sizeof(float) * 2 * (size_t)B * Dh, 256);
  off = align_up(off + sizeof(float) * 2 * (size_t)B * txt_chunks(n_cap) * Dh, 256);
  return off;
}

template <typename T>
pvlm_status launch_cossim(int nslots, int64_t voff0, int64_t voff1, int64_t toff0, int64_t toff1,
                          int B, int64_t m_cap, const int32_t* m, int Dh, int64_t n_cap,
                          const int32_t* n_txt, const T* hv, const T* ht, float* outp, float* inv,
                          float* u, float* part, int32_t* status, hipStream_t stream) {
  const int64_t nw = (int64_t)nslots * B * n_cap;
  hipLaunchKernelGGL(txt_norm_kernel<T>, dim3((unsigned)((nw + 3) / 4)), dim3(256), 0, stream, ht,
                     toff0, toff1, n_txt, nslots, B, n_cap, Dh, inv, status);
  PVLM_LAUNCHED();
  const int nchunk = txt_chunks(n_cap);
  hipLaunchKernelGGL(txt_dir_part_kernel<T>, dim3((Dh / 8 + 63) / 64, nchunk, nslots * B), dim3(64), 0,
                     stream, ht, toff0, toff1, n_txt, B, n_cap, Dh, nchunk, inv, part);
  PVLM_LAUNCHED();
  hipLaunchKernelGGL(txt_dir_sum_kernel, dim3((Dh + 255) / 256, nslots * B), dim3(256), 0, stream, part,
                     Dh, nchunk, u);
  PVLM_LAUNCHED();
  const int64_t vw = (int64_t)B * m_cap;
  hipLaunchKernelGGL(vis_kernel<T>, dim3((unsigned)((vw + 3) / 4)), dim3(256), 0, stream, hv, voff0,
                     voff1, m, nslots, B, m_cap, Dh, u, outp, status);
  PVLM_LAUNCHED();
  return PVLM_OK;
}

// nslots == 2: score from layers 0 and L of [L+1]-layer stacks; nslots == 1:
// the criterion of a single layer (L ignored, stacks hold one layer).
pvlm_status run_cossim(int nslots, int L, int B, int64_t m_cap, const int32_t* m, pvlm_dtype hdt,
                       int Dh, int64_t n_cap, const int32_t* n_txt, const void* hs_vis,
                       const void* hs_txt, float* outp, void* ws, size_t ws_bytes,
                       int32_t* status, hipStream_t stream) {
  if (!m || !n_txt || !hs_vis || !hs_txt || !outp) return PVLM_ERR_NULL;
  if (hdt != PVLM_F32 && hdt != PVLM_BF16) return PVLM_ERR_UNSUPPORTED;
  if (B < 1 || m_cap < 1 || n_cap < 1 || Dh < 8 || Dh % 8 != 0) return PVLM_ERR_SHAPE;
  if (m_cap > ((int64_t)1 << 30) || n_cap > ((int64_t)1 << 30)) return PVLM_ERR_SHAPE;
  if (nslots == 2 && L < 1) return PVLM_ERR_SHAPE;
  const size_t need = cossim_ws(B, Dh, n_cap);
  if (!ws || ws_bytes < need) return PVLM_ERR_WORKSPACE;
  char* w = static_cast<char*>(ws);
  float* inv = reinterpret_cast<float*>(w);
  float* u = reinterpret_cast<float*>(w + align_up(sizeof(float) * 2 * (size_t)B * n_cap, 256));
  float* part = reinterpret_cast<float*>(
      w + align_up(align_up(sizeof(float) * 2 * (size_t)B * n_cap, 256) + sizeof(float) * 2 * (size_t)B * Dh,
                   256));
  const int64_t vls = (int64_t)B * m_cap * Dh, tls = (int64_t)B * n_cap * Dh;
  const int64_t l1 = nslots == 2 ? L : 0;
  if (hdt == PVLM_BF16)
    return launch_cossim<uint16_t>(nslots, 0, l1 * vls, 0, l1 * tls, B, m_cap, m, Dh, n_cap, n_txt,
                                   static_cast<const uint16_t*>(hs_vis),
                                   static_cast<const uint16_t*>(hs_txt), outp, inv, u, part, status,
                                   stream);
  return launch_cossim<float>(nslots, 0, l1 * vls, 0, l1 * tls, B, m_cap, m, Dh, n_cap, n_txt,
                              static_cast<const float*>(hs_vis), static_cast<const float*>(hs_txt),
                              outp, inv, u, part, status, stream);
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
    const int64_t total = (int64_t)B * m_cap;
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
