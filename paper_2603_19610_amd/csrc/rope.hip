// Rotary embedding of the verify rows and their append to the KV cache
// (gfx950).  The target verifies the gamma + 1 speculated positions in one
// forward (ParallelVLM Sec. 2.2, Sec. 4.2): their queries and new keys are
// rotated by their positions (1-D RoPE, or the three-axis M-RoPE of the
// Qwen2.5-VL target) and the new key and value rows are written behind each
// sequence's context, where verify attention reads them.
//
// One thread per rotation pair (i, i + D/2) of one row; consecutive threads
// take consecutive pairs, so a row's loads and stores are contiguous.  Rows are
// q rows, then k rows, then v rows (copied) of every (b, t).  The angle
// p * base^(-2i/D) reaches ~1e5 rad for long contexts, so it and its sine and
// cosine are taken in float64 (fp32 would lose ~1e-2 rad there); the work is a
// few thousand rows, latency- rather than throughput-bound.
#include "common.h"

namespace pvlm {
namespace {

struct RArgs {
  const void* q_in;
  const void* k_in;
  const void* v_in;
  const int32_t* pos;
  const int32_t* ctx_len;
  void* q_out;
  void* k_cache;
  void* v_cache;
  int32_t* status;
  const int32_t* table;  // paged caches: [B][max_pages] pool page per logical page; NULL: padded
  int64_t n_pages;
  int max_pages, shift;
  int64_t n_cap, total;
  double log2_base;
  int B, T, Hq, Hkv, D, s0, s01, mrope;
};

template <typename E>
__device__ __forceinline__ double load_e(const void* p, size_t i) {
  if constexpr (sizeof(E) == 4) return static_cast<const float*>(p)[i];
  else return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
}
template <typename E>
__device__ __forceinline__ void store_e(void* p, size_t i, double x) {
  if constexpr (sizeof(E) == 4) static_cast<float*>(p)[i] = static_cast<float>(x);
  else static_cast<uint16_t*>(p)[i] = f32_to_bf16(static_cast<float>(x));
}

template <typename E>
__global__ void __launch_bounds__(256) rope_append_kernel(RArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= a.total) return;
  const int half = a.D >> 1;
  const int i = (int)(idx % half);
  const int64_t row = idx / half;
  const int heads = a.Hq + 2 * a.Hkv;
  const int h = (int)(row % heads);
  const int64_t bt = row / heads;
  const int t = (int)(bt % a.T);
  const int b = (int)(bt / a.T);
  int ctx = a.ctx_len[b];
  if (ctx < 0 || (int64_t)ctx + a.T > a.n_cap) {
    if (t == 0 && h == 0 && i == 0) dev_flag(a.status, PVLM_DEV_RANGE);
    ctx = ctx < 0 ? 0 : (int)(a.n_cap - a.T);
  }
  const void* src;
  void* dst;
  size_t so, d_off;
  if (h < a.Hq) {
    so = (size_t)((bt * a.Hq + h) * a.D);
    d_off = so;
    src = a.q_in;
    dst = a.q_out;
  } else {
    const int g = h < a.Hq + a.Hkv ? h - a.Hq : h - a.Hq - a.Hkv;
    so = (size_t)((bt * a.Hkv + g) * a.D);
    const int64_t lr = (int64_t)ctx + t;  // logical cache row
    if (a.table) {  // pool [n_pages][Hkv][page][D]
      const int pg = a.table[(size_t)b * a.max_pages + (lr >> a.shift)];
      if (pg < 0 || pg >= a.n_pages) {
        if (i == 0) dev_flag(a.status, PVLM_DEV_RANGE);
        return;
      }
      d_off = (size_t)(((((int64_t)pg * a.Hkv + g) << a.shift) + (lr & ((1 << a.shift) - 1))) * a.D);
    } else {
      d_off = (size_t)((((int64_t)b * a.Hkv + g) * a.n_cap + lr) * a.D);
    }
    const bool is_k = h < a.Hq + a.Hkv;
    src = is_k ? a.k_in : a.v_in;
    dst = is_k ? a.k_cache : a.v_cache;
    if (!is_k) {  // values are appended as they are
      if constexpr (sizeof(E) == 4) {
        static_cast<float*>(dst)[d_off + i] = static_cast<const float*>(src)[so + i];
        static_cast<float*>(dst)[d_off + i + half] = static_cast<const float*>(src)[so + i + half];
      } else {
        static_cast<uint16_t*>(dst)[d_off + i] = static_cast<const uint16_t*>(src)[so + i];
        static_cast<uint16_t*>(dst)[d_off + i + half] =
            static_cast<const uint16_t*>(src)[so + i + half];
      }
      return;
    }
  }
  // the pair's position: one component per section under M-RoPE
  const int axis = a.mrope ? (i < a.s0 ? 0 : (i < a.s01 ? 1 : 2)) : 0;
  const double p = (double)a.pos[((int64_t)axis * a.B + b) * a.T + t];
  const double ang = p * exp2(-2.0 * i / a.D * a.log2_base);
  double sn, cs;
  sincos(ang, &sn, &cs);
  const double x1 = load_e<E>(src, so + i), x2 = load_e<E>(src, so + i + half);
  store_e<E>(dst, d_off + i, x1 * cs - x2 * sn);
  store_e<E>(dst, d_off + i + half, x2 * cs + x1 * sn);
}

}  // namespace
}  // namespace pvlm

using namespace pvlm;

namespace {
pvlm_status rope_run(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D, int64_t n_cap,
                     double base, const int32_t* sections, const int32_t* pos, const void* q_in,
                     const void* k_in, const void* v_in, const int32_t* ctx_len, void* q_out,
                     void* k_cache, void* v_cache, const int32_t* table, int64_t n_pages,
                     int max_pages, int shift, int32_t* status, hipStream_t stream) {
  if (!pos || !q_in || !k_in || !v_in || !ctx_len || !q_out || !k_cache || !v_cache)
    return PVLM_ERR_NULL;
  if (dt != PVLM_F32 && dt != PVLM_BF16) return PVLM_ERR_UNSUPPORTED;
  if (B < 1 || T < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || D < 2 || D % 2 != 0 || D > 1024 ||
      n_cap < T || n_cap > ((int64_t)1 << 30) || !(base > 1.0 && base < 1e300))
    return PVLM_ERR_SHAPE;
  // one thread per rotation pair, in one launch of at most 2^32 - 256 work-items
  const int64_t heads = (int64_t)Hq + 2 * (int64_t)Hkv;
  if (heads > 65536 || (int64_t)B * T * heads * (D / 2) > ((int64_t)1 << 32) - 256)
    return PVLM_ERR_SHAPE;
  RArgs a;
  a.mrope = sections != nullptr;
  if (a.mrope) {
    if (sections[0] < 0 || sections[1] < 0 || sections[2] < 0 ||
        sections[0] + sections[1] + sections[2] != D / 2)
      return PVLM_ERR_SHAPE;
    a.s0 = sections[0];
    a.s01 = sections[0] + sections[1];
  } else {
    a.s0 = a.s01 = D / 2;
  }
  a.q_in = q_in;
  a.k_in = k_in;
  a.v_in = v_in;
  a.pos = pos;
  a.ctx_len = ctx_len;
  a.q_out = q_out;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.status = status;
  a.table = table;
  a.n_pages = n_pages;
  a.max_pages = max_pages;
  a.shift = shift;
  a.n_cap = n_cap;
  a.log2_base = std::log2(base);
  a.B = B;
  a.T = T;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.D = D;
  a.total = (int64_t)B * T * heads * (D / 2);
  const unsigned grid = (unsigned)((a.total + 255) / 256);
  if (dt == PVLM_F32)
    hipLaunchKernelGGL(rope_append_kernel<float>, dim3(grid), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(rope_append_kernel<uint16_t>, dim3(grid), dim3(256), 0, stream, a);
  PVLM_LAUNCHED();
  return PVLM_OK;
}
}  // namespace

extern "C" pvlm_status pvlm_rope_append(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                        int64_t n_cap, double base, const int32_t* sections,
                                        const int32_t* pos, const void* q_in, const void* k_in,
                                        const void* v_in, const int32_t* ctx_len, void* q_out,
                                        void* k_cache, void* v_cache, int32_t* status,
                                        hipStream_t stream) {
  return rope_run(dt, B, T, Hq, Hkv, D, n_cap, base, sections, pos, q_in, k_in, v_in, ctx_len,
                  q_out, k_cache, v_cache, nullptr, 0, 0, 0, status, stream);
}

extern "C" pvlm_status pvlm_rope_append_paged(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                              int page_size, int max_pages, int64_t n_pages,
                                              double base, const int32_t* sections,
                                              const int32_t* pos, const void* q_in,
                                              const void* k_in, const void* v_in,
                                              const int32_t* page_table, const int32_t* ctx_len,
                                              void* q_out, void* k_pool, void* v_pool,
                                              int32_t* status, hipStream_t stream) {
  if (!page_table) return PVLM_ERR_NULL;
  const int shift = page_shift_of(page_size);
  if (shift < 0 || max_pages < 1 || n_pages < 1 || n_pages > INT32_MAX) return PVLM_ERR_SHAPE;
  return rope_run(dt, B, T, Hq, Hkv, D, (int64_t)max_pages << shift, base, sections, pos, q_in,
                  k_in, v_in, ctx_len, q_out, k_pool, v_pool, page_table, n_pages, max_pages,
                  shift, status, stream);
}
