// Compact draft cache gather (gfx950): the draft holds [V*, X] (ParallelVLM
// Sec. 4.2, Stage I): the kept visual rows in ascending index order followed
// by the text (tail) rows, for every layer and KV head, K and V alike.  Pure
// bit copy with 16-byte loads/stores; a cache row is D * elem bytes (256 B for
// bf16, D = 128), i.e. 16 lanes per row.  One launch covers all layers of a
// stacked cache.
#include "common.h"

namespace pvlm {
namespace {

struct GArgs {
  const uint4* k;
  const uint4* v;
  const int32_t* idx;
  const int32_t* kk;
  const int32_t* tail_begin;
  const int32_t* tail_len;
  uint4* kd;
  uint4* vd;
  int32_t* status;
  const int32_t* table;  // paged source: [B][max_pages] pool page per logical page; NULL: padded
  int64_t n_pages;
  int max_pages, shift;
  int64_t n_cap, dst_cap;
  int B, Hkv, k_cap, row_vec;  // row_vec = 16-byte vectors per cache row
};

// grid: x = dst-row blocks, y = KV head, z = layer * B + batch.
__global__ void __launch_bounds__(256) gather_kernel(GArgs a) {
  const int b = blockIdx.z % a.B, g = blockIdx.y;
  const size_t lb = blockIdx.z;  // layer * B + b
  const int rows_per_block = 256 / a.row_vec;
  const int r = blockIdx.x * rows_per_block + threadIdx.x / a.row_vec;
  const int c = threadIdx.x % a.row_vec;
  int kb = a.kk[b], tb = a.tail_begin[b], tl = a.tail_len[b];
  bool bad = false;
  if (kb < 0 || kb > a.k_cap) {
    bad = true;
    kb = kb < 0 ? 0 : a.k_cap;
  }
  if (kb > a.dst_cap) {
    bad = true;
    kb = (int)a.dst_cap;
  }
  if (tb < 0 || tb > a.n_cap) {
    bad = true;
    tb = tb < 0 ? 0 : (int)a.n_cap;
  }
  if (tl < 0 || (int64_t)tb + tl > a.n_cap || (int64_t)kb + tl > a.dst_cap) {
    bad = true;
    int64_t lim = a.n_cap - tb < a.dst_cap - kb ? a.n_cap - tb : a.dst_cap - kb;
    tl = tl < 0 ? 0 : (int)(tl < lim ? tl : lim);
  }
  if (bad && blockIdx.x == 0 && g == 0 && lb == (size_t)b && threadIdx.x == 0)
    dev_flag(a.status, PVLM_DEV_RANGE);
  if (r >= kb + tl) return;
  int src;
  if (r < kb) {
    src = a.idx[(size_t)b * a.k_cap + r];
    if (src < 0 || src >= a.n_cap) {
      if (c == 0 && lb == (size_t)b) dev_flag(a.status, PVLM_DEV_RANGE);
      return;
    }
  } else {
    src = tb + (r - kb);
  }
  const size_t bg = lb * a.Hkv + g;
  size_t si;
  if (a.table) {  // pool [n_layers][n_pages][Hkv][page][D]; one table serves every layer
    const int pg = a.table[(size_t)b * a.max_pages + (src >> a.shift)];
    if (pg < 0 || pg >= a.n_pages) {
      if (c == 0) dev_flag(a.status, PVLM_DEV_RANGE);
      return;
    }
    const size_t l = lb / a.B;
    si = ((((l * a.n_pages + pg) * a.Hkv + g) << a.shift) + (src & ((1 << a.shift) - 1))) *
             a.row_vec + c;
  } else {
    si = (bg * a.n_cap + src) * a.row_vec + c;
  }
  const size_t di = (bg * a.dst_cap + r) * a.row_vec + c;
  // a pure stream: every source row is read once and every destination row
  // written once, so both go through the non-temporal cache policy
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 kv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a.k) + si);
  const u32x4 vv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a.v) + si);
  __builtin_nontemporal_store(kv, reinterpret_cast<u32x4*>(a.kd) + di);
  __builtin_nontemporal_store(vv, reinterpret_cast<u32x4*>(a.vd) + di);
}

}  // namespace
}  // namespace pvlm

using namespace pvlm;

namespace {
pvlm_status gather_run(pvlm_dtype dt, int n_layers, int B, int Hkv, int D, int64_t n_cap,
                       const void* k_cache, const void* v_cache, const int32_t* table,
                       int64_t n_pages, int max_pages, int shift, const int32_t* idx,
                       const int32_t* k, int32_t k_cap, const int32_t* tail_begin,
                       const int32_t* tail_len, int64_t dst_cap, void* k_dst, void* v_dst,
                       int32_t* status, hipStream_t stream) {
  if (!k_cache || !v_cache || !k || !tail_begin || !tail_len || !k_dst || !v_dst)
    return PVLM_ERR_NULL;
  if (k_cap > 0 && !idx) return PVLM_ERR_NULL;
  if (dt != PVLM_F32 && dt != PVLM_BF16) return PVLM_ERR_UNSUPPORTED;
  if (n_layers < 1 || B < 1 || Hkv < 1 || n_cap < 1 || k_cap < 0 || dst_cap < 0)
    return PVLM_ERR_SHAPE;
  if (n_cap > ((int64_t)1 << 30) || dst_cap > ((int64_t)1 << 30) || (int64_t)n_layers * B > 65535 ||
      Hkv > 65535)
    return PVLM_ERR_SHAPE;
  const int esize = dt == PVLM_F32 ? 4 : 2;
  const int row_bytes = D * esize;
  if (D < 1 || row_bytes % 16 != 0 || row_bytes / 16 > 256 || 256 % (row_bytes / 16) != 0)
    return PVLM_ERR_UNSUPPORTED;
  if (dst_cap == 0) return PVLM_OK;
  GArgs a;
  a.k = static_cast<const uint4*>(k_cache);
  a.v = static_cast<const uint4*>(v_cache);
  a.idx = idx;
  a.kk = k;
  a.tail_begin = tail_begin;
  a.tail_len = tail_len;
  a.kd = static_cast<uint4*>(k_dst);
  a.vd = static_cast<uint4*>(v_dst);
  a.status = status;
  a.table = table;
  a.n_pages = n_pages;
  a.max_pages = max_pages;
  a.shift = shift;
  a.n_cap = n_cap;
  a.dst_cap = dst_cap;
  a.B = B;
  a.Hkv = Hkv;
  a.k_cap = k_cap;
  a.row_vec = row_bytes / 16;
  const int rows_per_block = 256 / a.row_vec;
  const int64_t xb = (dst_cap + rows_per_block - 1) / rows_per_block;
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)xb, Hkv, n_layers * B), dim3(256), 0, stream, a);
  PVLM_LAUNCHED();
  return PVLM_OK;
}
}  // namespace

extern "C" pvlm_status pvlm_gather_kv(pvlm_dtype dt, int n_layers, int B, int Hkv, int D,
                                      int64_t n_cap, const void* k_cache, const void* v_cache,
                                      const int32_t* idx, const int32_t* k, int32_t k_cap,
                                      const int32_t* tail_begin, const int32_t* tail_len,
                                      int64_t dst_cap, void* k_dst, void* v_dst, int32_t* status,
                                      hipStream_t stream) {
  return gather_run(dt, n_layers, B, Hkv, D, n_cap, k_cache, v_cache, nullptr, 0, 0, 0, idx, k,
                    k_cap, tail_begin, tail_len, dst_cap, k_dst, v_dst, status, stream);
}

extern "C" pvlm_status pvlm_gather_kv_paged(pvlm_dtype dt, int n_layers, int B, int Hkv, int D,
                                            int page_size, int max_pages, int64_t n_pages,
                                            const void* k_pool, const void* v_pool,
                                            const int32_t* page_table, const int32_t* idx,
                                            const int32_t* k, int32_t k_cap,
                                            const int32_t* tail_begin, const int32_t* tail_len,
                                            int64_t dst_cap, void* k_dst, void* v_dst,
                                            int32_t* status, hipStream_t stream) {
  if (!page_table) return PVLM_ERR_NULL;
  const int shift = page_shift_of(page_size);
  if (shift < 0 || max_pages < 1 || n_pages < 1 || n_pages > INT32_MAX) return PVLM_ERR_SHAPE;
  return gather_run(dt, n_layers, B, Hkv, D, (int64_t)max_pages << shift, k_pool, v_pool,
                    page_table, n_pages, max_pages, shift, idx, k, k_cap, tail_begin, tail_len,
                    dst_cap, k_dst, v_dst, status, stream);
}
