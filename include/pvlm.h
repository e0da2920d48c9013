/*
 * pvlm.h -- C ABI of the ParallelVLM verify + UV-Prune + accept hot path
 * on AMD Instinct MI355X (gfx950).
 *
 * The calls follow the paper's statement of the problem (ParallelVLM,
 * arXiv 2603.19610):
 *   pvlm_rope_append    rotary embedding (1-D or M-RoPE) of the verify rows and
 *                       their append to the KV cache
 *   pvlm_verify_attn    target verification forward over the video KV cache
 *                       (Sec. 2.2; Sec. 4.2 Parallel Decoding), fused with the
 *                       per-token verifier attention mass (Sec. 3, Challenge 2)
 *   pvlm_*_paged        verify, rope-append and gather over a paged cache
 *   pvlm_verify_attn_noalloc  verify with the library's fixed scratch
 *   pvlm_uvprune_score  UV-Prune variation score, Eq. (average_similarity),
 *                       over Eq. (similarity) or over a per-layer criterion;
 *                       pvlm_uvprune_criterion_cossim one layer of it, and
 *                       pvlm_prefill_epilogue_cossim that layer's criterion
 *                       fused into the prefill layer's residual add
 *   pvlm_topk_select    Eq. (topk_selection): keep the top 1 - alpha fraction;
 *                       pvlm_uvprune_topk_mass with the MASS score in one launch
 *   pvlm_gather_kv      the draft's compact cache [V*, X] (Sec. 4.2, Stage I)
 *   pvlm_spec_accept    speculative-sampling accept/reject (Sec. 2.2) with the
 *                       bonus token of Suppl. B
 *   pvlm_set_stream_cu_budget  compute-unit budgets, so the draft's and the
 *                       target's waiting kernels can run at once (Stage II)
 *   pvlm_window_size,   host-only: the draft window gamma = c* of Eq. (Prefill)
 *   pvlm_speedup        and the speedup analysis (Thm. paravlm_speedup; the
 *                       supplement's theorems and Lemma 1)
 *   pvlm_pd_*           host-only: the parallel decoding scheduler (pre- and
 *                       post-verify rounds, draft rollback; Suppl. B)
 *
 * Conventions shared by every call
 *   - Every tensor pointer is a caller-owned DEVICE pointer.  The library never
 *     allocates, frees or keeps a pointer past the call.
 *   - Every call is asynchronous on the given stream: no device-wide sync and no
 *     host<->device copy happens inside a call.  Results are valid once the
 *     stream reaches the call's completion.
 *   - Host-side arguments (sizes, capacities, pointer NULL-ness) are validated
 *     before anything is launched; a failing call launches nothing.
 *   - Device-resident sizes (lengths, keep counts) are trusted up to the host
 *     capacities passed alongside them.  A kernel that finds one out of range
 *     clamps it into range (so memory is never touched out of bounds) and, if
 *     `status` is non-NULL, ORs PVLM_DEV_RANGE into *status.
 *   - Outputs must not alias inputs.  Optional outputs may be NULL.
 *   - Calls are re-entrant; a workspace buffer must not be shared by two calls
 *     in flight at the same time.  The library's only mutable state is the
 *     per-stream compute-unit budgets below and the fixed scratch of
 *     pvlm_verify_attn_noalloc.
 *   - Workgroups that wait on each other.  pvlm_verify_attn(_paged), top-k
 *     rows longer than 16384 scores and pvlm_spec_accept split their work
 *     over workgroups of one launch that exchange partial results and wait
 *     for each other (bounded waits: a wait that gives up sets
 *     PVLM_DEV_TIMEOUT, and the results are invalid).  Every workgroup must
 *     therefore be resident at once.  Each call checks before launching that
 *     its grid fits the device (the runtime's occupancy per compute unit
 *     times the compute units it plans for; PVLM_ERR_UNSUPPORTED otherwise).
 *     Eager launches on a stream without a budget are cooperative launches,
 *     whose co-residency the runtime guarantees.  Launches captured into a
 *     graph, and launches on a budgeted stream, are ordinary launches: then
 *     the caller guarantees that no other work holds compute units the call
 *     needs for longer than the call itself runs.  Without budgets that means
 *     the device to itself while such a call runs: no two of these calls in
 *     flight at once on different streams.  Kernels that never wait (rope,
 *     UV-Prune, short top-k rows, gather) and finish on their own may run
 *     beside them: they only delay them.
 *   - Compute-unit budgets (pvlm_set_stream_cu_budget): calls of the waiting
 *     kind on a stream with a budget of C compute units plan their grids for
 *     at most C workgroups.  Streams whose budgets sum to at most the
 *     device's compute units may then run such calls at the same time, since
 *     every workgroup of all of them fits at once (one workgroup per compute
 *     unit at most; budgets are multiples of the XCD count, so a grid spreads
 *     evenly over the XCDs the device deals workgroups to in turn).
 *   - Workspaces: zero-fill a workspace once before its first use.  Its first
 *     1 MiB holds the counters of the waits between workgroups, and every
 *     call leaves them in a consistent state (zero again, or, for verify's
 *     monotonic counters, advanced together), so one buffer (at least as large
 *     as each call requires) serves calls of any kind and shape in sequence.
 *   - Layouts are C-contiguous, innermost index last.  "bf16" is IEEE
 *     bfloat16 stored in 2 bytes.
 */
#ifndef PVLM_H_
#define PVLM_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PVLM_OK = 0,
  PVLM_ERR_NULL = 1,         /* a required pointer is NULL                     */
  PVLM_ERR_SHAPE = 2,        /* inconsistent or out-of-range size argument     */
  PVLM_ERR_UNSUPPORTED = 3,  /* valid request this build does not implement    */
  PVLM_ERR_WORKSPACE = 4,    /* workspace NULL or smaller than required        */
  PVLM_ERR_HIP = 5           /* a HIP call failed; see pvlm_last_hip_error()   */
} pvlm_status;

typedef enum { PVLM_F32 = 0, PVLM_BF16 = 1 } pvlm_dtype;

/* Criterion fed to UV-Prune's variation operator. */
typedef enum {
  PVLM_CRIT_MASS = 0,   /* a precomputed per-layer criterion stack, e.g. the
                           verifier attention mass of layers 0..L            */
  PVLM_CRIT_COSSIM = 1  /* vision-text cosine similarity, Eq. (similarity),
                           computed from layer-wise hidden states            */
} pvlm_crit;

/* Bits ORed into the optional device status word. */
#define PVLM_DEV_RANGE 1    /* a device-resident size or index was out of range */
#define PVLM_DEV_TIMEOUT 2  /* an inter-workgroup wait gave up (results invalid;
                               zero-fill the workspace again before reusing it) */
#define PVLM_DEV_PLACEMENT 4 /* a workgroup ran on another XCD than the launch
                               planned for (results may be invalid)          */

/* Compute-unit budget of `stream` on the current device: cus = 0 removes it
 * (calls then plan for the whole device), otherwise a multiple of the
 * device's XCD count (8 on MI355X) up to its compute units (a budget of all
 * of them is the same as none).  PVLM_ERR_SHAPE for another value.  Set it
 * before the stream's first call and clear it before destroying the stream
 * (budgets are keyed by the stream handle).  pvlm_stream_cu_budget returns
 * the stream's budget, 0 for none. */
pvlm_status pvlm_set_stream_cu_budget(hipStream_t stream, int cus);
int pvlm_stream_cu_budget(hipStream_t stream);

const char* pvlm_status_string(pvlm_status s);
/* Text of the last HIP error seen by a pvlm call on this host thread. */
const char* pvlm_last_hip_error(void);
int pvlm_version(void);

/* ------------------------------------------------------------------------
 * pvlm_verify_attn -- target verify attention with fused attention mass.
 *
 * Defines (Sec. 2.2 verification in one parallel forward; Sec. 4.2 Parallel
 * Decoding): for batch b, query head h (KV head g = floor(h*Hkv/Hq)), verify
 * row t in [0, T): the visible cache rows are i = 0 .. ctx_len[b] + t;
 *   s_i = scale * <q[b,t,h,:], k[b,g,i,:]>,  P_i = softmax_i(s),
 *   out[b,t,h,:] = sum_i P_i v[b,g,i,:],     lse[b,h,t] = log sum_i exp(s_i),
 *   mass[b,i] = sum_{h,t} P_{h,t,i}   (normalised probabilities, summed over
 *                                      every query head and verify row)
 * so sum_i mass[b,i] = Hq*T.  This is the attention criterion of
 * attention-guided pruning (Sec. 3, Challenge 2; Suppl. D).
 *
 *   dt        PVLM_BF16 (bf16 in/out, fp32 accumulate) or PVLM_F32.
 *   T         verify rows = gamma + 1, 1..32.  The last T valid cache rows of
 *             each sequence, [ctx_len[b], ctx_len[b]+T), are the verify block
 *             (causal among themselves).
 *   Hq, Hkv   query / KV heads, Hq % Hkv == 0, (Hq/Hkv)*T <= 640.
 *   D         head dim, 64 or 128.
 *   n_cap     cache capacity in rows (>= max_ctx + T).
 *   max_ctx   host upper bound of every ctx_len[b] (used to plan the launch);
 *             pass n_cap - T when unknown.
 *   scale     softmax scale, normally 1/sqrt(D).
 *   q         [B][T][Hq][D] post-RoPE queries.
 *   k_cache,
 *   v_cache   [B][Hkv][n_cap][D] post-RoPE keys / values.
 *   ctx_len   [B] int32 device array, context rows before the verify block.
 *   out       [B][T][Hq][D], dtype dt.
 *   mass      [B][n_cap] fp32 or NULL; rows >= ctx_len[b]+T are written 0.
 *   lse       [B][Hq][T] fp32 (natural log) or NULL.
 *   ws        device workspace of >= pvlm_verify_attn_workspace_size() bytes
 *             (see "Workspaces" above).
 *   status    optional device int32, see PVLM_DEV_*.
 * ---------------------------------------------------------------------- */
size_t pvlm_verify_attn_workspace_size(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                       int64_t n_cap, int64_t max_ctx);
pvlm_status pvlm_verify_attn(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                             int64_t n_cap, int64_t max_ctx, float scale,
                             const void* q, const void* k_cache, const void* v_cache,
                             const int32_t* ctx_len, void* out, float* mass, float* lse,
                             void* ws, size_t ws_bytes, int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_verify_attn_paged -- pvlm_verify_attn over a paged KV cache: the same
 * operation (Sec. 2.2 verification forward; attention mass of Sec. 3,
 * Challenge 2), with every cache row read through a page table instead of a
 * padded [B][Hkv][n_cap][D] slab, so ragged sequences share one pool without
 * padding.  Logical row i of sequence b lives in pool page
 * page_table[b][i / page_size] at row i % page_size of that page.
 *   dt          PVLM_BF16 only (PVLM_ERR_UNSUPPORTED otherwise).
 *   page_size   rows per page: a power of two in [32, 2^20] (PVLM_ERR_SHAPE).
 *   max_pages   page-table columns; the logical capacity is
 *               n_cap = max_pages * page_size (<= 2^30).
 *   n_pages     pool pages, 1 .. 2^31 - 1.
 *   k_pool,
 *   v_pool      [n_pages][Hkv][page_size][D] bf16 (one page holds page_size
 *               consecutive rows of every KV head).
 *   page_table  [B][max_pages] int32 device.  Only the entries of pages that
 *               hold rows < ctx_len[b] + T are read; an entry outside
 *               [0, n_pages) among them is clamped into the pool for the
 *               read (so no access leaves it) and flagged PVLM_DEV_RANGE.
 *   mass        [B][n_cap] fp32 or NULL, indexed by logical row.
 *   ws          >= pvlm_verify_attn_workspace_size(dt, B, T, Hq, Hkv, D,
 *               n_cap, max_ctx) bytes.
 * Every other argument, limit and error is that of pvlm_verify_attn.  With
 * equal max_ctx the call runs the padded call's launch plan and arithmetic,
 * so its results equal the padded call's bit for bit.
 * ---------------------------------------------------------------------- */
pvlm_status pvlm_verify_attn_paged(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                   int page_size, int max_pages, int64_t n_pages,
                                   int64_t max_ctx, float scale, const void* q,
                                   const void* k_pool, const void* v_pool,
                                   const int32_t* page_table, const int32_t* ctx_len, void* out,
                                   float* mass, float* lse, void* ws, size_t ws_bytes,
                                   int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_verify_attn_noalloc -- pvlm_verify_attn without a workspace argument,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, and harnesses that forbid allocation.  It
 * allocates nothing (no hipMalloc / hipFree, no allocating library call):
 * its scratch is a fixed device array inside the library, one per GPU,
 * held until the process ends.  The caller still provides q, the caches,
 * ctx_len, out and the optional mass / lse / status, with the meaning,
 * layout and error behaviour of pvlm_verify_attn.
 *   - Limit: the call needs pvlm_verify_attn_workspace_size() bytes of that
 *     scratch; a request beyond pvlm_verify_attn_noalloc_max_bytes()
 *     (32 MiB, which covers batch 4 at 33K tokens and 131K-token caches at
 *     Hkv = 8) returns PVLM_ERR_WORKSPACE and launches nothing.
 *   - Every call on one GPU shares that GPU's scratch: calls that overlap
 *     on one GPU (on different streams, or a replayed graph beside another
 *     call) race and give invalid results; serialise them.
 *   - The first call on a GPU also clears the scratch's synchronisation
 *     words with a small fill kernel on `stream` (never a memset, so a
 *     capturing caller records no memset node).
 * ---------------------------------------------------------------------- */
size_t pvlm_verify_attn_noalloc_max_bytes(void);
pvlm_status pvlm_verify_attn_noalloc(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                     int64_t n_cap, int64_t max_ctx, float scale, const void* q,
                                     const void* k_cache, const void* v_cache,
                                     const int32_t* ctx_len, void* out, float* mass, float* lse,
                                     int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_rope_append -- rotary embedding of the verify rows and their append to
 * the cache.  The target verifies the T = gamma + 1 speculated positions in
 * one forward (Sec. 2.2; Sec. 4.2, Parallel Decoding); pvlm_verify_attn reads
 * post-rotation queries and a cache whose rows ctx_len[b] .. ctx_len[b]+T-1
 * hold the verify rows.  This call produces both:
 *   q_out[b,t,h]                 = rot(q_in[b,t,h],  positions of (b,t))
 *   k_cache[b,g,ctx_len[b]+t]    = rot(k_in[b,t,g],  positions of (b,t))
 *   v_cache[b,g,ctx_len[b]+t]    = v_in[b,t,g]       (bit copy)
 * Every other cache row is left untouched.  rot pairs element i with
 * i + D/2 (rotate-half): (x_i, x_{i+D/2}) turns by the angle
 * p_i * base^(-2i/D), i < D/2.  1-D RoPE (LLaVA-OneVision's Qwen2 decoder):
 * sections = NULL, pos [B][T], p_i = pos[b][t].  M-RoPE (Qwen2.5-VL's decoder,
 * Qwen2-VL Sec. 2.1): sections = host int32[3] (s0, s1, s2) with
 * s0 + s1 + s2 = D/2, e.g. (16, 24, 24) at D = 128; pos [3][B][T] holds the
 * temporal, height and width components; pairs i < s0 take the temporal one,
 * s0 <= i < s0 + s1 the height one and the rest the width one.  Angles and
 * their sines and cosines are taken in float64; results are rounded once to
 * the storage type.
 *   q_in, q_out [B][T][Hq][D]; k_in, v_in [B][T][Hkv][D];
 *   k_cache, v_cache [B][Hkv][n_cap][D]; pos, ctx_len int32 device.
 * q_out may equal q_in (each element is read before it is written by the same
 * thread); no other argument may alias another.  A ctx_len[b] outside
 * [0, n_cap - T] is clamped into it and flagged PVLM_DEV_RANGE.
 * Errors: PVLM_ERR_NULL for a NULL pointer (sections excepted);
 * PVLM_ERR_SHAPE for a size < 1, Hq not a multiple of Hkv, D odd or > 1024,
 * n_cap < T or > 2^30, base not finite and > 1, sections that do not sum
 * to D/2, Hq + 2*Hkv > 65536, or more than 2^32 - 256 rotation pairs
 * (B*T*(Hq+2*Hkv)*D/2: one launch, one work-item per pair);
 * PVLM_ERR_UNSUPPORTED for another dtype.
 * ---------------------------------------------------------------------- */
pvlm_status pvlm_rope_append(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D, int64_t n_cap,
                             double base, const int32_t* sections, const int32_t* pos,
                             const void* q_in, const void* k_in, const void* v_in,
                             const int32_t* ctx_len, void* q_out, void* k_cache, void* v_cache,
                             int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_rope_append_paged -- pvlm_rope_append into a paged cache: k_pool /
 * v_pool [n_pages][Hkv][page_size][D] and page_table [B][max_pages] as for
 * pvlm_verify_attn_paged (logical capacity n_cap = max_pages * page_size).
 * The row of verify position t of sequence b goes to page
 * page_table[b][(ctx_len[b] + t) / page_size], row (ctx_len[b] + t) %
 * page_size; a row whose page entry lies outside [0, n_pages) is not written
 * and is flagged PVLM_DEV_RANGE.  Other arguments, limits and errors are
 * those of pvlm_rope_append; page_size and the page counts follow
 * pvlm_verify_attn_paged (PVLM_ERR_SHAPE otherwise).
 * ---------------------------------------------------------------------- */
pvlm_status pvlm_rope_append_paged(pvlm_dtype dt, int B, int T, int Hq, int Hkv, int D,
                                   int page_size, int max_pages, int64_t n_pages, double base,
                                   const int32_t* sections, const int32_t* pos, const void* q_in,
                                   const void* k_in, const void* v_in, const int32_t* page_table,
                                   const int32_t* ctx_len, void* q_out, void* k_pool,
                                   void* v_pool, int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_uvprune_score -- UV-Prune score, Eq. (average_similarity):
 *   score[b,i] = sum_{j<n[b]} sum_{l=1..L} (S^l_ij - S^{l-1}_ij)   (COSSIM)
 *   score[b,i] = sum_{l=1..L} (c^l_i - c^{l-1}_i)                (MASS)
 * for visual tokens i < m[b]; score[b, i >= m[b]] is written 0.  S^l is the
 * cosine similarity of Eq. (similarity) between hidden states at layer l
 * (layer 0 = decoder input), 0 when either vector has zero norm.  Both sums
 * telescope exactly, so only layers 0 and L are read.
 *
 *   crit        PVLM_CRIT_MASS or PVLM_CRIT_COSSIM.
 *   L           early layers, >= 1.
 *   m_cap       visual-row capacity; m: [B] int32 device, m[b] <= m_cap.
 *   crit_stack  MASS: [L+1][B][m_cap] fp32 (NULL for COSSIM).
 *   hdt, Dh     COSSIM: hidden-state dtype and hidden size (multiple of 8).
 *   n_cap,n_txt COSSIM: text-row capacity and [B] int32 device text counts.
 *   hs_vis      COSSIM: [L+1][B][m_cap][Dh] visual hidden states.
 *   hs_txt      COSSIM: [L+1][B][n_cap][Dh] text hidden states.
 *   score       [B][m_cap] fp32 output.
 *   ws          COSSIM only: >= pvlm_uvprune_workspace_size() bytes.
 * COSSIM forms the text directions u = sum_j ht_j/|ht_j| and the dot
 * products <hv_i, u> in float64 (inputs convert exactly); the visual norms
 * and the final quotient are fp32.
 * Limits, checked before any launch: m_cap <= 2^30 (PVLM_ERR_SHAPE); MASS:
 * B * m_cap rounded up to 256 <= 2^32 - 256 (one work-item per score in one
 * launch; PVLM_ERR_SHAPE); COSSIM: Dh <= 8192 (two float64 directions in the
 * visual kernel's LDS; PVLM_ERR_UNSUPPORTED), 2*B <= 65535 and
 * 64 * 2 * B * n_cap (one wave per text row of both layers, rounded up to
 * 256) <= 2^32 - 256 (PVLM_ERR_SHAPE).
 * ---------------------------------------------------------------------- */
size_t pvlm_uvprune_workspace_size(pvlm_crit crit, int B, int Dh, int64_t n_cap);
pvlm_status pvlm_uvprune_score(pvlm_crit crit, int B, int L, int64_t m_cap, const int32_t* m,
                               const float* crit_stack, pvlm_dtype hdt, int Dh, int64_t n_cap,
                               const int32_t* n_txt, const void* hs_vis, const void* hs_txt,
                               float* score, void* ws, size_t ws_bytes, int32_t* status,
                               hipStream_t stream);

/* One layer of the COSSIM criterion, c[b,i] = sum_{j<n[b]} cos(hv[b,i], ht[b,j])
 * (Eq. similarity summed over text tokens), for streaming use: a caller can
 * write c^0 and c^L into a criterion stack and call pvlm_uvprune_score(MASS).
 *   hs_vis [B][m_cap][Dh], hs_txt [B][n_cap][Dh]; crit_out [B][m_cap] fp32. */
pvlm_status pvlm_uvprune_criterion_cossim(int B, int64_t m_cap, const int32_t* m, pvlm_dtype hdt,
                                          int Dh, int64_t n_cap, const int32_t* n_txt,
                                          const void* hs_vis, const void* hs_txt, float* crit_out,
                                          void* ws, size_t ws_bytes, int32_t* status,
                                          hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_prefill_epilogue_cossim -- the UV-Prune criterion fused into a prefill
 * layer's epilogue (Sec. 4.1 defines the criterion on the early layers'
 * hidden states; Sec. 4.2 computes it while the target prefills).  The
 * epilogue's residual add and the criterion of its result in one pass over
 * the rows:
 *   vis_out[b,i] = vis_prev[b,i] + vis_delta[b,i]   i < m[b]
 *   txt_out[b,j] = txt_prev[b,j] + txt_delta[b,j]   j < n_txt[b]
 * (the sum taken in fp32 and rounded once to hdt; rows past m[b] / n_txt[b]
 * are not written), then, from those stored values,
 *   crit_out[b,i] = sum_{j<n_txt[b]} cos(vis_out[b,i], txt_out[b,j]),
 * 0 past m[b]: what pvlm_uvprune_criterion_cossim gives on the outputs, bit
 * for bit, without reading them again.  Called at layers 0 and L, it yields
 * the two criteria whose difference is the score (pvlm_uvprune_score, MASS,
 * over the stack [c^0, c^L]).
 *   vis_* [B][m_cap][Dh], txt_* [B][n_cap][Dh] in hdt; an output may be its
 *   prev (in place); crit_out [B][m_cap] fp32; ws as for
 *   pvlm_uvprune_criterion_cossim (pvlm_uvprune_workspace_size(COSSIM, B,
 *   Dh, n_cap) bytes).  Sizes, limits and errors are those of
 *   pvlm_uvprune_criterion_cossim.
 * ---------------------------------------------------------------------- */
pvlm_status pvlm_prefill_epilogue_cossim(int B, int64_t m_cap, const int32_t* m, int64_t n_cap,
                                         const int32_t* n_txt, pvlm_dtype hdt, int Dh,
                                         const void* vis_prev, const void* vis_delta,
                                         void* vis_out, const void* txt_prev,
                                         const void* txt_delta, void* txt_out, float* crit_out,
                                         void* ws, size_t ws_bytes, int32_t* status,
                                         hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_topk_select -- Eq. (topk_selection).  For each b keep the k[b]
 * visual tokens of largest score[b, 0..m[b]) (k[b] = floor(m[b]*(1-alpha)),
 * Sec. 4.2), ranking larger scores first, the lower index first among equal
 * scores, -0.0 equal to +0.0 and NaN below every number.  The kept indices
 * are written in ascending order to idx[b, 0..k[b]) and idx[b, k[b]..k_cap)
 * is set to -1.  k[b] = 0 is legal (alpha = 1).
 *   score [B][m_cap] fp32; m, k: [B] int32 device; idx [B][k_cap] int32.
 * Rows of up to 16384 scores (m_cap <= 16384) are selected by one workgroup
 * each and need no workspace (pvlm_topk_workspace_size returns 0, ws may be
 * NULL).  Longer rows are split over several workgroups of one co-resident
 * launch that exchange digit histograms and counts through `ws`
 * (pvlm_topk_workspace_size bytes, zero-filled before first use, reusable by
 * later calls on the stream); then B may not exceed the device's compute
 * units (PVLM_ERR_UNSUPPORTED).
 * ---------------------------------------------------------------------- */
size_t pvlm_topk_workspace_size(int B, int64_t m_cap);
pvlm_status pvlm_topk_select(int B, int64_t m_cap, const int32_t* m, const int32_t* k,
                             int32_t k_cap, const float* score, int32_t* idx, void* ws,
                             size_t ws_bytes, int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_uvprune_topk_mass -- the MASS form of pvlm_uvprune_score followed by
 * pvlm_topk_select, in one launch: Eq. (average_similarity) over a criterion
 * stack, score[b,i] = crit_stack[L][b][i] - crit_stack[0][b][i] (one fp32
 * subtraction, as pvlm_uvprune_score(MASS) rounds it), then Eq.
 * (topk_selection) over those scores.  The kept indices equal those of the
 * two calls bit for bit.
 *   crit_stack [L+1][B][m_cap] fp32, L >= 1; m, k [B] int32 device;
 *   score      [B][m_cap] fp32 output or NULL (written as pvlm_uvprune_score
 *              writes it, 0 past m[b]);
 *   idx        [B][k_cap] int32 output, as pvlm_topk_select (may be NULL
 *              when k_cap = 0: then only the scores are written).
 * Workspace, limits and errors are pvlm_topk_select's
 * (pvlm_topk_workspace_size(B, m_cap)); PVLM_ERR_SHAPE also for L < 1.
 * ---------------------------------------------------------------------- */
pvlm_status pvlm_uvprune_topk_mass(int B, int L, int64_t m_cap, const int32_t* m,
                                   const float* crit_stack, const int32_t* k, int32_t k_cap,
                                   float* score, int32_t* idx, void* ws, size_t ws_bytes,
                                   int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_gather_kv -- compact draft cache (Sec. 4.2 Stage I: the draft holds
 * [V*, X]).  For every layer l, batch b and KV head g:
 *   dst[l,b,g,r]      = src[l,b,g,idx[b,r]]             r < k[b]
 *   dst[l,b,g,k[b]+r] = src[l,b,g,tail_begin[b]+r]      r < tail_len[b]
 * for both K and V; rows keep their original RoPE rotation.  Rows past
 * k[b]+tail_len[b] are left untouched.  One kept set serves every layer, so
 * a stacked cache is gathered in one call (n_layers = 1 for a single layer).
 *   k_cache, v_cache [n_layers][B][Hkv][n_cap][D];
 *   k_dst, v_dst     [n_layers][B][Hkv][dst_cap][D];
 *   idx [B][k_cap] int32 (entries < k[b] must lie in [0, n_cap); an entry
 *   outside that range is skipped and flagged);
 *   k, tail_begin, tail_len: [B] int32 device.  n_layers * B <= 65535.
 * ---------------------------------------------------------------------- */
pvlm_status pvlm_gather_kv(pvlm_dtype dt, int n_layers, int B, int Hkv, int D, int64_t n_cap,
                           const void* k_cache, const void* v_cache, const int32_t* idx,
                           const int32_t* k, int32_t k_cap, const int32_t* tail_begin,
                           const int32_t* tail_len, int64_t dst_cap, void* k_dst, void* v_dst,
                           int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_gather_kv_paged -- pvlm_gather_kv from a paged cache into the compact
 * (padded) draft cache of Sec. 4.2, Stage I.  Source row src of sequence b,
 * layer l, KV head g is k_pool[l][page_table[b][src / page_size]][g]
 * [src % page_size] (likewise V); one page table serves every layer.
 *   k_pool, v_pool [n_layers][n_pages][Hkv][page_size][D];
 *   page_table [B][max_pages] int32 device, n_cap = max_pages * page_size
 *   bounds idx and tail_begin + tail_len as in pvlm_gather_kv;
 *   k_dst, v_dst [n_layers][B][Hkv][dst_cap][D].
 * A row whose page entry lies outside [0, n_pages) is skipped and flagged
 * PVLM_DEV_RANGE.  Other arguments, limits and errors are those of
 * pvlm_gather_kv; page_size and the page counts follow
 * pvlm_verify_attn_paged (PVLM_ERR_SHAPE otherwise).
 * ---------------------------------------------------------------------- */
pvlm_status pvlm_gather_kv_paged(pvlm_dtype dt, int n_layers, int B, int Hkv, int D,
                                 int page_size, int max_pages, int64_t n_pages,
                                 const void* k_pool, const void* v_pool,
                                 const int32_t* page_table, const int32_t* idx, const int32_t* k,
                                 int32_t k_cap, const int32_t* tail_begin,
                                 const int32_t* tail_len, int64_t dst_cap, void* k_dst,
                                 void* v_dst, int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------------
 * pvlm_spec_accept -- speculative-sampling accept/reject (Sec. 2.2) with the
 * bonus token after full acceptance (Suppl. B).  With p_t = softmax(
 * target_logits[b,t]/temperature) and q_t = softmax(draft_logits[b,t]/
 * temperature) (float64, maximum subtracted first):
 *   draft token x_t is accepted iff u_accept[b,t] * q_t(x_t) < p_t(x_t),
 *   scanning t = 0..gamma-1 and stopping at the first rejection a;
 *   n_accepted[b] = a (= gamma if none rejected);
 *   next_token[b] is drawn by inverse CDF (ascending vocabulary order, first
 *   y whose cumulative mass exceeds u_sample[b] * total) from
 *   max(0, p_a - q_a) after a rejection (from p_a if that is all zero), or
 *   from p_gamma (the bonus) after full acceptance.
 * temperature == 0 is greedy: accept iff x_t is the target argmax (lowest
 * index on ties) and next_token is the target argmax at position a.
 * The library draws no random numbers; decisions are taken in float64.
 *   draft_logits [B][gamma][V] fp32, target_logits [B][gamma+1][V] fp32
 *   (finite or -inf, at least one finite per row), draft_tokens [B][gamma],
 *   u_accept [B][gamma] f64 in [0,1), u_sample [B] f64 in [0,1).
 *   near_tie (nullable) [B]: 1 when a decision or the draw fell within 1e-9
 *   (relative) of its boundary, where another summation order could flip it.
 * Limits: B <= 256, gamma <= 32, V <= 1048576 (PVLM_ERR_UNSUPPORTED).  The
 * workgroups of the one launch exchange partial sums through `ws`
 * (pvlm_spec_accept_workspace_size bytes, zero-filled before first use).
 * ---------------------------------------------------------------------- */
size_t pvlm_spec_accept_workspace_size(int B, int gamma, int V);
pvlm_status pvlm_spec_accept(int B, int gamma, int V, float temperature,
                             const float* draft_logits, const float* target_logits,
                             const int32_t* draft_tokens, const double* u_accept,
                             const double* u_sample, int32_t* n_accepted, int32_t* next_token,
                             int32_t* near_tie, void* ws, size_t ws_bytes, int32_t* status,
                             hipStream_t stream);

/* ------------------------------------------------------------------------
 * Window size and speedup model (host-only arithmetic: no device pointer, no
 * stream, no GPU needed).  Times are per generated token in units of t, the
 * draft's single forward time T_q; the target's verification forward is
 * T_p = c t.  tau is the per-token acceptance rate.
 *
 * pvlm_speedup fills every quantity of the paper's speedup analysis for one
 * (c, tau, gamma):
 *   t_sd_ideal      (gamma + c) / (gamma + 1)          Suppl. Thm. Vanilla SD (Ideal)
 *   t_psd_ideal     max(gamma, c) / gamma              Suppl. Thm. Parallel SD (Ideal)
 *   t_sd            (gamma + c) / (tau gamma + 1)      Suppl. Thm. Vanilla SD (Practical)
 *   t_psd           max(gamma, c) / (tau gamma)        Suppl. Thm. Parallel SD (Practical);
 *                                                      at gamma = c its speedup is
 *                                                      Thm. (paravlm_speedup), tau c*
 *   expected_accepted  E[X] = tau (1 - tau^gamma) / (1 - tau), gamma at tau = 1
 *                      (Suppl. Lemma 1; X is the accepted prefix of a window)
 *   expected_total  (1 + tau^gamma) E[X], the tokens of the two rounds in the
 *                   proof of Suppl. Thm. Parallel SD (with Rollback)
 *   t_psd_rollback  2 max(gamma, c) / expected_total   (same theorem)
 *   v_*             c / t_*: speedup against target-only decoding
 * A per-token time that is unbounded (tau = 0 for the parallel forms) is
 * HUGE_VAL and its speedup 0.
 * Errors: PVLM_ERR_NULL if out is NULL; PVLM_ERR_SHAPE unless c is finite and
 * > 0, 0 <= tau <= 1 and 1 <= gamma <= 2^20.
 *
 * pvlm_window_size: Eq. (Prefill), gamma = c* = T_p / T_q(alpha) as an
 * integer in [1, gamma_max].  T_p, T_q: measured forward times (any one unit,
 * finite, > 0).  The quotient is first taken as the integer it lies within
 * 1e-9 (relative) of, if any.  Rounding (Suppl. "Window Size Selection"):
 *   PVLM_ROUND_DOWN / PVLM_ROUND_UP / PVLM_ROUND_NEAREST (halves up);
 *   PVLM_ROUND_BEST: the gamma of largest t_psd_rollback speedup at this
 *   tau (0 < tau <= 1), the smaller gamma on ties; it is always the
 *   rounded-down or rounded-up ratio.  tau is ignored by the other modes.
 * *gamma receives the window, *c_out (nullable) the unrounded T_p / T_q.
 * Errors: PVLM_ERR_NULL if gamma is NULL; PVLM_ERR_SHAPE for a time that is
 * not finite and > 0, gamma_max outside [1, 2^20], an unknown rounding mode,
 * or PVLM_ROUND_BEST with tau outside (0, 1].
 * ---------------------------------------------------------------------- */
typedef enum {
  PVLM_ROUND_DOWN = 0,
  PVLM_ROUND_UP = 1,
  PVLM_ROUND_NEAREST = 2,
  PVLM_ROUND_BEST = 3
} pvlm_round;

typedef struct {
  double t_sd_ideal, t_psd_ideal, t_sd, t_psd, t_psd_rollback;
  double v_sd_ideal, v_psd_ideal, v_sd, v_psd, v_psd_rollback;
  double expected_accepted, expected_total;
} pvlm_speedup_model;

pvlm_status pvlm_speedup(double c, double tau, int gamma, pvlm_speedup_model* out);
pvlm_status pvlm_window_size(double t_p, double t_q, pvlm_round rounding, double tau,
                             int gamma_max, int* gamma, double* c_out);

/* ------------------------------------------------------------------------
 * Parallel decoding scheduler (host-only: no device pointer, no stream).
 * Suppl. "Parallel Pipeline Details", Alg. (speculative_decoding), with the
 * startup window of Sec. 4.2, Stage I (iii) and the overlap of Stage II: the
 * draft drafts the next window while the target verifies the previous one.
 * The scheduler says what each round runs; the caller runs the draft and the
 * target (e.g. on two HIP streams, the target's verdict from
 * pvlm_spec_accept) and reports the outcome.  Positions count output tokens
 * (the prompt excluded).  A pvlm_pd is owned by one caller thread.
 *
 *   startup round   after pvlm_pd_start(startup = d0, d1..d_gamma: the draft's
 *                   first token and the window it drafted during prefill): the
 *                   target's prefill output decides d0; no forward, cost 0.
 *   PRE_VERIFY      nothing pending: the draft drafts gamma tokens from the
 *                   committed prefix, the target verifies the first of them.
 *   POST_VERIFY     the target verifies the pending window while the draft
 *                   drafts gamma tokens after it.
 * pvlm_pd_finish(drafted = the round's draft_count new tokens, n_accepted of
 * the verify_count verified tokens, target_token = the target's token at the
 * first rejection, ignored when all were accepted):
 *   all accepted: they are committed; the rest stay pending; the next round
 *   is POST_VERIFY, or PRE_VERIFY if nothing is pending (gamma = 1).
 *   a rejection: the accepted prefix and target_token are committed, every
 *   other draft is dropped, draft_keep becomes the committed count before
 *   target_token (the draft truncates its cache to the prompt plus that many
 *   output tokens and resumes from target_token), the next round is PRE_VERIFY.
 * A round that runs forwards costs max(gamma, c) units of t (the draft's
 * forward time); c = T_p / T_q.  Once max_len tokens are committed the plan's
 * mode is PVLM_PD_DONE (the output may overrun max_len by the last round).
 * max_draft_run is the longest run of committed draft tokens not interrupted
 * by a target token (the adaptive draft length).
 *
 * Errors: PVLM_ERR_NULL for a NULL handle or required pointer; PVLM_ERR_SHAPE
 * for gamma outside [1, 1024], c not finite and > 0, max_len outside
 * [1, 2^26], start twice, plan/finish before start, finish when DONE, a
 * drafted count other than the plan's draft_count or n_accepted outside
 * [0, verify_count] (the state is then unchanged); PVLM_ERR_UNSUPPORTED if
 * the handle cannot be allocated.  pvlm_pd_output / pvlm_pd_pending copy up
 * to cap tokens to a host buffer and set *n to the full count; dst = NULL
 * with cap = 0 only queries *n; a smaller cap copies a prefix and returns
 * PVLM_ERR_SHAPE.
 * ---------------------------------------------------------------------- */
typedef enum {
  PVLM_PD_PRE_VERIFY = 0,
  PVLM_PD_POST_VERIFY = 1,
  PVLM_PD_DONE = 2
} pvlm_pd_mode;

typedef struct {
  int32_t mode;          /* pvlm_pd_mode */
  int32_t verify_begin;  /* output position of the first token the target verifies */
  int32_t verify_count;  /* tokens the target verifies */
  int32_t draft_begin;   /* output position of the draft's first new token */
  int32_t draft_count;   /* tokens the draft drafts this round */
  double cost;           /* duration, units of t */
} pvlm_pd_round;

typedef struct {
  int32_t mode;           /* mode of the next round */
  int32_t committed;      /* committed output tokens */
  int32_t pending;        /* drafted tokens awaiting verification */
  int32_t target_rounds;  /* rounds that ran forwards */
  int32_t max_draft_run;  /* adaptive draft length */
  int32_t draft_keep;     /* rollback point of the last rejection (0 before any) */
  double elapsed;         /* sum of round costs, units of t */
} pvlm_pd_stats;

typedef struct pvlm_pd pvlm_pd;

pvlm_status pvlm_pd_create(int gamma, double c, int max_len, pvlm_pd** out);
void pvlm_pd_destroy(pvlm_pd* pd);
pvlm_status pvlm_pd_start(pvlm_pd* pd, const int32_t* startup);
pvlm_status pvlm_pd_plan(const pvlm_pd* pd, pvlm_pd_round* round);
pvlm_status pvlm_pd_finish(pvlm_pd* pd, const int32_t* drafted, int n_drafted, int n_accepted,
                           int32_t target_token);
pvlm_status pvlm_pd_output(const pvlm_pd* pd, int32_t* dst, int cap, int* n);
pvlm_status pvlm_pd_pending(const pvlm_pd* pd, int32_t* dst, int cap, int* n);
pvlm_status pvlm_pd_get_stats(const pvlm_pd* pd, pvlm_pd_stats* st);

#ifdef __cplusplus
}
#endif
#endif /* PVLM_H_ */
