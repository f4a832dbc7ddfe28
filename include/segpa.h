/*
 * segpa.h - SegPagedAttention with per-head page selection on AMD MI355X (gfx950).
 *
 * C ABI of libsegpa.so. Every pointer argument marked "device" is a HIP device
 * pointer; every size and scalar is host data. The library never allocates,
 * frees or retains caller memory past a call, except that the optional
 * profiling hooks keep host-side event records between
 * seg_paged_attn_profile_begin and seg_paged_attn_profile_end. Its only device
 * memory of its own is the static scratch of seg_paged_attn_fwd_noalloc.
 *
 * What is computed follows RedKnot (arXiv 2606.06256):
 *   - Section 4.3 and Algorithm 2 (SegPagedAttention): the KV cache of one
 *     layer is stored per KV head as head segments; a segment maps to
 *     consecutive virtual pages (segment table) and each virtual page to a
 *     physical page (page table). Each KV head attends only to its own selected
 *     page list, in one fused launch over all heads, without a mask.
 *   - Algorithm 2, policy step: a global head keeps the full page range; a
 *     local head keeps sink pages and recent-window pages, where the window of
 *     query position i is W(i) = S_sink U [max(0, i - w), i] (Section 4.2).
 *   - Section 4.4: attention over a key set split into parts, merged with
 *     log-sum-exp, equals attention over the union (used for split-KV).
 *
 * Terms.
 *   B = num_requests, Hq = num_q_heads, Hkv = num_kv_heads, G = Hq / Hkv,
 *   D = head_dim, P = page_size, pps = pages_per_segment.
 *   A unit is one (request r, KV head g) head stream, index u = r * Hkv + g.
 *   Query head h reads KV head h / G.
 *   ctx_lens[r] = L_r is the number of KV tokens of request r including its
 *   current query chunk; the stream has n_pages(r) = ceil(L_r / P) logical
 *   pages, page j holding tokens j*P .. j*P+P-1 (the last page may be partial).
 *   Request r has n_q(r) = q_indptr[r+1] - q_indptr[r] query tokens; query i of
 *   the chunk sits at position L_r - n_q(r) + i and sees selected tokens at
 *   positions <= its own (causal, aligned to the end of the context).
 *
 * Translate (Algorithm 2): logical page j of unit (r, g) lives in segment
 *   s = j / pps at offset o = j % pps;
 *   virtual = seg_table[(r * Hkv + g) * max_segments + s] + o  (entry -1: unmapped)
 *   physical = page_table[virtual].
 *
 * Physical page layout (both pools bf16, page stride P * D elements, 16-byte
 * aligned base): a page holds P/16 tiles of 16 tokens; tile t of a page starts
 * at element t * 16 * D.
 *   K tile: [D/8][16][8]  element (token u, dim d) at ((d / 8) * 16 + u) * 8 + d % 8
 *   V tile: [D][16]       element (token u, dim d) at d * 16 + u
 * These are the operand layouts of the gfx950 matrix-core instructions used by
 * the kernels, so every tile arrives in registers with contiguous loads.
 *
 * Selected pages: CSR over units. sel_indptr[u] .. sel_indptr[u+1]-1 index
 * sel_pages, which holds logical page ids, strictly ascending within a unit and
 * < n_pages(r). A unit with no pages is legal: its outputs are O = 0 and
 * LSE = -inf. Pages that are not selected never enter the softmax (true
 * eviction, Section 5.4).
 *
 * Outputs: out bf16 [total_q, Hq, D] (round to nearest even), with
 * total_q = q_indptr[B]; lse fp32 [total_q, Hq], natural log of the softmax
 * denominator including the max (may be NULL). MergeHeads of Algorithm 2 is the
 * identity in this layout.
 *
 * Execution. All calls except seg_paged_attn_validate are asynchronous and
 * stream-ordered on `stream` (a hipStream_t; NULL = the null stream): results
 * are valid when the stream reaches the end of the call. Host-checkable
 * argument errors return before anything is launched. Kernels never read out
 * of bounds on bad table or list contents: an out-of-range page id, unmapped
 * segment or out-of-range physical page is skipped (contributes nothing);
 * seg_paged_attn_validate reports such data synchronously. Calls that share a
 * workspace must not overlap. Every call except seg_paged_attn_validate only
 * launches kernels on `stream` (no memset, no copy, no host synchronisation;
 * the profiling hooks, when on, add event records), so a caller can capture
 * them in a HIP graph and replay it.
 */
#ifndef SEGPA_H
#define SEGPA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPA_OK = 0,
  SPA_ERR_INVALID_ARG = -1,  /* null pointer, bad dimension, inconsistent sizes */
  SPA_ERR_UNSUPPORTED = -2,  /* valid but not implemented here (e.g. D not 64/128) */
  SPA_ERR_WORKSPACE = -3,    /* workspace null or smaller than required */
  SPA_ERR_CAPACITY = -4,     /* sel_capacity below B * Hkv * max_segments * pps */
  SPA_ERR_HIP = -5,          /* a HIP runtime call or launch failed */
  SPA_ERR_BAD_DATA = -6      /* validate(): table or page-list content is invalid */
} spa_status_t;

/* Largest B * Hkv per call. */
#define SPA_MAX_UNITS 8192

typedef struct {
  int32_t num_requests;       /* B >= 1 */
  int32_t num_q_heads;        /* Hq, a multiple of Hkv, Hq / Hkv <= 16 */
  int32_t num_kv_heads;       /* Hkv >= 1 */
  int32_t head_dim;           /* D: 64 or 128 */
  int32_t page_size;          /* P: 16, 32, 64, 128 or 256 tokens */
  int32_t pages_per_segment;  /* pps >= 1 */
  int32_t max_segments;       /* inner dimension of seg_table, >= 1 */
  int32_t max_q_len;          /* host upper bound of n_q(r) over all requests, >= 1 */
  int32_t total_q;            /* rows of q and out (= q_indptr[B]), >= 0 */
  int32_t reserved0;
  int64_t num_virtual_pages;  /* length of page_table */
  int64_t num_phys_pages;     /* pages in each pool; num_phys_pages * P / 16 < 2^28 */
  float softmax_scale;        /* <= 0 selects 1 / sqrt(D) */
} spa_dims_t;

typedef enum {
  SPA_SEL_ALL = 0,          /* every page: U_h = V_h (global head of Algorithm 2) */
  SPA_SEL_HEAD_CLASS = 1,   /* Algorithm 2 policy: global -> all pages; local -> pages
                               overlapping S_sink or any W(i) of the chunk's queries */
  SPA_SEL_RANDOM_HASH = 2,  /* forced pages + the other pages with the smallest
                               SplitMix64 keys (seeded sample without replacement) */
  SPA_SEL_TOPK_MEANKEY = 3  /* forced pages + the other pages with the highest
                               score (q_bar . ksum_p) / n_valid(p), q_bar = sum of the
                               G query heads of the request's last query token */
} spa_sel_mode_t;

typedef struct {
  int32_t mode;               /* spa_sel_mode_t */
  int32_t n_sink_tokens;      /* HEAD_CLASS: |S_sink|, the first positions of the stream */
  int32_t window_tokens;      /* HEAD_CLASS: w */
  int32_t forced_head_pages;  /* RANDOM_HASH/TOPK: pages 0 .. f-1 always selected */
  int32_t forced_tail_pages;  /* RANDOM_HASH/TOPK: the last f pages always selected */
  int32_t reserved;
  uint64_t seed;              /* RANDOM_HASH */
  const int8_t* head_policy;  /* HEAD_CLASS: device [Hkv], 1 = global, 0 = local */
  const int32_t* budget_pages;/* RANDOM_HASH/TOPK: device [B], pages per unit of request r */
} spa_select_params_t;

/*
 * Bytes of workspace that seg_paged_attn_select (for `sel_mode`) and
 * seg_paged_attn_fwd need for these dims on the current device. Returns 0 on
 * invalid dims. The workspace is scratch owned by the caller; its content
 * between calls does not matter.
 */
size_t seg_paged_attn_workspace_size(const spa_dims_t* dims, int32_t sel_mode);

/*
 * SelectVisibleState (Section 4.4 adapter interface; Algorithm 2 policy,
 * Translate-ready metadata): the selected logical pages of every unit.
 *
 * Count of unit u (request r, KV head g), n = n_pages(r):
 *   ALL: n.  HEAD_CLASS: global n; local |[0, ceil(min(n_sink, L)/P)) U
 *   [floor(max(0, L - n_q - w) / P), n)|.  RANDOM_HASH / TOPK:
 *   min(n, max(budget_pages[r], |forced|)), forced = [0, fh) U [n - ft, n).
 * RANDOM_HASH key of page p: sm(sm(seed) ^ (r << 40 | g << 32 | p)) with
 *   sm(x) = SplitMix64 output function applied to x + 0x9E3779B97F4A7C15;
 *   smaller keys first, equal keys to the lower index.
 * TOPK_MEANKEY score in float64 from page_ksum (see page_summary); higher
 *   first, equal scores to the lower index. page_ksum may be NULL otherwise.
 *
 * In:  ctx_lens device [B]; q device bf16 [total_q, Hq, D] and q_indptr device
 *      [B+1] (q is read by TOPK only; q_indptr by HEAD_CLASS and TOPK, may be
 *      NULL for ALL/RANDOM_HASH); seg_table device [B*Hkv*max_segments];
 *      page_table device [num_virtual_pages] (both read by TOPK only).
 * Out: sel_indptr device [B*Hkv+1]; sel_pages device [sel_capacity], logical
 *      ids ascending per unit. sel_capacity must be at least
 *      B * Hkv * max_segments * pps.
 * ctx_lens[r] must not exceed max_segments * pps * P (larger values are
 * clamped to that many pages).
 */
spa_status_t seg_paged_attn_select(const spa_dims_t* dims, const spa_select_params_t* params,
                                   const int32_t* ctx_lens, const void* q, const int32_t* q_indptr,
                                   const float* page_ksum, const int32_t* seg_table,
                                   const int32_t* page_table, int32_t* sel_indptr,
                                   int32_t* sel_pages, int64_t sel_capacity, void* workspace,
                                   size_t workspace_bytes, void* stream);

/*
 * Execute / FusedVarlenAttention + MergeHeads (Algorithm 2): softmax attention
 * of every query row over the selected pages of its unit, in one fused launch
 * over all units, then a log-sum-exp combine of split partial results
 * (Section 4.4). bf16 inputs, fp32 accumulation, bf16 output.
 *
 * In:  q device bf16 [total_q, Hq, D]; q_indptr device [B+1]; ctx_lens device
 *      [B]; k_pool, v_pool device bf16 [num_phys_pages, P * D] in the tile
 *      layout above; seg_table device [B*Hkv*max_segments]; page_table device
 *      [num_virtual_pages]; sel_indptr device [B*Hkv+1]; sel_pages device
 *      [sel_capacity] (entries past sel_capacity are never read).
 * Out: out device bf16 [total_q, Hq, D]; lse device fp32 [total_q, Hq] or NULL.
 * Shapes: max_q_len * G < 128 runs the split-KV decode kernel (the query rows
 * of a unit in blocks of 16, one matrix-core tile each); larger chunks run the
 * chunked-prefill kernel.
 * Debug: with the environment variable SEGPA_VALIDATE set (and not "0"), the
 * call first runs the checks of seg_paged_attn_validate synchronously (so it
 * then synchronises the stream and cannot be captured in a graph) and returns
 * SPA_ERR_BAD_DATA without launching when the tables or lists are invalid.
 */
spa_status_t seg_paged_attn_fwd(const spa_dims_t* dims, const void* q, const int32_t* q_indptr,
                                const int32_t* ctx_lens, const void* k_pool, const void* v_pool,
                                const int32_t* seg_table, const int32_t* page_table,
                                const int32_t* sel_indptr, const int32_t* sel_pages,
                                int64_t sel_capacity, void* out, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream);

/*
 * seg_paged_attn_fwd for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops or harnesses that forbid hipMalloc):
 * the same arguments, outputs, kernels and errors, minus workspace and
 * workspace_bytes. The split-KV partials go to a scratch array inside the
 * library instead: SPA_NOALLOC_SCRATCH_BYTES of device memory on each GPU the
 * call runs on (a static device array of the library's code object, present
 * on a GPU once the library's code is loaded there, at the latest by the first
 * call, and held until the process ends). The call allocates nothing. A shape whose partials need more than that returns
 * SPA_ERR_WORKSPACE before anything is launched: the decode path needs
 * (W + B * Hkv * ceil(max_q_len * G / 16)) * (16 * D + 16) * 4 bytes (rounded
 * up to 256 twice), with W = 4 waves per compute unit (1024 on MI355X), e.g.
 * up to about 3,000 (unit, 16-row block) pairs at D = 128; the chunked-prefill
 * path keeps no partials. The scratch is not cleared: no call reads what an
 * earlier call left there. All calls on one GPU share that GPU's scratch, so
 * calls that overlap in time on one GPU (other streams, other host threads)
 * race; the caller must order them, e.g. on one stream.
 */
#define SPA_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
spa_status_t seg_paged_attn_fwd_noalloc(const spa_dims_t* dims, const void* q,
                                        const int32_t* q_indptr, const int32_t* ctx_lens,
                                        const void* k_pool, const void* v_pool,
                                        const int32_t* seg_table, const int32_t* page_table,
                                        const int32_t* sel_indptr, const int32_t* sel_pages,
                                        int64_t sel_capacity, void* out, float* lse, void* stream);

/*
 * Appending tokens to the head-segmented KV pool (BuildState, Section 4.4,
 * over the head segments of Section 4.3), with an optional refresh of the key
 * sums of every page that received a token.
 * Request r's new tokens new_indptr[r] .. new_indptr[r+1]-1 take positions
 * ctx_lens[r], ctx_lens[r] + 1, ... of each KV head's stream; position t is
 * slot t % P of logical page t / P, translated through seg_table and
 * page_table as in Algorithm 2. A token whose segment is unmapped, or whose
 * position lies past the segment table, is dropped. ctx_lens is read, not
 * updated: the caller adds the appended counts.
 * In:  ctx_lens device int32 [B] (tokens stored before the append);
 *      new_indptr device int32 [B+1] (0, non-decreasing, new_indptr[B] = n_new);
 *      k_new, v_new device bf16 [n_new, Hkv, D]; seg_table, page_table as for
 *      seg_paged_attn_fwd.
 * In/out: k_pool, v_pool device bf16 [num_phys_pages, P * D] (tile layout);
 *      page_ksum device fp32 [num_phys_pages, D] or NULL: for each page that
 *      received a token, the float32 rounding of the sum of its valid keys
 *      (valid = min(P, new length - page start)), as seg_paged_attn_page_summary.
 * A page written by this call must belong to one (request, KV head) only
 * (segments shared between requests are read-only); two units writing one
 * page is a data race.
 * Errors: INVALID_ARG for n_new < 0, a null pointer needed for n_new > 0, or
 * misaligned pools or page_ksum. Asynchronous on stream; n_new = 0 launches
 * nothing.
 */
spa_status_t seg_paged_attn_append(const spa_dims_t* dims, const int32_t* ctx_lens,
                                   const int32_t* new_indptr, const void* k_new, const void* v_new,
                                   int64_t n_new, const int32_t* seg_table,
                                   const int32_t* page_table, void* k_pool, void* v_pool,
                                   float* page_ksum, void* stream);

/*
 * RoPE positional alignment of cached keys (Section 4.2): a key cached at
 * offline position p_off and reused at online position p_on is replaced by
 * R(p_on) R(p_off)^-1 K(p_off), which is the rotation by delta = p_on - p_off.
 * Each listed physical page of k_pool is rotated in place by its delta; every
 * token slot of the page is rotated. Plane i pairs head dimension i with
 * i + D/2 and turns by delta * rope_base^(-2 i / D). Arithmetic in float64,
 * one rounding to bf16 (to nearest, ties to even).
 * In:  pages device int32 [n]: distinct physical page ids (an id outside
 *      [0, num_phys_pages) is skipped; an id listed twice is a data race);
 *      deltas device int32 [n]; rope_base > 1 (10000 and 1e6 are common).
 * In/out: k_pool device bf16 [num_phys_pages, P * D] in the tile layout.
 * Errors: INVALID_ARG for a null pointer with n > 0, n < 0 or n >= 2^31, a
 * rope_base that is not finite or <= 1, or a misaligned k_pool.
 * Asynchronous on stream; n = 0 launches nothing.
 */
spa_status_t seg_paged_attn_rope_align(const spa_dims_t* dims, void* k_pool, const int32_t* pages,
                                       const int32_t* deltas, int64_t n, double rope_base,
                                       void* stream);

/*
 * Page key summary for TOPK_MEANKEY (a content rule of this library; the
 * paper states none): page_ksum[p][d] = float32 rounding of the sum over the first
 * page_valid_tokens[p] tokens of physical page p of K[token][d], accumulated in
 * float64 (exact when the page's nonzero magnitudes span less than 2^40).
 * In:  k_pool device bf16 [num_phys_pages, P * D]; page_valid_tokens device
 *      int32 [num_phys_pages] (0..P; values outside are clamped).
 * Out: page_ksum device fp32 [num_phys_pages, D].
 */
spa_status_t seg_paged_attn_page_summary(const spa_dims_t* dims, const void* k_pool,
                                         const int32_t* page_valid_tokens, float* page_ksum,
                                         void* stream);

/*
 * Attention mass of the chunk tokens (the probability pass feeding
 * SelectImportantTokens, Algorithm 1; the token-importance signal of the
 * sparse FFN, Section 4.4). For token t of request r's query chunk (query
 * position L_r - n_q(r) + t) and KV head g:
 *   mass[q_indptr[r] + t][g] = sum over query heads h of group g and chunk
 *     queries i >= t of exp(scale * q[i][h] . k_t - lse[i][h]),
 * where token t counts only if its logical page is in unit (r, g)'s selected
 * list (as for seg_paged_attn_fwd: the same softmax, normalised by the
 * forward's lse, so with the fwd's lse each row's weights over its attended
 * keys sum to 1). A token whose page is not selected, unmapped, or whose
 * position is negative has mass 0 for that head. A row whose lse is not
 * finite contributes nothing. bf16 products, fp32 accumulation in a fixed
 * order (results are reproducible bit for bit).
 * In:  q, q_indptr, ctx_lens, k_pool, seg_table, page_table, sel_indptr,
 *      sel_pages, sel_capacity as for seg_paged_attn_fwd (v_pool is not read);
 *      lse device fp32 [total_q, Hq] from seg_paged_attn_fwd over the same
 *      selected pages (natural log).
 * Out: mass device fp32 [total_q, Hkv]. Rows outside every request's chunk
 *      are not written.
 * Errors: INVALID_ARG for a null pointer, q or k_pool not 16-byte aligned,
 * lse or mass not 4-byte aligned. Asynchronous on stream; total_q = 0
 * launches nothing.
 */
spa_status_t seg_paged_attn_token_mass(const spa_dims_t* dims, const void* q,
                                       const int32_t* q_indptr, const int32_t* ctx_lens,
                                       const void* k_pool, const int32_t* seg_table,
                                       const int32_t* page_table, const int32_t* sel_indptr,
                                       const int32_t* sel_pages, int64_t sel_capacity,
                                       const float* lse, float* mass, void* stream);

/*
 * SelectImportantTokens (Algorithm 1) by cumulative attention mass (Section
 * 4.4): per request, the smallest set of chunk tokens whose mass reaches tau
 * of the chunk's total, together with the most recent `recent` tokens (the
 * keep-recent-N rule of the sparse-FFN settings, Section 5).
 * Token mass m_t = float32 sum of mass[q_indptr[r] + t][0 .. mass_cols-1] in
 * column order (mass_cols = Hkv for the output of seg_paged_attn_token_mass,
 * 1 for per-token masses); a sum that is negative or NaN counts as 0.
 * Tokens are ranked by m_t descending, equal masses by position ascending;
 * with M_k the float64 sum of the masses ranked before token k and T the
 * float64 total, token k is kept iff T > 0 and M_k < tau * T (the ranked
 * prefix that first reaches tau * T). Tokens t >= n_q(r) - recent are kept
 * as well. The sums are formed in a parallel order: a result can differ from
 * a sequential summation only where a partial sum lies within float64
 * rounding of tau * T.
 * In:  q_indptr device [B+1]; mass device fp32 [total_q, mass_cols]
 *      (1 <= mass_cols <= 4096); 0 < tau <= 1; recent >= 0.
 * Out: keep device uint8 [total_q] (1 kept, 0 not); kept device int32
 *      [total_q] or NULL: the kept rows (absolute row ids) of request r in
 *      ascending order at kept[q_indptr[r] ..], keep_count[r] of them (later
 *      entries untouched); keep_count device int32 [B]; token_mass device fp32
 *      [total_q] or NULL: m_t.
 * Requires max_q_len <= 16384 (else UNSUPPORTED): a request's chunk is
 * sorted in one workgroup's LDS. The 99%-mass fraction of a chunk is
 * keep_count / n_q with tau = 0.99 and recent = 0.
 * Errors: INVALID_ARG for a null required pointer, tau outside (0, 1],
 * recent < 0, mass_cols outside [1, 4096], misaligned 4-byte outputs.
 */
spa_status_t seg_paged_attn_select_tokens(const spa_dims_t* dims, const int32_t* q_indptr,
                                          const float* mass, int32_t mass_cols, double tau,
                                          int32_t recent, uint8_t* keep, int32_t* kept,
                                          int32_t* keep_count, float* token_mass, void* stream);

/*
 * Synchronous check of table and list contents (debug aid). Checks q_indptr
 * (monotone, n_q <= min(max_q_len, L)), ctx_lens (0 <= L <= max_segments*pps*P),
 * sel_indptr (starts at 0, monotone), every selected page (in [0, n_pages),
 * strictly ascending in its unit, segment mapped, virtual page in range,
 * physical page in range). Returns SPA_OK or SPA_ERR_BAD_DATA; *bad_code (may
 * be NULL) receives a nonzero code naming the first failed check class and
 * *bad_index the smallest offending index of that class. Needs 64 bytes of
 * workspace.
 */
spa_status_t seg_paged_attn_validate(const spa_dims_t* dims, const int32_t* ctx_lens,
                                     const int32_t* q_indptr, const int32_t* seg_table,
                                     const int32_t* page_table, const int32_t* sel_indptr,
                                     const int32_t* sel_pages, int64_t sel_capacity,
                                     int32_t* bad_code,
                                     int64_t* bad_index, void* workspace, size_t workspace_bytes,
                                     void* stream);

/* Static text for a status code. */
const char* seg_paged_attn_status_string(spa_status_t status);

/*
 * Optional per-kernel timing (measurement aid, not thread-safe). Between begin
 * and end every kernel launch of the library is bracketed by HIP events on the
 * launch stream. end() waits for those events and fills, for up to `cap`
 * kernel kinds, the kind name (static string), the number of launches and the
 * summed milliseconds; it returns the number of kinds (or < 0 on error).
 */
spa_status_t seg_paged_attn_profile_begin(void);
int32_t seg_paged_attn_profile_end(const char** names, int32_t* launches, double* total_ms,
                                   int32_t cap);

#ifdef __cplusplus
}
#endif

#endif /* SEGPA_H */
