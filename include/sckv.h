/*
 * sckv.h -- C ABI of libsckv.so: the data-parallel hot path of sentinel-token
 * context compression (Ren, Jia and Zhu, "Context Compression for
 * Auto-regressive Transformers with Sentinel Tokens", EMNLP 2023) on one
 * AMD Instinct MI355X (gfx950).
 *
 * Vocabulary (Section 3.1 of the paper).  A transformed sequence holds normal
 * tokens and two kinds of sentinel tokens placed around each span whose
 * key/value memory will be compressed: <CL> opens the span, <CR> closes it.
 * A span is given by the pair (cl, cr) of the indices of its <CL> and <CR>
 * in the transformed sequence (cl < cr); the tokens strictly between them
 * are its enclosed tokens.  cr >= L_meta means the span is still open.
 * Attention rule (Sections 1 and 3.1): a <CL> attends only to itself; every
 * other token attends causally to earlier normal and <CR> tokens and to
 * itself, except that a token after a <CR> does not attend to the tokens
 * enclosed by that <CR>'s span, and no token other than itself attends to a
 * <CL>.
 *
 * Key/value cache (Section 2, "Complexity of Attention Mechanism"): a tensor
 * of shape (M, 2, b, H, L_cap, d_head) -- layers, {key, value}, batch, heads,
 * row capacity, head dimension -- contiguous, row-major, in device memory.
 * Row r of sequence s holds the token whose original index is tok_idx[s][r]
 * and whose (tied) position id is pos_ids[s][r]; rows [0, kv_len[s]) are
 * valid.  After compaction the surviving rows keep their original index and
 * position id (Section 3, "Manipulating Key-Value Memory for Inference-time
 * Compression": the memory of enclosed tokens is freed).
 *
 * Span metadata ("vu").  For every original index t of a sequence,
 *   vu[t] = t            if t is a <CL>,
 *   vu[t] = cr           if t is enclosed by the span closed by the <CR> at cr,
 *   vu[t] = INT32_MAX    otherwise (normal tokens outside spans, <CR>s).
 * Row i may attend to column j  <=>  j <= i <= vu[j]  and  (vu[i] != i or
 * j == i).  The key/value row of token t is still needed by a normal token at
 * index P or later  <=>  vu[t] >= P  and t is not a <CL>  <=>  vu[t] >= P
 * for t < P.
 *
 * Conventions for every entry point:
 *   - pointers named *_host are host memory; every other pointer is device
 *     memory of the calling process's current HIP device;
 *   - the caller owns every buffer; the library keeps no state besides a
 *     thread-local error message and never allocates or frees memory; all
 *     work is enqueued on `stream` (0 = the null stream) and no call waits
 *     for the device, except sckv_span_meta, whose copy from pageable host
 *     memory can block the calling thread (see there);
 *   - element types: SCKV_F32 (float) or SCKV_BF16 (bfloat16, stored as
 *     16-bit words); accumulation is always fp32;
 *   - supported head dimensions: 64 and 80;
 *   - device buffers must be 16-byte aligned;
 *   - arguments are checked on the host before any HIP call; a failed check
 *     returns SCKV_EINVAL / SCKV_ESPAN / SCKV_EUNSUP and enqueues nothing; a
 *     HIP error returns SCKV_EHIP; sckv_last_error() describes the last
 *     failure of the calling thread.  No C++ exception crosses this ABI.
 */
#ifndef SCKV_H
#define SCKV_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { SCKV_F32 = 0, SCKV_BF16 = 1 } sckv_dtype;

enum {
  SCKV_OK = 0,
  SCKV_EINVAL = 1,  /* bad size, stride, pointer or dtype            */
  SCKV_ESPAN = 2,   /* spans unsorted, overlapping or out of range    */
  SCKV_ECAP = 3,    /* (status bit) cache capacity exhausted          */
  SCKV_EHIP = 4,    /* a HIP runtime call failed                      */
  SCKV_EUNSUP = 5   /* valid but unsupported shape (e.g. d_head)      */
};

/* Device status bits written by kernels that cannot report synchronously
 * (bitwise OR into a caller-owned int32; nullable where noted). */
#define SCKV_STATUS_CAP 1      /* an append found kv_len >= L_cap: skipped */
#define SCKV_STATUS_TOKEN 2    /* a token index outside [0, L_meta): skipped */

/* Thread-local description of the last failure ("" if none). */
const char* sckv_last_error(void);

/* Library version string. */
const char* sckv_version(void);

/* ---------------------------------------------------------------------------
 * Span metadata and tied position ids.
 * Paper: Section 3.1 (sentinel tokens and the modified mask) and Section 3.1
 * "Input Transformation" (spans must not overlap; <CL> and <CR> take the
 * position of the token before them).
 *
 * cl_host, cr_host : [b][s_max] int32, host.  Spans of sequence s are
 *                    (cl[s][k], cr[s][k]) for k < n_host[s].
 * n_host           : [b] int32, host, 0 <= n <= s_max.
 * Checks (SCKV_ESPAN): 0 <= cl < L_meta, cl < cr, cr_k < cl_{k+1}.
 * spans_dev        : [2*b*s_max + b] int32, device scratch that receives a
 *                    copy of cl, cr and n (must stay allocated until the
 *                    enqueued kernel has run).
 * Host behaviour   : cl, cr and n are packed into a temporary pageable host
 *                    buffer and copied with hipMemcpyAsync on `stream`.  A
 *                    copy from pageable memory is staged by the HIP runtime
 *                    before the call returns, so this call can block the
 *                    calling thread until work already queued on `stream`
 *                    has drained; when it returns, the host arrays and the
 *                    temporary buffer are no longer read and may be reused.
 *                    It is the only entry point that can block the host; a
 *                    prompt calls it once per batch (a few KB).
 * vu               : [b][L_meta] int32 out (definition above).
 * pos              : [b][L_meta] int32 out, nullable: normal tokens get
 *                    consecutive positions 0,1,2,...; a sentinel at t gets
 *                    pos[t-1] (0 at t = 0).
 * ------------------------------------------------------------------------- */
int sckv_span_meta(const int32_t* cl_host, const int32_t* cr_host, const int32_t* n_host,
                   int32_t s_max, int32_t b, int32_t L_meta, int32_t* spans_dev,
                   int32_t* vu, int32_t* pos, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Rotary position embedding at tied positions (rotate-half form over the full
 * head dimension, angle pos * theta^(-2i/d) for pair (i, i + d/2)).
 * Paper: Section 1 and Section 4.1 "Models" (rotary models are supported) with
 * the position tie of Section 3.1 "Input Transformation".
 *
 * x, y  : (b, H, n rows, d_head) with (b,h) slice strides x_stride_bh,
 *         y_stride_bh (elements); rows are contiguous d_head elements.
 *         y == x rotates in place.  Row t of a slice of sequence s is
 *         rotated at position pos[s][tok0 + t].
 * theta : > 0 rotates; == 0 copies x to y unchanged.
 * ------------------------------------------------------------------------- */
int rope_apply(const void* x, void* y, int32_t b, int32_t H, int32_t n, int64_t x_stride_bh,
               int64_t y_stride_bh, int32_t d_head, sckv_dtype dt, const int32_t* pos,
               int32_t L_meta, int32_t tok0, float theta, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * rope_apply into a cache at a per-sequence row: row t of x (token tok0 + t)
 * goes to row row0[s] + t of y.  Used to append a block of the prompt to the
 * compacted cache (Section 3, "Manipulating Key-Value Memory": a long prompt
 * is processed block by block and freed progressively).
 * row0   : [b] device; typically the output of kv_extend.
 * y_rows : rows of each y slice (L_cap); y_stride_bh >= y_rows * d_head.
 * A sequence with row0 < 0 or row0 + n > y_rows is not written and sets
 * SCKV_STATUS_CAP in status (nullable).
 * ------------------------------------------------------------------------- */
int rope_apply_at(const void* x, void* y, const int32_t* row0, int32_t y_rows, int32_t b,
                  int32_t H, int32_t n, int64_t x_stride_bh, int64_t y_stride_bh, int32_t d_head,
                  sckv_dtype dt, const int32_t* pos, int32_t L_meta, int32_t tok0, float theta,
                  int32_t* status, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Causal attention under the <CL>/<CR> span-exclusion mask (prefill).
 * Paper: Section 1 (tokens after <CR> do not see the enclosed tokens) and
 * Section 3.1 (<CL> sees only itself; normal tokens see earlier <CR> and
 * normal tokens).
 *
 * O[s,h,i,:] = sum_j softmax_j(scale * q_i . k_j  over allowed j) * v_j
 * q, o  : (b, H, L, d_head), (b,h) slice strides q_stride_bh, o_stride_bh.
 * k, v  : (b, H, >= L rows, d_head) with slice stride kv_stride_bh (e.g. the
 *         layer slices kv[m,0], kv[m,1] of the cache, stride L_cap*d_head);
 *         column j of sequence s is original token j.
 * vu    : [b][L_meta] span metadata from sckv_span_meta, L <= L_meta.
 * ws    : device workspace of at least sckv_prefill_workspace_bytes(b, L)
 *         bytes (overwritten).
 * Limits: 1 <= L <= 32768.  Key columns that no row of a query block may see
 * are never read.
 * ------------------------------------------------------------------------- */
size_t sckv_prefill_workspace_bytes(int32_t b, int32_t L);
int span_masked_prefill_attn(const void* q, const void* k, const void* v, void* o, int32_t b,
                             int32_t H, int32_t L, int32_t d_head, int64_t q_stride_bh,
                             int64_t kv_stride_bh, int64_t o_stride_bh, sckv_dtype dt,
                             float scale, const int32_t* vu, int32_t L_meta, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * The same attention with the visibility plan built once per prompt.  The
 * plan (for every query block, the key columns its rows may see) depends only
 * on vu, b and L, the same for every layer and head (Section 3.1: the mask is
 * a function of the token types), so a model runs sckv_prefill_plan once and
 * span_masked_prefill_attn_planned per layer.
 *
 * sckv_prefill_plan: vu, L_meta, b, L and ws as for span_masked_prefill_attn;
 *   writes the plan into ws (stream-ordered).
 * span_masked_prefill_attn_planned: the arguments of span_masked_prefill_attn;
 *   ws must hold a plan from sckv_prefill_plan for the same vu, b and L,
 *   not overwritten since.  It only reads ws, so calls on one plan may run
 *   concurrently.  With a workspace that holds no such plan the outputs are
 *   unspecified, but nothing outside ws, q, k, v and o is accessed.
 * span_masked_prefill_attn = sckv_prefill_plan + span_masked_prefill_attn_planned.
 * Errors: as span_masked_prefill_attn.
 * ------------------------------------------------------------------------- */
int sckv_prefill_plan(const int32_t* vu, int32_t L_meta, int32_t b, int32_t L, void* ws,
                      size_t ws_bytes, hipStream_t stream);
int span_masked_prefill_attn_planned(const void* q, const void* k, const void* v, void* o,
                                     int32_t b, int32_t H, int32_t L, int32_t d_head,
                                     int64_t q_stride_bh, int64_t kv_stride_bh,
                                     int64_t o_stride_bh, sckv_dtype dt, float scale,
                                     const int32_t* vu, int32_t L_meta, void* ws,
                                     size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * The same masked attention for one block of the prompt whose keys and
 * values are in a (compacted) cache: block-wise processing of a prompt that
 * does not fit, freeing closed spans after each block (Section 3,
 * "Manipulating Key-Value Memory for Inference-time Compression").
 *
 * q, o     : (b, H, nq, d_head): the block's queries, tokens tok0 .. tok0+nq-1.
 * k_cache, v_cache : (b, H, L_cap, d_head) layer slices, slice stride
 *            kv_stride_bh >= L_cap * d_head.  Row r of sequence s holds token
 *            tok_idx[s][r]; rows [0, row0[s]) are earlier blocks' surviving
 *            rows (ascending tokens, all < tok0) and rows row0[s] + i hold
 *            token tok0 + i (written by rope_apply_at; tok_idx by kv_extend).
 * row0     : [b] device; a sequence with row0 < 0 or row0 + nq > L_cap gets
 *            NaN outputs, nothing is read, and SCKV_STATUS_CAP is set in
 *            status (nullable).
 * Output row i equals row tok0 + i of span_masked_prefill_attn over the
 * whole prompt whenever the cache holds every row that row may see (which
 * kv_compact at the block boundaries guarantees).
 * ws       : >= sckv_prefill_cached_workspace_bytes(b, nq, L_cap) bytes.
 * Limits: nq <= L_cap <= 32768; L_meta < 2^24 - 1.
 * ------------------------------------------------------------------------- */
size_t sckv_prefill_cached_workspace_bytes(int32_t b, int32_t nq, int32_t L_cap);
int span_masked_prefill_attn_cached(const void* q, const void* k_cache, const void* v_cache,
                                    void* o, int32_t b, int32_t H, int32_t nq, int32_t d_head,
                                    int64_t q_stride_bh, int64_t kv_stride_bh,
                                    int64_t o_stride_bh, sckv_dtype dt, float scale,
                                    const int32_t* vu, int32_t L_meta, int32_t tok0,
                                    const int32_t* row0, const int32_t* tok_idx, int32_t L_cap,
                                    void* ws, size_t ws_bytes, int32_t* status,
                                    hipStream_t stream);

/* The cached attention with its plan built once per block: the plan (for
 * every query block, the cache rows its rows may see) depends on vu, tok0,
 * row0, tok_idx, L_cap, b and nq, not on the layer, so block-wise processing
 * runs sckv_prefill_cached_plan once per block and the planned call per layer.
 * sckv_prefill_cached_plan: arguments as for span_masked_prefill_attn_cached;
 *   writes the plan into ws (stream-ordered).
 * span_masked_prefill_attn_cached_planned: the arguments of
 *   span_masked_prefill_attn_cached; ws must hold a plan from
 *   sckv_prefill_cached_plan for the same vu, tok0, row0, tok_idx contents,
 *   L_cap, b and nq, not overwritten since.  With a workspace that holds no
 *   such plan the outputs are unspecified, but nothing outside ws and the
 *   argument buffers is accessed.
 * Errors: as span_masked_prefill_attn_cached. */
int sckv_prefill_cached_plan(const int32_t* vu, int32_t L_meta, int32_t tok0, const int32_t* row0,
                             const int32_t* tok_idx, int32_t L_cap, int32_t b, int32_t nq,
                             void* ws, size_t ws_bytes, hipStream_t stream);
int span_masked_prefill_attn_cached_planned(const void* q, const void* k_cache,
                                            const void* v_cache, void* o, int32_t b, int32_t H,
                                            int32_t nq, int32_t d_head, int64_t q_stride_bh,
                                            int64_t kv_stride_bh, int64_t o_stride_bh,
                                            sckv_dtype dt, float scale, const int32_t* vu,
                                            int32_t L_meta, int32_t tok0, const int32_t* row0,
                                            const int32_t* tok_idx, int32_t L_cap, void* ws,
                                            size_t ws_bytes, int32_t* status, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Free the key/value rows of closed spans, in place, keeping the survivors in
 * their order (stable stream compaction).
 * Paper: Section 3, "Manipulating Key-Value Memory for Inference-time
 * Compression" (the memory of enclosed tokens is freed) and Section 2 (cache
 * layout).
 *
 * kv        : (M, 2, b, H, L_cap, d_head) cache, rows moved in place.
 * kv_out    : nullable; if set, the same shape: surviving rows are written to
 *             their compacted place in kv_out and kv is left untouched.
 * kv_len    : [b] in/out.  tok_idx, pos_ids: [b][L_cap] in/out (compacted in
 *             place in both modes).
 * next_tok  : [b] original index P of each sequence's next query: row r,
 *             holding token t = tok_idx[r], is kept iff t is not a <CL>
 *             (vu[t] != t) and vu[t] >= P (a row whose t lies outside
 *             [0, L_meta) is kept).
 * kept_src_row : [b][L_cap] out: source row of each surviving row, -1 after
 *             the new kv_len.
 * ------------------------------------------------------------------------- */
int kv_compact(void* kv, void* kv_out, int32_t M, int32_t b, int32_t H, int32_t L_cap,
               int32_t d_head, sckv_dtype dt, int32_t* kv_len, int32_t* tok_idx,
               int32_t* pos_ids, const int32_t* next_tok, const int32_t* vu, int32_t L_meta,
               int32_t* kept_src_row, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * One decode step of one layer over the compacted cache.
 * Paper: Section 1 and Section 2 (attention reads the whole key/value memory;
 * its size drives decode latency) and Section 4.3 (generation continues from
 * the compressed cache).
 *
 * Precondition: rows [0, kv_len[s]) hold only tokens that token t =
 * cur_tok[s] may attend to, i.e. no row holds a <CL> or a token enclosed by
 * a span whose <CR> is before t.  The kernel attends to every such row
 * without a mask, so the caller runs kv_compact (next_tok = cur_tok) after
 * the prompt and after every step whose token was a <CR>, before the next
 * decode step; rows appended by other steps keep the precondition.
 *
 * For each sequence s with current token t = cur_tok[s]:
 *   - if vu[s][t] == t (t is a <CL>): o[s,h] = v_new[s,h] and nothing is
 *     written to the cache;
 *   - else: q and k_new are rotated at position pos[s][t] when
 *     rope_theta > 0; the new key/value pair is written at row kv_len[s] of
 *     k_cache/v_cache; o[s,h] = softmax(scale * q . K[0..kv_len]) V[0..kv_len]
 *     over the kv_len[s] + 1 rows.  kv_len itself is not changed (all layers
 *     of a step share it; see kv_commit).
 *   - kv_len[s] >= L_cap sets SCKV_STATUS_CAP, writes NaN to o[s] and
 *     appends nothing; t outside [0, L_meta) sets SCKV_STATUS_TOKEN likewise.
 * q, k_new, v_new, o : (b, H, d_head) contiguous.
 * k_cache, v_cache   : (b, H, L_cap, d_head) layer slices (kv[m,0], kv[m,1]).
 * kv_len, cur_tok    : [b].   vu, pos: [b][L_meta].
 * ws     : device workspace >= sckv_decode_workspace_bytes(b, H, L_cap, d_head)
 *          holding the split-K partials (overwritten; calls that share a
 *          workspace must be ordered, e.g. enqueued on one stream).
 * status : nullable int32, status bits OR-ed in.
 * Launch shape: with b*H >= 512 one workgroup per (sequence, head) covers
 * all its rows and writes o (the workspace is not touched); with fewer, the
 * rows are cut into balanced chunks of at most about 1024 rows, one
 * workgroup each, and a second kernel merges the chunk partials
 * (log-sum-exp) into o.  bf16 scores are computed on the matrix cores with
 * q carried as two bf16 terms (about fp32 accuracy).
 * ------------------------------------------------------------------------- */
size_t sckv_decode_workspace_bytes(int32_t b, int32_t H, int32_t L_cap, int32_t d_head);
int compacted_decode_attn(const void* q, const void* k_new, const void* v_new, void* k_cache,
                          void* v_cache, const int32_t* kv_len, const int32_t* cur_tok,
                          const int32_t* vu, const int32_t* pos, int32_t L_meta, void* o,
                          int32_t b, int32_t H, int32_t L_cap, int32_t d_head, sckv_dtype dt,
                          float scale, float rope_theta, void* ws, size_t ws_bytes,
                          int32_t* status, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * compacted_decode_attn without any allocation, for callers that cannot
 * allocate device memory or pass a workspace: code being captured into a
 * HIP graph, tight serving loops, harnesses that forbid hipMalloc.
 *
 * Same arguments, semantics, precondition, status bits and outputs as
 * compacted_decode_attn, minus ws / ws_bytes: the split-K partials of a
 * launch with fewer than 512 (sequence, head) slices go to a scratch array
 * of SCKV_NOALLOC_SCRATCH_BYTES bytes inside the library, one per device,
 * held from the library's load until the process ends.  The call allocates
 * and frees nothing; its first call on a device looks up that device's
 * array address once.
 * Limit: with b*H < 512, sckv_decode_workspace_bytes(b, H, L_cap, d_head)
 * must not exceed SCKV_NOALLOC_SCRATCH_BYTES (511 slices of up to 65536
 * rows fit, at either head size); larger shapes return SCKV_EUNSUP and
 * enqueue nothing.  With b*H >= 512 the scratch array is not used.
 * Every call on a device shares its array and overwrites what the previous
 * call left there (nothing in it needs clearing); calls that may overlap on
 * one device (two host threads, or two streams without ordering) race and
 * must not be made.
 * ------------------------------------------------------------------------- */
#define SCKV_NOALLOC_SCRATCH_BYTES (16u << 20)
int compacted_decode_attn_noalloc(const void* q, const void* k_new, const void* v_new,
                                  void* k_cache, void* v_cache, const int32_t* kv_len,
                                  const int32_t* cur_tok, const int32_t* vu, const int32_t* pos,
                                  int32_t L_meta, void* o, int32_t b, int32_t H, int32_t L_cap,
                                  int32_t d_head, sckv_dtype dt, float scale, float rope_theta,
                                  int32_t* status, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Local-attention comparator (the "Local Attention" baseline of Section 4.1:
 * a token attends only to a window of the most recent tokens), at a fixed
 * budget of W cached rows: rows [0, W) of each slice are a ring holding the
 * W most recent tokens, token t at row t mod W.  For each sequence with
 * current token t = cur_tok[s], the new key (rotated at pos[s][t] when
 * rope_theta > 0) and value replace row t mod W (the token t - W) and
 * o[s,h] = attention of q over the W tokens t-W+1 .. t.  cur_tok is not
 * changed.  A <CL> step (vu[s][t] == t) outputs v_new and writes nothing.
 * The ring must be full (t >= W: the W rows hold tokens t-W .. t-1 when the
 * call is made, e.g. after a prompt of at least W tokens was loaded into
 * it); every ring row other than the replaced one is attended as it stands.
 * Same launch shapes and workspace as compacted_decode_attn; bf16 only;
 * 0 < W < L_cap.
 * ------------------------------------------------------------------------- */
int local_decode_attn(const void* q, const void* k_new, const void* v_new, void* k_cache,
                      void* v_cache, int32_t W, const int32_t* cur_tok, const int32_t* vu,
                      const int32_t* pos, int32_t L_meta, void* o, int32_t b, int32_t H,
                      int32_t L_cap, int32_t d_head, sckv_dtype dt, float scale,
                      float rope_theta, void* ws, size_t ws_bytes, int32_t* status,
                      hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Append bookkeeping for a block of n prompt tokens tok0 .. tok0+n-1 (all of
 * them, sentinels included; kv_compact frees what the block closes): for
 * each sequence, row0_out[s] = kv_len[s], rows kv_len[s] + i get
 * tok_idx = tok0 + i and pos_ids = pos[s][tok0 + i], and kv_len[s] += n.
 * A sequence without room (kv_len + n > L_cap) is left unchanged, gets
 * row0_out[s] = -1 and sets SCKV_STATUS_CAP in status (nullable).
 * Paper: Section 3, "Manipulating Key-Value Memory" (progressive freeing).
 * ------------------------------------------------------------------------- */
int kv_extend(int32_t* kv_len, int32_t* tok_idx, int32_t* pos_ids, int32_t* row0_out,
              const int32_t* pos, int32_t L_meta, int32_t tok0, int32_t n, int32_t b,
              int32_t L_cap, int32_t* status, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Close a decode step after all layers: for each sequence, unless its current
 * token t = cur_tok[s] is a <CL> (vu[s][t] == t), record row kv_len[s]
 * (tok_idx = t, pos_ids = pos[s][t]) and increment kv_len[s]; then increment
 * cur_tok[s].  Capacity or token-range violations set status bits and skip
 * the record.
 * Paper: Section 3, "Manipulating Key-Value Memory" (the cache holds only rows
 * later tokens may see) with the position tie of "Input Transformation".
 * ------------------------------------------------------------------------- */
int kv_commit(int32_t* kv_len, int32_t* tok_idx, int32_t* pos_ids, int32_t* cur_tok,
              const int32_t* vu, const int32_t* pos, int32_t L_meta, int32_t b, int32_t L_cap,
              int32_t* status, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* SCKV_H */
