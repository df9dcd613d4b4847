/*
 * linattn.h - strict-prefix linear-attention prefill for one tensor-parallel
 * rank's heads on one MI355X (gfx950).
 *
 * C ABI.  Every buffer is a plain pointer; "device" pointers are HIP device
 * memory on the current device, "host" pointers are ordinary host memory.
 * Streams and events are passed as void* (a hipStream_t / hipEvent_t; NULL
 * stream = the null stream).  No C++ exception crosses this boundary.
 *
 * Notation follows the paper (section 2.2, "State position and scheduler
 * position"): N is a prompt length, C the checkpoint interval (the paper's
 * cache block, Table 1), B the prefix a restored state represents and p the
 * scheduler's computed-token count.  Prefix lengths are counts and token
 * indices are zero based; a state for prefix [0, B) continues from B.
 *
 * The recurrence is the gated delta rule (the paper names Flash Linear
 * Attention kernels but does not write it out; the form below is the one the
 * library is specified with).  Per sequence and head, with state S (dk x dv):
 *
 *   LA_GDR_LITERAL:        S_t = exp(g_t) S_{t-1} + beta_t k_t (v_t - S_{t-1}^T k_t)^T
 *   LA_GDR_DECAYED_DELTA:  S_t = exp(g_t) S_{t-1} + beta_t k_t (v_t - exp(g_t) S_{t-1}^T k_t)^T
 *   o_t = scale * S_t^T q_t
 *
 * Data layout ("packed varlen"): the tokens of all sequences are
 * concatenated; sequence i owns rows cu_seqlens[i] .. cu_seqlens[i+1]-1.
 *   q, k   [T_total, H, dk]   io dtype (bf16 or fp32), row-major
 *   v, o   [T_total, H, dv]   io dtype
 *   g, beta[T_total, H]       fp32 (g <= 0 keeps every exponent <= 0; not checked)
 *   states [n, H, dk, dv]     fp32 (recurrent state, checkpoints, final state)
 * q, k, v, o, states and the workspace must be 16-byte aligned.
 *
 * Errors: a problem visible on the host (shape, dtype, alignment, an empty
 * suffix, a misaligned restored state, a short workspace) returns a status
 * before anything is launched and leaves every output untouched.  A failed
 * launch returns LA_ERR_HIP; la_last_error_message() then describes it.
 * All work is queued on the given stream in order; nothing synchronises the
 * host.  Outputs must not alias inputs.  The library allocates nothing and
 * keeps no pointer after a call returns.
 */
#ifndef LINATTN_H
#define LINATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum la_status {
    LA_OK = 0,
    LA_ERR_INVALID_ARG = 1,       /* null/misaligned pointer, bad size, bad table      */
    LA_ERR_UNSUPPORTED = 2,       /* valid but not built: head dims, chunk size         */
    LA_ERR_EMPTY_SUFFIX = 3,      /* resume with B_i == N_i (nothing to schedule)       */
    LA_ERR_MISALIGNED_STATE = 4,  /* resume with B_i not a multiple of C                */
    LA_ERR_HIP = 5,               /* HIP runtime reported an error                      */
    LA_ERR_WORKSPACE = 6          /* workspace smaller than la_prefill_workspace_bytes  */
} la_status;

typedef enum la_dtype { LA_F32 = 0, LA_BF16 = 1 } la_dtype;

typedef enum la_variant {
    LA_GDR_LITERAL = 0,           /* prediction S_{t-1}^T k_t                 */
    LA_GDR_DECAYED_DELTA = 1      /* prediction exp(g_t) S_{t-1}^T k_t        */
} la_variant;

/* Problem shape shared by the prefill entry points. */
typedef struct la_shape {
    int32_t n_seqs;          /* >= 1                                                 */
    int32_t n_heads;         /* H >= 1: this rank's heads                            */
    int32_t dk, dv;          /* head dims; built: dk, dv in {64, 128}                */
    int32_t chunk;           /* tokens per chunk; built: 64                          */
    int32_t ckpt_interval;   /* C >= 1: checkpoints at absolute multiples of C       */
    int32_t io_dtype;        /* la_dtype of q, k, v, o                               */
    int32_t variant;         /* la_variant                                           */
    float scale;             /* output scale (1.0 in the paper's setting)            */
} la_shape;

/*
 * strict_prefix_boundary - the repaired lookup rule (paper, section 2.2 and
 * section 3.2; the worked examples of Table 4).
 *
 * Restricting the lookup to the prompt without its last token selects
 * B = C * floor((N - 1) / C); the scheduler then computes the nonempty
 * suffix [B, N).  In a general cache the checkpoint must also be available:
 * with a contiguous cached prefix of `available_tokens` tokens,
 *     B = min(C * floor((N - 1) / C), C * floor(available_tokens / C)).
 * B = 0 means a cold start.  Writes B to *boundary_out.
 * Errors: LA_ERR_INVALID_ARG if n_tokens < 1, interval < 1,
 * available_tokens < 0 or boundary_out is NULL (nothing is written).
 * Host only; touches no device.
 */
la_status strict_prefix_boundary(int64_t n_tokens, int64_t interval,
                                 int64_t available_tokens, int64_t *boundary_out);

/*
 * la_prefill_workspace_bytes - size of the device workspace la_prefill and
 * la_prefill_resume need for `total_tokens` tokens over shape->n_seqs
 * sequences.  Returns 0 for an invalid or unsupported shape.  Host only.
 */
size_t la_prefill_workspace_bytes(const la_shape *shape, int64_t total_tokens);

/*
 * la_prefill - cold chunked prefill, the computation a cold recomputation
 * runs (paper, sections 2.2 and 5.5), emitting fp32 state checkpoints at
 * cache-block boundaries (the matched checkpoint schedule of section 4).
 *
 * Sequence i covers absolute positions [0, N_i) with N_i = cu[i+1] - cu[i]
 * (N_i = 0 is allowed: no output rows, zero final state).
 *   q, k, v, g, beta, o   device, layouts above
 *   cu_seqlens_dev/host   int32 [n_seqs + 1], same values on both sides;
 *                         cu[0] = 0, non-decreasing (host copy is validated)
 *   final_state           device fp32 [n_seqs, H, dk, dv] or NULL
 *   ckpt_out              device fp32 [rows, H, dk, dv] or NULL.  The state
 *                         for prefix [0, P) at every P = j*C <= N_i goes to
 *                         row ckpt_offsets[i] + (j - 1).
 *   ckpt_offsets_dev/host int32 [n_seqs] row offsets (required iff ckpt_out)
 *   workspace, ws_bytes   device scratch of la_prefill_workspace_bytes()
 *   stream                hipStream_t
 */
la_status la_prefill(const la_shape *shape,
                     const void *q, const void *k, const void *v,
                     const float *g, const float *beta,
                     const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                     void *o, float *final_state,
                     float *ckpt_out, const int32_t *ckpt_offsets_dev,
                     const int32_t *ckpt_offsets_host,
                     void *workspace, size_t ws_bytes, void *stream);

/*
 * la_prefill_resume - continue from restored states (paper, section 2.2:
 * computed = B, scheduled = N - B; section 5.2 reports exactly this first
 * batch after the repair).
 *
 * The token arrays hold only the suffixes: sequence i's rows are the tokens
 * at absolute positions [B_i, N_i), with N_i - B_i = cu[i+1] - cu[i].
 *   start_pos_dev/host  int64 [n_seqs]: B_i, the prefix the restored state
 *                       represents AND the position of the first scheduled
 *                       token (one number, so the two cannot disagree).
 *   state_in            device fp32 [n_seqs, H, dk, dv]: the state for prefix
 *                       [0, B_i) (zeros where B_i = 0).
 * Checkpoints are those at P = j*C with B_i < P <= N_i, to rows
 * ckpt_offsets[i] + (j - B_i / C - 1).  Other arguments as la_prefill.
 * Errors: LA_ERR_EMPTY_SUFFIX if some N_i - B_i == 0 (the pre-fix failure of
 * section 3.2 needs exactly such a call); LA_ERR_MISALIGNED_STATE if some
 * B_i is not a multiple of C (no checkpoint represents that prefix).
 */
la_status la_prefill_resume(const la_shape *shape,
                            const void *q, const void *k, const void *v,
                            const float *g, const float *beta,
                            const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                            const int64_t *start_pos_dev, const int64_t *start_pos_host,
                            const float *state_in,
                            void *o, float *final_state,
                            float *ckpt_out, const int32_t *ckpt_offsets_dev,
                            const int32_t *ckpt_offsets_host,
                            void *workspace, size_t ws_bytes, void *stream);

/*
 * la_checkpoint_rows - the checkpoint row numbering of one call, so that
 * callers need not re-derive it.  Sequence i (suffix length
 * cu[i+1] - cu[i], starting at absolute position B_i = start_pos_host[i], or
 * 0 when start_pos_host is NULL) owns the checkpoints at the absolute
 * multiples P of C with B_i < P <= B_i + len_i (section 2.2: the state for
 * prefix [0, P)), numbered consecutively from offsets_out[i]; the sequences'
 * blocks follow one another in order.  Writes offsets_out[n_seqs] and the
 * total row count.  Host only; errors: LA_ERR_INVALID_ARG for a decreasing
 * cu_seqlens, C < 1, a negative start or more than 2^31 rows.
 */
la_status la_checkpoint_rows(int32_t n_seqs, const int32_t *cu_seqlens_host, const int64_t *start_pos_host,
                             int64_t interval, int32_t *offsets_out, int64_t *total_rows_out);

/*
 * la_prefill_form - which kernels a prefill call of this shape runs.  The
 * form depends on the shape alone (never on the lengths), so a resume always
 * runs the arithmetic of the call that wrote its checkpoint:
 *   LA_FORM_FUSED_SCAN        bf16, checkpoint intervals below 8 chunks:
 *                             the chunk preparation, then one fused scan
 *                             (recurrence, output, checkpoints) per
 *                             (sequence, head);
 *   LA_FORM_FUSED_TWO_LEVEL   bf16, intervals of 8 chunks or more (C > 448):
 *                             the preparation, segment maps, the sequential
 *                             combine over segments and the fused replay;
 *   LA_FORM_TILE_SCAN_OUT     fp32, dk = 64: per-chunk operands, then one
 *                             scan wave and one output wave per 16 columns;
 *   LA_FORM_SPLIT_DK_SCAN     fp32, dk = 128: per-chunk operands, a scan
 *                             whose waves split dk, and the output kernel.
 * LA_FORM_NONE for an invalid or unsupported shape.  Host only.
 */
typedef enum la_form {
    LA_FORM_NONE = 0,
    LA_FORM_FUSED_SCAN = 1,
    LA_FORM_FUSED_TWO_LEVEL = 2,
    LA_FORM_TILE_SCAN_OUT = 3,
    LA_FORM_SPLIT_DK_SCAN = 4
} la_form;
la_form la_prefill_form(const la_shape *shape);

/*
 * la_prefill_scan_columns - state columns per workgroup of the fused scan
 * that a bf16 prefill call of this shape and these sequence lengths runs
 * (the single-level scan, or the replay of the two-level form).  The width
 * is a scheduling choice made from the chains' chunk counts: narrow
 * workgroups shorten each chunk's step, so the longest (sequence, head)
 * chains may run in 32-column workgroups while the others run in 64-column
 * ones.  Every column's arithmetic is the same at all widths, so no result
 * depends on it.  cu_seqlens_host: n_seqs + 1 prefix offsets, as for
 * la_prefill.  Returns 32, 64 or 128: the width of every chain, or 64 when
 * the call mixes 32 and 64; narrow_chains_out (may be NULL) receives the
 * number of chains, the longest, that run at 32 columns.  Returns 0 (and
 * 0 chains) for fp32, an invalid or unsupported shape, or invalid offsets.
 * Host only; reads nothing but its arguments.
 */
int la_prefill_scan_columns(const la_shape *shape, const int32_t *cu_seqlens_host, int64_t *narrow_chains_out);

/*
 * la_prefill_paged - a prefill (cold or resumed) whose checkpoints go
 * straight into pool pages and whose starting states come straight from pool
 * pages: the save of section 3.1 and the restore of a reload (sections 3.2
 * and 5.5, Table 5) folded into the prefill, with the pool and page layout
 * of la_state_save_paged / la_state_restore_paged (one page = one head's
 * [dk, dv] fp32 state).
 *
 *   pages->pool            device fp32 [n_pages, dk*dv], 16-byte aligned.
 *   pages->ckpt_page_ids   device int32 [rows * H] or NULL (no checkpoints):
 *                          checkpoint row r, head h (rows numbered by
 *                          ckpt_offsets exactly as ckpt_out's in
 *                          la_prefill_resume) is written to page
 *                          ckpt_page_ids[r * H + h]; -1 writes nothing.
 *   pages->state_page_ids  device int32 [n_seqs * H], required with
 *                          start_pos (a resume), NULL for a cold call:
 *                          (sequence i, head h) starts from page
 *                          state_page_ids[i * H + h], the state for prefix
 *                          [0, B_i); -1 starts from the zero state (B_i = 0).
 *   pages->err_count       device int32 or NULL: incremented once per page
 *                          id outside [-1, n_pages).  Such a checkpoint is
 *                          not written; such a start uses the zero state.
 * start_pos_dev/host NULL make a cold call.  ckpt_offsets are required with
 * ckpt_page_ids.  The pool must not alias the other buffers; a page read as
 * a starting state must not also be written as a checkpoint in the same
 * call.  Other arguments, results and errors as la_prefill_resume.
 */
typedef struct {
    float *pool;
    int64_t n_pages;
    const int32_t *ckpt_page_ids;
    const int32_t *state_page_ids;
    int32_t *err_count;
} la_pages;

la_status la_prefill_paged(const la_shape *shape, const la_pages *pages,
                           const void *q, const void *k, const void *v,
                           const float *g, const float *beta,
                           const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                           const int64_t *start_pos_dev, const int64_t *start_pos_host,
                           void *o, float *final_state,
                           const int32_t *ckpt_offsets_dev, const int32_t *ckpt_offsets_host,
                           void *workspace, size_t ws_bytes, void *stream);

/*
 * la_prefill_paged_noalloc - la_prefill_paged without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).  The call
 * allocates nothing: its workspace is a 64 MiB static device array inside
 * the library, one per device, held until the process ends (its address is
 * looked up once per device, on the first call there).  Calls whose
 * workspace (la_prefill_workspace_bytes for the shape and cu_seqlens[n_seqs]
 * tokens) exceeds 64 MiB return LA_ERR_WORKSPACE before any launch.  Every
 * call on a device shares that device's array, and nothing in it has to
 * start at zero (each call writes what it reads); calls that overlap on one
 * device (e.g. on two streams) race and must not be issued.  Arguments,
 * results and other errors as la_prefill_paged.
 */
la_status la_prefill_paged_noalloc(const la_shape *shape, const la_pages *pages,
                                   const void *q, const void *k, const void *v,
                                   const float *g, const float *beta,
                                   const int32_t *cu_seqlens_dev, const int32_t *cu_seqlens_host,
                                   const int64_t *start_pos_dev, const int64_t *start_pos_host,
                                   void *o, float *final_state,
                                   const int32_t *ckpt_offsets_dev, const int32_t *ckpt_offsets_host,
                                   void *stream);

/*
 * la_decode_step - decode continuation: advance every (sequence, head) by one
 * generated token from its fp32 state (the recurrent state of section 2.1,
 * continued after a cold prefill or a reload; sections 5.1, 5.4 and 5.5
 * compare 64-, 256- and 128-token continuations).
 *
 * q, k: [n_seqs, H, dk]; v: [n_seqs, H, dv] in shape->io_dtype; g, beta:
 * [n_seqs, H] fp32; state: [n_seqs, H, dk, dv] fp32, read and overwritten
 * with the state after the token (16-byte aligned); o: [n_seqs, H, dv] in
 * io_dtype, o = scale * S_new^T q.  The recurrence is the prefill's
 * (shape->variant selects the prediction), token by token in fp32.
 * shape->chunk and ckpt_interval are validated as for the prefill and
 * otherwise unused.  All buffers device, caller-owned; outputs must not
 * alias inputs other than state.  Errors: INVALID_ARG (NULL pointer,
 * misaligned state), UNSUPPORTED (dk, dv outside {64, 128}), HIP.
 */
la_status la_decode_step(const la_shape *shape,
                         const void *q, const void *k, const void *v,
                         const float *g, const float *beta,
                         float *state, void *o, void *stream);

/*
 * la_state_save_paged - scatter states into a paged fp32 pool (the paper's
 * page rows, section 3.1 and Table 5; a save must complete before dependent
 * reuse, so order the reuse on the same stream or behind an event).
 *
 * Item n of `states` ([n_items, page_elems] fp32, device) goes to
 * pool page page_ids[n] ([n_pages, page_elems] fp32, device).  Id -1 skips
 * the item; any other id outside [0, n_pages) skips it and increments
 * *err_count_dev (device int32, may be NULL).  Duplicate destination ids in
 * one call are a caller error (unspecified winner).  page_elems must be a
 * positive multiple of 4; states and pool 16-byte aligned.
 */
la_status la_state_save_paged(const float *states, int64_t n_items, int64_t page_elems,
                              float *pool, int64_t n_pages, const int32_t *page_ids_dev,
                              int32_t *err_count_dev, void *stream);

/*
 * la_state_restore_paged - gather states from the pool (the reload of
 * section 3.2 / 5.5).  states[n] = pool[page_ids[n]]; id -1 writes a zero
 * state (cold start); any other out-of-range id leaves states[n] untouched
 * and increments *err_count_dev.  Sizes and alignment as the save.
 */
la_status la_state_restore_paged(const float *pool, int64_t n_pages,
                                 const int32_t *page_ids_dev, float *states,
                                 int64_t n_items, int64_t page_elems,
                                 int32_t *err_count_dev, void *stream);

/*
 * la_hybrid_boundary - the position a hybrid cache resumes from: attention
 * KV blocks and recurrent checkpoints restored together at one B.  A reload
 * moves both kinds of entries (section 2.1; Table 5), and the attention
 * prefix must end where the checkpoint's prefix ends (sections 1 and 6).
 *
 * B is the strict-prefix boundary (section 2.2) over the shorter of the two
 * cached prefixes: the largest multiple of C with B <= N - 1, B <=
 * kv_cached_tokens (the first KV blocks, of kv_block_tokens tokens each,
 * that are cached contiguously) and B <= state_cached_tokens (checkpoints
 * exist at every multiple of C up to it).  *kv_blocks_out = B /
 * kv_block_tokens, the blocks that cover [0, B).  Errors: INVALID_ARG for
 * N < 1, C < 1, kv_block_tokens < 1, negative cached lengths or NULL
 * outputs; MISALIGNED_STATE when kv_block_tokens does not divide C (no
 * checkpoint position falls on a block boundary).
 */
la_status la_hybrid_boundary(int64_t n_tokens, int64_t interval, int64_t kv_block_tokens,
                             int64_t kv_cached_tokens, int64_t state_cached_tokens,
                             int64_t *boundary_out, int64_t *kv_blocks_out);

/*
 * la_hybrid_restore - restore, in one launch, every sequence's attention KV
 * blocks of the prefix [0, B_i) and its recurrent state pages of the
 * checkpoint at B_i (the joint reload of section 2.1 and Table 5, at the
 * boundary la_hybrid_boundary gives).
 *
 * kv: the attention KV pages of this rank, opaque bytes.
 *   pool     [n_pool_blocks, block_bytes]: device memory, or pinned host
 *            memory mapped into the device (the CPU tier of section 2.1).
 *   cache    [n_cache_blocks, block_bytes] device: the engine's KV cache.
 *   src_ids, dst_ids  device int32 [n_seqs, max_blocks]: block j < B_i /
 *            block_tokens of sequence i goes from pool[src_ids[i][j]] to
 *            cache[dst_ids[i][j]]; either id -1 skips it, ids out of range
 *            skip it and count.  block_bytes a positive multiple of 16.
 * boundary_dev/host  int64 [n_seqs]: B_i, a multiple of block_tokens with
 *            B_i / block_tokens <= max_blocks (MISALIGNED_STATE / INVALID_ARG
 *            before any launch otherwise).
 * State pages (page_elems fp32 each, one head's state, as la_state_restore_paged):
 *   state_pool [n_state_pages, page_elems]: device or pinned host memory;
 *   state_page_ids_dev int32 [n_seqs * n_heads]; states [n_seqs * n_heads,
 *   page_elems] device: id -1 writes the zero state, ids out of range leave
 *   the item untouched and count.  n_heads = 0 restores no state.
 * err_count_dev (device int32, may be NULL) counts every out-of-range id.
 * Pools given as pinned host memory are checked with
 * hipPointerGetAttributes before any launch (pageable memory: INVALID_ARG).
 * The caller owns every buffer; cache and states must not alias the pools.
 */
typedef struct {
    const void *pool;
    int64_t n_pool_blocks;
    void *cache;
    int64_t n_cache_blocks;
    int64_t block_bytes;
    int64_t block_tokens;
    const int32_t *src_ids;
    const int32_t *dst_ids;
    int64_t max_blocks;
} la_kv_blocks;

la_status la_hybrid_restore(const la_kv_blocks *kv, int32_t n_seqs, int32_t n_heads, int64_t page_elems,
                            const int64_t *boundary_dev, const int64_t *boundary_host,
                            const float *state_pool, int64_t n_state_pages,
                            const int32_t *state_page_ids_dev, float *states,
                            int32_t *err_count_dev, void *stream);

/*
 * la_state_save_host / la_state_restore_host - the host-memory tier: the
 * same page scatter and gather as la_state_save_paged / la_state_restore_paged
 * with the pool in pinned host memory (the paper's CPU reload path, section
 * 2.1 and Table 5; section 3.1 requires a save to complete before the pages
 * are reused, and section 5.5 times CPU reloads).
 *
 * host_pool: [n_pages, page_elems] fp32 in pinned host memory mapped into the
 * device's address space (hipHostMalloc, or a torch tensor allocated with
 * pin_memory=True), 16-byte aligned; the kernels move pages over the host
 * link directly.  Both ends of the pool are checked with
 * hipPointerGetAttributes before any launch: pageable or unmapped memory
 * returns INVALID_ARG.  states, page ids and err_count are device memory,
 * with the meanings, -1 / out-of-range handling and alignment of the
 * device-pool calls.  The copy is asynchronous on `stream`; if done_event
 * (a hipEvent_t, may be NULL) is given it is recorded after the copy, so the
 * host may poll or wait on it before reading saved pages (save) or before
 * overwriting pages being restored (restore).
 */
la_status la_state_save_host(const float *states, int64_t n_items, int64_t page_elems,
                             float *host_pool, int64_t n_pages, const int32_t *page_ids_dev,
                             int32_t *err_count_dev, void *stream, void *done_event);
la_status la_state_restore_host(const float *host_pool, int64_t n_pages, const int32_t *page_ids_dev,
                                float *states, int64_t n_items, int64_t page_elems,
                                int32_t *err_count_dev, void *stream, void *done_event);

/* Name of a status code (static string). */
const char *la_status_string(la_status status);

/* Description of the last error returned on this thread (static per thread). */
const char *la_last_error_message(void);

/*
 * la_trace_set_events - profiling hook.  When `events` holds at least 4
 * hipEvent_t (created by the caller), every later la_prefill,
 * la_prefill_resume and la_prefill_paged call on this thread records, on the
 * call's stream, events[0] before its first kernel, events[1] after the
 * chunk-preparation kernel, events[2] after the segment maps and their
 * combine (two-level forms; directly after events[1] otherwise) and
 * events[3] after the last scan kernel (the fused scan, the segment replay,
 * or the fp32 scan and output kernels).  The events are overwritten by each
 * call.  n_events = 0 (or events = NULL) switches it off.
 */
void la_trace_set_events(void *const *events, int32_t n_events);

#ifdef __cplusplus
}
#endif

#endif /* LINATTN_H */
