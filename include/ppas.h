/*
 * ppas.h -- C ABI of libppas.so: one mixed scheduler step's attention over a
 * paged KV cache on an AMD Instinct MI355X (gfx950).
 *
 * A scheduler iteration batches prefill chunks and single-token decode rows of
 * different requests under one token budget (P-PAS paper, Section 2: continuous
 * batching with chunked prefill; Section 6.2: prefill and decode tokens sharing
 * an iteration). Prefill and decode store each token's key and value in the KV
 * cache (Section 2), which is paged (Section 7, PagedAttention). A step is two
 * calls on one stream: ppas_kv_append writes the step's new keys/values into
 * the pages (or ppas_rope_kv_append, which first rotates the new query and key
 * rows by their positions), then ppas_attn_step computes the attention of
 * every query row.
 *
 * Conventions shared by every entry point
 *   - bf16 means IEEE bfloat16 bit patterns (uint16 in memory).
 *   - Device pointers are HIP device memory on the current device; host pointers
 *     are ordinary host memory. The caller owns every buffer. The library
 *     allocates no device memory; it keeps a pool of pinned host buffers that
 *     hold its work lists (read by the kernels directly), released at process
 *     exit, and ppas_attn_step_noalloc uses one fixed device array per device.
 *   - No state is shared between calls other than that pool and that array:
 *     planning choices and profiling events are arguments of the calls that
 *     use them.
 *   - All device work is enqueued on `hip_stream` (a hipStream_t, NULL = the
 *     null stream) and the call returns without synchronising the host. Calls
 *     on the same stream execute in order; append before attending.
 *   - Every argument is validated on the host before anything is enqueued; a
 *     failed validation enqueues nothing. No C++ exception crosses the ABI.
 *   - Compiled shapes: head_dim 128, page_size 16, n_q_heads / n_kv_heads == 8
 *     (grouped-query attention; query head h reads KV head h / 8). Anything else
 *     returns PPAS_EUNSUPPORTED.
 *
 * Layouts
 *   q, out      [T][n_q_heads][128] bf16, row t = query token t of the step.
 *   k_new,v_new [T][n_kv_heads][128] bf16, the step's new keys/values, same rows.
 *   k_pages     [num_pages][n_kv_heads][16][16][8] bf16: per page and KV head,
 *               16 chunks of 8 consecutive features; chunk c holds the 16
 *               tokens' features 8c..8c+7, token after token (chunk-major).
 *   v_pages     [num_pages][n_kv_heads][128][16] bf16: per page and KV head,
 *               128 feature rows of 16 contiguous tokens.
 *   block_table [n_seqs][bt_stride] int32: entry j of request s is the physical
 *               page holding its positions 16j..16j+15. Entries past the
 *               request's last page are ignored (conventionally -1).
 *   seqs        host array of n_seqs descriptors (query_start, n_query,
 *               cached_len). Request s owns rows query_start..query_start+n-1,
 *               at positions cached_len..cached_len+n-1; query_start must start
 *               at 0 and be contiguous (query_start[s+1] = query_start[s] + n[s]),
 *               so T = sum of n_query. n_query == 1 is a decode row.
 */
#ifndef PPAS_H
#define PPAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum ppas_status {
  PPAS_OK = 0,
  PPAS_EINVAL = -1,        /* malformed argument: null pointer, bad descriptor, bad stride */
  PPAS_ERANGE = -2,        /* a block-table entry outside [0, num_pages), a length overflow, or a step
                               too large for the int32 work list */
  PPAS_ENOSPACE = -3,      /* workspace smaller than ppas_attn_workspace_bytes(), or a step too large
                               for the fixed array of ppas_attn_step_noalloc */
  PPAS_EHIP = -4,          /* a HIP runtime call or kernel launch failed */
  PPAS_EUNSUPPORTED = -5   /* shape outside the compiled set, or no gfx950 device */
} ppas_status;

typedef struct ppas_shape {
  int32_t n_q_heads;    /* query heads (16 for the Qwen2.5-3B attention shape) */
  int32_t n_kv_heads;   /* KV heads; n_q_heads / n_kv_heads must be 8 */
  int32_t head_dim;     /* must be 128 */
  int32_t page_size;    /* tokens per page; must be 16 */
  int32_t num_pages;    /* pages in each of the K and V pools */
  float scale;          /* softmax scale applied to q.k (1/sqrt(head_dim) by convention) */
} ppas_shape;

typedef struct ppas_seq {
  int32_t query_start;  /* first query row of this request in q/out/k_new/v_new */
  int32_t n_query;      /* new tokens of this request in the step, >= 1 */
  int32_t cached_len;   /* tokens already in the cache before this step, >= 0 */
} ppas_seq;

/*
 * Planning choices of one call (this library's own tuning, not a quantity of
 * the paper). A zeroed struct, or NULL where a pointer is taken, selects the
 * automatic choice for every field.
 */
typedef struct ppas_plan_opts {
  int32_t prefill_split;    /* > 0: at most this many keys per prefill work item (rounded up to a
                               multiple of 64); 0: about two prefill items per compute unit */
  int32_t decode_split;     /* > 0: at most this many keys per decode work item (rounded up to a
                               multiple of 32, capped at 16384); 0: automatic */
  int32_t tile_positions;   /* 16 or 32: prefill tiles of that many positions (four- or eight-wave
                               kernel); 0: chosen per step. Any other value is PPAS_EINVAL */
  int32_t num_cus;          /* > 0: plan for a device with this many compute units; 0: the current
                               device's count (ppas_plan_items: 256) */
} ppas_plan_opts;

/*
 * HIP events (hipEvent_t handles created by the caller) that a call's kernel
 * launches record as they start and end, so a kernel's own duration can be
 * read with hipEventElapsedTime. Each pair is either both NULL (not recorded)
 * or both set (PPAS_EINVAL otherwise).
 *   start, stop              the call's main kernel: the packed attention
 *                            launch, or the page-write launch of an append
 *   merge_start, merge_stop  the split-merge launch of an attention call; not
 *                            recorded when the call merges no split row
 *                            (ppas_step_plan_info tells whether it does)
 */
typedef struct ppas_events {
  void* start;
  void* stop;
  void* merge_start;
  void* merge_stop;
} ppas_events;

/* Human-readable name of a status code. Never NULL; the string is static. */
const char* ppas_status_string(ppas_status status);

/*
 * Host-only check of a step description (no HIP call; usable without a GPU).
 * The description is the one of a scheduler iteration in Section 2: each
 * request contributes n_query new tokens (a prefill chunk, or one decode
 * token) after cached_len tokens already in the KV cache, stored in pages
 * (Section 7, PagedAttention) that the block table names. The checks
 * themselves are this library's own:
 * the shape (PPAS_EUNSUPPORTED outside the compiled set, PPAS_EINVAL for
 * non-positive sizes or a non-finite scale), each descriptor (n_query >= 1,
 * cached_len >= 0, contiguous query_start from 0, cached_len + n_query fitting in
 * int32: PPAS_EINVAL / PPAS_ERANGE), bt_stride >= ceil((cached_len+n_query)/16)
 * for every request (PPAS_EINVAL), and, when block_table_host is not NULL, that
 * every entry a request uses lies in [0, num_pages) (PPAS_ERANGE) and that no
 * two requests write the same (page, slot) in this step (PPAS_EINVAL). The cost
 * grows with the pages the requests use, not with num_pages.
 * n_seqs == 0 is a valid empty step.
 */
ppas_status ppas_validate_step(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                               const int32_t* block_table_host, int32_t bt_stride);

/*
 * Append the step's new keys and values to the paged cache (Section 2: the
 * processed tokens' keys and values are stored in the KV cache).
 * For every request s and i < n_query: position p = cached_len + i,
 * page = block_table[s][p / 16], slot = p % 16;
 *   k_pages[page][g][d / 8][slot][d % 8] = k_new[query_start + i][g][d]
 *   v_pages[page][g][:][slot] = v_new[query_start + i][g][:]   for every KV head g.
 * Bit-exact copies; no other byte of the pools is written. One kernel launch
 * for any number of requests. block_table_dev is the device copy of the table;
 * block_table_host (nullable) is a host copy used only for validation (range
 * and overlap checks are skipped when it is NULL, and out-of-range device
 * entries then give undefined results).
 * Returns PPAS_OK or a validation / PPAS_EHIP status.
 */
ppas_status ppas_kv_append(const ppas_shape* shape, void* k_pages, void* v_pages,
                           const void* k_new, const void* v_new,
                           const ppas_seq* seqs, int32_t n_seqs,
                           const int32_t* block_table_dev, int32_t bt_stride,
                           const int32_t* block_table_host, void* hip_stream);

/*
 * Rotary position embedding of the step's new rows, fused with the append.
 * The paper does not describe positional encoding; the operation is the
 * standard rotary embedding (RoPE) in rotate-half form over the whole head,
 * applied to the new query and key rows of a decoder block's attention
 * (Section 6.1) before they are used and cached. For every request s and
 * i < n_query: row r = query_start + i at position p = cached_len + i; for
 * every pair j < 64 the angle is a = p * rope_theta^(-2j/128), and a head row x
 * becomes (x_j cos a - x_{j+64} sin a) at j and (x_{j+64} cos a + x_j sin a) at
 * j + 64.
 *   q [T][n_q_heads][128] bf16: every query head row r is rotated in place.
 *   k_new [T][n_kv_heads][128] bf16: rotated and written to k_pages at (page,
 *     slot) exactly as ppas_kv_append writes keys; k_new itself is not modified.
 *   v_new: copied to v_pages unrotated, bit-exact, as ppas_kv_append does.
 * Angles are reduced in fp64, cos/sin taken in fp32, the rotation computed in
 * fp32 and rounded to bf16 nearest-even. Nothing else in q or the pools is
 * written. rope_theta must be finite and > 0 (else PPAS_EINVAL); q must not
 * be NULL. Validation, ownership and errors otherwise as ppas_kv_append. Call
 * it in place of ppas_kv_append, before ppas_attn_step, on the same stream.
 */
ppas_status ppas_rope_kv_append(const ppas_shape* shape, float rope_theta, void* q,
                                void* k_pages, void* v_pages,
                                const void* k_new, const void* v_new,
                                const ppas_seq* seqs, int32_t n_seqs,
                                const int32_t* block_table_dev, int32_t bt_stride,
                                const int32_t* block_table_host, void* hip_stream);

/*
 * Device workspace that ppas_attn_step needs for this step description on the
 * current device, with the automatic planning choices. This sizing call is the
 * library's own (the paper describes no workspace): the workspace holds the
 * fp32 partial results of rows whose keys are split across workgroups of the
 * launch (at least 256 bytes). Depends only on the shape, the descriptors and
 * the device's compute-unit count. Returns 0 if the description is invalid.
 */
size_t ppas_attn_workspace_bytes(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs);

/*
 * Attention of every query row of the step (Section 2 chunked prefill and
 * decode; Section 6.2 mixed iterations). For request s, row i at position
 * p = cached_len + i, query head h and KV head g = h / 8:
 *   out[query_start+i][h][:] = sum_{j<=p} softmax_j(scale * q[.][h] . K_s[j][g]) V_s[j][g][:]
 * where K_s/V_s are request s's keys/values at positions 0..p read from the
 * pages through block_table (the step's own keys must already be appended).
 * Prefill rows (n_query > 1) are causal within their chunk and see the whole
 * cached prefix; decode rows (n_query == 1) see cached_len + 1 keys. Inputs bf16,
 * fp32 accumulation, output rounded to bf16 (nearest even).
 * All rows of all requests run in one packed launch; rows whose keys were split
 * across workgroups are merged by a second, small launch.
 * workspace: device buffer of at least ppas_attn_workspace_bytes() bytes, owned
 * by the caller, not read before being written; it must not be used by another
 * call still in flight. The work list travels in pinned host memory from a pool
 * the library owns, read by the kernels directly; a buffer of the pool is
 * reused only after the launches that read it have completed. Because the work
 * list is staged per call, a call cannot be captured into a HIP graph and
 * replayed. Calls from several threads or on several streams are safe (each
 * with its own workspace). Equivalent to creating a step plan with default
 * options, ppas_attn_step_planned, and destroying the plan.
 * Returns PPAS_OK, a validation status, PPAS_ENOSPACE or PPAS_EHIP.
 */
ppas_status ppas_attn_step(const ppas_shape* shape, void* out, const void* q,
                           const void* k_pages, const void* v_pages,
                           const ppas_seq* seqs, int32_t n_seqs,
                           const int32_t* block_table_dev, int32_t bt_stride,
                           const int32_t* block_table_host,
                           void* workspace, size_t workspace_bytes, void* hip_stream);

/*
 * Step plans. One scheduler iteration runs every decoder layer over the same
 * batch of requests (Section 2: an iteration processes the batch's tokens
 * through the model; Section 6.1 profiles one decoder block of it), so the
 * host work of a step (validation, the attention work list, the page-write
 * list) is the same for every layer. A plan holds that work once, for as many
 * launches as the caller makes with it: ppas_kv_append_planned,
 * ppas_rope_kv_append_planned and ppas_attn_step_planned then only launch
 * kernels. The plan keeps the shape, the descriptors' work and bt_stride; each
 * planned call takes the layer's device buffers and block table (same stride).
 *
 * ppas_step_plan_create validates as ppas_validate_step does (with the range
 * and overlap checks when block_table_host is not NULL), plans with `opts`
 * (NULL = automatic) for the current device, and stores the lists in pinned
 * host memory from the library's pool. *plan receives the handle (NULL on
 * error). Returns PPAS_OK, a validation status, PPAS_ERANGE for a step too
 * large for the int32 work list, PPAS_EUNSUPPORTED without a gfx950 device, or
 * PPAS_EHIP.
 */
typedef struct ppas_step_plan ppas_step_plan;

ppas_status ppas_step_plan_create(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                                  const int32_t* block_table_host, int32_t bt_stride,
                                  const ppas_plan_opts* opts, ppas_step_plan** plan);

/* What a plan launches (host only). */
typedef struct ppas_plan_info {
  int32_t n_items;          /* workgroups of the packed attention launch */
  int32_t n_merge;          /* split-merge items (0: no merge launch) */
  int32_t tile_positions;   /* 16 or 32 */
  int32_t n_append;         /* (request, page) workgroups of a page-write launch */
  uint64_t workspace_bytes; /* workspace ppas_attn_step_planned needs */
} ppas_plan_info;

ppas_status ppas_step_plan_info(const ppas_step_plan* plan, ppas_plan_info* info);

/* As ppas_kv_append, with the plan's descriptors and validation; events may be NULL. */
ppas_status ppas_kv_append_planned(const ppas_step_plan* plan, void* k_pages, void* v_pages,
                                   const void* k_new, const void* v_new,
                                   const int32_t* block_table_dev, const ppas_events* events,
                                   void* hip_stream);

/* As ppas_rope_kv_append, with the plan's descriptors and validation; events may be NULL. */
ppas_status ppas_rope_kv_append_planned(const ppas_step_plan* plan, float rope_theta, void* q,
                                        void* k_pages, void* v_pages,
                                        const void* k_new, const void* v_new,
                                        const int32_t* block_table_dev, const ppas_events* events,
                                        void* hip_stream);

/*
 * As ppas_attn_step, with the plan's descriptors, validation and work list
 * (workspace of at least ppas_plan_info.workspace_bytes); events may be NULL.
 * Calls with one plan may run on several streams at once, each with its own
 * workspace.
 */
ppas_status ppas_attn_step_planned(const ppas_step_plan* plan, void* out, const void* q,
                                   const void* k_pages, const void* v_pages,
                                   const int32_t* block_table_dev,
                                   void* workspace, size_t workspace_bytes,
                                   const ppas_events* events, void* hip_stream);

/*
 * Release a plan (NULL is a no-op). Does not wait: the plan's pinned memory
 * returns to the pool and is reused only after every launch made with the plan
 * has completed.
 */
void ppas_step_plan_destroy(ppas_step_plan* plan);

/*
 * Work-list introspection for tests (host only, no HIP call). Plans the step
 * with `opts` (NULL = automatic; num_cus 0 = 256 compute units) and writes at
 * most `capacity` items of 8 int32 each to `items_out` (kind, seq, kv_head, row0,
 * pos0, npos, key_lo, key_hi per item, in launch order; kind 0 = prefill tile,
 * 1 = decode row). Returns the number of items, or a negative ppas_status
 * (PPAS_EINVAL also for an invalid opts field).
 */
int32_t ppas_plan_items(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                        const ppas_plan_opts* opts, int32_t* items_out, int32_t capacity);

/*
 * The fused gate-up projection of a decoder block's MLP, the other prefill
 * operation the paper profiles next to attention (Section 6.1: cumulative time
 * of eight 2k chunks against one 16k chunk, Fig. 4b; SM throughput, L2 hit rate
 * and DRAM throughput at both chunk sizes, Table 6). The gate and up
 * projections read the same hidden states and run as one linear layer whose
 * weight stacks the gate rows over the up rows:
 *   y[t][n] = sum_k x[t][k] * w[n][k]      t < n_tokens, n < n_out
 * x [n_tokens][hidden] bf16 (the chunk's normalised hidden states), w
 * [n_out][hidden] bf16 (row-major, gate rows 0..n_out/2-1 then up rows; any
 * n_out >= 1 is accepted), y [n_tokens][n_out] bf16, all device memory owned by
 * the caller. fp32 accumulation, output rounded to bf16 nearest-even; the
 * activation that follows is not applied. When a call's 256 x 256 output
 * tiles are fewer than the device's compute units, the reduction over hidden
 * is split across several workgroups per tile; their fp32 partial sums go to
 * the caller's workspace (ppas_gateup_workspace_bytes, device memory, not read
 * before written, not shared with a call still in flight) and a second launch
 * adds them in a fixed order. A workspace smaller than that (NULL with 0 bytes
 * included) gives fewer splits, down to none: results are deterministic for a
 * given shape and workspace size, and every split count stays within the same
 * rounding bound. The kernels run on hip_stream (events: start on the first
 * launch, stop on the last, as for the other calls; may be NULL); no host sync.
 * hidden must be a positive multiple of 64 (PPAS_EUNSUPPORTED otherwise);
 * n_tokens == 0 is a no-op; NULL pointers (a NULL workspace with a non-zero
 * size included) or non-positive sizes are PPAS_EINVAL; n_tokens or n_out above
 * 2^31 - 513, or more than 2^31 - 1 output tiles of 256 x 256, is PPAS_ERANGE.
 */
ppas_status ppas_gateup_proj(const void* x, const void* w, void* y, int32_t n_tokens, int32_t hidden,
                             int32_t n_out, void* workspace, size_t workspace_bytes,
                             const ppas_events* events, void* hip_stream);

/* Workspace ppas_gateup_proj uses for this shape on the current device (0 when
 * it does not split the reduction, or for an invalid shape). The library's own
 * sizing call: the paper describes no workspace. */
size_t ppas_gateup_workspace_bytes(int32_t n_tokens, int32_t hidden, int32_t n_out);

/*
 * The same projection with the MLP's gated activation applied on the way out:
 * the paper profiles the projection (Section 6.1, Fig. 4b, Table 6); in the
 * Qwen2.5 models it measures, the MLP then multiplies the SiLU of the gate half
 * by the up half, and doing that in the projection's epilogue writes half the
 * bytes and saves a pass over them (the library's own fusion). With n_inter
 * intermediate features and w [2 n_inter][hidden] (gate rows 0..n_inter-1, then
 * the up rows of the same features):
 *   y[t][f] = silu(g) * u,  g = sum_k x[t][k] w[f][k],  u = sum_k x[t][k] w[n_inter + f][k],
 *   silu(g) = g / (1 + e^-g),  t < n_tokens, f < n_inter
 * y [n_tokens][n_inter] bf16; g and u are accumulated in fp32 as in
 * ppas_gateup_proj, silu(g) * u is evaluated in fp32 and rounded to bf16
 * nearest-even. Workspace, splits, events, streams and status codes as for
 * ppas_gateup_proj with n_out = 2 n_inter; n_inter above (2^31 - 513) / 2 is
 * PPAS_ERANGE.
 */
ppas_status ppas_gateup_act(const void* x, const void* w, void* y, int32_t n_tokens, int32_t hidden,
                            int32_t n_inter, void* workspace, size_t workspace_bytes,
                            const ppas_events* events, void* hip_stream);

/* Workspace ppas_gateup_act uses for this shape on the current device (0 when it
 * does not split the reduction, or for an invalid shape). The library's own
 * sizing call. */
size_t ppas_gateup_act_workspace_bytes(int32_t n_tokens, int32_t hidden, int32_t n_inter);

/*
 * A plain streaming read of `bytes` bytes of device memory at `buf`: the
 * device's attainable HBM read rate, the measured ceiling beside the spec peak
 * for the memory-bound kernels above (the library's own measurement aid, not a
 * step of the method). Every 16-byte word is read once with nontemporal loads by
 * one 256-thread workgroup per compute unit, each wave reading contiguous 8 KB
 * runs; the XOR of all words, as four uint32 lanes, is XORed into the 16 bytes
 * of device memory at `sink` (zero it first to receive the XOR itself), so the
 * reads cannot be elided and the result is checkable. `buf` and `bytes` must be multiples of 16 and `sink`
 * 4-byte aligned (PPAS_EINVAL otherwise); bytes == 0 is a no-op. Enqueued on
 * hip_stream without a host sync; the launch records `events` if given.
 */
ppas_status ppas_stream_read(const void* buf, size_t bytes, void* sink, const ppas_events* events,
                             void* hip_stream);

/*
 * For callers that cannot allocate memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc. Computes exactly what
 * ppas_attn_step computes, with the same plan and kernels (bit-identical
 * output), but takes no workspace and uses neither a caller buffer nor the
 * library's pinned host pool: the step's work list (32 bytes per work item)
 * and, after it, the fp32 partials of rows split across workgroups live in a
 * fixed device array of PPAS_NOALLOC_SCRATCH_BYTES that every device the call
 * runs on holds until the process ends. The call allocates nothing
 * (no hipMalloc, hipFree, hipHostMalloc); the first call on a device looks up
 * that device's array (hipGetSymbolAddress).
 *
 * The work list is copied from host memory to the array with hipMemcpyAsync on
 * hip_stream during the call, then the attention and merge launches follow on
 * the same stream. Every call on one device shares that device's array, which
 * keeps the last call's contents (nothing in it needs to start at zero): calls
 * ordered on one stream are safe, but calls that overlap in time on one device
 * (other streams, other threads) race and give undefined results.
 *
 * A step whose work list and partials do not fit the array returns
 * PPAS_ENOSPACE and enqueues nothing (steps of up to ~40 MB of partials fit,
 * e.g. two 1,024-token chunks plus 48 decode rows of 20k-30k keys).
 * Arguments, validation and other errors as ppas_attn_step.
 */
#define PPAS_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

ppas_status ppas_attn_step_noalloc(const ppas_shape* shape, void* out, const void* q,
                                   const void* k_pages, const void* v_pages,
                                   const ppas_seq* seqs, int32_t n_seqs,
                                   const int32_t* block_table_dev, int32_t bt_stride,
                                   const int32_t* block_table_host, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* PPAS_H */
