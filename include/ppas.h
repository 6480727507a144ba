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
 *     allocates no device memory; it keeps a small pinned host staging ring for
 *     uploading its work list, released at process exit.
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
  PPAS_ENOSPACE = -3,      /* workspace smaller than ppas_attn_workspace_bytes() */
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

/* Human-readable name of a status code. Never NULL; the string is static. */
const char* ppas_status_string(ppas_status status);

/*
 * Host-only check of a step description (no HIP call; usable without a GPU).
 * Checks the shape (PPAS_EUNSUPPORTED outside the compiled set, PPAS_EINVAL for
 * non-positive sizes or a non-finite scale), each descriptor (n_query >= 1,
 * cached_len >= 0, contiguous query_start from 0, cached_len + n_query fitting in
 * int32: PPAS_EINVAL / PPAS_ERANGE), bt_stride >= ceil((cached_len+n_query)/16)
 * for every request (PPAS_EINVAL), and, when block_table_host is not NULL, that
 * every entry a request uses lies in [0, num_pages) (PPAS_ERANGE) and that no
 * two requests write the same (page, slot) in this step (PPAS_EINVAL).
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
 * Bit-exact copies; no other byte of the pools is written. block_table_dev is
 * the device copy of the table; block_table_host (nullable) is a host copy used
 * only for validation (range and overlap checks are skipped when it is NULL,
 * and out-of-range device entries then give undefined results).
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
 * current device: fp32 partial results of rows whose keys are split across
 * workgroups (at least 256 bytes). Depends only on the shape, the descriptors
 * and the device's compute-unit count. Returns 0 if the description is invalid.
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
 * call still in flight. The work list itself travels in pinned host memory the
 * library owns (a ring of eight staging buffers per device, read by the kernels
 * directly); a call waits on the device only when the buffer it would reuse is
 * still being read by a launch eight calls back. Because the work list is staged
 * per call, a call cannot be captured into a HIP graph and replayed. Calls from
 * several threads or on several streams are safe (each with its own workspace).
 * Returns PPAS_OK, a validation status, PPAS_ENOSPACE or PPAS_EHIP.
 */
ppas_status ppas_attn_step(const ppas_shape* shape, void* out, const void* q,
                           const void* k_pages, const void* v_pages,
                           const ppas_seq* seqs, int32_t n_seqs,
                           const int32_t* block_table_dev, int32_t bt_stride,
                           const int32_t* block_table_host,
                           void* workspace, size_t workspace_bytes, void* hip_stream);

/*
 * Work-list introspection for tests (host only, no HIP call). Plans the step for
 * a device with `num_cus` compute units and writes at most `capacity` items of 8
 * int32 each to `items_out` (kind, seq, kv_head, row0, pos0, npos, key_lo,
 * key_hi per item, in launch order; kind 0 = prefill tile, 1 = decode row).
 * Returns the number of items, or a negative ppas_status.
 */
int32_t ppas_plan_items(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                        int32_t num_cus, int32_t* items_out, int32_t capacity);

/*
 * Planner tuning (process-wide; 0 restores the automatic choice). prefill_split
 * and decode_split cap the keys one workgroup processes for a prefill tile /
 * a decode row (rounded to multiples of 64 / 32). Affects plans made after the
 * call, including ppas_attn_workspace_bytes. Returns PPAS_EINVAL for negative
 * values.
 */
ppas_status ppas_set_split_keys(int32_t prefill_split, int32_t decode_split);

/*
 * Planner tuning (process-wide). The packed launch comes in two shapes: prefill
 * tiles of 16 positions on four-wave workgroups, or of 32 positions on
 * eight-wave workgroups (each staged K/V block then serves twice the rows). By
 * default (0) each step picks 32 only when its 32-position tiles reach two per
 * compute unit and decode rows are a small share of its work; 16 or 32 forces
 * the shape. Affects plans made after the call, including
 * ppas_attn_workspace_bytes and ppas_plan_items (whose npos then reaches 32).
 * Returns PPAS_EINVAL for any other value.
 */
ppas_status ppas_set_tile_positions(int32_t tile_positions);

/*
 * Profiling hook (process-wide). When both are non-NULL, the following calls
 * have their kernel launches record `start_event` when the kernel starts and
 * `stop_event` when it ends (hipEvent_t handles created by the caller;
 * hipExtLaunchKernel's events), so a kernel's own duration can be read with
 * hipEventElapsedTime: in ppas_attn_step the packed attention kernel (not the
 * split merge), in ppas_kv_append and ppas_rope_kv_append their page-write
 * kernel (start at the first launch, stop at the last when a call needs several
 * launches for over 64 requests). Pass NULLs to stop recording. The events are
 * re-recorded by every call; the caller owns and destroys them.
 * Returns PPAS_EINVAL if exactly one of them is NULL.
 */
ppas_status ppas_set_profile_events(void* start_event, void* stop_event);

#ifdef __cplusplus
}
#endif

#endif /* PPAS_H */
