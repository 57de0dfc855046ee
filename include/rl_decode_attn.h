/*
 * rl_decode_attn.h - C ABI of the MI355X (gfx950) decode-attention library.
 *
 * Operation.  One decode step of one attention layer for a batch of sequences
 * that each add one query token, over a paged KV cache: for every sequence b and
 * query head h,
 *
 *     out[b,h,:] = sum_{t < seq_lens[b]} softmax_t(scale * q[b,h,:] . k_t) * v_t
 *
 * where k_t, v_t are token t of KV head kv_head_of_q[h] of sequence b.  This is
 * the computation that dominates the rollout stage the paper schedules: rollout
 * time is set by autoregressive decode whose long-tail sequences dominate
 * (Sec. 2.3), decode cost grows with the attended history H_dec and the per-token
 * KV footprint b_kv (App. A.1.2, rollout model), and GRPO groups of responses
 * share one prompt (Sec. 2.1).  The paper states no attention formula; the
 * readings used by this library are:
 *   - seq_lens[b] counts every cached token including the current one; its K/V
 *     are already in the cache (the library never writes the cache);
 *   - seq_lens[b] == 0 yields an all-zero output row;
 *   - token t of sequence b is slot t % page_size of pool page
 *     block_table[b * max_pages_per_seq + t / page_size]; entries past
 *     ceil(seq_lens[b] / page_size) and slots past the end are never read;
 *   - scale defaults to 1/sqrt(head_dim);
 *   - fp8 caches use the OCP E4M3FN encoding, and the value of an element is
 *     decode(byte) * scale[page][kv_head] (one fp32 scale per page and KV head,
 *     separately for K and V).
 *
 * Conventions.
 *   - Every pointer given to rl_decode_attn_run is DEVICE memory owned by the
 *     caller and must stay valid until the work queued on `stream` completes.
 *     The library allocates no device memory and never synchronises the stream.
 *   - Errors are status codes; nothing throws across this interface.  Argument
 *     checks that need no device access happen before any launch; a failure
 *     there launches nothing.
 *   - A handle owns host memory only; it may be shared by threads, but two calls
 *     that can overlap (different streams) need different workspaces.
 */
#ifndef RL_DECODE_ATTN_H
#define RL_DECODE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RLDA_F32 = 0,          /* IEEE binary32 */
  RLDA_BF16 = 1,         /* bfloat16 (upper half of binary32) */
  RLDA_FP8_E4M3FN = 2    /* OCP 8-bit E4M3, no infinities, max 448 */
} rlda_dtype;

typedef enum {
  RLDA_OK = 0,
  RLDA_ERR_INVALID_ARG = -1,   /* inconsistent sizes, null or misaligned pointer */
  RLDA_ERR_UNSUPPORTED = -2,   /* valid request outside the built kernel set */
  RLDA_ERR_HIP = -3,           /* a HIP runtime call or a launch failed */
  RLDA_ERR_WORKSPACE = -4,     /* workspace missing or smaller than required */
  RLDA_ERR_ALLOC = -5,         /* host allocation for the handle failed */
  RLDA_ERR_SCRATCH = -6        /* beyond the static scratch of rl_decode_attn_run_noalloc */
} rlda_status;

typedef struct rlda_handle* rl_decode_attn_t;

/*
 * Static description of the attention layer and cache.  Supported sets:
 *   (q, kv, out) = (f32, f32, f32)               head_dim 64 or 128,
 *                                                group size G = Hq/Hkv with G*head_dim <= 128
 *   (q, kv, out) = (bf16, bf16 | fp8, f32 | bf16) head_dim 64 or 128, 1 <= G <= 16
 * page_size must be 16.
 */
typedef struct {
  int32_t num_q_heads;            /* Hq >= 1, at most 256 */
  int32_t num_kv_heads;           /* Hkv >= 1, divides Hq */
  int32_t head_dim;               /* d: 64 or 128 */
  int32_t page_size;              /* P: 16 */
  int32_t max_batch;              /* largest batch passed to run, 1..8192 */
  int32_t max_pages_per_seq;      /* block_table row length (elements); max_batch *
                                     (max_pages_per_seq + 2) * num_kv_heads <= 2^31 - 1,
                                     else RLDA_ERR_UNSUPPORTED                       */
  rlda_dtype q_dtype, kv_dtype, out_dtype;
  const int32_t* kv_head_of_q;    /* HOST array [Hq] copied at create; NULL = h / G.
                                     Every KV head must receive exactly G query heads. */
  float softmax_scale;            /* 0 = 1/sqrt(head_dim) */
  int64_t kv_stride_page;         /* element strides of the K and V caches; d is      */
  int64_t kv_stride_head;         /* contiguous.  All three 0 = dense layout           */
  int64_t kv_stride_slot;         /* [page][kv_head][slot][d].  Must keep each row     */
                                  /* 16-byte aligned; slot stride >= head_dim.         */
  int32_t num_work_ranges;        /* 0 = fill the GPU (default).  > 0 forces how many
                                     equal-cost shares the KV work is cut into (tuning and
                                     tests of the split/merge path); at most 4096.     */
} rl_decode_attn_config;

/* Validate `cfg` and create a handle (host memory only; no HIP call).
 * Returns RLDA_ERR_INVALID_ARG / RLDA_ERR_UNSUPPORTED without creating one. */
rlda_status rl_decode_attn_create(const rl_decode_attn_config* cfg, rl_decode_attn_t* out_handle);

/* Bytes of device workspace a run with this handle needs (host-only). */
rlda_status rl_decode_attn_workspace_size(rl_decode_attn_t handle, size_t* bytes);

/*
 * Queue the attention for `batch` sequences on `stream` (a hipStream_t; NULL =
 * the null stream).  Device arrays, all row-major:
 *   q            [batch][Hq][d]                   q_dtype
 *   k_cache,     pool of `num_pages` pages,        kv_dtype, strides from the config
 *   v_cache
 *   k_scale,     [num_pages][Hkv] fp32             fp8 caches only, else NULL
 *   v_scale
 *   block_table  [batch][max_pages_per_seq] int32  page ids in [0, num_pages)
 *   seq_lens     [batch] int32                     0 <= L <= max_pages_per_seq*16
 *   out          [batch][Hq][d]                    out_dtype
 *   workspace    >= rl_decode_attn_workspace_size bytes, 256-byte aligned, zero-filled
 *                before its first use.  It holds per-segment counters that every run
 *                returns to zero, partial results (each stored with a tag of the call
 *                that wrote it), and the contract-flag word (its first 32-bit word,
 *                which accumulates).  A counter that is not zero when a run begins (a
 *                workspace that was not zero-filled, or another run using it at the
 *                same time) raises flag bit 3: the run counts more pieces than the
 *                segment has, or merges a partial it did not write.  The rows of the
 *                affected segments are then unspecified, and the counters stay dirty
 *                until the workspace is zero-filled again.  Calls that may overlap in
 *                time need separate workspaces.
 * Pointers q, k_cache, v_cache and out must be 16-byte aligned; with num_pages == 0
 * (all sequences empty) the cache and scale pointers may be NULL.
 * Device-side contract violations (a page id outside the pool, a length beyond
 * the block-table row) never read outside the given arrays: the offending page
 * or tokens are skipped, the output row is unspecified, and a flag is raised that
 * rl_decode_attn_read_flags reports.
 */
rlda_status rl_decode_attn_run(rl_decode_attn_t handle, int32_t batch, int32_t num_pages, const void* q,
                               const void* k_cache, const void* v_cache, const float* k_scale,
                               const float* v_scale, const int32_t* block_table, const int32_t* seq_lens,
                               void* out, void* workspace, size_t workspace_bytes, void* stream);

/* As rl_decode_attn_run, and records the caller's hipEvent_t `event_begin` /
 * `event_end` on `stream` immediately before and after the attention kernel (the
 * run's only kernel), so callers can time it alone.  Both events are required. */
rlda_status rl_decode_attn_run_profiled(rl_decode_attn_t handle, int32_t batch, int32_t num_pages, const void* q,
                                        const void* k_cache, const void* v_cache, const float* k_scale,
                                        const float* v_scale, const int32_t* block_table,
                                        const int32_t* seq_lens, void* out, void* workspace,
                                        size_t workspace_bytes, void* stream, void* event_begin,
                                        void* event_end);

/*
 * rl_decode_attn_run without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  Same operation, kernel and arguments as rl_decode_attn_run, except:
 *   - the flags, segment counters and partial results live in a static device
 *     array of the library (about 8.6 MiB; one copy on each GPU the library runs
 *     on, held until the process ends), found on the first call on each device;
 *   - limits of that array: batch * num_kv_heads <= 65536 and head_dim <= 128
 *     (else RLDA_ERR_SCRATCH, nothing launched), and the work is cut into at most
 *     512 shares (the default: one per CU on MI355X, two for fp8 caches and
 *     for bf16 caches at head_dim 64);
 *   - flags: NULL, or a caller-owned device uint32_t (4-byte aligned) that receives
 *     the contract bits of rl_decode_attn_read_flags (OR-ed in; the caller clears
 *     it).  With NULL they go to a word of the static array that nothing reads.
 * The array starts zeroed and every call that completes leaves its counters at
 * zero, so nothing needs clearing between calls.  Every call on one GPU shares that
 * GPU's array: calls that may overlap in time (different streams) race on it and
 * must not be issued (flag bit 3 reports it when they meet).
 * No device memory is allocated or freed; one kernel, asynchronous.
 */
rlda_status rl_decode_attn_run_noalloc(rl_decode_attn_t handle, int32_t batch, int32_t num_pages, const void* q,
                                       const void* k_cache, const void* v_cache, const float* k_scale,
                                       const float* v_scale, const int32_t* block_table, const int32_t* seq_lens,
                                       void* out, uint32_t* flags, void* stream);

/*
 * Shared-prompt (GRPO group) variant of rl_decode_attn_run.  GRPO samples a group
 * of responses for each prompt (Sec. 2.1), and every response of a group attends
 * to the prompt's KV pages.  Sequences [i*group_size, min((i+1)*group_size, batch))
 * form group i; the first prefix_pages[i] entries of their block-table rows name
 * the same pool pages (the prompt), each holding page_size valid tokens.  The
 * result is that of rl_decode_attn_run on the same arguments (up to rounding
 * order), but prompt pages are read fewer times.  Two ways, chosen on the host:
 *   - packed (at least two members fit the 16 rows of one MFMA tile: 2G <= 16,
 *     group_size >= 2, batch <= 4096, max_pages_per_seq <= 32767, and the prompt
 *     bytes packing reads again, (packs per group - 1) * groups * Hkv *
 *     prompt_pages_hint * 32 * head_dim * bytes(kv), below 240 MiB): one kernel.
 *     Up to min(7, 16/G) consecutive members of a group form a pack whose rows
 *     share one tile; the pack's segment streams the prompt pages once with every
 *     member's rows, then each member's own pages with only its rows unmasked.
 *     Each prompt page is read once per pack and KV head.
 *   - otherwise: a prompt pass multiplies each prompt page against the query rows
 *     of up to 64/G members at once (up to four 16-row MFMA tiles), and the
 *     attention over the remaining pages of each sequence starts from the prompt
 *     pass's (max, sum, output) state.  Each prompt page is read once per group
 *     and KV head.
 *   group_size    >= 1, host value
 *   prefix_pages  [ceil(batch / group_size)] int32, device memory
 *   prompt_pages_hint  host value: the caller's estimate of the prompt pages (e.g. the
 *                 largest prefix_pages entry); only chooses between the two ways;
 *                 <= 0: unknown (packed when the other conditions hold)
 * The prompt pages are read from the block-table row of the group's first
 * sequence; the other members' first prefix_pages[i] entries are not read (a
 * member whose entries differ is computed as if they matched).  A group's prompt
 * is clamped to the full pages of its shortest member,
 * min(prefix_pages[i], min over members of floor(seq_lens[b] / 16)), and a clamp
 * raises flag bit 2; prefix_pages[i] = 0 shares nothing for group i.
 * Supported for bf16 and fp8 caches (RLDA_ERR_UNSUPPORTED for f32).
 * workspace: >= rl_decode_attn_grouped_workspace_size bytes, same rules as for
 * rl_decode_attn_run (the same workspace serves both calls).  One kernel (packed)
 * or two (the prompt pass, then the attention over the rest) are queued on
 * `stream`.  event_begin / event_end (hipEvent_t): both NULL, or both given to be
 * recorded before the first and after the last kernel.
 */
rlda_status rl_decode_attn_run_grouped(rl_decode_attn_t handle, int32_t batch, int32_t num_pages, int32_t group_size,
                                       const int32_t* prefix_pages, int32_t prompt_pages_hint, const void* q,
                                       const void* k_cache, const void* v_cache, const float* k_scale,
                                       const float* v_scale,
                                       const int32_t* block_table, const int32_t* seq_lens, void* out,
                                       void* workspace, size_t workspace_bytes, void* stream, void* event_begin,
                                       void* event_end);

/* Bytes of device workspace rl_decode_attn_run_grouped needs with this handle:
 * rl_decode_attn_workspace_size plus max_batch*(Hq*(head_dim+2)+1)*4 (rounded up)
 * for the prompt pass's per-row results (host-only). */
rlda_status rl_decode_attn_grouped_workspace_size(rl_decode_attn_t handle, size_t* bytes);

/*
 * Append one decode step's K and V rows to the paged cache: the write that
 * precedes each step's attention, since every live request adds one token per
 * step (App. A.1.2, decode steps and the per-token footprint b_kv).  For every
 * sequence b with 1 <= seq_lens[b] <= max_pages_per_seq*16, token
 * t = seq_lens[b] - 1 (seq_lens counts the new token, as for rl_decode_attn_run)
 * is written to slot t % 16 of page block_table[b][t / 16] for every KV head:
 *   k_new, v_new  [batch][Hkv][d]  q_dtype: bf16 for bf16 and fp8 caches, f32 for f32
 *   k_cache, v_cache, k_scale, v_scale, block_table, seq_lens: as for rl_decode_attn_run
 *   (the caches and, for fp8, the scales are written).
 * bf16 and f32 caches store the rows as given.  fp8 caches keep each (page, KV head)
 * scale covering every row written so far (the paper fixes no rule; this is the
 * library's):
 *   - slot 0 (a new page): scale = amax / 448, amax = the row's largest |value|;
 *   - a later slot: if amax > 448 * scale, scale = amax / 448 and the page's earlier
 *     rows are re-encoded, byte = E4M3(decode(byte) * (old scale / new scale)); a
 *     stored scale that is not positive and finite counts as 0 (earlier rows become 0);
 *   - the row is stored as E4M3(value / scale), zero bytes when scale is 0;
 * all in fp32, E4M3 rounding to nearest even and saturating at 448.
 * The pages one call writes must each belong to one sequence.  A length outside
 * [0, capacity] or an out-of-pool page id skips that sequence and raises the flag
 * rl_decode_attn_run would; seq_lens[b] == 0 skips silently.  workspace: as for
 * rl_decode_attn_run (only its flag word is used).  One kernel, asynchronous.
 */
rlda_status rl_decode_attn_append(rl_decode_attn_t handle, int32_t batch, int32_t num_pages, const void* k_new,
                                  const void* v_new, void* k_cache, void* v_cache, float* k_scale, float* v_scale,
                                  const int32_t* block_table, const int32_t* seq_lens, void* workspace,
                                  size_t workspace_bytes, void* stream);

/*
 * Multi-token queries: attention for prefill chunks, or for verifying a few
 * drafted tokens (any query rows that are the last tokens of their sequences).
 * Rollout prefills the prompt tokens before decoding (Sec. 3; the prefill cost of
 * App. A.1.2, whose attention term grows with the square of the prompt length).
 * Sequence b has n_b = q_start[b+1] - q_start[b] query rows q[q_start[b] + i],
 * 0 <= i < n_b: its last n_b cached tokens (their K/V already in the cache), so
 * row i is at position seq_lens[b] - n_b + i and attends causally to positions
 * 0 .. seq_lens[b] - n_b + i:
 *   out[q_start[b] + i][h] = sum_{t <= pos} softmax_t(scale * q[.][h] . k_t) v_t.
 * n_b = 1 for every sequence is rl_decode_attn_run (up to rounding order).
 *   q            [total_q][Hq][d]   q_dtype (bf16)
 *   q_start      [batch + 1] int32, device memory, 0 <= q_start[b] <= q_start[b+1] <= total_q
 *   out          [total_q][Hq][d]   out_dtype; rows no sequence names are not written
 *   total_q      host value: rows of q and out
 *   max_q_len    host value, 0 or an upper bound on every n_b.  When
 *                1 <= max_q_len <= 16 and max_q_len * G <= 64 (and batch * Hkv *
 *                (max_pages_per_seq + 2) * ceil(max_q_len * G / 16) < 2^31), the call runs
 *                on the decode kernel's page stream (the n_b * G rows of each
 *                (sequence, KV head) as 16-row MFMA tiles, one wave holding two of
 *                them against each page when batch <= 2048, up to four segments
 *                that each stream the pages, long sequences split across
 *                workgroups; workspace as
 *                for rl_decode_attn_run, counters included); a sequence with
 *                n_b > max_q_len then gets no rows and raises flag bit 1.  Otherwise
 *                the (token, head) pairs of one (sequence, KV head) are processed 128
 *                at a time by one workgroup as 32x32 MFMA tiles (each K/V page read
 *                once per 128 rows), batch <= 4096, and only the flag word of the
 *                workspace is used.
 *   other arrays and `workspace` as for rl_decode_attn_run.
 * Supported for bf16 and fp8 caches (RLDA_ERR_UNSUPPORTED for f32, and when q
 * holds 2^31 bytes or more).  Device-side checks: a sequence with inconsistent
 * q_start entries gets no rows (flag bit 1); n_b > seq_lens[b] raises flag bit 1
 * and rows at negative positions are zero; lengths beyond capacity and
 * out-of-pool pages as for rl_decode_attn_run.  One kernel, asynchronous;
 * event_begin / event_end (hipEvent_t): both NULL, or both given to be recorded
 * around it.
 */
rlda_status rl_decode_attn_run_multi(rl_decode_attn_t handle, int32_t batch, int32_t num_pages, int32_t total_q,
                                     int32_t max_q_len, const void* q, const void* k_cache, const void* v_cache,
                                     const float* k_scale, const float* v_scale, const int32_t* block_table,
                                     const int32_t* seq_lens, const int32_t* q_start, void* out, void* workspace,
                                     size_t workspace_bytes, void* stream, void* event_begin, void* event_end);

/* Flags raised by device-side contract checks since the workspace was zeroed
 * (bit 0: page id outside [0, num_pages); bit 1: seq_len beyond capacity;
 * bit 2: a group's shared prompt clamped to its shortest member; bit 3: a
 * segment counter was not zero when the run began, so the run counted more pieces
 * than a segment has or merged a partial it had not written: the workspace was not
 * zero-filled, or runs overlapped on it).
 * SYNCHRONISES `stream` (waits for queued work, copies 4 bytes to the host). */
rlda_status rl_decode_attn_read_flags(rl_decode_attn_t handle, const void* workspace, void* stream,
                                      uint32_t* flags);

/* Destroy a handle; NULL is allowed. */
rlda_status rl_decode_attn_destroy(rl_decode_attn_t handle);

/* Static description of a status code. */
const char* rl_decode_attn_strerror(rlda_status status);

#ifdef __cplusplus
}
#endif

#endif /* RL_DECODE_ATTN_H */
