/*
 * hbm_probe.h - read-bandwidth reference kernels for gfx950 (libhbm_probe.so).
 *
 * The decode-attention path is bound by HBM reads: every call streams each cached
 * KV byte once (the per-token footprint b_kv of App. A.1.2 times the tokens
 * attended).  These kernels measure what a plain reader reaches on the same
 * GPU, so that the attention kernel's rate has a measured ceiling beside the
 * 8 TB/s data-sheet peak.  They do no arithmetic beyond folding the loaded words
 * together, and write (almost) nothing.
 *
 * Conventions: every pointer is device memory owned by the caller; the kernels
 * are queued on `stream` (a hipStream_t; NULL = the null stream) and nothing is
 * synchronised or allocated.  Return value: 0 on success, -1 for an invalid
 * argument (nothing launched), -3 when the launch failed.
 */
#ifndef HBM_PROBE_H
#define HBM_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` (a multiple of 16) of `buf` once with `blocks` workgroups of
 * `threads` threads (a multiple of 64, at most 512), each lane keeping a ring of
 * `unroll` (1, 2, 4, 8 or 16) 16-byte non-temporal loads in flight.  `sink` holds
 * at least `blocks` 32-bit words; a word is written only if a lane's folded value equals an
 * internal sentinel. */
int hbm_probe_stream_read(const void* buf, uint64_t bytes, uint32_t* sink, int blocks, int threads, int unroll,
                          void* stream);

/* Read `ntiles` pairs of tiles: for entry e, `tile_bytes` (1024, 2048, 3072 or
 * 4096) bytes at byte offset tile_offsets[e] of `k_pool` and the same of `v_pool`.
 * Every offset must keep the tile inside both pools (not checked on the device).
 * The list is cut into equal contiguous shares, one per wave of the grid (`blocks`
 * workgroups of `threads` threads), and each wave keeps a ring of `depth` (1 to 4)
 * pairs in flight.  `sink` as for hbm_probe_stream_read. */
int hbm_probe_tile_gather(const void* k_pool, const void* v_pool, const int64_t* tile_offsets, int64_t ntiles,
                          int tile_bytes, uint32_t* sink, int blocks, int threads, int depth, void* stream);

/* The tile gather with run-time balancing: entries [0, nstatic) are cut into equal
 * contiguous shares, one per wave; the remaining ntiles - nstatic entries (a
 * multiple of `chunk`, depth <= chunk <= 64) form chunks that waves claim one at a
 * time with an atomicAdd on counter[0] once their share is done, the load ring
 * running on across chunks.  `counter` is one 32-bit word of device memory that must
 * be zero before the first launch; each launch leaves it zero (and launches on one
 * counter must not overlap).  Shares must hold at least `depth` entries (nstatic /
 * waves >= depth) or none.  depth 2 to 4; other arguments as for
 * hbm_probe_tile_gather. */
int hbm_probe_tile_gather_balanced(const void* k_pool, const void* v_pool, const int64_t* tile_offsets, int64_t ntiles,
                                   int64_t nstatic, int chunk, uint32_t* counter, int tile_bytes, uint32_t* sink,
                                   int blocks, int threads, int depth, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HBM_PROBE_H */
