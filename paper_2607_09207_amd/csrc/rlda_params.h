// Internal launch parameters shared by the host entry points and the kernels.
#pragma once
#include <stddef.h>
#include <stdint.h>

namespace rlda {

constexpr int kPage = 16;          // tokens per KV page
constexpr int kWaves = 4;          // waves per workgroup: one per SIMD, one workgroup per CU
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxQHeads = 256;
constexpr int kMaxBatch = 8192;
constexpr int kMaxRanges = 4096;   // upper bound on work ranges (= workgroups)
constexpr int kMaxGroup = 16;      // query heads per KV head packed in one MFMA tile
constexpr int kMaxRowChunks = 4;   // multi-token rows through the decode kernel: up to 4 x 16 per (sequence, KV head)
#ifndef RLDA_MAX_ROW_TILES
#define RLDA_MAX_ROW_TILES 2       // 16-row tiles a wave holds against each page on that path (1 or 2)
#endif
constexpr int kMaxRowTiles = RLDA_MAX_ROW_TILES;
#ifndef RLDA_START_COST
#define RLDA_START_COST 2          // work-split cost of a segment's start, in pages
#endif
constexpr int kStartCost = RLDA_START_COST;
constexpr int kMaxRowsQLen = 16;   // ... and at most 16 rows per sequence (a full page's token count, clamped
                                   // to 31, less a row's causal shift of up to 15 still covers the page)

// Bits of the device-side contract flag word.
constexpr uint32_t kFlagBadPage = 1u;
constexpr uint32_t kFlagBadLen = 2u;
constexpr uint32_t kFlagPrefixClamped = 4u;
constexpr uint32_t kFlagStaleState = 8u;   // a counter or a partial this call did not write (workspace not zeroed)

// Static scratch of rl_decode_attn_run_noalloc (one copy per GPU, in the kernel
// source): the flag word, then segment counters for batch * Hkv <= kScratchMaxSegments,
// then two partial slots of kMaxGroup rows per work range for up to
// kScratchMaxRanges ranges at head_dim 128.
constexpr int kScratchMaxRanges = 512;
constexpr int kScratchMaxSegments = 65536;
constexpr size_t kScratchCountersOff = 256;
constexpr size_t kScratchMlOff = kScratchCountersOff + sizeof(uint32_t) * kScratchMaxSegments;
constexpr size_t kScratchAccOff = kScratchMlOff + sizeof(float) * 4 * kScratchMaxRanges * kMaxGroup * 2;
constexpr size_t kScratchBytes = kScratchAccOff + sizeof(float) * 2 * kScratchMaxRanges * kMaxGroup * 128;
static_assert(kScratchMlOff % 256 == 0 && kScratchAccOff % 256 == 0, "scratch regions stay 256-byte aligned");

struct Params {
  const void* q;               // [batch][Hq][D]
  const void* k;               // KV pools (byte addressed through the strides)
  const void* v;
  const float* k_scale;        // [num_pages][Hkv] (fp8 only)
  const float* v_scale;
  const int32_t* block_table;  // [batch][max_pages]
  const int32_t* seq_lens;     // [batch]
  void* out;                   // [batch][Hq][D]
  float* part_acc;             // [2 * nranges][part_rows][D]  unnormalised partial outputs
  float* part_ml;              // [2 * nranges][part_rows][4]  (running max in log2 units, sum, call tag, 0)
  int32_t part_rows;           // query rows per (sequence, KV head) segment: G, or n_max * G for multi-token rows
  uint32_t* counters;          // [max_batch * Hkv * 4] finished pieces per split segment; zero between runs
  uint32_t call_tag;           // this call's tag, published with each partial (never 0 or all-ones)
  uint32_t* flags;             // contract-violation bits
  int64_t stride_page;         // bytes
  int64_t stride_head;         // bytes
  int32_t stride_slot;         // bytes
  int32_t batch;
  int32_t num_pages;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;               // G = Hq / Hkv
  int32_t max_pages;           // block-table row length
  int32_t nranges;             // workgroups = equal-cost shares of the flattened work
  float scale_log2;            // softmax scale * log2(e)
  int32_t out_bf16;            // 0: fp32 output, 1: bf16 output
  // Shared-prompt (grouped) runs; all null / 0 otherwise.
  const int32_t* prefix_pages; // [ngroups] requested prompt pages per group (device)
  int32_t* gprefix;            // [ngroups] prompt pages after the clamp (written by the prompt pass)
  float* pfx_acc;              // [batch][Hq][D] prompt-pass unnormalised outputs
  float* pfx_ml;               // [batch][Hq][2] prompt-pass (max in log2 units, sum)
  int32_t group_size;          // sequences per group; 0: not grouped
  int32_t pfx_mblock;          // members per prompt-pass job (rows = members * G <= 64)
  int32_t pfx_nblocks;         // jobs per (group, KV head)
  int32_t pfx_splits;          // workgroups per job (their states meet in the partial slots)
  int32_t pfx_slots;           // capacity of part_acc / part_ml in 64-row prompt-pass slots
  int32_t pack;                // packed grouped runs: members per pack (their rows share the MFMA tiles)
  int32_t pack_units;          // packed grouped runs: packs in the batch
  // KV append (rl_decode_attn_append): the step's new rows, [batch][Hkv][D] in the q dtype.
  const void* k_in;
  const void* v_in;
  // Multi-token queries (rl_decode_attn_run_multi): q and out are [total_q][Hq][D].
  const int32_t* q_start;      // [batch + 1] query-row offsets
  int32_t total_q;
  int32_t max_q_len;           // decode-kernel path: rows per sequence allowed (n_b <= max_q_len)
  int32_t row_chunks;          // decode-kernel path: segments per (sequence, KV head), ceil(max_q_len * G / (16 * tiles))
  int16_t q_head[kMaxQHeads];  // q_head[g * G + i] = i-th query head of KV head g
};

enum class KvKind { F32, BF16, FP8 };

// Kernel launchers (rlda_kernels.hip).  Return hipSuccess or the launch error.
// The kernel is bracketed by ev_begin / ev_end when they are non-null.
int launch_decode(KvKind kind, int head_dim, int group, const Params& p, void* stream, void* ev_begin,
                  void* ev_end);
// Prompt pass of a grouped run (one workgroup per (group, KV head, member block)),
// followed by the attention kernel.
int launch_grouped(KvKind kind, int head_dim, int group, const Params& p, int ngroups, void* stream,
                   void* ev_begin, void* ev_end);
// Decode with two workgroups per CU for the half-size pages (fp8, and bf16 at d = 64;
// two waves per SIMD; batch <= kTwoWgMaxBatch, nranges twice the CUs): eight waves
// per CU keep twice the tiles in flight.
int launch_decode_two(KvKind kind, int head_dim, const Params& p, void* stream, void* ev_begin, void* ev_end);
// KV append: one wave per (sequence, KV head).
int launch_append(KvKind kind, int head_dim, const Params& p, void* stream);
// Device address of the static scratch on the current device (kScratchBytes bytes),
// looked up once per device; 0 on success.
int noalloc_scratch(void** ptr);
// Multi-token queries (rlda_multi.hip): one workgroup per (128-row query block, KV head).
int launch_multi(KvKind kind, int head_dim, const Params& p, int grid, void* stream, void* ev_begin, void* ev_end);
// Multi-token queries with at most 16 * tiles rows per (sequence, KV head) segment
// (tiles 1 or 2): the decode kernel's page stream, each row masked causally (bf16 / fp8).
int launch_decode_rows(KvKind kind, int head_dim, int tiles, const Params& p, void* stream, void* ev_begin,
                       void* ev_end);
// Grouped runs with the members of a group packed into the rows of the MFMA tiles
// (pack members per (pack, KV head) segment): the decode kernel's page stream, the
// prompt pages streamed once per pack, each member's own pages after them.
int launch_decode_packed(KvKind kind, int head_dim, int tiles, const Params& p, void* stream, void* ev_begin,
                         void* ev_end);
#ifndef RLDA_MQ_TILES
#define RLDA_MQ_TILES 1            // 32-row MFMA tiles per wave in the multi-token kernel
#endif
constexpr int kMultiTiles = RLDA_MQ_TILES;
constexpr int kMultiRows = 128 * kMultiTiles;   // query rows (token, head pairs) per workgroup of the multi-token kernel
constexpr int kMultiMaxBatch = 4096;   // its per-sequence LDS tables stay within 48 KiB of LDS per workgroup
constexpr int kPackMaxBatch = 4096;    // packed grouped runs: per-sequence and per-pack LDS tables of this size
constexpr int kPackMaxMembers = 7;     // ... members per pack (3 bits of the page descriptor, 7 = every member)
constexpr int kPackMaxPages = 32767;   // ... pages per sequence (16-bit LDS entries)
constexpr int kTwoWgMaxBatch = 512;      // two workgroups per CU (fp8, bf16 d = 64 decode): per-sequence LDS tables of this size
constexpr int kTwoTileMaxBatch = 2048;   // two-tile multi-token rows: per-sequence LDS tables of this size
                                         // leave room for 32-row merge slots

}  // namespace rlda
