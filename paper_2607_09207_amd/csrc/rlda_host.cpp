// Host side of the decode-attention C ABI: argument validation, workspace
// layout, work-range sizing and the launch.  create/workspace_size/destroy and
// every argument check of run make no HIP call.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <new>

#include "rl_decode_attn.h"
#include "rlda_params.h"

struct rlda_handle {
  rl_decode_attn_config cfg;
  int32_t group;
  int64_t stride_page, stride_head, stride_slot;   // elements
  int32_t ws_ranges;                               // work ranges the workspace is sized for
  float scale;
  int16_t q_head[rlda::kMaxQHeads];
  rlda::KvKind kind;
};

namespace {

constexpr size_t kAlign = 256;
constexpr int kDefaultWsRanges = 1024;   // default work ranges = CU count (256 on MI355X)
constexpr int64_t kPackedExtraBytes = 240ll << 20;   // grouped runs: packed below this many re-read prompt bytes

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int elem_bytes(rlda_dtype t) { return t == RLDA_F32 ? 4 : t == RLDA_BF16 ? 2 : 1; }

struct WsLayout {
  size_t flags, counters, part_ml, part_acc, total;
  size_t gprefix, pfx_ml, pfx_acc, grouped_total;   // grouped runs only
};

WsLayout layout_of(const rlda_handle* h) {
  const rl_decode_attn_config& c = h->cfg;
  WsLayout w;
  w.flags = 0;
  w.counters = align_up(sizeof(uint32_t));
  // Counters: one per (sequence, KV head) segment, or per 16-row chunk of one in
  // multi-token runs through the decode kernel.
  w.part_ml = align_up(w.counters + sizeof(uint32_t) * (size_t)c.max_batch * c.num_kv_heads * rlda::kMaxRowChunks);
  // Partial slots: two per work range, 16 rows each (G rows in decode runs, up to
  // 16 rows of a segment in multi-token runs).
  w.part_acc = align_up(w.part_ml + sizeof(float) * 4 * (size_t)h->ws_ranges * rlda::kMaxGroup * 2);
  w.total = align_up(w.part_acc + sizeof(float) * 2 * (size_t)h->ws_ranges * rlda::kMaxGroup * c.head_dim);
  w.gprefix = w.total;
  w.pfx_ml = align_up(w.gprefix + sizeof(int32_t) * (size_t)c.max_batch);
  w.pfx_acc = align_up(w.pfx_ml + sizeof(float) * 2 * (size_t)c.max_batch * c.num_q_heads);
  w.grouped_total = align_up(w.pfx_acc + sizeof(float) * (size_t)c.max_batch * c.num_q_heads * c.head_dim);
  return w;
}

// Device properties cached per device id (multiprocessor count).
std::mutex g_dev_mu;
int g_cu_count[64];

int cu_count(int dev) {
  std::lock_guard<std::mutex> lk(g_dev_mu);
  if (dev < 0 || dev >= 64) return 0;
  if (g_cu_count[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    g_cu_count[dev] = n;
  }
  return g_cu_count[dev];
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Call tags: published with every partial so that a merge can tell a piece of this
// call from a stale one.  Consecutive calls get well-spread values (a multiplicative
// hash of a process-wide sequence number); 0 and all-ones, what zeroed or
// never-written memory holds, are skipped.
std::atomic<uint32_t> g_call_seq{0};

uint32_t next_call_tag() {
  for (;;) {
    const uint32_t t = (g_call_seq.fetch_add(1, std::memory_order_relaxed) * 2654435761u) ^ 0xA5A5A5A5u;
    if (t != 0u && t != 0xFFFFFFFFu) return t;
  }
}

}  // namespace

extern "C" {

rlda_status rl_decode_attn_create(const rl_decode_attn_config* cfg, rl_decode_attn_t* out_handle) {
  if (!cfg || !out_handle) return RLDA_ERR_INVALID_ARG;
  *out_handle = nullptr;
  const rl_decode_attn_config& c = *cfg;
  if (c.num_q_heads < 1 || c.num_q_heads > rlda::kMaxQHeads || c.num_kv_heads < 1 ||
      c.num_q_heads % c.num_kv_heads != 0)
    return RLDA_ERR_INVALID_ARG;
  if (c.max_batch < 1 || c.max_batch > rlda::kMaxBatch || c.max_pages_per_seq < 1 ||
      (int64_t)c.max_pages_per_seq * rlda::kPage > INT32_MAX)
    return RLDA_ERR_INVALID_ARG;
  if (c.num_work_ranges < 0 || c.num_work_ranges > rlda::kMaxRanges) return RLDA_ERR_INVALID_ARG;
  if (!(c.softmax_scale >= 0.f) || isinf(c.softmax_scale)) return RLDA_ERR_INVALID_ARG;
  if (c.q_dtype < RLDA_F32 || c.q_dtype > RLDA_FP8_E4M3FN || c.kv_dtype < RLDA_F32 ||
      c.kv_dtype > RLDA_FP8_E4M3FN || c.out_dtype < RLDA_F32 || c.out_dtype > RLDA_FP8_E4M3FN)
    return RLDA_ERR_INVALID_ARG;
  if (c.page_size != rlda::kPage) return RLDA_ERR_UNSUPPORTED;
  if (c.head_dim != 64 && c.head_dim != 128) return RLDA_ERR_UNSUPPORTED;
  // The kernel numbers (sequence, KV head, page) units, and prices their work with
  // kStartCost more per (sequence, KV head), in 32-bit integers.
  if ((int64_t)c.max_batch * (c.max_pages_per_seq + rlda::kStartCost) * c.num_kv_heads > INT32_MAX)
    return RLDA_ERR_UNSUPPORTED;
  const int G = c.num_q_heads / c.num_kv_heads;

  rlda::KvKind kind;
  if (c.q_dtype == RLDA_F32 && c.kv_dtype == RLDA_F32 && c.out_dtype == RLDA_F32) {
    if (G * c.head_dim > 128) return RLDA_ERR_UNSUPPORTED;
    kind = rlda::KvKind::F32;
  } else if (c.q_dtype == RLDA_BF16 && (c.kv_dtype == RLDA_BF16 || c.kv_dtype == RLDA_FP8_E4M3FN) &&
             (c.out_dtype == RLDA_F32 || c.out_dtype == RLDA_BF16)) {
    if (G > rlda::kMaxGroup) return RLDA_ERR_UNSUPPORTED;
    kind = c.kv_dtype == RLDA_BF16 ? rlda::KvKind::BF16 : rlda::KvKind::FP8;
  } else {
    return RLDA_ERR_UNSUPPORTED;
  }

  // Strides (elements).  Rows must stay 16-byte aligned and not overlap.
  int64_t sp = c.kv_stride_page, sh = c.kv_stride_head, ss = c.kv_stride_slot;
  if (sp == 0 && sh == 0 && ss == 0) {
    ss = c.head_dim;
    sh = (int64_t)rlda::kPage * c.head_dim;
    sp = (int64_t)c.num_kv_heads * sh;
  }
  const int eb = elem_bytes(c.kv_dtype);
  if (sp <= 0 || sh <= 0 || ss < c.head_dim) return RLDA_ERR_INVALID_ARG;
  if ((sp * eb) % 16 || (sh * eb) % 16 || (ss * eb) % 16) return RLDA_ERR_INVALID_ARG;
  if ((ss * eb) * (rlda::kPage - 1) + (int64_t)c.head_dim * eb > INT32_MAX) return RLDA_ERR_UNSUPPORTED;

  // Head map: every KV head gets exactly G query heads.
  int16_t q_head[rlda::kMaxQHeads];
  int fill[rlda::kMaxQHeads];
  memset(fill, 0, sizeof fill);
  for (int h = 0; h < c.num_q_heads; ++h) {
    const int g = c.kv_head_of_q ? c.kv_head_of_q[h] : h / G;
    if (g < 0 || g >= c.num_kv_heads || fill[g] >= G) return RLDA_ERR_INVALID_ARG;
    q_head[g * G + fill[g]++] = (int16_t)h;
  }

  rlda_handle* hd = new (std::nothrow) rlda_handle;
  if (!hd) return RLDA_ERR_ALLOC;
  hd->cfg = c;
  hd->cfg.kv_head_of_q = nullptr;   // copied into q_head
  hd->group = G;
  hd->stride_page = sp;
  hd->stride_head = sh;
  hd->stride_slot = ss;
  hd->ws_ranges = c.num_work_ranges > 0 ? c.num_work_ranges : kDefaultWsRanges;
  hd->scale = c.softmax_scale > 0.f ? c.softmax_scale : (float)(1.0 / sqrt((double)c.head_dim));
  memcpy(hd->q_head, q_head, sizeof q_head);
  hd->kind = kind;
  *out_handle = hd;
  return RLDA_OK;
}

rlda_status rl_decode_attn_workspace_size(rl_decode_attn_t h, size_t* bytes) {
  if (!h || !bytes) return RLDA_ERR_INVALID_ARG;
  *bytes = layout_of(h).total;
  return RLDA_OK;
}

rlda_status rl_decode_attn_grouped_workspace_size(rl_decode_attn_t h, size_t* bytes) {
  if (!h || !bytes) return RLDA_ERR_INVALID_ARG;
  *bytes = layout_of(h).grouped_total;
  return RLDA_OK;
}

}  // extern "C"

namespace {

// Device memory a plain run keeps its flags, counters and partials in, when it is
// not the caller's workspace (the no-allocation entry point's static scratch).
struct RunMem {
  uint32_t* flags;
  uint32_t* counters;
  float* part_ml;
  float* part_acc;
  int ranges_cap;   // work ranges the partial slots are sized for
};

// group_size == 0: plain run; > 0: grouped run with prefix_pages.  With `mem` the
// run uses it instead of a workspace (plain runs only).
rlda_status run_impl(rl_decode_attn_t h, int32_t batch, int32_t num_pages, int32_t group_size,
                     const int32_t* prefix_pages, int32_t prompt_pages_hint, const void* q, const void* k_cache, const void* v_cache,
                     const float* k_scale, const float* v_scale, const int32_t* block_table,
                     const int32_t* seq_lens, void* out, void* workspace, size_t workspace_bytes, void* stream,
                     void* ev_begin, void* ev_end, const RunMem* mem = nullptr) {
  if (!h) return RLDA_ERR_INVALID_ARG;
  const rl_decode_attn_config& c = h->cfg;
  const bool grouped = group_size > 0;
  if (batch < 0 || batch > c.max_batch || num_pages < 0 || group_size < 0) return RLDA_ERR_INVALID_ARG;
  if (grouped && h->kind == rlda::KvKind::F32) return RLDA_ERR_UNSUPPORTED;
  if (batch == 0) return RLDA_OK;
  if (!q || !block_table || !seq_lens || !out) return RLDA_ERR_INVALID_ARG;
  // An empty pool (every sequence empty) may come with null cache pointers.
  if (num_pages > 0 && (!k_cache || !v_cache)) return RLDA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out)) return RLDA_ERR_INVALID_ARG;
  if (((uintptr_t)block_table & 3u) || ((uintptr_t)seq_lens & 3u)) return RLDA_ERR_INVALID_ARG;
  if (grouped && (!prefix_pages || ((uintptr_t)prefix_pages & 3u))) return RLDA_ERR_INVALID_ARG;
  const bool fp8 = h->kind == rlda::KvKind::FP8;
  if (fp8 && num_pages > 0 && (!k_scale || !v_scale || ((uintptr_t)k_scale & 3u) || ((uintptr_t)v_scale & 3u)))
    return RLDA_ERR_INVALID_ARG;
  const WsLayout wl = layout_of(h);
  if (mem) {
    if (grouped) return RLDA_ERR_UNSUPPORTED;
  } else {
    if (!workspace || ((uintptr_t)workspace % kAlign)) return RLDA_ERR_WORKSPACE;
    if (workspace_bytes < (grouped ? wl.grouped_total : wl.total)) return RLDA_ERR_WORKSPACE;
  }

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return RLDA_ERR_HIP;
  // One workgroup (one wave per SIMD) per CU by default: a second workgroup on a
  // CU would lose instruction arbitration to the first and finish its share later.
  // fp8 pages, and bf16 pages at d = 64, are half the bytes of bf16 ones at d = 128,
  // and four waves per CU cannot keep enough of them in flight: such plain runs of
  // up to kTwoWgMaxBatch sequences take two workgroups per CU (two waves per SIMD,
  // within 256 registers each).
  const bool half_pages = h->kind == rlda::KvKind::FP8 || (h->kind == rlda::KvKind::BF16 && c.head_dim == 64);
  const bool two = !grouped && half_pages && batch <= rlda::kTwoWgMaxBatch;
  int ranges = c.num_work_ranges;
  if (ranges == 0) {
    ranges = cu_count(dev);
    if (ranges <= 0) return RLDA_ERR_HIP;
    if (two) ranges *= 2;
  }
  const int ranges_cap = mem ? mem->ranges_cap : h->ws_ranges;
  if (ranges > ranges_cap) ranges = ranges_cap;
  if (ranges > rlda::kMaxRanges) ranges = rlda::kMaxRanges;
  // Never more shares than (sequence, KV head, page) units could exist.
  const int64_t max_units = (int64_t)batch * c.num_kv_heads * c.max_pages_per_seq;
  if (ranges > max_units) ranges = (int)max_units;

  char* ws = (char*)workspace;
  rlda::Params p;
  memset(&p, 0, sizeof p);
  p.q = q;
  p.k = k_cache;
  p.v = v_cache;
  p.k_scale = k_scale;
  p.v_scale = v_scale;
  p.block_table = block_table;
  p.seq_lens = seq_lens;
  p.out = out;
  p.flags = mem ? mem->flags : (uint32_t*)(ws + wl.flags);
  p.counters = mem ? mem->counters : (uint32_t*)(ws + wl.counters);
  p.call_tag = next_call_tag();
  p.part_ml = mem ? mem->part_ml : (float*)(ws + wl.part_ml);
  p.part_acc = mem ? mem->part_acc : (float*)(ws + wl.part_acc);
  p.part_rows = h->group;
  const int eb = elem_bytes(c.kv_dtype);
  p.stride_page = h->stride_page * eb;
  p.stride_head = h->stride_head * eb;
  p.stride_slot = (int32_t)(h->stride_slot * eb);
  p.batch = batch;
  p.num_pages = num_pages;
  p.num_q_heads = c.num_q_heads;
  p.num_kv_heads = c.num_kv_heads;
  p.group = h->group;
  p.max_pages = c.max_pages_per_seq;
  p.nranges = ranges;
  p.scale_log2 = h->scale * 1.4426950408889634f;
  p.out_bf16 = c.out_dtype == RLDA_BF16;
  memcpy(p.q_head, h->q_head, sizeof p.q_head);
  if (!grouped) {
    const int e = two ? rlda::launch_decode_two(h->kind, c.head_dim, p, stream, ev_begin, ev_end)
                      : rlda::launch_decode(h->kind, c.head_dim, h->group, p, stream, ev_begin, ev_end);
    if (e != hipSuccess) return RLDA_ERR_HIP;
    return RLDA_OK;
  }
  p.prefix_pages = prefix_pages;
  p.group_size = group_size;
  // Packed: up to 16 / G members of a group share the rows of one MFMA tile, so
  // one segment streams the prompt pages once for all of them and then each
  // member's own pages.  One launch, no prompt pass.
  const int tiles = 1;
  const int pack = std::min(std::min(rlda::kPackMaxMembers, rlda::kMaxGroup / h->group), group_size);
  const int ngroups = (batch + group_size - 1) / group_size, per_group = (group_size + pack - 1) / pack;
  // Packed runs read each prompt page once per pack, the prompt pass once per group
  // at a fixed cost (a second launch, its merge).  With the caller's prompt length
  // in hand, the prompt pass is taken once the extra prompt bytes of packing exceed
  // kPackedExtraBytes (measured on the GRPO workload, 32 groups of 8, two KV heads,
  // G = 6: packed 6% faster at 2048-token prompts, 14% slower at 4096; equal
  // times near 2600).
  const int64_t page_bytes = 2 * (int64_t)rlda::kPage * c.head_dim * elem_bytes(c.kv_dtype);
  const int64_t extra = prompt_pages_hint > 0 ? (int64_t)(per_group - 1) * ngroups * c.num_kv_heads *
                                                    prompt_pages_hint * page_bytes
                                              : 0;
  if (pack >= 2 && batch <= rlda::kPackMaxBatch && c.max_pages_per_seq <= rlda::kPackMaxPages &&
      extra < kPackedExtraBytes) {
    const int last = batch - (ngroups - 1) * group_size;
    p.pack = pack;
    p.pack_units = (ngroups - 1) * per_group + (last + pack - 1) / pack;
    p.total_q = batch;
    p.row_chunks = 1;
    p.part_rows = std::min(pack * h->group, rlda::kMaxGroup * tiles);
    const int64_t cap_ranges = (int64_t)h->ws_ranges * rlda::kMaxGroup / p.part_rows;
    if (p.nranges > cap_ranges) p.nranges = (int)std::max<int64_t>(cap_ranges, 1);
    if (rlda::launch_decode_packed(h->kind, c.head_dim, tiles, p, stream, ev_begin, ev_end) != hipSuccess)
      return RLDA_ERR_HIP;
    return RLDA_OK;
  }
  p.gprefix = (int32_t*)(ws + wl.gprefix);
  p.pfx_ml = (float*)(ws + wl.pfx_ml);
  p.pfx_acc = (float*)(ws + wl.pfx_acc);
  // Prompt-pass jobs: up to 64 query rows (4 MFMA tiles) of G heads per member.
  p.pfx_mblock = group_size < 64 / h->group ? group_size : 64 / h->group;
  p.pfx_nblocks = (group_size + p.pfx_mblock - 1) / p.pfx_mblock;
  const int64_t jobs = (int64_t)ngroups * c.num_kv_heads * p.pfx_nblocks;
  if (jobs * rlda::kMaxRanges > INT32_MAX) return RLDA_ERR_UNSUPPORTED;
  // Split each job over several workgroups until the prompt pass fills the CUs,
  // within the partial-slot capacity the workspace has (64-row slots).
  const int64_t slots = 2 * (int64_t)h->ws_ranges * rlda::kMaxGroup / 64;
  int64_t split = jobs >= ranges ? 1 : ranges / jobs;
  if (split > 8) split = 8;
  if (split * jobs > slots) split = slots / jobs;
  p.pfx_splits = split < 1 ? 1 : (int)split;
  p.pfx_slots = (int)(slots < INT32_MAX ? slots : INT32_MAX);
  if (rlda::launch_grouped(h->kind, c.head_dim, h->group, p, ngroups, stream, ev_begin, ev_end) != hipSuccess)
    return RLDA_ERR_HIP;
  return RLDA_OK;
}

}  // namespace

extern "C" {

rlda_status rl_decode_attn_run(rl_decode_attn_t h, int32_t batch, int32_t num_pages, const void* q,
                               const void* k_cache, const void* v_cache, const float* k_scale,
                               const float* v_scale, const int32_t* block_table, const int32_t* seq_lens,
                               void* out, void* workspace, size_t workspace_bytes, void* stream) {
  return run_impl(h, batch, num_pages, 0, nullptr, -1, q, k_cache, v_cache, k_scale, v_scale, block_table, seq_lens,
                  out, workspace, workspace_bytes, stream, nullptr, nullptr);
}

rlda_status rl_decode_attn_run_profiled(rl_decode_attn_t h, int32_t batch, int32_t num_pages, const void* q,
                                        const void* k_cache, const void* v_cache, const float* k_scale,
                                        const float* v_scale, const int32_t* block_table,
                                        const int32_t* seq_lens, void* out, void* workspace,
                                        size_t workspace_bytes, void* stream, void* event_begin,
                                        void* event_end) {
  if (!event_begin || !event_end) return RLDA_ERR_INVALID_ARG;
  return run_impl(h, batch, num_pages, 0, nullptr, -1, q, k_cache, v_cache, k_scale, v_scale, block_table, seq_lens,
                  out, workspace, workspace_bytes, stream, event_begin, event_end);
}

rlda_status rl_decode_attn_run_noalloc(rl_decode_attn_t h, int32_t batch, int32_t num_pages, const void* q,
                                       const void* k_cache, const void* v_cache, const float* k_scale,
                                       const float* v_scale, const int32_t* block_table, const int32_t* seq_lens,
                                       void* out, uint32_t* flags, void* stream) {
  if (!h) return RLDA_ERR_INVALID_ARG;
  const rl_decode_attn_config& c = h->cfg;
  if (batch < 0 || batch > c.max_batch || num_pages < 0) return RLDA_ERR_INVALID_ARG;
  if ((uintptr_t)flags & 3u) return RLDA_ERR_INVALID_ARG;
  // The static scratch holds counters for batch * Hkv segments and partial slots of
  // 16 rows of at most 128 elements; checked before any HIP call.
  if ((int64_t)batch * c.num_kv_heads > rlda::kScratchMaxSegments || c.head_dim > 128) return RLDA_ERR_SCRATCH;
  if (batch == 0) return RLDA_OK;
  void* base = nullptr;
  if (rlda::noalloc_scratch(&base) != 0) return RLDA_ERR_HIP;
  char* sc = (char*)base;
  const RunMem mem = {flags ? flags : (uint32_t*)sc, (uint32_t*)(sc + rlda::kScratchCountersOff),
                      (float*)(sc + rlda::kScratchMlOff), (float*)(sc + rlda::kScratchAccOff),
                      rlda::kScratchMaxRanges};
  return run_impl(h, batch, num_pages, 0, nullptr, -1, q, k_cache, v_cache, k_scale, v_scale, block_table, seq_lens,
                  out, nullptr, 0, stream, nullptr, nullptr, &mem);
}

rlda_status rl_decode_attn_run_grouped(rl_decode_attn_t h, int32_t batch, int32_t num_pages, int32_t group_size,
                                       const int32_t* prefix_pages, int32_t prompt_pages_hint, const void* q,
                                       const void* k_cache,
                                       const void* v_cache, const float* k_scale, const float* v_scale,
                                       const int32_t* block_table, const int32_t* seq_lens, void* out,
                                       void* workspace, size_t workspace_bytes, void* stream, void* event_begin,
                                       void* event_end) {
  if (group_size < 1 || (!event_begin) != (!event_end)) return RLDA_ERR_INVALID_ARG;
  return run_impl(h, batch, num_pages, group_size, prefix_pages, prompt_pages_hint, q, k_cache, v_cache, k_scale,
                  v_scale, block_table, seq_lens, out, workspace, workspace_bytes, stream, event_begin, event_end);
}

rlda_status rl_decode_attn_append(rl_decode_attn_t h, int32_t batch, int32_t num_pages, const void* k_new,
                                  const void* v_new, void* k_cache, void* v_cache, float* k_scale, float* v_scale,
                                  const int32_t* block_table, const int32_t* seq_lens, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  if (!h) return RLDA_ERR_INVALID_ARG;
  const rl_decode_attn_config& c = h->cfg;
  if (batch < 0 || batch > c.max_batch || num_pages < 0) return RLDA_ERR_INVALID_ARG;
  if (batch == 0) return RLDA_OK;
  if (!k_new || !v_new || !block_table || !seq_lens) return RLDA_ERR_INVALID_ARG;
  if (num_pages > 0 && (!k_cache || !v_cache)) return RLDA_ERR_INVALID_ARG;
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) || !aligned16(v_cache))
    return RLDA_ERR_INVALID_ARG;
  if (((uintptr_t)block_table & 3u) || ((uintptr_t)seq_lens & 3u)) return RLDA_ERR_INVALID_ARG;
  if (h->kind == rlda::KvKind::FP8 && num_pages > 0 &&
      (!k_scale || !v_scale || ((uintptr_t)k_scale & 3u) || ((uintptr_t)v_scale & 3u)))
    return RLDA_ERR_INVALID_ARG;
  const WsLayout wl = layout_of(h);
  if (!workspace || ((uintptr_t)workspace % kAlign)) return RLDA_ERR_WORKSPACE;
  if (workspace_bytes < wl.total) return RLDA_ERR_WORKSPACE;
  rlda::Params p;
  memset(&p, 0, sizeof p);
  p.k = k_cache;
  p.v = v_cache;
  p.k_scale = k_scale;
  p.v_scale = v_scale;
  p.k_in = k_new;
  p.v_in = v_new;
  p.block_table = block_table;
  p.seq_lens = seq_lens;
  p.flags = (uint32_t*)((char*)workspace + wl.flags);
  const int eb = elem_bytes(c.kv_dtype);
  p.stride_page = h->stride_page * eb;
  p.stride_head = h->stride_head * eb;
  p.stride_slot = (int32_t)(h->stride_slot * eb);
  p.batch = batch;
  p.num_pages = num_pages;
  p.num_q_heads = c.num_q_heads;
  p.num_kv_heads = c.num_kv_heads;
  p.group = h->group;
  p.max_pages = c.max_pages_per_seq;
  if (rlda::launch_append(h->kind, c.head_dim, p, stream) != hipSuccess) return RLDA_ERR_HIP;
  return RLDA_OK;
}

rlda_status rl_decode_attn_run_multi(rl_decode_attn_t h, int32_t batch, int32_t num_pages, int32_t total_q,
                                     int32_t max_q_len, const void* q, const void* k_cache, const void* v_cache,
                                     const float* k_scale, const float* v_scale, const int32_t* block_table,
                                     const int32_t* seq_lens, const int32_t* q_start, void* out, void* workspace,
                                     size_t workspace_bytes, void* stream, void* event_begin, void* event_end) {
  if (!h) return RLDA_ERR_INVALID_ARG;
  const rl_decode_attn_config& c = h->cfg;
  if (batch < 0 || batch > c.max_batch || num_pages < 0 || total_q < 0 || max_q_len < 0) return RLDA_ERR_INVALID_ARG;
  if ((!event_begin) != (!event_end)) return RLDA_ERR_INVALID_ARG;
  if (h->kind == rlda::KvKind::F32) return RLDA_ERR_UNSUPPORTED;
  // Few rows per sequence: the decode kernel's page stream, which splits long
  // sequences across workgroups.  The rows of a (sequence, KV head), at most 64,
  // are held by a wave as one or two 16-row tiles against each page; more than 32
  // take two segments.  Otherwise the 128-row MFMA kernel.
  const int64_t rows = (int64_t)max_q_len * h->group;
  int tiles = rows > rlda::kMaxGroup && batch <= rlda::kTwoTileMaxBatch ? rlda::kMaxRowTiles : 1;
  int64_t row_chunks = (rows + rlda::kMaxGroup * tiles - 1) / (rlda::kMaxGroup * tiles);
  const bool rows_path = max_q_len >= 1 && max_q_len <= rlda::kMaxRowsQLen &&
                         rows <= (int64_t)rlda::kMaxGroup * rlda::kMaxRowChunks &&
                         (int64_t)batch * (c.max_pages_per_seq + rlda::kStartCost) * c.num_kv_heads * row_chunks <= INT32_MAX;
  if (!rows_path && batch > rlda::kMultiMaxBatch) return RLDA_ERR_UNSUPPORTED;
  // The kernels address q with 32-bit byte offsets.
  if ((int64_t)total_q * c.num_q_heads * c.head_dim * 2 > INT32_MAX) return RLDA_ERR_UNSUPPORTED;
  if (batch == 0 || total_q == 0) return RLDA_OK;
  if (!q || !block_table || !seq_lens || !q_start || !out) return RLDA_ERR_INVALID_ARG;
  if (num_pages > 0 && (!k_cache || !v_cache)) return RLDA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out)) return RLDA_ERR_INVALID_ARG;
  if (((uintptr_t)block_table & 3u) || ((uintptr_t)seq_lens & 3u) || ((uintptr_t)q_start & 3u))
    return RLDA_ERR_INVALID_ARG;
  if (h->kind == rlda::KvKind::FP8 && num_pages > 0 &&
      (!k_scale || !v_scale || ((uintptr_t)k_scale & 3u) || ((uintptr_t)v_scale & 3u)))
    return RLDA_ERR_INVALID_ARG;
  const WsLayout wl = layout_of(h);
  if (!workspace || ((uintptr_t)workspace % kAlign)) return RLDA_ERR_WORKSPACE;
  if (workspace_bytes < wl.total) return RLDA_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  rlda::Params p;
  memset(&p, 0, sizeof p);
  p.q = q;
  p.k = k_cache;
  p.v = v_cache;
  p.k_scale = k_scale;
  p.v_scale = v_scale;
  p.block_table = block_table;
  p.seq_lens = seq_lens;
  p.q_start = q_start;
  p.total_q = total_q;
  p.max_q_len = max_q_len;
  p.out = out;
  p.flags = (uint32_t*)(ws + wl.flags);
  const int eb = elem_bytes(c.kv_dtype);
  p.stride_page = h->stride_page * eb;
  p.stride_head = h->stride_head * eb;
  p.stride_slot = (int32_t)(h->stride_slot * eb);
  p.batch = batch;
  p.num_pages = num_pages;
  p.num_q_heads = c.num_q_heads;
  p.num_kv_heads = c.num_kv_heads;
  p.group = h->group;
  p.max_pages = c.max_pages_per_seq;
  p.scale_log2 = h->scale * 1.4426950408889634f;
  p.out_bf16 = c.out_dtype == RLDA_BF16;
  memcpy(p.q_head, h->q_head, sizeof p.q_head);
  if (rows_path) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return RLDA_ERR_HIP;
    int ranges = c.num_work_ranges > 0 ? c.num_work_ranges : cu_count(dev);
    if (ranges <= 0) return RLDA_ERR_HIP;
    // Partial slots hold one segment's rows each; the workspace has room for
    // 2 * ws_ranges * 16 rows.  A workspace sized for fewer ranges than two-tile
    // slots need falls back to one tile per segment.
    if (tiles == 2 && (int64_t)h->ws_ranges * rlda::kMaxGroup / std::min<int64_t>(rows, 32) < 1) {
      tiles = 1;
      row_chunks = (rows + rlda::kMaxGroup - 1) / rlda::kMaxGroup;
    }
    p.row_chunks = (int)row_chunks;
    p.part_rows = (int)std::min<int64_t>(rows, (int64_t)rlda::kMaxGroup * tiles);
    const int64_t cap_ranges = (int64_t)h->ws_ranges * rlda::kMaxGroup / p.part_rows;
    if (ranges > cap_ranges) ranges = (int)cap_ranges;
    if (ranges > rlda::kMaxRanges) ranges = rlda::kMaxRanges;
    const int64_t max_units = (int64_t)batch * c.num_kv_heads * row_chunks * c.max_pages_per_seq;
    if (ranges > max_units) ranges = (int)max_units;
    if (ranges < 1) ranges = 1;
    p.nranges = ranges;
    p.counters = (uint32_t*)(ws + wl.counters);
    p.call_tag = next_call_tag();
    p.part_ml = (float*)(ws + wl.part_ml);
    p.part_acc = (float*)(ws + wl.part_acc);
    if (rlda::launch_decode_rows(h->kind, c.head_dim, tiles, p, stream, event_begin, event_end) != hipSuccess)
      return RLDA_ERR_HIP;
    return RLDA_OK;
  }
  // One workgroup per (row block, KV head): a sequence's n_b * G rows take at most
  // n_b * G / rows_per_block + 1 blocks, so this grid covers every consistent q_start.
  const int64_t blocks = ((int64_t)total_q * h->group + rlda::kMultiRows - 1) / rlda::kMultiRows + batch;
  // Four KV heads: each XCD takes one KV head of one of two sequence classes, and
  // the grid holds 8 blocks per row block so that either class fits (see the kernel).
  const int64_t grid = blocks * (c.num_kv_heads == 4 ? 8 : c.num_kv_heads);
  if (grid > INT32_MAX) return RLDA_ERR_UNSUPPORTED;
  if (rlda::launch_multi(h->kind, c.head_dim, p, (int)grid, stream, event_begin, event_end) != hipSuccess)
    return RLDA_ERR_HIP;
  return RLDA_OK;
}

rlda_status rl_decode_attn_read_flags(rl_decode_attn_t h, const void* workspace, void* stream, uint32_t* flags) {
  if (!h || !workspace || !flags) return RLDA_ERR_INVALID_ARG;
  uint32_t v = 0;
  if (hipMemcpyAsync(&v, (const char*)workspace + layout_of(h).flags, sizeof v, hipMemcpyDeviceToHost,
                     (hipStream_t)stream) != hipSuccess)
    return RLDA_ERR_HIP;
  if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return RLDA_ERR_HIP;
  *flags = v;
  return RLDA_OK;
}

rlda_status rl_decode_attn_destroy(rl_decode_attn_t h) {
  delete h;
  return RLDA_OK;
}

const char* rl_decode_attn_strerror(rlda_status s) {
  switch (s) {
    case RLDA_OK: return "ok";
    case RLDA_ERR_INVALID_ARG: return "invalid argument";
    case RLDA_ERR_UNSUPPORTED: return "unsupported configuration";
    case RLDA_ERR_HIP: return "HIP runtime error";
    case RLDA_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case RLDA_ERR_ALLOC: return "host allocation failed";
    case RLDA_ERR_SCRATCH: return "request exceeds the static scratch of the no-allocation entry point";
  }
  return "unknown status";
}

}  // extern "C"
