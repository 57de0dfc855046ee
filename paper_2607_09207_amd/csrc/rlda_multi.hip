// Multi-token queries (prefill chunks) over the paged KV cache, for gfx950.
//
// Rollout runs prefill over the prompt tokens before it decodes them (Sec. 3,
// rollout); the prefill cost model (App. A.1.2) charges its attention with a term
// quadratic in the prompt length, so unlike decode this operation is a dense
// contraction and runs on the matrix cores.  Sequence b brings n_b query rows (its
// last n_b cached tokens, K/V already in the cache); row i attends causally to
// positions 0 .. seq_lens[b] - n_b + i.
//
// Work.  The query rows of one (sequence, KV head) are its n_b * G (token, query
// head) pairs, token-major, so every K/V row read serves all G heads sharing that
// KV head.  A workgroup takes 128 of them: each of its 4 waves owns one 32-row
// MFMA tile.  Workgroups are numbered heaviest first over the whole call (the row
// blocks that attend to the most keys are dispatched first), so the slots of the
// GPU fill longest-job-first.
//
// Keys.  The workgroup walks its causal key range in blocks of 32 keys (two
// pages).  Each wave brings one page of K or V of every block (page ids come
// through the scalar cache one block before that): bf16 pages at d = 128 by
// buffer-load DMA straight into LDS, two blocks ahead; other caches through
// registers one block ahead (fp8 converted exactly to bf16 on the way).  Per block:
//   S^T[key][row] = K Q^T    v_mfma_f32_32x32x16_bf16, K from LDS, Q in registers;
//   online softmax per row (lanes l and l^32 hold one row), with the reference
//   maximum moved only when a score exceeds it by more than 2^8;
//   O^T[d][row] += V^T P^T   the score registers are the P^T operand as they are;
//                            V^T comes from the row-major V block through the
//                            LDS transpose read (ds_read_b64_tr_b16).
// The causal mask is evaluated only on blocks that reach a row's limit.  fp8 K
// scales multiply the scores and V scales multiply P, per page.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rlda_device.h"
#include "rlda_params.h"

namespace rlda {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

#ifndef RLDA_MQ_KPAD
#define RLDA_MQ_KPAD 16                       // LDS row padding of the K block (bytes)
#endif
#ifndef RLDA_MQ_VPAD
#define RLDA_MQ_VPAD 32                       // ... of the V block
#endif
constexpr int kTile = 32;                     // rows (and keys) of one MFMA tile
constexpr int kNT = kMultiTiles;              // 32-row tiles per wave
#ifndef RLDA_MQ_KEY_TILES
#define RLDA_MQ_KEY_TILES 1                   // 32-key score tiles per key block
#endif
constexpr int kKH = RLDA_MQ_KEY_TILES;
constexpr int kKeys = kTile * kKH;            // keys per block (2 kKH pages)

#ifndef RLDA_MQ_WAVES_D64
#define RLDA_MQ_WAVES_D64 4                   // waves per SIMD at d = 64 (about 100 registers)
#endif
#ifndef RLDA_MQ_PREFETCH
#define RLDA_MQ_PREFETCH 1                    // blocks loaded ahead into registers (register staging)
#endif
#ifndef RLDA_MQ_DMA
#define RLDA_MQ_DMA 1                         // bf16, d = 128: pages go to LDS by buffer-load DMA
#endif

// Workgroup barrier for the DMA path: wait until at most N vector-memory
// operations of this wave are outstanding (the DMAs of the newest block) and its
// LDS operations are done, then s_barrier.  __syncthreads would wait for every
// outstanding DMA (its release fence counts them as stores).  The asm's memory
// clobber keeps the compiler from moving memory accesses across it.
template <int N>
__device__ __forceinline__ void dma_barrier() {
  static_assert(N >= 0 && N < 16, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}
static_assert(kTile * kNT * kWaves == kMultiRows, "a workgroup's rows are its waves' tiles");

template <int D, bool FP8>
struct MqShape {
  static constexpr int KS = D / 16;           // 32x32x16 k-steps of K Q^T
  static constexpr int DT = D / 32;           // 32-wide output tiles of O^T
  static constexpr int EB = FP8 ? 1 : 2;      // bytes per cached element
  // bf16 pages at d = 128 are copied to LDS by the buffer-load DMA (no registers,
  // no LDS writes by the waves) into unpadded rows whose 16-byte chunks are
  // permuted per row (see chunk_pos); other caches are staged through registers
  // (fp8 is converted on the way) into padded rows.
  static constexpr bool DMA = !FP8 && D == 128 && RLDA_MQ_DMA;
  static constexpr int NBUF = DMA ? 3 : 2;    // LDS block buffers
  // Waves per SIMD (register budget 512 / waves).  With the V operands read after
  // the softmax, three fit (168 registers): the DMA path without staging registers,
  // the register path with one block of staging in flight.  At d = 64 the state is
  // about 100 registers, and four fit.
#ifdef RLDA_MQ_WAVES
  static constexpr int WAVES = RLDA_MQ_WAVES;
#else
  static constexpr int WAVES = kNT == 1 ? (D == 64 ? RLDA_MQ_WAVES_D64 : 3) : 1;
#endif
  static constexpr int KRS = DMA ? 2 * D : 2 * D + RLDA_MQ_KPAD;   // LDS row stride of the K block (bytes)
  static constexpr int VRS = DMA ? 2 * D : 2 * D + RLDA_MQ_VPAD;   // ... of the V block
  static constexpr int CPR = D * EB / 16;     // 16-byte chunks per cached row
  static constexpr int LPL = kPage * CPR / 64; // 16-byte loads per lane to stage one page
};

// Max / sum of a value with the one 32 lanes away (the other half of a score
// row), both halves getting the result: v_permlane32_swap of x with itself leaves
// the lower halves of x in one result and the upper halves in the other.
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ bf16x4 lds_tr_read(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(__attribute__((address_space(3))) char*)p);
}

template <int D, bool FP8>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads),
                          amdgpu_waves_per_eu(MqShape<D, FP8>::WAVES, MqShape<D, FP8>::WAVES)))
void multi_query_kernel(const Params p) {
  using S = MqShape<D, FP8>;
  // Two block buffers: block kb is computed from one while block kb + 1 is written
  // to the other.
  __shared__ __align__(16) char s_k[S::NBUF][kKeys * S::KRS];
  __shared__ __align__(16) char s_v[S::NBUF][kKeys * S::VRS];
  __shared__ float s_scale[S::NBUF][4 * kKH];   // fp8: K scales of the block's pages, then V's
  __shared__ int32_t s_bad[S::NBUF][2 * kKH];   // page of the block not in the pool (contributes nothing)
  __shared__ int32_t s_scan[kWaves], s_emax[kWaves];
  __shared__ int16_t s_qh[kMaxQHeads];
  __shared__ uint8_t s_cls[64];   // sequence classes (XCD placement, batches of at most 64)
  // Per sequence: {L - n_b (position of query token 0), n_b G rows} (rows 0 when
  // its offsets are inconsistent).
  extern __shared__ int2 s_sq[];   // [batch], then s_key [batch]

  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  const int batch = p.batch, Hkv = p.num_kv_heads, G = p.group, Hq = p.num_q_heads;
  const int cap = p.max_pages * kPage;
  // Ordering key of each sequence's row blocks: its key count L when they are
  // dispatched together, -1 when each row block is ordered by its own key count.
  int32_t* s_key = (int32_t*)(s_sq + batch);

  // 1. Rows of every sequence and the number of row blocks (identical in every
  //    workgroup).  Inconsistent offsets give a sequence no rows; they, and lengths
  //    out of range or shorter than the rows, raise the flag.
  int nitems = 0, emax = 0;   // emax: the most keys any sequence's rows see
  {
    int sum = 0, bad = 0, lmax = 0;
    for (int b = tid; b < batch; b += kThreads) {
      const int q0 = p.q_start[b], q1 = p.q_start[b + 1];
      const bool ok = q0 >= 0 && q1 >= q0 && q1 <= p.total_q;
      const int n = ok ? q1 - q0 : 0;
      int L = p.seq_lens[b];
      if (!ok || L < 0 || L > cap || n > L) bad = 1;
      L = min(max(L, 0), cap);
      const int rows = (int)min((int64_t)n * G, (int64_t)INT32_MAX - kMultiRows);
      s_sq[b] = make_int2(L - n, rows);
      sum += (rows + kMultiRows - 1) / kMultiRows;
      if (rows > 0) lmax = max(lmax, L);
    }
    if (__builtin_amdgcn_ballot_w64(bad) != 0 && blockIdx.x == 0 && lane == 0) atomicOr(p.flags, kFlagBadLen);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      sum += __shfl_xor(sum, o);
      lmax = max(lmax, __shfl_xor(lmax, o));
    }
    if (lane == 0) {
      s_scan[wave] = sum;
      s_emax[wave] = lmax;
    }
    for (int e = tid; e < Hq; e += kThreads) s_qh[e] = p.q_head[e];
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      nitems += s_scan[w];
      emax = max(emax, s_emax[w]);
    }
    // A sequence whose rows see at most an eighth of the largest job's keys apart
    // is dispatched as a group (its row blocks then read its pages together).
    for (int b = tid; b < batch; b += kThreads) {
      const int2 sq = s_sq[b];
      const int n = sq.y / G;
      s_key[b] = (sq.y > 0 && 8 * (int64_t)n <= emax) ? max(0, sq.x + n) : -1;
    }
    __syncthreads();
  }
  const int64_t items = (int64_t)nitems * Hkv;
  if (blockIdx.x == 0 && tid == 0 && items > (int64_t)gridDim.x) atomicOr(p.flags, kFlagBadLen);

  // 2. The (sequence b, row block rb, KV head g) items of this workgroup.  Row block
  //    rb of sequence b covers rows [128 rb, r1), r1 = min(128 (rb + 1), n_b G), and
  //    reads the keys below E = max(0, L - n_b + (r1 - 1) / G + 1), its cost.
  //    Placement: workgroups are dispatched round-robin over the 8 XCDs (block u on
  //    XCD u % 8), and the row blocks of one (sequence, KV head) read the same pages,
  //    so they are kept on one XCD, whose L2 then serves the repeats:
  //      Hkv a multiple of 8: XCD x takes KV heads (x + b) % 8, + 8, ... of every
  //                           sequence b;
  //      Hkv = 4:             XCD x takes KV head (x + b) % 4 of the sequences b of
  //                           class x / 4, the two classes balanced by work (rank by
  //                           estimated keys, snake order; batches above 64: b mod 2),
  //                           the grid holding 8 blocks per (sequence, row block) so
  //                           that either class fits;
  //      otherwise:           one set over the whole grid, no placement.
  //    Within its set each XCD dispatches heaviest first (keys descending; ties by
  //    sequence, then last row block first, then KV head), so the slots of the XCD
  //    fill longest-job-first.  The row blocks of a sequence whose rows span at most
  //    an eighth of the largest job's keys all take the sequence's key count L: they
  //    run together and read the sequence's pages side by side, once from HBM; block t of the XCD takes item t of its set (blocks
  //    past the set's end return).  Item t is found by a binary search on the key count: with
  //    C(x) the items having at least x keys (a closed form per sequence, summed
  //    across the wave), its key count x* is the largest x with C(x) > t.  Every wave
  //    finds it (no barrier).
  const int u = blockIdx.x, xcd = u & 7;
  const bool by_head = Hkv % 8 == 0, by_class = Hkv == 4;
  const int ncls = by_class ? 8 / Hkv : 1, my_cls = by_class ? xcd / Hkv : 0;
  const int hx = by_head ? Hkv / 8 : (by_class ? 1 : Hkv);   // KV heads per (b, rb) in the set
  const int t_first = (by_head || by_class) ? u >> 3 : u;
  if (by_class && batch <= 64) {
    // Class of each sequence: sort by estimated keys (descending; bitonic across the
    // lanes of wave 0), then deal the ranks out in snake order 0, 1, .., K-1, K-1, .., 0.
    if (wave == 0) {
      float key = -1.f;
      int id = lane;
      if (lane < batch) {
        const int2 sq = s_sq[lane];
        const int nrb = (sq.y + kMultiRows - 1) / kMultiRows;
        key = (float)nrb * ((float)max(sq.x, 0) + 0.5f * (float)(sq.y / G) + 1.f);
      }
#pragma unroll
      for (int k = 2; k <= 64; k <<= 1)
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
          const float ok = __shfl_xor(key, j);
          const int oid = __shfl_xor(id, j);
          const bool mine_first = key > ok || (key == ok && id < oid);
          const bool keep = (((lane & j) == 0) == ((lane & k) == 0)) ? mine_first : !mine_first;
          if (!keep) {
            key = ok;
            id = oid;
          }
        }
      const int rr = lane % (2 * ncls);
      if (id < batch) s_cls[id] = (uint8_t)(rr < ncls ? rr : 2 * ncls - 1 - rr);
    }
    __syncthreads();
  }
  auto in_set = [&](int b) {
    return !by_class || (batch <= 64 ? (int)s_cls[b] : b % ncls) == my_cls;
  };
  // Row blocks of sequence `sq` with at least x keys (E is non-decreasing in rb).
  auto at_least = [&](int2 sq, int key, int x) -> int {
    const int rows = sq.y;
    const int nrb = (rows + kMultiRows - 1) / kMultiRows;
    if (x <= 0) return nrb;
    if (key >= 0) return key >= x ? nrb : 0;   // dispatched as a group
    const int64_t k = (int64_t)x - sq.x - 1;   // x >= 1: E >= x iff (r1 - 1) / G >= k
    if (k <= 0) return nrb;
    const int64_t thr = (int64_t)G * k + 1;   // ... iff r1 >= thr
    if (rows < thr) return 0;
    return nrb - (int)((thr + kMultiRows - 1) / kMultiRows - 1);
  };
  auto count = [&](int x) {
    int c = 0;
    for (int b = lane; b < batch; b += 64)
      if (in_set(b)) c += at_least(s_sq[b], s_key[b], x);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o);
    return c;   // the same in every lane
  };
  const int set_items = count(0) * hx;

  if (t_first >= set_items) return;
  const int v = t_first / hx, hsub = t_first - v * hx;
  int b = 0, rb = 0;
  {
    int lo = 0, hi = cap + 1, chi = 0;   // C(lo) > v >= C(hi) = chi
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      const int c = count(mid);
      if (c > v) {
        lo = mid;
      } else {
        hi = mid;
        chi = c;
      }
    }
    // Among the items with exactly lo keys, the (v - chi)-th in sequence order.
    int j = v - chi, found = 0;
    for (int b0 = 0; b0 < batch && !found; b0 += 64) {
      const int bb = b0 + lane;
      int c1 = 0, c2 = 0, nrb = 0;
      if (bb < batch && in_set(bb)) {
        const int2 sq = s_sq[bb];
        const int key = s_key[bb];
        c1 = at_least(sq, key, lo);
        c2 = at_least(sq, key, lo + 1);
        nrb = (sq.y + kMultiRows - 1) / kMultiRows;
      }
      const int eq = c1 - c2;
      int incl = eq;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
      const uint64_t hit = __builtin_amdgcn_ballot_w64(j >= incl - eq && j < incl);
      if (hit) {
        const int src = __builtin_ctzll(hit);
        b = __builtin_amdgcn_readlane(bb, src);
        rb = __builtin_amdgcn_readlane(nrb - c2 - 1, src) - (j - __builtin_amdgcn_readlane(incl - eq, src));
        found = 1;
      } else {
        j -= __builtin_amdgcn_readlane(incl, 63);
      }
    }
    b = uni(b);
    rb = uni(rb);
  }
  // The KV head: rotated by the sequence, so that every XCD serves every head (the
  // head fixes the page tiles' offset, and with it their HBM channels).
  const int g = by_head ? ((xcd + b) & 7) + 8 * hsub : (by_class ? (xcd + b) % Hkv : hsub);
  const int q0 = p.q_start[b];
  const int2 sqb = s_sq[b];
  const int n = sqb.y / G;
  const int L = sqb.x + n;
  const int rows = n * G;
  const int r0 = rb * kMultiRows, r1 = min(r0 + kMultiRows, rows);
  const int base_pos = L - n;                                   // position of query token 0
  const int E = max(0, base_pos + (r1 - 1) / G + 1);            // keys the workgroup reads
  const int nkb = (E + kKeys - 1) / kKeys;
  const int wr0 = r0 + kTile * kNT * wave, wr1 = min(wr0 + kTile * kNT, r1);
  const int Ew = wr0 < wr1 ? max(0, base_pos + (wr1 - 1) / G + 1) : 0;       // keys this wave needs
  const int Ew_full = wr0 < wr1 ? max(0, base_pos + wr0 / G + 1) : 0;       // ... visible to all its rows

  // This lane's query rows, one per tile: lanes i and i + 32 share row wr0 + 32 t + i.
  const int i = lane & 31, hh = lane >> 5;
  bool live[kNT];
  int qi[kNT], head[kNT], lim[kNT];
#pragma unroll
  for (int t = 0; t < kNT; ++t) {
    const int row = wr0 + kTile * t + i;
    live[t] = row < wr1;
    qi[t] = live[t] ? row / G : 0;
    head[t] = live[t] ? s_qh[g * G + (row - qi[t] * G)] : 0;
    lim[t] = live[t] ? base_pos + qi[t] + 1 : 0;               // keys [0, lim) are visible
  }

  // Q operands (B of K Q^T): lane 32h + i holds its row's elements [16s + 8h, 16s + 8h + 8).
  bf16x8 qop[kNT][S::KS];
  {
    const __amdgpu_buffer_rsrc_t rq = make_rsrc_uni(p.q, (uint32_t)p.total_q * (uint32_t)Hq * D * 2u);
#pragma unroll
    for (int t = 0; t < kNT; ++t) {
      const int off = live[t] ? ((q0 + qi[t]) * Hq + head[t]) * D * 2 : kPastRange;
#pragma unroll
      for (int s = 0; s < S::KS; ++s)
        qop[t][s] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rq, off + 16 * (2 * s + hh), 0, 0));
    }
  }

  // Staging: wave w brings pages (w & 1) + 2h, h < kKH, of each block's K (w < 2)
  // or V (w >= 2).
  const int which = wave >> 1, pgw = wave & 1;
  const char* pool = (const char*)(which ? p.v : p.k);
  const float* scl = which ? p.v_scale : p.k_scale;
  // Register sets of the blocks in flight: block kb is loaded into set kb % PD
  // PD blocks before it is computed (global latency is several blocks' work).
  constexpr int PD = RLDA_MQ_PREFETCH;
  u32x4 stg[PD][kKH][S::LPL];
  float stg_scale[PD][kKH];
  int stg_bad[PD][kKH];
  // Page ids come through the scalar cache (the block table is read-only here),
  // one block ahead of the loads that use them; the index is clamped into the row
  // so the load is always in bounds (pages past the keys are not used).
  typedef const __attribute__((address_space(4))) int32_t bt_elem;
  bt_elem* bt_row = (bt_elem*)(const void*)(p.block_table + (int64_t)b * p.max_pages);
  auto page_index = [&](int kb, int h) { return 2 * kKH * kb + pgw + 2 * h; };
  auto page_ids = [&](int kb, int* pid) {
#pragma unroll
    for (int h = 0; h < kKH; ++h) pid[h] = bt_row[min(page_index(kb, h), p.max_pages - 1)];
  };
  auto stage_load = [&](int kb, int set, const int* pid) {
#pragma unroll
    for (int h = 0; h < kKH; ++h) {
      const int j = page_index(kb, h);   // page index in the sequence
      int tok = min(max(E - j * kPage, 0), kPage);
      stg_bad[set][h] = 0;
      if (tok > 0) {
        if ((unsigned)pid[h] >= (unsigned)p.num_pages) {
          if (lane == 0) atomicOr(p.flags, kFlagBadPage);
          tok = 0;
          stg_bad[set][h] = 1;
        }
      }
      const int64_t po = tok > 0 ? (int64_t)pid[h] * p.stride_page + (int64_t)g * p.stride_head : 0;
      const uint32_t nrec = tok > 0 ? (uint32_t)((tok - 1) * p.stride_slot + D * S::EB) : 0u;
      const __amdgpu_buffer_rsrc_t r = make_rsrc_uni(pool + po, nrec);
#pragma unroll
      for (int k = 0; k < S::LPL; ++k) {
        const int ci = lane + 64 * k, rr = ci / S::CPR, c = ci % S::CPR;
        stg[set][h][k] = __builtin_amdgcn_raw_buffer_load_b128(r, rr * p.stride_slot + 16 * c, 0, 0);
      }
      if constexpr (FP8) stg_scale[set][h] = tok > 0 ? scl[(int64_t)pid[h] * Hkv + g] : 0.f;
    }
  };
  auto stage_write = [&](int set, int buf) {
    char* dst = which ? s_v[buf] : s_k[buf];
    const int RS = which ? S::VRS : S::KRS;
#pragma unroll
    for (int h = 0; h < kKH; ++h) {
#pragma unroll
      for (int k = 0; k < S::LPL; ++k) {
        const int ci = lane + 64 * k, rr = ci / S::CPR, c = ci % S::CPR;
        char* rowp = dst + (kPage * (pgw + 2 * h) + rr) * RS;
        if constexpr (!FP8) {
          *(u32x4*)(rowp + 16 * c) = stg[set][h][k];
        } else {   // 16 E4M3 values -> 16 bf16 (exact)
          uint32_t w[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if constexpr (kFp8Direct) {
              w[2 * e] = fp8x2_to_bf16x2(stg[set][h][k][e], false);
              w[2 * e + 1] = fp8x2_to_bf16x2(stg[set][h][k][e], true);
            } else {
              const f32x2 a = fp8x2_to_f32(stg[set][h][k][e], false), bb = fp8x2_to_f32(stg[set][h][k][e], true);
              w[2 * e] = pack_bf16(a[0], a[1]);
              w[2 * e + 1] = pack_bf16(bb[0], bb[1]);
            }
          }
          *(u32x4*)(rowp + 32 * c) = u32x4{w[0], w[1], w[2], w[3]};
          *(u32x4*)(rowp + 32 * c + 16) = u32x4{w[4], w[5], w[6], w[7]};
        }
      }
      if (lane == 0) {
        if constexpr (FP8) s_scale[buf][2 * kKH * which + pgw + 2 * h] = stg_scale[set][h];
        if (which == 0) s_bad[buf][pgw + 2 * h] = stg_bad[set][h];
      }
    }
  };

  // DMA path: 16-byte chunk c of row r (the row's slot in its page) sits at chunk
  // position c ^ (r & 15) in K rows and c ^ 4 (r & 3) in V rows, so that the
  // score operand reads (16 rows, one chunk) and the transpose reads (4 rows, 4
  // chunks, two 16-lane groups) each touch all 64 banks once.  Lane l of the k-th
  // DMA of a page fills slot 64k + l of the page, row (64k + l) / 16, position
  // (64k + l) % 16, so it fetches the chunk that belongs there.
  auto chunk_pos = [](bool v_rows, int r, int c) { return c ^ (v_rows ? 4 * (r & 3) : (r & 15)); };
  int bad_pages = 0;   // DMA path: the flag is raised after the loop (no atomics between the DMAs)
  auto dma_issue = [&](int kb, int buf, const int* pid) {
    char* dst = which ? s_v[buf] : s_k[buf];
#pragma unroll
    for (int h = 0; h < kKH; ++h) {
      const int j = page_index(kb, h);
      int tok = min(max(E - j * kPage, 0), kPage);
      int badp = 0;
      if (tok > 0 && (unsigned)pid[h] >= (unsigned)p.num_pages) {
        tok = 0;
        badp = 1;
      }
      bad_pages |= badp;
      const int64_t po = tok > 0 ? (int64_t)pid[h] * p.stride_page + (int64_t)g * p.stride_head : 0;
      const uint32_t nrec = tok > 0 ? (uint32_t)((tok - 1) * p.stride_slot + D * S::EB) : 0u;
      const __amdgpu_buffer_rsrc_t r = make_rsrc_uni(pool + po, nrec);
      char* page_base = dst + kPage * (pgw + 2 * h) * S::KRS;
#pragma unroll
      for (int k = 0; k < S::LPL; ++k) {
        const int sl = 64 * k + lane, rr = sl / S::CPR, c = chunk_pos(which != 0, rr, sl % S::CPR);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            r, (__attribute__((address_space(3))) void*)(page_base + 1024 * k), 16, rr * p.stride_slot + 16 * c, 0, 0, 0);
      }
      if (which == 0 && lane == 0) s_bad[buf][pgw + 2 * h] = badp;
    }
  };

  f32x16 acc[kNT][S::DT];
  float m[kNT], l[kNT];
#pragma unroll
  for (int t = 0; t < kNT; ++t) {
#pragma unroll
    for (int c = 0; c < S::DT; ++c) acc[t][c] = f32x16{};
    m[t] = neg_inf();
    l[t] = 0.f;
  }

  // P^T operands of the current block per tile: key tile kh, key step kk.
  bf16x8 pb[kNT][kKH][2];
  // Online softmax of tile t on block kb: updates (m, l), rescales the tile's
  // accumulators when m moves and leaves the block's P^T operands in pb[t].
  auto softmax = [&](int t, int kb, int buf, const f32x16* sc) {
    // Lane 32h + i holds S^T[key 32kh + 8(j/4) + 4h + j%4][row i] of key tile kh,
    // j < 16: page 2kh for j < 8, 2kh + 1 above.
    float km[2 * kKH], vm[2 * kKH];
    int bad = 0;
#pragma unroll
    for (int q = 0; q < 2 * kKH; ++q) {
      km[q] = FP8 ? p.scale_log2 * s_scale[buf][q] : p.scale_log2;
      vm[q] = FP8 ? s_scale[buf][2 * kKH + q] : 1.f;
      bad |= s_bad[buf][q];
    }
    // bf16: one positive factor for the whole block, so the maximum is taken on the
    // raw scores and the factor enters the exponent's fma; fp8: per-page factors.
    float sv[kKH][16];
#pragma unroll
    for (int kh = 0; kh < kKH; ++kh)
#pragma unroll
      for (int j = 0; j < 16; ++j) sv[kh][j] = FP8 ? sc[kh][j] * km[2 * kh + (j >> 3)] : sc[kh][j];
    if ((kb + 1) * kKeys > Ew_full || bad) {
#pragma unroll
      for (int kh = 0; kh < kKH; ++kh)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int key = kb * kKeys + kTile * kh + 8 * (j >> 2) + 4 * hh + (j & 3);
          if (key >= lim[t] || s_bad[buf][2 * kh + (j >> 3)]) sv[kh][j] = neg_inf();
        }
    }
    float mx = neg_inf();
#pragma unroll
    for (int kh = 0; kh < kKH; ++kh) {
#pragma unroll
      for (int j = 0; j < 16; j += 2) mx = fmaxf(fmaxf(mx, sv[kh][j]), sv[kh][j + 1]);
    }
    mx = pair_max(mx);
    if constexpr (!FP8) mx *= km[0];
    // Lazy rescale: the reference maximum moves only when a score exceeds it by
    // more than 2^kRescaleLog2 (always when it is still -inf and a score is not).
    // A row whose keys are all masked so far keeps m = -inf and alpha = 1.
    const bool up = mx > m[t] + kRescaleLog2;
    if (__builtin_amdgcn_ballot_w64(up) != 0) {
      const float alpha = up ? __builtin_amdgcn_exp2f(m[t] - mx) : 1.f;
      l[t] *= alpha;
      m[t] = up ? mx : m[t];
#pragma unroll
      for (int c = 0; c < S::DT; ++c) acc[t][c] *= alpha;
    }
    const float mu = (m[t] == neg_inf()) ? 0.f : m[t];
    const float fk = FP8 ? 1.f : km[0];
#pragma unroll
    for (int kh = 0; kh < kKH; ++kh) {
      float pr[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        pr[j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[kh][j], fk, -mu));
        l[t] += pr[j];
      }
      // P^T operand of key step kk: K position 8h + e is key 16kk + 8(e/4) + 4h + e%4
      // of the key tile.
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const float v = vm[2 * kh + kk];
        const u32x4 w = {pack_bf16(pr[8 * kk] * v, pr[8 * kk + 1] * v), pack_bf16(pr[8 * kk + 2] * v, pr[8 * kk + 3] * v),
                         pack_bf16(pr[8 * kk + 4] * v, pr[8 * kk + 5] * v), pack_bf16(pr[8 * kk + 6] * v, pr[8 * kk + 7] * v)};
        pb[t][kh][kk] = __builtin_bit_cast(bf16x8, w);
      }
    }
  };
  // Operand reads.  K rows of block buffer `buf` for S^T = K Q^T: lane 32h + i
  // reads key i, elements [16s + 8h, 16s + 8h + 8).  V^T operands: the transpose read gives lane (16-lane group q, index c) the 4 keys
  // k0 .. k0+3 of column d = 16 (q & 1) + c of a 32-column tile, when lane c' of the
  // group addresses key k0 + c'/4, columns 4 (c' % 4) .. +3; operand kk*DT + t is
  // key step kk, column tile t.
  auto read_k = [&](bf16x8* ka, int buf, int kh) {
    const int R = kTile * kh + i;
    const char* kl = s_k[buf] + R * S::KRS;
#pragma unroll
    for (int s = 0; s < S::KS; ++s) {
      const int c = 2 * s + hh;
      ka[s] = *(const bf16x8*)(kl + 16 * (S::DMA ? chunk_pos(false, R, c) : c));
    }
  };
  const int lr = (lane & 15) >> 2, lc = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  auto read_v = [&](bf16x8* va, int buf, int kh) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int R = kTile * kh + 16 * kk + 4 * hh + lr;   // and R + 8: the same R & 3
      const char* vr = s_v[buf] + R * S::VRS;
#pragma unroll
      for (int t = 0; t < S::DT; ++t) {
        // column 32t + lc: chunk (32t + lc) / 8, byte 2 ((32t + lc) % 8) = 8 (lane & 1) in it
        const int c = 4 * t + (lc >> 3);
        const int off = S::DMA ? 16 * chunk_pos(true, R, c) + 8 * (lane & 1) : 2 * (32 * t + lc);
        const bf16x4 x0 = lds_tr_read(vr + off);
        const bf16x4 x1 = lds_tr_read(vr + 8 * S::VRS + off);
        va[kk * S::DT + t] = bf16x8{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
      }
    }
  };
  static_assert(S::KS == 2 * S::DT, "as many V^T operands as score k-steps");

  // Block kb in LDS buffer buf: scores, softmax, P V, for the wave's row tiles.
  auto compute_block = [&](int kb, int buf) {
    if (kb * kKeys < Ew) {
      // Each K and V operand read serves every row tile of the wave.
      f32x16 sc[kNT][kKH];
      bf16x8 va[kKH][S::KS];
#pragma unroll
      for (int kh = 0; kh < kKH; ++kh) {
        bf16x8 ka[S::KS];
        read_k(ka, buf, kh);
#pragma unroll
        for (int t = 0; t < kNT; ++t) sc[t][kh] = f32x16{};
#pragma unroll
        for (int s = 0; s < S::KS; ++s)
#pragma unroll
          for (int t = 0; t < kNT; ++t)
            sc[t][kh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[s], qop[t][s], sc[t][kh], 0, 0, 0);
      }
#pragma unroll
      for (int t = 0; t < kNT; ++t) softmax(t, kb, buf, sc[t]);
#pragma unroll
      for (int kh = 0; kh < kKH; ++kh) read_v(va[kh], buf, kh);
#pragma unroll
      for (int kh = 0; kh < kKH; ++kh)
#pragma unroll
        for (int s = 0; s < S::KS; ++s)
#pragma unroll
          for (int t = 0; t < kNT; ++t)
            acc[t][s % S::DT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[kh][s], pb[t][kh][s / S::DT],
                                                                        acc[t][s % S::DT], 0, 0, 0);
    }
  };

  // 3. Key blocks.
  if constexpr (S::DMA) {
    // Iteration kb starts the DMA of block kb + 2 into buffer (kb + 2) % 3 (read
    // last in iteration kb - 1), computes block kb, then waits until only block
    // kb + 2's DMAs are outstanding (block kb + 1 has landed) before the barrier.
    // Past the keys the DMAs read nothing, so every iteration issues the same count.
    constexpr int kDmaPerBlock = S::LPL * kKH;
    {
      int pid[kKH];
      page_ids(0, pid);
      dma_issue(0, 0, pid);
      page_ids(1, pid);
      dma_issue(1, 1, pid);
    }
    int pid_next[kKH];
    page_ids(2, pid_next);
    dma_barrier<kDmaPerBlock>();
    for (int kb0 = 0; kb0 < nkb; kb0 += 3) {
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const int kb = kb0 + u;
        if (kb < nkb) {
          dma_issue(kb + 2, (u + 2) % 3, pid_next);
          compute_block(kb, u);
          page_ids(kb + 3, pid_next);
          dma_barrier<kDmaPerBlock>();
        }
      }
    }
    if (bad_pages && lane == 0) atomicOr(p.flags, kFlagBadPage);
  } else {
    // Blocks 0 .. PD-1 are loaded before the loop, block 0 is written to LDS, and
    // iteration kb loads block kb + PD (past the wave's keys nothing is read, but
    // the loads are issued so that every iteration has the same loads in flight),
    // computes block kb and writes block kb + 1 to the other buffer.  The loop is
    // unrolled PD times so that each register set is fixed.
    {
      int pid[kKH];
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        page_ids(u, pid);
        stage_load(u, u, pid);
      }
    }
    int pid_next[kKH];
    page_ids(PD, pid_next);
    stage_write(0, 0);
    __syncthreads();
    for (int kb0 = 0; kb0 < nkb; kb0 += PD) {
#pragma unroll
      for (int u = 0; u < PD; ++u) {
        const int kb = kb0 + u;
        if (kb < nkb) {
          const int buf = kb & 1;
          stage_load(kb + PD, u, pid_next);
          compute_block(kb, buf);
          if (kb + 1 < nkb) stage_write((u + 1) % PD, buf ^ 1);
          // The next page ids are read here: a scalar load shares its completion
          // counter with the LDS reads, so issued earlier it would hold up the
          // first MFMA's operand wait; here the barrier's wait covers it.
          page_ids(kb + PD + 1, pid_next);
          __syncthreads();
        }
      }
    }
  }

  // 4. Normalise and write: lane 32h + i holds O^T[d = 32c + 8jj + 4h + 0..3][its row].
#pragma unroll
  for (int t = 0; t < kNT; ++t) {
    const float lt = pair_sum(l[t]);
    if (!live[t]) continue;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    const int64_t ob = ((int64_t)(q0 + qi[t]) * Hq + head[t]) * D;
#pragma unroll
    for (int c = 0; c < S::DT; ++c)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int d = 32 * c + 8 * jj + 4 * hh;
        const float o0 = acc[t][c][4 * jj] * inv, o1 = acc[t][c][4 * jj + 1] * inv;
        const float o2 = acc[t][c][4 * jj + 2] * inv, o3 = acc[t][c][4 * jj + 3] * inv;
        if (p.out_bf16)
          *(u32x2*)((uint16_t*)p.out + ob + d) = u32x2{pack_bf16(o0, o1), pack_bf16(o2, o3)};
        else
          *(f32x4*)((float*)p.out + ob + d) = f32x4{o0, o1, o2, o3};
      }
  }
}

template <int D, bool FP8>
int launch_multi_t(const Params& p, int grid, void* stream, void* ev_begin, void* ev_end) {
  hipStream_t st = (hipStream_t)stream;
  if (ev_begin && hipEventRecord((hipEvent_t)ev_begin, st) != hipSuccess) return -1;
  const size_t lds = (sizeof(int2) + sizeof(int32_t)) * (size_t)p.batch;
  hipLaunchKernelGGL((multi_query_kernel<D, FP8>), dim3(grid), dim3(kThreads), lds, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  if (ev_end && hipEventRecord((hipEvent_t)ev_end, st) != hipSuccess) return -1;
  return 0;
}

}  // namespace

int launch_multi(KvKind kind, int head_dim, const Params& p, int grid, void* stream, void* ev_begin, void* ev_end) {
  switch (kind) {
    case KvKind::BF16:
      return head_dim == 128 ? launch_multi_t<128, false>(p, grid, stream, ev_begin, ev_end)
                             : launch_multi_t<64, false>(p, grid, stream, ev_begin, ev_end);
    case KvKind::FP8:
      return head_dim == 128 ? launch_multi_t<128, true>(p, grid, stream, ev_begin, ev_end)
                             : launch_multi_t<64, true>(p, grid, stream, ev_begin, ev_end);
    case KvKind::F32:
      break;
  }
  return -1;
}

}  // namespace rlda
