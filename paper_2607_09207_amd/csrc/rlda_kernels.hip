// Decode attention over a paged KV cache for gfx950 (MI355X).
//
// One launch does the whole operation (the attention step the paper's rollout
// model charges through the history term H_dec and the per-token footprint b_kv,
// App. A.1.2):
//
//   1. Work plan.  Every workgroup scans seq_lens into page-count prefix sums in
//      LDS.  The work is the flattened list of (sequence, KV head, page) units,
//      priced one per page plus a fixed start cost per (sequence, KV head);
//      workgroup u owns the u-th of nranges equal-cost shares of it.  Long
//      sequences are therefore cut across many workgroups and short ones packed
//      together: every workgroup streams the same work however long the tail of
//      the length distribution is (Sec. 2.3 on long-tail decode).
//   2. Page gather.  Each of the 4 waves of a workgroup takes a quarter of the
//      share and walks it as one continuous stream of pages: its lanes decode 64
//      positions at a time (sequence, KV head, page id, valid tokens, segment
//      start/end flags) one chunk ahead of use, and the wave keeps 3 pages in
//      flight in registers with buffer loads whose range check returns zero past
//      a page's last valid token, so masked slots cost no memory traffic and
//      never yield NaN.  A segment's Q operand is loaded with its first page.
//      Segment boundaries inside the stream cost no pipeline restart.
//   3. Scores and softmax.  All G query heads that share the KV head are packed
//      into one 16-row MFMA tile: S^T = K Q^T with v_mfma_f32_16x16x32_bf16; the
//      online softmax keeps a running reference max and sum per head in log2
//      units, and moves the reference (rescaling the accumulator) only when a
//      score exceeds it by more than 8, i.e. a probability above 2^8.
//   4. PV.  O^T += V^T P^T with v_mfma_f32_16x16x16_bf16: the score tile's output
//      registers are already the P^T operand, and V's operand is assembled from
//      4 row loads per lane, so neither operand goes through LDS.
//   5. Merge.  A segment a wave covered whole is normalised and written by that
//      wave.  The cut pieces (at most 2 per wave) are merged through LDS.  A piece
//      of a segment that is split across workgroups stores its unnormalised
//      partial with device-scope (sc1) stores, which write through the XCD's L2;
//      after they complete, the workgroup bumps the segment's counter.  The
//      workgroup that completes the count reads every piece of the segment with
//      device-scope loads, merges them in piece order with log-sum-exp weights,
//      writes the output and resets the counter.  Each partial carries the
//      call's tag, so a merge that meets a piece this call did not publish (a
//      counter left non-zero in the workspace) raises a flag.  No workgroup waits
//      for another, and no device-scope fence (a whole-L2 writeback and
//      invalidate per XCD) is issued.
// fp8 (OCP E4M3FN) caches are converted exactly to bf16 for the MFMA; the K
// scale multiplies the scores and the V scale multiplies P.  fp32 caches use a
// VALU path.
// The same kernel serves multi-token rows (a few query rows per sequence, each
// masked at its causal position, up to two 16-row tiles per wave) and packed
// GRPO groups (the members of a group in the rows of one tile, the shared prompt
// pages streamed once per pack); see decode_attention_kernel.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "rlda_device.h"
#include "rlda_params.h"

// Flags, segment counters and partial slots of rl_decode_attn_run_noalloc, for
// callers that cannot allocate device memory (layout in rlda_params.h).  Each GPU
// the library runs on holds its own copy until the process ends.  In host code the
// name stands for a host-side handle, never a device address: the address comes
// from hipGetSymbolAddress (noalloc_scratch below).
static __device__ __align__(256) unsigned char scratch[rlda::kScratchBytes];

namespace rlda {
namespace {

#ifndef RLDA_MFMA_DEPTH
#define RLDA_MFMA_DEPTH 3                    // pages in flight per wave, MFMA path
#endif
#ifndef RLDA_MFMA_DEPTH_FP8
#define RLDA_MFMA_DEPTH_FP8 RLDA_MFMA_DEPTH  // ... with fp8 pages (half the bytes each)
#endif
constexpr int kChunk = 64;                   // page ids fetched per vector load

template <int BYTES>
struct RowLoad;
template <>
struct RowLoad<16> {
  typedef u32x4 type;
  template <int CP = kLoadNT>
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CP);
  }
};
template <>
struct RowLoad<8> {
  typedef u32x2 type;
  template <int CP = kLoadNT>
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, CP);
  }
};
template <>
struct RowLoad<4> {
  typedef uint32_t type;
  template <int CP = kLoadNT>
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, CP);
  }
};

__device__ __forceinline__ uint32_t word_of(u32x4 v, int i) { return v[i]; }
__device__ __forceinline__ uint32_t word_of(u32x2 v, int i) { return v[i]; }
__device__ __forceinline__ uint32_t word_of(uint32_t v, int) { return v; }

// Max / sum over the four 16-lane groups of a wave (lanes l, l^16, l^32, l^48).
__device__ __forceinline__ float group_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ __forceinline__ float group_sum(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}



// ---------------------------------------------------------------- helpers

__device__ __forceinline__ int64_t owner_of(int64_t x, int W, int64_t C) {
  // Largest u with floor(u*C/W) <= x: the share holding cost x.
  return ((x + 1) * (int64_t)W - 1) / C;
}

// Write N consecutive output elements o[0..N) * inv of row (b, qh) starting at d0.
template <int D, int N>
__device__ __forceinline__ void store_row(const Params& p, int b, int qh, int d0, const float* o, float inv) {
  const int64_t base = ((int64_t)b * p.num_q_heads + qh) * D + d0;
  if (p.out_bf16) {
    uint32_t* dst = (uint32_t*)((uint16_t*)p.out + base);
#pragma unroll
    for (int k = 0; k < N / 2; ++k) dst[k] = pack_bf16(o[2 * k] * inv, o[2 * k + 1] * inv);
  } else {
    float* dst = (float*)p.out + base;
#pragma unroll
    for (int k = 0; k < N; k += 4) *(f32x4*)(dst + k) = f32x4{o[k] * inv, o[k + 1] * inv, o[k + 2] * inv, o[k + 3] * inv};
  }
}
template <int D, int DPT = D / 16>
__device__ __forceinline__ void store_out(const Params& p, int b, int qh, int d0, const float* o, float inv) {
  store_row<D, DPT>(p, b, qh, d0, o, inv);
}

// Query heads of each KV head (a copy of Params::q_head, filled at kernel start):
// s_qhead[g * G + i] is the i-th query head of KV head g.
__shared__ int16_t s_qhead[kMaxQHeads];

// Partials of split segments live in the workspace: slot sl of query row h holds
// (m, l, call tag, 0) at part_ml[(sl*R + h)*4] and the unnormalised output at
// part_acc[(sl*R + h)*D ...], sl < 2*nranges, R = part_rows (G, or the rows of a
// multi-token segment).  They are written and read with the
// sc1 cache policy (device scope: write-through past the XCD's L2 and read from
// the coherent level), so workgroups on different XCDs exchange them without L2
// writeback or invalidate.
constexpr int kDeviceScope = 16;             // buffer cache-policy bit sc1
struct PartialRsrc {
  __amdgpu_buffer_rsrc_t acc, ml;
  template <int D>
  __device__ __forceinline__ static PartialRsrc of(const Params& p) {
    const uint32_t slots = 2u * (uint32_t)p.nranges * (uint32_t)p.part_rows;
    return {make_rsrc_uni(p.part_acc, slots * D * 4u), make_rsrc_uni(p.part_ml, slots * 16u)};
  }
};

// Online log-sum-exp merge of one partial (mj, lj, v[]) into (M, Ls, o[]).
template <int N>
__device__ __forceinline__ void lse_merge(float& M, float& Ls, float* o, float mj, float lj, const float* v) {
  if (mj == neg_inf()) return;
  const float Mn = fmaxf(M, mj);
  const float a_old = __builtin_amdgcn_exp2f(M - Mn), a_new = __builtin_amdgcn_exp2f(mj - Mn);
  Ls = Ls * a_old + lj * a_new;
#pragma unroll
  for (int e = 0; e < N; ++e) o[e] = o[e] * a_old + v[e] * a_new;
  M = Mn;
}

// Merge the pieces of segment (b, g) held by workgroups u_first..u_last: the piece
// of workgroup k is in slot 2k+1 when it continues past k's share, else in slot 2k.
// Loads are issued kBatch pieces at a time (one round trip per batch), then merged
// in piece order with a running maximum.  Thread (h, d0) merges its DPT outputs.
template <int D, int kBatch, int DPT>
__device__ __forceinline__ void merge_batches(const Params& p, const PartialRsrc& rs, int h, int d0, int64_t u_first,
                                              int64_t u_last, float& M, float& Ls, float* o) {
  const int G = p.part_rows;
  bool stale = false;
  for (int64_t k0 = u_first; k0 <= u_last; k0 += kBatch) {
    u32x4 ml[kBatch];
    float v[kBatch][DPT];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int64_t k = min(k0 + i, u_last);   // past the last piece: re-read it, unused
      const int sl = (int)((k < u_last) ? 2 * k + 1 : 2 * k);
      ml[i] = __builtin_amdgcn_raw_buffer_load_b128(rs.ml, (sl * G + h) * 16, 0, kDeviceScope);
#pragma unroll
      for (int c = 0; c < DPT; c += 4)
        *(u32x4*)&v[i][c] = __builtin_amdgcn_raw_buffer_load_b128(rs.acc, ((sl * G + h) * D + d0 + c) * 4, 0,
                                                                   kDeviceScope);
    }
#pragma unroll
    for (int i = 0; i < kBatch; ++i)
      if (k0 + i <= u_last) {
        stale |= ml[i][2] != p.call_tag;
        lse_merge<DPT>(M, Ls, o, __uint_as_float(ml[i][0]), __uint_as_float(ml[i][1]), v[i]);
      }
  }
  // A piece this call has not published: the segment's counter was not zero when the
  // call began (a workspace that was not zero-filled, or calls overlapping on it).
  if (__builtin_amdgcn_ballot_w64(stale) != 0 && (threadIdx.x & 63) == 0) atomicOr(p.flags, kFlagStaleState);
}

// A segment cut into many pieces (a long sequence over few workgroups' worth of
// other work) is merged 16 pieces per round trip (8 when a thread holds 16 outputs);
// the common 2-4 pieces, 4 at a time.
template <int D, int DPT = D / 16>
__device__ __forceinline__ void merge_pieces(const Params& p, int orow, int qh, int h, int d0, int64_t u_first,
                                             int64_t u_last) {
  const PartialRsrc rs = PartialRsrc::of<D>(p);
  float M = neg_inf(), Ls = 0.f, o[DPT];
#pragma unroll
  for (int e = 0; e < DPT; ++e) o[e] = 0.f;
  if (u_last - u_first >= 4)
    merge_batches<D, (DPT <= 8 ? 16 : 8), DPT>(p, rs, h, d0, u_first, u_last, M, Ls, o);
  else
    merge_batches<D, 4, DPT>(p, rs, h, d0, u_first, u_last, M, Ls, o);
  store_out<D, DPT>(p, orow, qh, d0, o, Ls > 0.f ? 1.f / Ls : 0.f);
}

// ---------------------------------------------------------------- MFMA policy
// Lane l = 16q + i (q = lane group 0..3, i = 0..15).
// K fragment: lane l holds row (token) i of the page, the 8-element chunks
//   bf16: chunk 4s+q for k-step s;  fp8: chunks 8(s/2)+2q+(s%2).
//   Each load instruction of the wave then covers one 64-byte sector per row.
// V fragment: lane l holds rows 4q..4q+3, elements [D/16*i, D/16*(i+1)).
// Score tile (D layout of 16x16 MFMA): lane l holds S[token 4q+r][head i].
// Output tile dt: lane l holds O[head i][d = D/16*(4q+r) + dt].
template <int D, bool FP8>
struct Mfma {
  static constexpr int kD = D;
  static constexpr bool kFp8 = FP8;
  static constexpr int KS = D / 32;                  // 16x16x32 k-steps for QK
  static constexpr int DT = D / 16;                  // output tiles = V elements per row per lane
  static constexpr int EB = FP8 ? 1 : 2;             // bytes per KV element
  static constexpr int kEB = EB;
  static constexpr int kDepth = FP8 ? RLDA_MFMA_DEPTH_FP8 : RLDA_MFMA_DEPTH;
  static constexpr int KL = FP8 ? D / 64 : D / 32;   // 16-byte K loads per lane
  static constexpr int VB = DT * EB;                 // V bytes per row per lane
  typedef typename RowLoad<VB>::type VRow;

  struct Frag {
    u32x4 k[KL];
    VRow v[4];
  };

  // Q operand of one (sequence, KV head): lane 16q+i holds head i's chunks for the k-steps.
  struct QOp {
    bf16x8 v[KS];
  };
  static constexpr bool kQRing = true;   // the Q operand travels with the pages in flight

  f32x4 acc[DT];
  float m, l;
  QOp q;
  int koff[KL], voff[4], qoff[KS];
  // Multi-token rows: how many tokens this lane's row sits before its segment's
  // last query token (keys at or past valid_tokens - shift of a page are masked).
  int shift = 0;

  __device__ __forceinline__ static int chunk_of(int qg, int s) {
    return FP8 ? 8 * (s >> 1) + 2 * qg + (s & 1) : 4 * s + qg;
  }

  __device__ __forceinline__ void setup(const Params& p, int lane, int32_t ss) {
    const int i = lane & 15, qg = lane >> 4;
#pragma unroll
    for (int s = 0; s < KL; ++s) koff[s] = i * ss + (FP8 ? 64 * s + 16 * qg : 16 * chunk_of(qg, s));
#pragma unroll
    for (int r = 0; r < 4; ++r) voff[r] = (4 * qg + r) * ss + i * VB;
    (void)p;
  }

  // Q rows of KV head g of sequence b, issued (when `load`) together with the
  // first page of the segment.  Padding rows (i >= G) read past the descriptor's
  // range and get zeros, so no instruction touches the loaded values before they
  // are consumed and the loads stay in flight with the page's.
  __device__ __forceinline__ static void load_q(QOp& qo, const Params& p, int b, int g, int lane, bool load) {
    if (!load) return;
    const int i = lane & 15, qg = lane >> 4;
    const int G = p.group;
    const uint16_t* qb = (const uint16_t*)p.q + (int64_t)b * p.num_q_heads * D;
    const __amdgpu_buffer_rsrc_t r = make_rsrc_uni(qb, load ? (uint32_t)(p.num_q_heads * D * 2) : 0u);
    const int row = (i < G) ? s_qhead[g * G + i] * D * 2 : kPastRange;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qo.v[s] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, row + 16 * chunk_of(qg, s), 0, 0));
  }

  // Q operand of a multi-token segment: tile row i is row rr = r0 + i of the
  // (sequence, KV head), query head (rr % G) of query row q0 + rr / G; rows at or
  // past n * G read zeros.
  __device__ __forceinline__ static void load_q_multi(QOp& qo, const Params& p, int q0, int n, int g, int r0, int lane,
                                                      bool load) {
    if (!load) return;
    const int i = lane & 15, qg = lane >> 4, G = p.group, rr = r0 + i;
    const __amdgpu_buffer_rsrc_t r =
        make_rsrc_uni(p.q, (uint32_t)p.total_q * (uint32_t)p.num_q_heads * D * 2u);
    const int row = (rr < n * G) ? ((q0 + rr / G) * p.num_q_heads + s_qhead[g * G + rr % G]) * D * 2 : kPastRange;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qo.v[s] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, row + 16 * chunk_of(qg, s), 0, 0));
  }

  // Q operand of the prompt pass: row r of the tile (lane group i = r) is query
  // head (row % G) of sequence b_first + row / G with row = row0 + r; rows at or
  // past `rows` read zeros.
  __device__ __forceinline__ static void load_q_rows(QOp& qo, const Params& p, int g, int b_first, int rows, int row0,
                                                     int lane) {
    const int i = lane & 15, qg = lane >> 4;
    const int G = p.group, row = row0 + i;
    const __amdgpu_buffer_rsrc_t r = make_rsrc_uni(p.q, (uint32_t)p.batch * (uint32_t)p.num_q_heads * D * 2u);
    int off = kPastRange;
    if (row < rows) {
      const int b = b_first + row / G, h = s_qhead[g * G + row % G];
      off = (b * p.num_q_heads + h) * D * 2;
    }
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qo.v[s] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, off + 16 * chunk_of(qg, s), 0, 0));
  }

  // Start accumulating a new (sequence, KV head) with its Q operand.
  __device__ __forceinline__ void begin(const QOp& qo, const Params&, int, int, int) {
#pragma unroll
    for (int t = 0; t < DT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    m = neg_inf();
    l = 0.f;
    q = qo;
  }

  // State of a grouped run's prompt pass for one (sequence, KV head), loaded with
  // the segment's first page: lane 16q + i gets O[head i][D/16*(4q+r) + t] for
  // r < 4, t < D/16, and (m, l) of head i.
  struct PInit {
    u32x4 a[DT];
    u32x2 ml;
  };
  __device__ __forceinline__ static void load_prompt(PInit& pi, const Params& p, int b, int g, int lane, bool load) {
    if (!load) return;
    const int i = lane & 15, qg = lane >> 4;
    const int G = p.group, Hq = p.num_q_heads;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc_uni(p.pfx_acc + (int64_t)b * Hq * D, (uint32_t)(Hq * D * 4));
    const __amdgpu_buffer_rsrc_t rm = make_rsrc_uni(p.pfx_ml + (int64_t)b * Hq * 2, (uint32_t)(Hq * 8));
    const int h = (i < G) ? s_qhead[g * G + i] : 0;
    const int orow = (i < G) ? h * D * 4 : kPastRange, mrow = (i < G) ? h * 8 : kPastRange;
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int c = 0; c < DT; c += 4)
        pi.a[r * (DT / 4) + c / 4] = __builtin_amdgcn_raw_buffer_load_b128(ra, orow + (DT * (4 * qg + r) + c) * 4, 0, 0);
    pi.ml = __builtin_amdgcn_raw_buffer_load_b64(rm, mrow, 0, 0);
  }

  // Start a segment from the prompt pass's state (the first piece of a grouped
  // sequence's remaining pages).  The lane-group partial sums of l add up to the
  // prompt's sum: lane group 0 carries it.
  __device__ __forceinline__ void begin_prompt(const QOp& qo, const PInit& pi, int G, int lane) {
    const int i = lane & 15, qg = lane >> 4;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[t][r] = __uint_as_float(pi.a[r * (DT / 4) + t / 4][t % 4]);
    m = (i < G) ? __uint_as_float(pi.ml[0]) : neg_inf();
    l = (i < G && qg == 0) ? __uint_as_float(pi.ml[1]) : 0.f;
    q = qo;
  }

  template <int CP = kLoadNT>
  __device__ __forceinline__ void issue(Frag& f, __amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv) const {
#pragma unroll
    for (int s = 0; s < KL; ++s) f.k[s] = RowLoad<16>::template load<CP>(rk, koff[s]);
#pragma unroll
    for (int r = 0; r < 4; ++r) f.v[r] = RowLoad<VB>::template load<CP>(rv, voff[r]);
  }

  __device__ __forceinline__ static bf16x8 k_operand(const Frag& f, int s) {
    if constexpr (!FP8) {
      return __builtin_bit_cast(bf16x8, f.k[s]);
    } else {
      const u32x4 w = f.k[s >> 1];
      const uint32_t lo = w[2 * (s & 1)], hi = w[2 * (s & 1) + 1];
      if constexpr (kFp8Direct) {   // fp8 pairs straight to bf16 pairs (unit scale: exact)
        u32x4 o = {fp8x2_to_bf16x2(lo, false), fp8x2_to_bf16x2(lo, true), fp8x2_to_bf16x2(hi, false),
                   fp8x2_to_bf16x2(hi, true)};
        return __builtin_bit_cast(bf16x8, o);
      }
      f32x2 a = __builtin_amdgcn_cvt_pk_f32_fp8(lo, false);
      f32x2 b = __builtin_amdgcn_cvt_pk_f32_fp8(lo, true);
      f32x2 c = __builtin_amdgcn_cvt_pk_f32_fp8(hi, false);
      f32x2 d = __builtin_amdgcn_cvt_pk_f32_fp8(hi, true);
      u32x4 o = {pack_bf16(a[0], a[1]), pack_bf16(b[0], b[1]), pack_bf16(c[0], c[1]), pack_bf16(d[0], d[1])};
      return __builtin_bit_cast(bf16x8, o);
    }
  }

  // V^T operands of a page for the 16x16x16 products, one per 16-wide output tile:
  // lane 16q + i supplies V[rows 4q..4q+3][column D/16*i + t] of tile t (fp8
  // converted exactly to bf16).  They depend on the page only, so the tiles of a
  // wave that holds two share them.
  struct VOp {
    s16x4 a[DT];
  };
  __device__ __forceinline__ static VOp v_operand(const Frag& f) {
    VOp vo;
    if constexpr (!FP8) {
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const uint32_t w0 = word_of(f.v[0], t >> 1), w1 = word_of(f.v[1], t >> 1);
        const uint32_t w2 = word_of(f.v[2], t >> 1), w3 = word_of(f.v[3], t >> 1);
        uint32_t lo, hi;
        if ((t & 1) == 0) {
          lo = (w0 & 0xFFFFu) | (w1 << 16);
          hi = (w2 & 0xFFFFu) | (w3 << 16);
        } else {
          lo = (w0 >> 16) | (w1 & 0xFFFF0000u);
          hi = (w2 >> 16) | (w3 & 0xFFFF0000u);
        }
        vo.a[t] = __builtin_bit_cast(s16x4, u32x2{lo, hi});
      }
    } else if constexpr (kFp8Direct) {
#pragma unroll
      for (int u = 0; u < DT / 2; ++u) {   // element pair (2u, 2u+1) of each row
        // Bytes (row 0, row 1) of elements 2u and 2u+1 in one word, then each pair to
        // bf16: word 0 of the operands of tiles 2u and 2u+1; rows 2, 3 give word 1.
        const int sh = (u & 1) * 16;
        const uint32_t w0 = word_of(f.v[0], u >> 1) >> sh, w1 = word_of(f.v[1], u >> 1) >> sh;
        const uint32_t w2 = word_of(f.v[2], u >> 1) >> sh, w3 = word_of(f.v[3], u >> 1) >> sh;
        const uint32_t x01 = __builtin_amdgcn_perm(w1, w0, 0x05010400u);   // r0e0 r1e0 r0e1 r1e1
        const uint32_t x23 = __builtin_amdgcn_perm(w3, w2, 0x05010400u);
        vo.a[2 * u] = __builtin_bit_cast(s16x4, u32x2{fp8x2_to_bf16x2(x01, false), fp8x2_to_bf16x2(x23, false)});
        vo.a[2 * u + 1] = __builtin_bit_cast(s16x4, u32x2{fp8x2_to_bf16x2(x01, true), fp8x2_to_bf16x2(x23, true)});
      }
    } else {
#pragma unroll
      for (int u = 0; u < DT / 2; ++u) {   // element pair (2u, 2u+1) of each row
        f32x2 c[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) c[r] = fp8x2_to_f32(word_of(f.v[r], u >> 1), (u & 1) != 0);
#pragma unroll
        for (int e = 0; e < 2; ++e)
          vo.a[2 * u + e] = __builtin_bit_cast(s16x4, u32x2{pack_bf16(c[0][e], c[1][e]), pack_bf16(c[2][e], c[3][e])});
      }
    }
    return vo;
  }

  // Page with index `j` in its sequence; `valid_tokens` tokens of it count (for
  // multi-token rows: tokens of the page and after it, up to 31, less `shift`).
  template <bool MULTI = false>
  __device__ __forceinline__ void compute(const Frag& f, int lane, int valid_tokens, float kmul, float vmul) {
    compute_with<MULTI>(f, nullptr, lane, valid_tokens, kmul, vmul);
  }
  // ... with the page's V operands built once by the caller (vo), or here (null).
  template <bool MULTI = false>
  __device__ __forceinline__ void compute_with(const Frag& f, const VOp* vo, int lane, int valid_tokens, float kmul,
                                               float vmul) {
    const int qg = lane >> 4;
    f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k_operand(f, s), q.v[s], sc, 0, 0, 0);
    float sv[4];
    float mx = neg_inf();
    const int vt = MULTI ? valid_tokens - shift : valid_tokens;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      sv[r] = (4 * qg + r < vt) ? sc[r] * kmul : neg_inf();
      mx = fmaxf(mx, sv[r]);
    }
    mx = group_max(mx);
    // The reference maximum m only moves when a score exceeds it by more than
    // 2^kRescaleLog2: probabilities stay <= 2^kRescaleLog2 (exact in fp32, the
    // same relative rounding in bf16), and the accumulator rescale, which reads
    // and writes every accumulator register, is skipped on almost every page.
    const bool up = mx > m + kRescaleLog2;   // always when m is still -inf and mx is not
    if (__builtin_amdgcn_ballot_w64(up) != 0)
    {
      // Multi-token rows: a row whose keys are all masked so far keeps m = -inf
      // while other rows move, so alpha comes from `up` (1 otherwise).
      const float mn = up ? mx : m;
      const float alpha = MULTI ? (up ? __builtin_amdgcn_exp2f(m - mx) : 1.f)
                                : __builtin_amdgcn_exp2f(m - mn);   // 0 from -inf, 1 when unchanged
      l *= alpha;
      m = mn;
#pragma unroll
      for (int t = 0; t < DT; ++t) acc[t] *= alpha;
    }
    const float mu = (m == neg_inf()) ? 0.f : m;
    float pr[4];
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      pr[r] = __builtin_amdgcn_exp2f(sv[r] - mu);
      ps += pr[r];
    }
    l += ps;
    u32x2 pb2 = {pack_bf16(pr[0] * vmul, pr[1] * vmul), pack_bf16(pr[2] * vmul, pr[3] * vmul)};
    const s16x4 pb = __builtin_bit_cast(s16x4, pb2);
    const VOp v = vo ? *vo : v_operand(f);
#pragma unroll
    for (int t = 0; t < DT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(v.a[t], pb, acc[t], 0, 0, 0);
  }

  // Write this wave's state in canonical [head][d] form to LDS.
  __device__ __forceinline__ void to_lds(float (*sacc)[D + 4], float (*sml)[2], int lane) {
    const int i = lane & 15, qg = lane >> 4;
    const float lt = group_sum(l);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float* dst = &sacc[i][DT * (4 * qg + r)];
#pragma unroll
      for (int t = 0; t < DT; ++t) dst[t] = acc[t][r];
    }
    if (qg == 0) {
      sml[i][0] = m;
      sml[i][1] = lt;
    }
  }

  // A multi-token segment this wave covered entirely: tile row i is row
  // rr = r0 + i < n * G, output row q0 + rr / G, query head (rr % G) of KV head g.
  __device__ __forceinline__ void write_out_multi(const Params& p, int q0, int n, int g, int r0, int lane) const {
    const int i = lane & 15, qg = lane >> 4, G = p.group, rr = r0 + i;
    const float lt = group_sum(l);
    if (rr >= n * G) return;
    float o[4 * DT];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int t = 0; t < DT; ++t) o[r * DT + t] = acc[t][r];
    store_row<D, 4 * DT>(p, q0 + rr / G, s_qhead[g * G + rr % G], 4 * DT * qg, o, lt > 0.f ? 1.f / lt : 0.f);
  }

  // A piece this wave covered entirely: normalise and write its rows.
  __device__ __forceinline__ void write_out(const Params& p, int b, int g, int lane) const {
    const int i = lane & 15, qg = lane >> 4;
    const float lt = group_sum(l);
    if (i >= p.group) return;
    float o[4 * DT];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int t = 0; t < DT; ++t) o[r * DT + t] = acc[t][r];
    store_row<D, 4 * DT>(p, b, s_qhead[g * p.group + i], 4 * DT * qg, o, lt > 0.f ? 1.f / lt : 0.f);
  }
};

// ---------------------------------------------------------------- VALU policy (fp32 KV)
// Lane l = 4t + c: token slot t (0..15) of the page, chunk c (0..3) of D/4 values.
template <int D, int GM>
struct Valu {
  static constexpr int kD = D;
  static constexpr bool kFp8 = false;
  static constexpr int kEB = 4;
  static constexpr int kDepth = 2;
  static constexpr int CW = D / 4;
  static constexpr int NL = CW / 4;
  struct Frag {
    u32x4 k[NL];
    u32x4 v[NL];
  };
  struct QOp {};
  static constexpr bool kQRing = false;   // q is loaded when a segment begins
  struct PInit {};                        // grouped runs are not supported with fp32 caches

  float acc[GM][CW];
  float qv[GM][CW];
  float m[GM], l[GM];
  int off;

  __device__ __forceinline__ void setup(const Params&, int lane, int32_t ss) {
    off = (lane >> 2) * ss + (lane & 3) * CW * 4;
  }

  __device__ __forceinline__ static void load_q(QOp&, const Params&, int, int, int, bool) {}
  __device__ __forceinline__ static void load_prompt(PInit&, const Params&, int, int, int, bool) {}

  __device__ __forceinline__ void begin(const QOp&, const Params& p, int b, int g, int lane) {
    const int c = lane & 3;
    const int G = p.group;
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      m[h] = neg_inf();
      l[h] = 0.f;
      const float* qb = nullptr;
      if (h < G) qb = (const float*)p.q + ((int64_t)b * p.num_q_heads + s_qhead[g * G + h]) * D + c * CW;
#pragma unroll
      for (int j = 0; j < CW; ++j) {
        acc[h][j] = 0.f;
        qv[h][j] = qb ? qb[j] : 0.f;
      }
    }
  }

  __device__ __forceinline__ void issue(Frag& f, __amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv) const {
#pragma unroll
    for (int s = 0; s < NL; ++s) f.k[s] = RowLoad<16>::load(rk, off + 16 * s);
#pragma unroll
    for (int s = 0; s < NL; ++s) f.v[s] = RowLoad<16>::load(rv, off + 16 * s);
  }

  __device__ __forceinline__ void compute(const Frag& f, int lane, int valid_tokens, float kmul, float) {
    const int t = lane >> 2;
    const bool valid = t < valid_tokens;
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < CW; ++j) s += qv[h][j] * __uint_as_float(f.k[j >> 2][j & 3]);
      s += __shfl_xor(s, 1);
      s += __shfl_xor(s, 2);
      s = valid ? s * kmul : neg_inf();
      float mx = s;
#pragma unroll
      for (int o = 4; o < 64; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      const float mn = fmaxf(m[h], mx);
      const float mu = (mn == neg_inf()) ? 0.f : mn;
      const float alpha = __builtin_amdgcn_exp2f(m[h] - mu);
      const float pr = __builtin_amdgcn_exp2f(s - mu);
      l[h] = l[h] * alpha + pr;
      m[h] = mn;
#pragma unroll
      for (int j = 0; j < CW; ++j) acc[h][j] = acc[h][j] * alpha + pr * __uint_as_float(f.v[j >> 2][j & 3]);
    }
  }

  // Sum the per-token-slot partial sums over the 16 token slots (lanes 4t + c).
  __device__ __forceinline__ void reduce_tokens(float* lt) {
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      float a = l[h];
#pragma unroll
      for (int o = 4; o < 64; o <<= 1) a += __shfl_xor(a, o);
      lt[h] = a;
#pragma unroll
      for (int j = 0; j < CW; ++j) {
        float v = acc[h][j];
#pragma unroll
        for (int o = 4; o < 64; o <<= 1) v += __shfl_xor(v, o);
        acc[h][j] = v;
      }
    }
  }

  __device__ __forceinline__ void to_lds(float (*sacc)[D + 4], float (*sml)[2], int lane) {
    const int c = lane & 3;
    float lt[GM];
    reduce_tokens(lt);
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      if (lane < 4) {
#pragma unroll
        for (int j = 0; j < CW; ++j) sacc[h][c * CW + j] = acc[h][j];
      }
      if (lane == 0) {
        sml[h][0] = m[h];
        sml[h][1] = lt[h];
      }
    }
  }

  __device__ __forceinline__ void write_out(const Params& p, int b, int g, int lane) {
    const int c = lane & 3;
    float lt[GM];
    reduce_tokens(lt);
    if (lane >= 4) return;
#pragma unroll
    for (int h = 0; h < GM; ++h)
      if (h < p.group) store_row<D, CW>(p, b, s_qhead[g * p.group + h], c * CW, acc[h], lt[h] > 0.f ? 1.f / lt[h] : 0.f);
  }
};

// ---------------------------------------------------------------- stream metadata
// A wave walks its quarter [w0, w1) of the flattened (sequence, KV head, page) list
// as one continuous page stream.  Its lanes describe 64 consecutive positions at a
// time (lane k: position base + k), fetched one chunk ahead of use; the page ring
// runs on across chunks.
constexpr int kInfoTok = 31;            // valid tokens of the page (0: nothing to read)
constexpr int kInfoFirst = 1 << 5;      // first page of its (sequence, KV head)
constexpr int kInfoLast = 1 << 6;       // last page of its (sequence, KV head)
constexpr int kInfoStart = 1 << 7;      // first position of this wave's quarter
constexpr int kInfoEnd = 1 << 8;        // last position of this wave's quarter
constexpr int kInfoHeadShift = 9;       // KV head g: 8 bits
constexpr int kInfoSeqShift = 17;       // sequence b: 13 bits (b < 8192)
constexpr int kInfoPrompt = 1 << 30;    // grouped run: the sequence's prompt pass state seeds its first page
constexpr int kInfoChunkShift = 30;     // multi-token run: the segment's 16-row chunk (2 bits)
constexpr int kInfoActShift = 29;       // packed grouped run: the pack member whose rows the page serves (3 bits;
constexpr int kActAll = 7;              // kActAll: a prompt page, every member's rows); the pack index has 12 bits

// The page id is returned as read; it is checked where it is used, so that
// nothing waits for these loads until the chunk is consumed.
struct StreamChunk {
  int pid;      // page id from the block table (lanes past the quarter: -1)
  int info;     // bits above
};

// Positions fit in 32 bits: the host rejects max_batch * max_pages * Hkv (times
// the row chunks of a multi-token run) >= 2^31.
// Multi-token runs report, instead of a page's valid tokens, the tokens from the
// page's start to the sequence's end (up to 31), which the rows' causal masks
// need, and split a (sequence, KV head) with more than 16 rows into nrc segments
// of 16 rows that each stream the pages: segment gv = g * nrc + rc of a sequence,
// Hs = Hkv * nrc segments per sequence.
// Packed grouped runs: a unit is a pack of consecutive members of one GRPO group;
// its segment streams the group's prompt pages once (every member's rows take
// part), then each member's own pages in member order (only that member's rows).
template <bool MULTI, bool PACK>
__device__ __forceinline__ StreamChunk fetch_chunk(const Params& p, const int32_t* s_pre, const uint8_t* s_tail,
                                                   const int32_t* s_ppre, const uint16_t* s_nfull,
                                                   const int16_t* s_gpp, int nunits, int base, int w0, int w1,
                                                   int lane, int Hs, int nrc, int hint) {
  StreamChunk c = {-1, 0};
  const int pos = base + lane;
  if (pos < w1) {
    const int y = (int)((uint32_t)pos / (uint32_t)Hs);
    // `hint` is the unit of a position at or before `base`, so s_pre[hint] <= y.  A
    // chunk spans few units: gallop from it, then bisect.
    int lo = hint, hi = min(nunits, hint + 1);
    for (int step = 2; hi < nunits && s_pre[hi] <= y; step <<= 1) {
      lo = hi;
      hi = min(nunits, lo + step);
    }
    while (hi - lo > 1) {   // s_pre[lo] <= y < s_pre[hi]
      const int mid = (lo + hi) >> 1;
      if (s_pre[mid] <= y) lo = mid; else hi = mid;
    }
    const int b = lo, pre = s_pre[b], nb = s_pre[b + 1] - pre;
    const int off = pos - Hs * pre;
    const int gv = (int)((uint32_t)off / (uint32_t)nb), j = off - gv * nb;
    const int g = MULTI ? (int)((uint32_t)gv / (uint32_t)nrc) : gv;
    const int flags = (j == 0 ? kInfoFirst : 0) | (j == nb - 1 ? kInfoLast : 0) | (pos == w0 ? kInfoStart : 0) |
                      (pos == w1 - 1 ? kInfoEnd : 0) | (g << kInfoHeadShift) | (b << kInfoSeqShift);
    if constexpr (PACK) {
      const int b0 = s_ppre[b] >> 5, np = s_ppre[b] & 31, gs = p.group_size;
      const int grp = b0 / gs, pp = s_gpp[grp];
      int row, page, tok, act;
      if (j < pp) {   // a prompt page: the group's first sequence names it
        row = grp * gs;
        page = j;
        tok = kPage;
        act = kActAll;
      } else {
        int jj = j - pp, m = 0;
        while (m < np - 1) {
          const int t = s_nfull[b0 + m] - pp;
          if (jj < t) break;
          jj -= t;
          ++m;
        }
        row = b0 + m;
        page = pp + jj;
        tok = (page == s_nfull[row] - 1) ? s_tail[row] : kPage;
        act = m;
      }
      c.pid = p.block_table[(int64_t)row * p.max_pages + page];
      c.info = tok | flags | (act << kInfoActShift);
      return c;
    }
    const int tok = (j == nb - 1) ? s_tail[b] : (MULTI ? (j == nb - 2 ? min(kPage + s_tail[b], 31) : 31) : kPage);
    const int pp = MULTI ? 0 : s_ppre[b];   // prompt pages handled by the prompt pass (grouped runs)
    c.pid = p.block_table[(int64_t)b * p.max_pages + pp + j];
    c.info = tok | flags | (MULTI ? (gv - g * nrc) << kInfoChunkShift : (pp > 0 ? kInfoPrompt : 0));
  }
  return c;
}

// ---------------------------------------------------------------- the kernel

#ifndef RLDA_PROMPT_TEMPORAL
#define RLDA_PROMPT_TEMPORAL 1
#endif
constexpr bool kPromptTemporal = RLDA_PROMPT_TEMPORAL;

// The prompt-pass state a grouped run's segment may start from (section 7b of the
// attention kernel's users): only the launch that follows a prompt pass carries it.
struct NoPromptState {};
template <class Pol, bool PROMPT>
struct PromptState {
  typedef typename Pol::PInit type;
};
template <class Pol>
struct PromptState<Pol, false> {
  typedef NoPromptState type;
};

// MULTI: multi-token rows (rl_decode_attn_run_multi with at most 16 NT row_chunks
// rows per (sequence, KV head)): (b, g) has n_b * G rows, row r is query head
// (r % G) of query row q_start[b] + r / G and sees keys below L - n_b + r / G + 1;
// its rows are streamed as row_chunks segments of 16 NT rows, NT tiles of 16 rows
// per wave against each page.
// PACK (with MULTI): grouped runs with the members of a GRPO group packed into
// the rows of the tiles.  The units are packs instead of sequences; row r of a
// pack is query head (r % G) of member r / G, and a page counts for every row (a
// prompt page) or for one member's rows (its own pages).
// PROMPT: the attention launch of a grouped run's prompt-pass form; a sequence's
// first page then starts from the prompt pass's state.  Other launches carry no
// prompt state (about 100 registers fewer).
// WPE: waves per SIMD.  2: two workgroups per CU (batch <= kTwoWgMaxBatch, whose
// per-sequence LDS tables leave room for two), each wave within 256 registers.
template <class Pol, bool MULTI = false, int NT = 1, bool PACK = false, bool PROMPT = false, int WPE = 1>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads), amdgpu_waves_per_eu(WPE, WPE)))
void decode_attention_kernel(const Params p) {
  static_assert(NT == 1 || (MULTI && NT == 2), "two row tiles only for multi-token rows");
  static_assert(!PACK || MULTI, "packed grouped runs use the multi-token row machinery");
  static_assert(!(PACK && NT == 2), "packed grouped runs hold one tile");
  constexpr int D = Pol::kD;
  // Workgroup merge: kMR rows per slot (both tiles of a two-tile segment), kTPR
  // threads per row, DPT output elements per thread.
  constexpr int kMR = 16 * NT, kTPR = kThreads / kMR;
  constexpr int DPT = D / kTPR;
  static_assert(!(PROMPT && (MULTI || PACK)), "the prompt-pass state belongs to plain grouped launches");
  static_assert(WPE == 1 || (WPE == 2 && !MULTI && !PACK && !PROMPT), "two waves per SIMD: plain runs only");
  constexpr int kB = WPE == 2 ? kTwoWgMaxBatch : PACK ? kPackMaxBatch : (NT == 2 ? kTwoTileMaxBatch : kMaxBatch);
  // Units: sequences, or packs of group members (packed grouped runs).
  __shared__ int32_t s_pre[kB + 1];
  __shared__ uint8_t s_tail[kB];   // valid tokens of each sequence's last page
  // Grouped runs: leading pages covered by the prompt pass.  Multi-token runs:
  // (q_start[b] << 5) | n_b.  Packed grouped runs: (first member << 5) | members.
  __shared__ int32_t s_ppre[kB];
  // Packed grouped runs: pages of each sequence, and the clamped prompt pages of each group.
  __shared__ uint16_t s_nfull[PACK ? kB : 1];
  __shared__ int16_t s_gpp[PACK ? kB : 1];
  // Cut pieces: slot 2w holds wave w's piece that began before its quarter of the
  // share, slot 2w+1 its piece that continues past it.
  __shared__ __align__(16) float s_acc[2 * kWaves][kMR][D + 4];
  __shared__ __align__(16) float s_ml[2 * kWaves][kMR][2];
  // Non-empty units before each unit (the work split prices every segment's start).
  __shared__ uint16_t s_ne[kB + 1];
  __shared__ int32_t s_seg[2 * kWaves];
  __shared__ int32_t s_scan[kWaves], s_scan_ne[kWaves];
  __shared__ int32_t s_last[2];

  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  // The query-head map (kernel argument memory), loaded alongside the lengths.
  static_assert(kMaxQHeads <= kThreads, "one query head per thread");
  const int16_t qh0 = tid < p.num_q_heads ? p.q_head[tid] : (int16_t)0;
  const int W = p.nranges;
  // Share index.  Workgroups are dispatched round-robin over the 8 XCDs (block b
  // runs on XCD b % 8); each XCD gets a contiguous run of shares, so neighbouring
  // work (the sequences of a GRPO group reading the same prompt pages, the pieces
  // of one split segment) shares one L2.  A bijection of [0, W).
  const int u = [&] {
    const int b = blockIdx.x, x = b & 7, i = b >> 3, q = W >> 3, r = W & 7;
    return x * q + min(x, r) + i;
  }();
  const int batch = p.batch, Hkv = p.num_kv_heads, G = p.group;
  const int cap = p.max_pages * kPage;
  // Multi-token runs: nrc segments of 16 NT rows per (sequence, KV head), Hs per
  // sequence; a wave holds NT 16-row tiles against each page of a segment.
  // (Packed grouped runs have one row chunk: a pack's rows fit one segment.)
  const int nrc = (MULTI && !PACK) ? p.row_chunks : 1, Hs = Hkv * nrc;
  // Packed grouped runs: the pack member that each of this lane's tile rows belongs to.
  const int rmem = PACK ? (lane & 15) / G : 0, rmem2 = (PACK && NT == 2) ? (16 + (lane & 15)) / G : 0;
  constexpr int kSegRows = 16 * NT;
  // The 16 NT-row chunk of its (sequence, KV head) that a page's segment covers.
  auto chunk_of_info = [](int info) { return PACK ? 0 : (info >> kInfoChunkShift) & 3; };

  // Units of the flattened list: sequences, or packs (packed grouped runs).
  const int nunits = PACK ? p.pack_units : batch;
  // Packed grouped runs whose groups are aligned runs of the lanes (a power-of-two
  // group size up to 64 dividing the batch, a power-of-two pack size dividing it,
  // at most one sequence per thread): the group clamps and the pack sums are
  // shuffles across the members' lanes, so the prologue needs one barrier before
  // the scan instead of three.  Other shapes take the general prologue below.
  bool pack_lanes = false;
  if constexpr (PACK) {
    const int gs = p.group_size, P = p.pack;
    pack_lanes = batch <= kThreads && gs <= 64 && (gs & (gs - 1)) == 0 && P >= 1 && (P & (P - 1)) == 0 && P <= gs &&
                 batch % gs == 0 && nunits * P == batch;
  }
  if (PACK && pack_lanes) {
    const int gs = p.group_size, P = p.pack, b = tid;
    const bool live = b < batch;
    int L = live ? p.seq_lens[b] : 0;
    const int want = live ? p.prefix_pages[b / gs] : 0;
    const bool badl = live && (L < 0 || L > cap);
    L = min(max(L, 0), cap);
    const int nf = (L + kPage - 1) / kPage, tail = L - (nf - 1) * kPage;
    // The group's prompt: the requested pages clamped to its shortest member's full pages.
    int mn = live ? ((nf > 0 && tail < kPage) ? nf - 1 : nf) : 0x7fffffff;
    for (int o = 1; o < gs; o <<= 1) mn = min(mn, __shfl_xor(mn, o));
    const int pp = max(0, min(want, mn));
    // Pack b / P: the prompt once, then each member's own pages.
    int own = live ? nf - pp : 0;
    for (int o = 1; o < P; o <<= 1) own += __shfl_xor(own, o);
    const bool head = live && (b & (P - 1)) == 0;   // the lane of the pack's first member
    const int n = head ? pp + own : 0;
    if (live) {
      s_nfull[b] = (uint16_t)nf;
      s_tail[b] = (uint8_t)tail;
      if ((b & (gs - 1)) == 0) s_gpp[b / gs] = (int16_t)pp;
    }
    if (head) s_ppre[b / P] = (b << 5) | P;
    if (__builtin_amdgcn_ballot_w64(badl) != 0 && lane == 0 && u == 0) atomicOr(p.flags, kFlagBadLen);
    if (__builtin_amdgcn_ballot_w64(live && (b & (gs - 1)) == 0 && want != pp) != 0 && lane == 0 && u == 0)
      atomicOr(p.flags, kFlagPrefixClamped);
    // Prefix sums of the packs' pages and of the non-empty packs, in pack order
    // (= lane order of the packs' first members).
    int x = n, xn = n > 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o), yn = __shfl_up(xn, o);
      if (lane >= o) {
        x += y;
        xn += yn;
      }
    }
    if (lane == 63) {
      s_scan[wave] = x;
      s_scan_ne[wave] = xn;
    }
    if (tid < p.num_q_heads) s_qhead[tid] = qh0;
    if (tid < 2 * kWaves) s_seg[tid] = -1;
    __syncthreads();
    int run = x, rne = xn;   // inclusive
    for (int w = 0; w < wave; ++w) {
      run += s_scan[w];
      rne += s_scan_ne[w];
    }
    if (head) {
      s_ne[b / P] = (uint16_t)(rne - (n > 0));
      s_pre[b / P + 1] = run;
    }
    if (tid == kThreads - 1) s_ne[nunits] = (uint16_t)rne;
    if (tid == 0) {
      s_pre[0] = 0;
      s_ne[0] = 0;
    }
    __syncthreads();
  } else {
    if constexpr (PACK) {
      // Pages and last-page tokens of every sequence, then each group's prompt pages:
      // the requested count clamped to the full pages of its shortest member.  The
      // first requested counts are loaded together with the lengths.
      const int gs = p.group_size, ngroups = (batch + gs - 1) / gs;
      const int want0 = tid < ngroups ? p.prefix_pages[tid] : 0;
      int bad = 0;
      for (int b = tid; b < batch; b += kThreads) {
        int L = p.seq_lens[b];
        if (L < 0 || L > cap) bad = 1;
        L = min(max(L, 0), cap);
        const int nf = (L + kPage - 1) / kPage;
        s_nfull[b] = (uint16_t)nf;
        s_tail[b] = (uint8_t)(L - (nf - 1) * kPage);
      }
      if (bad && u == 0) atomicOr(p.flags, kFlagBadLen);
      __syncthreads();
      for (int i = tid; i < ngroups; i += kThreads) {
        int mn = 0x7fffffff;
        for (int b = i * gs; b < min(batch, (i + 1) * gs); ++b) {
          const int nf = s_nfull[b];
          mn = min(mn, (nf > 0 && s_tail[b] < kPage) ? nf - 1 : nf);   // full pages
        }
        const int want = i == tid ? want0 : p.prefix_pages[i], pp = max(0, min(want, mn));
        if (want != pp && u == 0) atomicOr(p.flags, kFlagPrefixClamped);
        s_gpp[i] = (int16_t)pp;
      }
      __syncthreads();
    }

    // 1. Page counts per unit and their prefix sums (identical in every workgroup).
    {
      const int per = (nunits + kThreads - 1) / kThreads;
      const int lo = min(tid * per, nunits), hi = min(lo + per, nunits);
      int sum = 0, cnt = 0, bad = 0;   // pages, non-empty units
      for (int b = lo; b < hi; ++b) {
        if constexpr (PACK) {
          // Pack b: members b0 .. b0 + np - 1 of group i; the prompt once, then each member's own pages.
          const int gs = p.group_size, P = p.pack, ppg = (gs + P - 1) / P;
          const int i = b / ppg, r = b - i * ppg;
          const int b0 = i * gs + r * P, np = min(P, min(batch, (i + 1) * gs) - b0);
          const int pp = s_gpp[i];
          int n = pp;
          for (int m = 0; m < np; ++m) n += s_nfull[b0 + m] - pp;
          s_ppre[b] = (b0 << 5) | np;
          s_pre[b + 1] = n;
          sum += n;
          cnt += n > 0;
          continue;
        }
        int L = p.seq_lens[b];
        if (L < 0 || L > cap) bad = 1;
        L = min(max(L, 0), cap);
        int nfull = (L + kPage - 1) / kPage;
        int pp = 0;
        if constexpr (MULTI) {
          // Inconsistent offsets, or more rows than the call allows: no rows.  More
          // rows than tokens: flagged; rows before position 0 see no key (zeros).
          const int q0 = p.q_start[b], q1 = p.q_start[b + 1];
          int nq = q1 - q0;
          if (q0 < 0 || q1 < q0 || q1 > p.total_q || nq > p.max_q_len) {
            bad = 1;
            nq = 0;
          }
          if (nq > L) bad = 1;
          if (nq == 0) nfull = 0;
          s_ppre[b] = nq > 0 ? (q0 << 5) | nq : 0;
        } else {
          // Grouped runs: the prompt pass covered the first pp pages (its clamp keeps
          // pp <= floor(L / 16)); this kernel streams the rest.
          pp = p.group_size > 0 ? min(max(p.gprefix[b / p.group_size], 0), L / kPage) : 0;
          s_ppre[b] = pp;
        }
        const int n = nfull - pp;
        s_pre[b + 1] = n;
        s_tail[b] = (uint8_t)(L - (nfull - 1) * kPage);   // 1..16 when nfull > 0
        sum += n;
        cnt += n > 0;
      }
      if (bad && u == 0) atomicOr(p.flags, kFlagBadLen);
      int x = sum, xn = cnt;
  #pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o), yn = __shfl_up(xn, o);
        if (lane >= o) {
          x += y;
          xn += yn;
        }
      }
      if (lane == 63) {
        s_scan[wave] = x;
        s_scan_ne[wave] = xn;
      }
      if (tid < p.num_q_heads) s_qhead[tid] = qh0;
      if (tid < 2 * kWaves) s_seg[tid] = -1;
      __syncthreads();
      int run = x - sum, rne = xn - cnt;
      for (int w = 0; w < wave; ++w) {
        run += s_scan[w];
        rne += s_scan_ne[w];
      }
      for (int b = lo; b < hi; ++b) {
        const int n = s_pre[b + 1];
        s_ne[b] = (uint16_t)rne;
        rne += n > 0;
        run += n;
        s_pre[b + 1] = run;
      }
      if (tid == kThreads - 1) s_ne[nunits] = (uint16_t)rne;   // the last thread's range ends at nunits
      if (tid == 0) {
        s_pre[0] = 0;
        s_ne[0] = 0;
      }
      __syncthreads();
    }
  }
  const int64_t T = uni64((int64_t)s_pre[nunits] * Hs);
  // Cost of the flattened list: one per position, and kStartCost more per segment
  // of a non-empty unit for its start (loading Q, opening and closing the state
  // cost about a page's time on the stream).  Unit b's segments begin at cost
  // K(b) = Hs (s_pre[b] + S s_ne[b]), each nb + S long: its start, then its pages.
  constexpr int S = kStartCost;
  const int64_t C = uni64((int64_t)Hs * (s_pre[nunits] + S * s_ne[nunits]));
  auto cost_of = [&](int64_t pos, int b, int gv) { return pos + (int64_t)S * (Hs * s_ne[b] + gv + 1); };

  // 2. Sequences with no pages left to stream: zero rows, or (grouped runs) the
  //    normalised prompt-pass result when the prompt is the whole sequence.
  for (int b = u; b < nunits; b += W) {
    if (s_pre[b + 1] != s_pre[b]) continue;
    if constexpr (MULTI) {
      // Rows of a sequence with no keys (none, or rows claimed past an empty cache).
      const int nq = s_ppre[b] & 31, q0 = s_ppre[b] >> 5;
      const int n = nq * p.num_q_heads * D;
      for (int e = tid; e < n; e += kThreads) {
        const int64_t idx = (int64_t)q0 * p.num_q_heads * D + e;
        if (p.out_bf16)
          ((uint16_t*)p.out)[idx] = 0;
        else
          ((float*)p.out)[idx] = 0.f;
      }
      continue;
    }
    const int n = p.num_q_heads * D;
    const bool prompt = s_ppre[b] > 0;
    for (int e = tid; e < n; e += kThreads) {
      float v = 0.f;
      if (prompt) {
        const int64_t row = (int64_t)b * p.num_q_heads + e / D;
        const float ls = p.pfx_ml[row * 2 + 1];
        v = ls > 0.f ? p.pfx_acc[(int64_t)b * n + e] / ls : 0.f;
      }
      if (p.out_bf16)
        ((uint16_t*)p.out)[(int64_t)b * n + e] = __builtin_bit_cast(uint16_t, (__bf16)v);
      else
        ((float*)p.out)[(int64_t)b * n + e] = v;
    }
  }

  // Never more shares than positions (C >= T >= Wn).  A share can still hold no
  // position when the shares are shorter than two costs.
  const int Wn = (int)min((int64_t)W, T);
  if (u >= Wn) return;

  // 3. This workgroup's share [r0, r1) of the flattened (sequence, KV head, page)
  //    list, and this wave's quarter [w0, w1) of it: equal parts of the cost
  //    [floor(u C / Wn), floor((u + 1) C / Wn)), each taken as the positions whose
  //    cost falls inside it.  Each wave walks its own pieces without waiting for
  //    the others; a piece inside its quarter is written directly.
  int w0, w1, wunit = 0;   // wunit: the unit of position w0 (when w0 < T)
  int64_t r0, r1;
  {
    // Lane i < 5 turns quarter boundary i into the first position of cost at least
    // that boundary: the unit holding it (K(b) <= B < K(b + 1)), then the segment
    // and the page within it (the segment's start cost maps to its first page).
    int rb = 0;
    if (lane <= kWaves) {
      const int64_t B0 = (int64_t)u * C / Wn, B1 = (int64_t)(u + 1) * C / Wn;
      const int64_t B = B0 + (B1 - B0) * lane / kWaves;
      if (B >= C) {
        rb = (int)T;
      } else {
        int lo = 0, hi = nunits;
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if ((int64_t)Hs * (s_pre[mid] + S * s_ne[mid]) <= B) lo = mid; else hi = mid;
        }
        const int pre = s_pre[lo], nb = s_pre[lo + 1] - pre;
        const int rem = (int)(B - (int64_t)Hs * (pre + S * s_ne[lo]));
        const int gv = rem / (nb + S), q = rem - gv * (nb + S);
        rb = Hs * pre + gv * nb + max(q - S, 0);
        wunit = lo;
      }
    }
    r0 = __builtin_amdgcn_readfirstlane(rb);
    r1 = __builtin_amdgcn_readlane(rb, kWaves);
    w0 = __builtin_amdgcn_readlane(rb, wave);
    w1 = __builtin_amdgcn_readlane(rb, wave + 1);
    wunit = __builtin_amdgcn_readlane(wunit, wave);
  }
  // Q operands of the NT tiles, loaded with a segment's first page.
  struct QN {
    typename Pol::QOp t[NT];
  };
  if (w0 < w1) {
    constexpr int kDepth = Pol::kDepth;
    Pol st, st2;   // st2: the second tile of a two-tile segment
    st.setup(p, lane, p.stride_slot);
    QN qring[kDepth];
    typedef typename PromptState<Pol, PROMPT>::type PInit;
    PInit pring[kDepth];
    bool began = false;   // the segment being accumulated began inside this quarter
    // Page ids and position info come kChunk positions per vector load: `cur` holds
    // the chunk starting at position cbase, `nxt` the one after it (fetched a whole
    // chunk ahead).  The ring runs across chunk boundaries, so it drains only at
    // the end of the quarter.
    const int cn = w1 - w0;   // positions of this quarter (relative index k)
    // The unit of a chunk's last position bounds the units of the next chunk from below.
    auto unit_of_info = [](int info) { return (info >> kInfoSeqShift) & (PACK ? 4095 : 8191); };
    auto fetch = [&](int base, int hint) {
      return base < w1 ? fetch_chunk<MULTI, PACK>(p, s_pre, s_tail, s_ppre, s_nfull, s_gpp, nunits, base, w0, w1, lane,
                                                  Hs, nrc, hint)
                       : StreamChunk{-1, 0};
    };
    StreamChunk cur = fetch(w0, wunit), nxt = {-1, 0};   // nxt: fetched once the first loads are out
    int cbase = 0;   // relative position of cur's first entry
    {
      typename Pol::Frag fr[kDepth];
      int sinfo[kDepth];
      float skm[kDepth], svm[kDepth];
      // Issue the loads of position w0 + k into pipeline slot `sl`.
      auto issue = [&](typename Pol::Frag& f, int& info_out, float& km_out, float& vm_out, QN& q_out,
                       PInit& pi_out, int k) {
        int pk = -1, info = 0;
        float ks = 1.f, vs = 1.f;
        if (k < cn) {
          // Within two positions of the consumer, so at most one chunk ahead of it.
          const bool in_cur = k < cbase + kChunk;
          const int l = in_cur ? k - cbase : k - cbase - kChunk;
          pk = __builtin_amdgcn_readlane(in_cur ? cur.pid : nxt.pid, l);
          info = __builtin_amdgcn_readlane(in_cur ? cur.info : nxt.info, l);
          if ((unsigned)pk >= (unsigned)p.num_pages) {   // not a page of the pool: contributes nothing
            if (lane == 0) atomicOr(p.flags, kFlagBadPage);
            pk = -1;
            info &= ~kInfoTok;
          }
        }
        const int tok = info & kInfoTok;
        const int g = (info >> kInfoHeadShift) & 255, b = (info >> kInfoSeqShift) & (PACK ? 4095 : 8191);
        if constexpr (Pol::kFp8) {
          // Scales of (page, KV head); no records (reads of zero) for an absent page.
          const int64_t si = (pk >= 0) ? (int64_t)pk * Hkv + g : 0;
          const uint32_t sb = (pk >= 0) ? 4u : 0u;
          ks = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(make_rsrc_uni(p.k_scale + si, sb), 0, 0, 0));
          vs = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(make_rsrc_uni(p.v_scale + si, sb), 0, 0, 0));
        }
        const int64_t po = (pk >= 0) ? (int64_t)pk * p.stride_page + (int64_t)g * p.stride_head : 0;
        const int ptok = MULTI ? min(tok, kPage) : tok;   // tokens of this page
        const uint32_t nrec = ptok > 0 ? (uint32_t)((ptok - 1) * p.stride_slot + D * Pol::kEB) : 0u;
        const __amdgpu_buffer_rsrc_t rk = make_rsrc_uni((const char*)p.k + po, nrec);
        const __amdgpu_buffer_rsrc_t rv = make_rsrc_uni((const char*)p.v + po, nrec);
        if constexpr (PACK && kPromptTemporal) {
          // A group's prompt page is read by each of its packs, which run at about
          // the same time on one XCD: keep it in the L2 for the other packs.
          if (((info >> kInfoActShift) & 7) == kActAll)
            st.template issue<0>(f, rk, rv);
          else
            st.issue(f, rk, rv);
        } else {
          st.issue(f, rk, rv);
        }
        if constexpr (MULTI) {
          const int qs = s_ppre[b], rb = kSegRows * chunk_of_info(info);
          const bool ld = (info & (kInfoFirst | kInfoStart)) != 0;
          Pol::load_q_multi(q_out.t[0], p, qs >> 5, qs & 31, g, rb, lane, ld);
          if constexpr (NT == 2) Pol::load_q_multi(q_out.t[NT - 1], p, qs >> 5, qs & 31, g, rb + 16, lane, ld);
        } else if constexpr (Pol::kQRing) {
          Pol::load_q(q_out.t[0], p, b, g, lane, (info & (kInfoFirst | kInfoStart)) != 0);
          if constexpr (PROMPT) Pol::load_prompt(pi_out, p, b, g, lane, (info & kInfoFirst) && (info & kInfoPrompt));
        }
        info_out = info;   // the scales are used as loaded, in compute
        km_out = ks;
        vm_out = vs;
      };
      // Consume pipeline slot `sl` (position w0 + k).
      auto compute = [&](const typename Pol::Frag& f, int info, float km, float vm, const QN& q,
                         const PInit& pi, int k) {
        if (k >= cn) return;
        const int g = (info >> kInfoHeadShift) & 255, b = (info >> kInfoSeqShift) & (PACK ? 4095 : 8191);
        if (info & (kInfoFirst | kInfoStart)) {
          bool seeded = false;
          if constexpr (Pol::kQRing && PROMPT) {
            if ((info & kInfoFirst) && (info & kInfoPrompt)) {
              st.begin_prompt(q.t[0], pi, G, lane);
              seeded = true;
            }
          }
          if (!seeded) st.begin(q.t[0], p, b, g, lane);
          if constexpr (MULTI && !PACK) {
            const int nq = s_ppre[b] & 31, r = kSegRows * chunk_of_info(info) + (lane & 15);
            st.shift = (r < nq * G) ? nq - 1 - r / G : 0;
            if constexpr (NT == 2) {
              st2.begin(q.t[NT - 1], p, b, g, lane);
              st2.shift = (r + 16 < nq * G) ? nq - 1 - (r + 16) / G : 0;
            }
          }
          if constexpr (PACK) {
            if constexpr (NT == 2) st2.begin(q.t[NT - 1], p, b, g, lane);
          }
          began = (info & kInfoFirst) != 0;
        }
        if constexpr (PACK) {
          // A member's own page counts for its rows only; a prompt page for every row.
          const int act = (info >> kInfoActShift) & 7, tok = info & kInfoTok;
          // A tile none of whose rows the page serves is skipped (its state would not change).
          if constexpr (NT == 1) {
            st.template compute<true>(f, lane, (act == kActAll || rmem == act) ? tok : 0, p.scale_log2 * km, vm);
          } else {
            const typename Pol::VOp vo = Pol::v_operand(f);
            if (act == kActAll || act * G < 16)
              st.template compute_with<true>(f, &vo, lane, (act == kActAll || rmem == act) ? tok : 0,
                                             p.scale_log2 * km, vm);
            if (act == kActAll || (act + 1) * G > 16)
              st2.template compute_with<true>(f, &vo, lane, (act == kActAll || rmem2 == act) ? tok : 0,
                                              p.scale_log2 * km, vm);
          }
        } else if constexpr (MULTI) {
          if constexpr (NT == 1) {
            st.template compute<true>(f, lane, info & kInfoTok, p.scale_log2 * km, vm);
          } else {
            const typename Pol::VOp vo = Pol::v_operand(f);
            st.template compute_with<true>(f, &vo, lane, info & kInfoTok, p.scale_log2 * km, vm);
            st2.template compute_with<true>(f, &vo, lane, info & kInfoTok, p.scale_log2 * km, vm);
          }
        } else
          st.compute(f, lane, info & kInfoTok, p.scale_log2 * km, vm);
        if (info & (kInfoLast | kInfoEnd)) {
          const bool ended = (info & kInfoLast) != 0;
          if (began && ended) {
            if constexpr (MULTI) {
              const int rb = kSegRows * chunk_of_info(info);
              st.write_out_multi(p, s_ppre[b] >> 5, s_ppre[b] & 31, g, rb, lane);
              if constexpr (NT == 2) st2.write_out_multi(p, s_ppre[b] >> 5, s_ppre[b] & 31, g, rb + 16, lane);
            } else {
              st.write_out(p, b, g, lane);
            }
          } else {
            const int slot = 2 * wave + (ended ? 0 : 1);
            st.to_lds(s_acc[slot], s_ml[slot], lane);
            if constexpr (NT == 2) st2.to_lds(s_acc[slot] + 16, s_ml[slot] + 16, lane);
            if (lane == 0) s_seg[slot] = b * Hs + (MULTI ? g * nrc + chunk_of_info(info) : g);
          }
        }
      };
      // Once position k (relative) is consumed: the last one of cur moves the ids on
      // by a chunk (its successor has been read from nxt already).
      auto advance = [&](int k) {
        if (k + 1 == cbase + kChunk && k + 1 < cn) {
          cur = nxt;
          cbase += kChunk;
          nxt = fetch(w0 + cbase + kChunk, unit_of_info(__builtin_amdgcn_readlane(cur.info, kChunk - 1)));
        }
      };
#pragma unroll
      for (int k = 0; k < kDepth - 1; ++k)
        if (k < cn) issue(fr[k], sinfo[k], skm[k], svm[k], qring[k], pring[k], k);
      // First read kChunk - kDepth + 1 positions from now.
      nxt = fetch(w0 + kChunk, unit_of_info(__builtin_amdgcn_readlane(cur.info, kChunk - 1)));
      int i = 0;
      // Steady state: every position issued lies inside the quarter.
      for (; i + 2 * kDepth - 2 < cn; i += kDepth) {
#pragma unroll
        for (int k = 0; k < kDepth; ++k) {
          const int si = (k + kDepth - 1) % kDepth;
          issue(fr[si], sinfo[si], skm[si], svm[si], qring[si], pring[si], i + k + kDepth - 1);
          compute(fr[k], sinfo[k], skm[k], svm[k], qring[k], pring[k], i + k);
          advance(i + k);
        }
      }
      // Drain: no loads are issued past the quarter, so none is left in flight.
      for (; i < cn; i += kDepth) {
#pragma unroll
        for (int k = 0; k < kDepth; ++k) {
          const int si = (k + kDepth - 1) % kDepth;
          if (i + k + kDepth - 1 < cn)
            issue(fr[si], sinfo[si], skm[si], svm[si], qring[si], pring[si], i + k + kDepth - 1);
          compute(fr[k], sinfo[k], skm[k], svm[k], qring[k], pring[k], i + k);
          advance(i + k);
        }
      }
    }
  }
  // The waves' pieces are in LDS; their global stores need not have completed.
  lds_barrier();

  // 4. Merge the cut pieces in position order.  The used slots holding one segment
  //    are consecutive; together they are either the whole segment (normalise and
  //    write) or this workgroup's piece of a segment cut at the share boundary
  //    (published as a partial).
  const int h = tid / kTPR, d0 = (tid % kTPR) * DPT;
  // Segment gv of sequence b: its rows, and the output row / query head of this
  // thread's row h (multi-token runs: row 16 NT rc + h of the (sequence, KV head)).
  auto seg_row = [&](int gv) { return kSegRows * (gv % nrc) + h; };
  auto seg_rows = [&](int b, int gv) {
    return MULTI ? min(kSegRows, (s_ppre[b] & 31) * G - kSegRows * (gv % nrc)) : G;
  };
  auto out_row = [&](int b, int gv) { return MULTI ? (s_ppre[b] >> 5) + seg_row(gv) / G : b; };
  auto out_head = [&](int gv) {
    return MULTI ? s_qhead[(gv / nrc) * G + seg_row(gv) % G] : s_qhead[gv * G + h];
  };
  int hand_seg[2] = {-1, -1};
  int nhand = 0;
  {
    int cur = -1;   // segment of the group being merged
    float M = neg_inf(), Ls = 0.f, o[DPT];
#pragma unroll
    for (int e = 0; e < DPT; ++e) o[e] = 0.f;
    // Close the group of segment `cur`: write it, or publish this workgroup's piece.
    // Lane j < 2 kWaves: slot j's segment and its first and last positions, read
    // for every slot at once (the merge below takes them with readlane).
    // Lane j < 2 kWaves: slot j's segment, its sequence and segment within the
    // sequence, and its first and last positions, read for every slot at once (the
    // merge below takes them with readlane).
    int lseg = -2, lb = 0, lg = 0, lstart = 0, lend = 0;
    if (lane < 2 * kWaves) {
      lseg = s_seg[lane];
      if (lseg >= 0) {
        lb = lseg / Hs;
        lg = lseg - lb * Hs;
        const int pre_b = s_pre[lb], nb = s_pre[lb + 1] - pre_b;
        lstart = Hs * pre_b + lg * nb;
        lend = lstart + nb;
      }
    }
    int jcur = 0;   // a slot of segment `cur`
    int qh_cur = 0;   // this thread's output query head in segment `cur` (read when the group opens)
    auto flush = [&]() {
      const int b = __builtin_amdgcn_readlane(lb, jcur), g = __builtin_amdgcn_readlane(lg, jcur);
      const int64_t seg_start = __builtin_amdgcn_readlane(lstart, jcur), seg_end = __builtin_amdgcn_readlane(lend, jcur);
      const bool whole = seg_start >= r0 && seg_end <= r1;
      if (h < seg_rows(b, g)) {
        if (whole) {
          store_out<D, DPT>(p, out_row(b, g), qh_cur, d0, o, Ls > 0.f ? 1.f / Ls : 0.f);
        } else {
          const PartialRsrc rs = PartialRsrc::of<D>(p);
          const int gs = (seg_end > r1) ? 2 * u + 1 : 2 * u;
          const int R = p.part_rows, hr = h;   // the row within the slot
#pragma unroll
          for (int c = 0; c < DPT; c += 4)
            __builtin_amdgcn_raw_buffer_store_b128(*(const u32x4*)&o[c], rs.acc, ((gs * R + hr) * D + d0 + c) * 4, 0,
                                                   kDeviceScope);
          if (tid % kTPR == 0)   // one thread per row stores its (m, l) and the call's tag
            __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(M), __float_as_uint(Ls), p.call_tag, 0u},
                                                   rs.ml, (gs * R + hr) * 16, 0, kDeviceScope);
        }
      }
      if (!whole && nhand < 2) hand_seg[nhand++] = cur;   // only the first and last group can be cut
    };
    // Slots in position order; the used slots of one segment are consecutive.  Every
    // slot's max/sum and partial output, and this thread's output head for every
    // slot's segment, are read from LDS before the first merge (unused slots read
    // values that are never used), so the merge waits for LDS once, not per slot.
    float ms[2 * kWaves], ls[2 * kWaves], vs[2 * kWaves][DPT];
    int qhs[2 * kWaves];
#pragma unroll
    for (int j = 0; j < 2 * kWaves; ++j) {
      ms[j] = s_ml[j][h][0];
      ls[j] = s_ml[j][h][1];
#pragma unroll
      for (int c = 0; c < DPT; c += 4) *(f32x4*)&vs[j][c] = *(const f32x4*)&s_acc[j][h][d0 + c];
      qhs[j] = out_head(__builtin_amdgcn_readlane(lg, j));
    }
#pragma unroll
    for (int j = 0; j <= 2 * kWaves; ++j) {
      const int sj = j < 2 * kWaves ? __builtin_amdgcn_readlane(lseg, j) : -2;   // -2: past the last slot
      if (sj == -1) continue;   // unused slot
      if (sj != cur) {
        if (cur >= 0) flush();
        cur = sj;
        jcur = j;
        if (sj >= 0) qh_cur = qhs[j];
        M = neg_inf();
        Ls = 0.f;
#pragma unroll
        for (int e = 0; e < DPT; ++e) o[e] = 0.f;
      }
      if (sj >= 0 && h < seg_rows(__builtin_amdgcn_readlane(lb, j), __builtin_amdgcn_readlane(lg, j)))
        lse_merge<DPT>(M, Ls, o, ms[j], ls[j], vs[j]);
    }
  }

  // 5. Segments cut at the share boundary: count this piece; the workgroup that
  //    completes the count merges every piece of the segment and resets the count.
  if (nhand == 0) return;
  __builtin_amdgcn_s_waitcnt(0);   // this wave's device-scope stores have completed
  __syncthreads();                 // ... and every other wave's
  if (tid < nhand) {
    const int sgi = hand_seg[tid];
    const int b = sgi / Hs, g = sgi - b * Hs;
    const int pre_b = s_pre[b], nb = s_pre[b + 1] - pre_b;
    const int64_t seg_start = (int64_t)Hs * pre_b + (int64_t)g * nb;
    const uint32_t npieces = (uint32_t)(owner_of(cost_of(seg_start + nb - 1, b, g), Wn, C) -
                                        owner_of(cost_of(seg_start, b, g), Wn, C) + 1);
    const uint32_t old = atomicAdd(p.counters + sgi, 1u);
    if (old >= npieces) atomicOr(p.flags, kFlagStaleState);   // more pieces than the segment has
    s_last[tid] = (old + 1u == npieces);
  }
  __syncthreads();
  for (int i = 0; i < nhand; ++i) {
    if (!s_last[i]) continue;
    const int sgi = hand_seg[i];
    const int b = sgi / Hs, g = sgi - b * Hs;
    const int pre_b = s_pre[b], nb = s_pre[b + 1] - pre_b;
    const int64_t seg_start = (int64_t)Hs * pre_b + (int64_t)g * nb;
    if (h < seg_rows(b, g))
      merge_pieces<D, DPT>(p, out_row(b, g), out_head(g), h, d0, owner_of(cost_of(seg_start, b, g), Wn, C),
                           owner_of(cost_of(seg_start + nb - 1, b, g), Wn, C));
    if (tid == 0) atomicExch(p.counters + sgi, 0u);
  }
}

// ---------------------------------------------------------------- prompt pass (grouped runs)
// One workgroup per job (group i, KV head g, member block): the job's query rows
// are the G heads of each of up to 64/G members (row = (member - first) * G +
// head index), packed into up to 4 MFMA tiles of 16 rows.  The 4 waves split the
// group's prompt pages; each page is loaded once and multiplied against every
// tile, so the group reads its prompt once per KV head instead of once per
// response.  The 4 waves' states are merged through LDS and each row's
// unnormalised (m, l, O) is stored for the attention kernel, which continues
// every member's softmax from it.  The job of block 0 of KV head 0 also stores
// the group's clamped prompt length.
constexpr int kPromptTiles = 4;

template <int D, bool FP8>
__global__ __attribute__((amdgpu_flat_work_group_size(kThreads, kThreads), amdgpu_waves_per_eu(1, 1)))
void prompt_kernel(const Params p) {
  using Pol = Mfma<D, FP8>;
  constexpr int R = kPromptTiles, kRows = 16 * R, kDepth = Pol::kDepth;
  __shared__ __align__(16) float s_acc[kWaves][kRows][D + 4];
  __shared__ __align__(16) float s_ml[kWaves][kRows][2];
  __shared__ int32_t s_min;

  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  const int Hkv = p.num_kv_heads, G = p.group, Hq = p.num_q_heads, n = p.group_size;
  const int cap = p.max_pages * kPage;
  const int job = blockIdx.x / p.pfx_splits, split = blockIdx.x - job * p.pfx_splits;
  const int mb = job % p.pfx_nblocks, ig = job / p.pfx_nblocks;
  const int g = ig % Hkv, gi = ig / Hkv;
  const int b0 = gi * n, b1 = min(b0 + n, p.batch);                        // members of group gi
  const int m0 = b0 + mb * p.pfx_mblock, m1 = min(m0 + p.pfx_mblock, b1);  // members of this job

  for (int e = tid; e < Hq; e += kThreads) s_qhead[e] = p.q_head[e];
  if (tid == 0) s_min = 0x7fffffff;
  __syncthreads();
  // Shared prompt: the requested pages, clamped to the full pages of the shortest member.
  {
    int mn = 0x7fffffff;
    for (int b = b0 + tid; b < b1; b += kThreads) mn = min(mn, min(max(p.seq_lens[b], 0), cap) / kPage);
    if (mn != 0x7fffffff) atomicMin(&s_min, mn);
  }
  __syncthreads();
  const int want = p.prefix_pages[gi];
  const int P = uni(max(0, min(want, s_min)));
  if (tid == 0 && g == 0 && mb == 0 && split == 0) {
    p.gprefix[gi] = P;
    if (want != P) atomicOr(p.flags, kFlagPrefixClamped);
  }
  const int rows = (m1 - m0) * G;
  // Workgroups per job: at least 32 pages each (8 per wave), at most the launched
  // p.pfx_splits; the others have nothing to do.  A split costs a device-scope
  // handoff, which only pays off for long prompts.
  const int S = uni(min(p.pfx_splits, max(1, (P + 31) / 32)));
  if (P == 0 || rows <= 0 || split >= S) return;
  const int nt = uni((rows + 15) / 16);   // tiles in use

  Pol t[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    t[r].setup(p, lane, p.stride_slot);
    typename Pol::QOp qo;
    Pol::load_q_rows(qo, p, g, m0, rows, 16 * r, lane);
    t[r].begin(qo, p, 0, 0, lane);
  }

  // This wave's prompt pages [j0, j1) (the job's pages cut into S * 4 ranges), read
  // from the group's first member's row.
  const int ws = split * kWaves + wave;
  const int j0 = ws * P / (S * kWaves), j1 = (ws + 1) * P / (S * kWaves);
  const int32_t* bt = p.block_table + (int64_t)b0 * p.max_pages;
  const int rec = (kPage - 1) * p.stride_slot + D * Pol::kEB;   // a full page
  for (int cb = j0; cb < j1; cb += kChunk) {
    const int cn = min(kChunk, j1 - cb);
    int pid = bt[cb + min(lane, cn - 1)];
    typename Pol::Frag fr[kDepth];
    float skm[kDepth], svm[kDepth];
    int sval[kDepth];
    // Every step issues the same loads (past the range with descriptors of no
    // records, which read nothing), so the loads stay in flight across steps.
    auto issue = [&](typename Pol::Frag& f, int& val, float& ks, float& vs, int k) {
      int pk = -1;
      if (k < cn) {
        pk = __builtin_amdgcn_readlane(pid, k);
        if ((unsigned)pk >= (unsigned)p.num_pages) {   // not a page of the pool: contributes nothing
          if (lane == 0) atomicOr(p.flags, kFlagBadPage);
          pk = -1;
        }
      }
      val = pk >= 0 ? kPage : 0;
      const int64_t po = (pk >= 0) ? (int64_t)pk * p.stride_page + (int64_t)g * p.stride_head : 0;
      const uint32_t nrec = pk >= 0 ? (uint32_t)rec : 0u;
      ks = 1.f;
      vs = 1.f;
      if constexpr (FP8) {
        const int64_t si = (pk >= 0) ? (int64_t)pk * Hkv + g : 0;
        const uint32_t sb = (pk >= 0) ? 4u : 0u;
        ks = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(make_rsrc_uni(p.k_scale + si, sb), 0, 0, 0));
        vs = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(make_rsrc_uni(p.v_scale + si, sb), 0, 0, 0));
      }
      t[0].issue(f, make_rsrc_uni((const char*)p.k + po, nrec), make_rsrc_uni((const char*)p.v + po, nrec));
    };
    auto compute = [&](const typename Pol::Frag& f, int val, float ks, float vs) {
#pragma unroll
      for (int r = 0; r < R; ++r)
        if (r < nt) t[r].compute(f, lane, val, p.scale_log2 * ks, vs);
    };
#pragma unroll
    for (int k = 0; k < kDepth - 1; ++k) issue(fr[k], sval[k], skm[k], svm[k], k);
    for (int i = 0; i < cn; i += kDepth) {
#pragma unroll
      for (int k = 0; k < kDepth; ++k) {
        const int si = (k + kDepth - 1) % kDepth;
        issue(fr[si], sval[si], skm[si], svm[si], i + k + kDepth - 1);
        if (i + k < cn) compute(fr[k], sval[k], skm[k], svm[k]);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) t[r].to_lds(s_acc[wave] + 16 * r, s_ml[wave] + 16 * r, lane);
  __syncthreads();

  // Merge the 4 waves' states: thread (row, quarter of d).
  constexpr int DQ = D / 4;
  const int row = tid >> 2, d0 = (tid & 3) * DQ;
  float M = neg_inf(), Ls = 0.f, o[DQ];
#pragma unroll
  for (int e = 0; e < DQ; ++e) o[e] = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    float v[DQ];
#pragma unroll
    for (int c = 0; c < DQ; c += 4) *(f32x4*)&v[c] = *(const f32x4*)&s_acc[w][row][d0 + c];
    lse_merge<DQ>(M, Ls, o, s_ml[w][row][0], s_ml[w][row][1], v);
  }
  if (S > 1) {
    // The job is split over S workgroups: publish this one's state in slot
    // job * S + split (device scope, rows of 64), count it, and let the workgroup
    // that completes the count merge the S states in split order.
    const __amdgpu_buffer_rsrc_t ra = make_rsrc_uni(p.part_acc, (uint32_t)p.pfx_slots * kRows * D * 4u);
    const __amdgpu_buffer_rsrc_t rm = make_rsrc_uni(p.part_ml, (uint32_t)p.pfx_slots * kRows * 8u);
    const int slot_row = (job * p.pfx_splits + split) * kRows + row;
#pragma unroll
    for (int c = 0; c < DQ; c += 4)
      __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(o[c]), __float_as_uint(o[c + 1]),
                                                   __float_as_uint(o[c + 2]), __float_as_uint(o[c + 3])},
                                             ra, (slot_row * D + d0 + c) * 4, 0, kDeviceScope);
    if ((tid & 3) == 0)
      __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(M), __float_as_uint(Ls)}, rm, slot_row * 8, 0,
                                            kDeviceScope);
    __builtin_amdgcn_s_waitcnt(0);   // this wave's device-scope stores have completed
    __syncthreads();                 // ... and every other wave's
    if (tid == 0) {
      const uint32_t old = atomicAdd(p.counters + job, 1u);
      if (old >= (uint32_t)S) atomicOr(p.flags, kFlagStaleState);   // more pieces than the job has
      s_min = (old + 1u == (uint32_t)S);
    }
    __syncthreads();
    if (!s_min) return;
    if (tid == 0) atomicExch(p.counters + job, 0u);
    M = neg_inf();
    Ls = 0.f;
#pragma unroll
    for (int e = 0; e < DQ; ++e) o[e] = 0.f;
    constexpr int kBatch = 4;
    for (int k0 = 0; k0 < S; k0 += kBatch) {
      u32x2 ml[kBatch];
      float v[kBatch][DQ];
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        const int sr = (job * p.pfx_splits + min(k0 + i, S - 1)) * kRows + row;   // past the last split: re-read, unused
        ml[i] = __builtin_amdgcn_raw_buffer_load_b64(rm, sr * 8, 0, kDeviceScope);
#pragma unroll
        for (int c = 0; c < DQ; c += 4)
          *(u32x4*)&v[i][c] = __builtin_amdgcn_raw_buffer_load_b128(ra, (sr * D + d0 + c) * 4, 0, kDeviceScope);
      }
#pragma unroll
      for (int i = 0; i < kBatch; ++i)
        if (k0 + i < S) lse_merge<DQ>(M, Ls, o, __uint_as_float(ml[i][0]), __uint_as_float(ml[i][1]), v[i]);
    }
  }
  if (row >= rows) return;
  const int b = m0 + row / G, h = s_qhead[g * G + row % G];
  const int64_t orow = (int64_t)b * Hq + h;
  float* dst = p.pfx_acc + orow * D + d0;
#pragma unroll
  for (int c = 0; c < DQ; c += 4) *(f32x4*)(dst + c) = f32x4{o[c], o[c + 1], o[c + 2], o[c + 3]};
  if ((tid & 3) == 0) *(f32x2*)(p.pfx_ml + orow * 2) = f32x2{M, Ls};
}

// ---------------------------------------------------------------- KV append
// One wave per (sequence, KV head): lane l owns elements [l * E, (l + 1) * E) of a
// row, E = D / 64.  bf16 / fp32 caches copy the new row into its slot.  fp8 caches
// keep the page's scale covering every row written so far: the first row of a page
// sets amax / 448; a later row with a larger amax raises the scale and re-encodes
// the earlier rows (decode, times old/new scale, round to nearest even).

// E4M3 (OCP FN) encoding of two fp32 values into the low 16 bits, round to nearest even.
__device__ __forceinline__ uint32_t e4m3x2(float a, float b) {
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false) & 0xFFFFu;
}

template <int D, KvKind KIND>
__global__ __launch_bounds__(kThreads) void append_kernel(const Params p) {
  constexpr int E = D / 64;
  const int lane = threadIdx.x & 63;
  const int item = uni((int)(blockIdx.x * kWaves + (threadIdx.x >> 6)));
  if (item >= p.batch * p.num_kv_heads) return;
  const int b = item / p.num_kv_heads, g = item - b * p.num_kv_heads;
  const int cap = p.max_pages * kPage;
  const int L = uni(p.seq_lens[b]);
  if (L < 1 || L > cap) {
    if ((L < 0 || L > cap) && lane == 0) atomicOr(p.flags, kFlagBadLen);
    return;
  }
  const int t = L - 1, slot = t % kPage;
  const int pid = uni(p.block_table[(int64_t)b * p.max_pages + t / kPage]);
  if ((unsigned)pid >= (unsigned)p.num_pages) {
    if (lane == 0) atomicOr(p.flags, kFlagBadPage);
    return;
  }
  const int64_t row0 = (int64_t)pid * p.stride_page + (int64_t)g * p.stride_head;   // bytes, slot 0
  const int64_t in_off = ((int64_t)item * D + lane * E);                               // elements

#pragma unroll
  for (int kv = 0; kv < 2; ++kv) {
    char* cache = (char*)(kv ? p.v : p.k);
    const void* in = kv ? p.v_in : p.k_in;
    if constexpr (KIND == KvKind::F32) {
      const float* src = (const float*)in + in_off;
      float* dst = (float*)(cache + row0 + (int64_t)slot * p.stride_slot) + lane * E;
#pragma unroll
      for (int e = 0; e < E; ++e) dst[e] = src[e];
    } else if constexpr (KIND == KvKind::BF16) {
      const uint16_t* src = (const uint16_t*)in + in_off;
      uint16_t* dst = (uint16_t*)(cache + row0 + (int64_t)slot * p.stride_slot) + lane * E;
#pragma unroll
      for (int e = 0; e < E; ++e) dst[e] = src[e];
    } else {
      float* scales = (float*)(kv ? p.v_scale : p.k_scale);
      const uint16_t* src = (const uint16_t*)in + in_off;
      float x[E];
      float amax = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        x[e] = __uint_as_float((uint32_t)src[e] << 16);
        amax = fmaxf(amax, fabsf(x[e]));
      }
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) amax = fmaxf(amax, __shfl_xor(amax, o));
      amax = __builtin_bit_cast(float, uni(__builtin_bit_cast(int, amax)));
      const int64_t si = (int64_t)pid * p.num_kv_heads + g;
      float s = 0.f;
      if (slot > 0) {
        s = scales[si];
        if (!(s > 0.f) || __builtin_isinf(s)) s = 0.f;
      }
      float s_new = s;
      if (slot == 0 || amax > 448.f * s) {
        s_new = amax / 448.f;
        // Earlier rows of the page (slot > 0 only): re-encode at the new scale.
        const float ratio = s > 0.f ? s / s_new : 0.f;
        for (int r = 0; r < slot; ++r) {
          uint8_t* rp = (uint8_t*)(cache + row0 + (int64_t)r * p.stride_slot) + lane * E;
          if constexpr (E == 2) {
            const uint32_t w = *(const uint16_t*)rp;
            const f32x2 v = fp8x2_to_f32(w, false);
            *(uint16_t*)rp = (uint16_t)(s > 0.f ? e4m3x2(v[0] * ratio, v[1] * ratio) : 0u);
          } else {
            const f32x2 v = fp8x2_to_f32((uint32_t)*rp, false);
            *rp = (uint8_t)(s > 0.f ? e4m3x2(v[0] * ratio, 0.f) & 0xFFu : 0u);
          }
        }
      }
      uint8_t* dst = (uint8_t*)(cache + row0 + (int64_t)slot * p.stride_slot) + lane * E;
      if constexpr (E == 2)
        *(uint16_t*)dst = (uint16_t)(s_new > 0.f ? e4m3x2(x[0] / s_new, x[1] / s_new) : 0u);
      else
        *dst = (uint8_t)(s_new > 0.f ? e4m3x2(x[0] / s_new, 0.f) & 0xFFu : 0u);
      if (lane == 0) scales[si] = s_new;
    }
  }
}

template <int D, KvKind KIND>
int launch_append_t(const Params& p, void* stream) {
  const int items = p.batch * p.num_kv_heads;
  hipLaunchKernelGGL((append_kernel<D, KIND>), dim3((items + kWaves - 1) / kWaves), dim3(kThreads), 0,
                     (hipStream_t)stream, p);
  return (int)hipGetLastError();
}

template <class Pol, bool MULTI = false, int NT = 1, bool PACK = false, bool PROMPT = false, int WPE = 1>
int launch(const Params& p, void* stream, void* ev_begin, void* ev_end) {
  hipStream_t st = (hipStream_t)stream;
  if (ev_begin && hipEventRecord((hipEvent_t)ev_begin, st) != hipSuccess) return -1;
  hipLaunchKernelGGL((decode_attention_kernel<Pol, MULTI, NT, PACK, PROMPT, WPE>), dim3(p.nranges), dim3(kThreads), 0, st,
                     p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  if (ev_end && hipEventRecord((hipEvent_t)ev_end, st) != hipSuccess) return -1;
  return 0;
}

template <int D, bool FP8>
int launch_prompt_then_decode(const Params& p, int ngroups, void* stream, void* ev_begin, void* ev_end) {
  hipStream_t st = (hipStream_t)stream;
  if (ev_begin && hipEventRecord((hipEvent_t)ev_begin, st) != hipSuccess) return -1;
  const int jobs = ngroups * p.num_kv_heads * p.pfx_nblocks;
  hipLaunchKernelGGL((prompt_kernel<D, FP8>), dim3(jobs * p.pfx_splits), dim3(kThreads), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  return launch<Mfma<D, FP8>, false, 1, false, true>(p, stream, nullptr, ev_end);
}

std::mutex g_scratch_mu;
void* g_scratch_ptr[64];

}  // namespace

int noalloc_scratch(void** ptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return -1;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    // With `dev` current: this device's copy of the array.
    void* a = nullptr;
    if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || !a) return -1;
    g_scratch_ptr[dev] = a;
  }
  *ptr = g_scratch_ptr[dev];
  return 0;
}

#define RLDA_DISPATCH(FN, ...)                                                  \
  switch (kind) {                                                               \
    case KvKind::BF16:                                                          \
      return head_dim == 128 ? FN<Mfma<128, false>>(__VA_ARGS__)                \
                             : FN<Mfma<64, false>>(__VA_ARGS__);                \
    case KvKind::FP8:                                                           \
      return head_dim == 128 ? FN<Mfma<128, true>>(__VA_ARGS__)                 \
                             : FN<Mfma<64, true>>(__VA_ARGS__);                 \
    case KvKind::F32:                                                           \
      if (head_dim == 128) return FN<Valu<128, 1>>(__VA_ARGS__);                \
      return group == 1 ? FN<Valu<64, 1>>(__VA_ARGS__) : FN<Valu<64, 2>>(__VA_ARGS__); \
  }                                                                             \
  return -1;

int launch_decode(KvKind kind, int head_dim, int group, const Params& p, void* stream, void* ev_begin,
                  void* ev_end) {
  RLDA_DISPATCH(launch, p, stream, ev_begin, ev_end)
}

template <class Pol>
int launch_rows(int tiles, const Params& p, void* stream, void* ev_begin, void* ev_end) {
  return tiles == 2 ? launch<Pol, true, 2>(p, stream, ev_begin, ev_end) : launch<Pol, true, 1>(p, stream, ev_begin, ev_end);
}

template <class Pol>
int launch_packed(int tiles, const Params& p, void* stream, void* ev_begin, void* ev_end) {
  return tiles == 1 ? launch<Pol, true, 1, true>(p, stream, ev_begin, ev_end) : -1;
}

int launch_decode_rows(KvKind kind, int head_dim, int tiles, const Params& p, void* stream, void* ev_begin,
                       void* ev_end) {
  switch (kind) {
    case KvKind::BF16:
      return head_dim == 128 ? launch_rows<Mfma<128, false>>(tiles, p, stream, ev_begin, ev_end)
                             : launch_rows<Mfma<64, false>>(tiles, p, stream, ev_begin, ev_end);
    case KvKind::FP8:
      return head_dim == 128 ? launch_rows<Mfma<128, true>>(tiles, p, stream, ev_begin, ev_end)
                             : launch_rows<Mfma<64, true>>(tiles, p, stream, ev_begin, ev_end);
    case KvKind::F32:
      break;
  }
  return -1;
}

int launch_decode_packed(KvKind kind, int head_dim, int tiles, const Params& p, void* stream, void* ev_begin,
                         void* ev_end) {
  switch (kind) {
    case KvKind::BF16:
      return head_dim == 128 ? launch_packed<Mfma<128, false>>(tiles, p, stream, ev_begin, ev_end)
                             : launch_packed<Mfma<64, false>>(tiles, p, stream, ev_begin, ev_end);
    case KvKind::FP8:
      return head_dim == 128 ? launch_packed<Mfma<128, true>>(tiles, p, stream, ev_begin, ev_end)
                             : launch_packed<Mfma<64, true>>(tiles, p, stream, ev_begin, ev_end);
    case KvKind::F32:
      break;
  }
  return -1;
}

int launch_decode_two(KvKind kind, int head_dim, const Params& p, void* stream, void* ev_begin, void* ev_end) {
  if (kind == KvKind::BF16)
    return head_dim == 64 ? launch<Mfma<64, false>, false, 1, false, false, 2>(p, stream, ev_begin, ev_end) : -1;
  if (kind != KvKind::FP8) return -1;
  return head_dim == 128 ? launch<Mfma<128, true>, false, 1, false, false, 2>(p, stream, ev_begin, ev_end)
                         : launch<Mfma<64, true>, false, 1, false, false, 2>(p, stream, ev_begin, ev_end);
}

int launch_append(KvKind kind, int head_dim, const Params& p, void* stream) {
  switch (kind) {
    case KvKind::BF16:
      return head_dim == 128 ? launch_append_t<128, KvKind::BF16>(p, stream) : launch_append_t<64, KvKind::BF16>(p, stream);
    case KvKind::FP8:
      return head_dim == 128 ? launch_append_t<128, KvKind::FP8>(p, stream) : launch_append_t<64, KvKind::FP8>(p, stream);
    case KvKind::F32:
      return head_dim == 128 ? launch_append_t<128, KvKind::F32>(p, stream) : launch_append_t<64, KvKind::F32>(p, stream);
  }
  return -1;
}

int launch_grouped(KvKind kind, int head_dim, int, const Params& p, int ngroups, void* stream, void* ev_begin,
                   void* ev_end) {
  switch (kind) {
    case KvKind::BF16:
      return head_dim == 128 ? launch_prompt_then_decode<128, false>(p, ngroups, stream, ev_begin, ev_end)
                             : launch_prompt_then_decode<64, false>(p, ngroups, stream, ev_begin, ev_end);
    case KvKind::FP8:
      return head_dim == 128 ? launch_prompt_then_decode<128, true>(p, ngroups, stream, ev_begin, ev_end)
                             : launch_prompt_then_decode<64, true>(p, ngroups, stream, ev_begin, ev_end);
    case KvKind::F32:
      break;
  }
  return -1;
}


}  // namespace rlda
