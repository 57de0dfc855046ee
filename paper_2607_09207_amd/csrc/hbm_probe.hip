// Achievable HBM read rate on gfx950: two read-only kernels that set the ceiling
// a bandwidth-bound kernel is measured against.  Not part of the attention path;
// the bench loads this library next to the attention library and reports the best
// rate each kernel reaches over a few launch shapes.
//
//   stream read  - a contiguous buffer read once, 16 bytes per lane per load, a
//                  ring of U loads in flight per lane, non-temporal (the data is
//                  not reused);
//   tile gather  - the decode kernel's access pattern without its arithmetic: a list
//                  of (K, V) tile pairs at byte offsets into two pools (one pair per
//                  (sequence, KV head, page) of a workload, in the order the decode
//                  kernel streams them), cut into equal contiguous shares, one per
//                  wave, with a ring of U tile pairs in flight per wave.
//   balanced gather - the same tiles and ring, but only the first `nstatic`
//                  entries are cut into equal shares; the rest is a pool of chunks
//                  of `chunk` entries that waves claim one at a time with an
//                  atomicAdd once their share is done (the next claim is made when
//                  a chunk starts, so the ring runs on across chunks).  It measures
//                  what run-time balancing of the tile stream could add.
// All fold every loaded word into a per-lane value and store it only when it
// equals a sentinel, so the loads cannot be removed and almost nothing is written.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hbm_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kSentinel = 0x9E3779B9u;

__device__ __forceinline__ uint32_t fold(u32x4 v) { return v[0] ^ v[1] ^ v[2] ^ v[3]; }

// Thread t of the grid reads elements t, t + N, t + 2N, ... (N threads) as a ring
// of U loads: the load U - 1 elements ahead is issued before each element is
// folded, so U loads stay in flight from the first element to the last.
template <int U>
__global__ __attribute__((amdgpu_flat_work_group_size(64, 512))) void stream_read_kernel(const u32x4* __restrict__ buf, uint64_t n16, uint32_t* __restrict__ sink) {
  const uint64_t N = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t i0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint64_t cnt = i0 < n16 ? (n16 - i0 + N - 1) / N : 0;   // elements of this thread
  const u32x4* p = buf + i0;
  u32x4 r[U];
  uint32_t acc = 0;
#pragma unroll
  for (int k = 0; k < U - 1; ++k)
    if ((uint64_t)k < cnt) r[k] = __builtin_nontemporal_load(p + k * N);
  uint64_t j = 0;
  for (; j + 2 * U - 2 < cnt; j += U) {   // every index issued here is below cnt
#pragma unroll
    for (int k = 0; k < U; ++k) {
      r[(k + U - 1) % U] = __builtin_nontemporal_load(p + (j + k + U - 1) * N);
      acc ^= fold(r[k]);
    }
  }
  for (; j < cnt; j += U) {
#pragma unroll
    for (int k = 0; k < U; ++k) {
      if (j + k + U - 1 < cnt) r[(k + U - 1) % U] = __builtin_nontemporal_load(p + (j + k + U - 1) * N);
      if (j + k < cnt) acc ^= fold(r[k]);
    }
  }
  if (acc == kSentinel) sink[blockIdx.x] = acc;
}

// Wave w of the grid reads entries [w*n/W, (w+1)*n/W) of the offset list: for each,
// the K tile and the V tile of `tile_bytes` at that byte offset, lane l loading bytes
// [16 l, 16 l + 16) of every 1 KiB of the tile (one load instruction of the wave
// covers 1 KiB contiguous).  The entries go through a ring of U: the tiles of entry
// e + U - 1 are issued before entry e is folded.
template <int U>
__global__ __attribute__((amdgpu_flat_work_group_size(64, 512))) void tile_gather_kernel(const char* __restrict__ k, const char* __restrict__ v,
                                   const int64_t* __restrict__ off, int64_t n, int tile_bytes,
                                   uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
  const int64_t w = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t e0 = w * n / waves, e1 = (w + 1) * n / waves;
  const int per = tile_bytes / 1024;   // 1 KiB load instructions per tile
  uint32_t acc = 0;
  u32x4 kv[U][2][4];
  auto issue = [&](u32x4 (&t)[2][4], int64_t e) {
    const int64_t o = off[e];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t b = o + (int64_t)c * 1024 + lane * 16;
      t[0][c] = c < per ? __builtin_nontemporal_load((const u32x4*)(k + b)) : u32x4{0, 0, 0, 0};
      t[1][c] = c < per ? __builtin_nontemporal_load((const u32x4*)(v + b)) : u32x4{0, 0, 0, 0};
    }
  };
  auto consume = [&](const u32x4 (&t)[2][4]) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc ^= fold(t[0][c]) ^ fold(t[1][c]);
  };
#pragma unroll
  for (int u = 0; u < U - 1; ++u)
    if (e0 + u < e1) issue(kv[u], e0 + u);
  int64_t e = e0;
  for (; e + 2 * U - 2 < e1; e += U) {   // every entry issued here is below e1
#pragma unroll
    for (int u = 0; u < U; ++u) {
      issue(kv[(u + U - 1) % U], e + u + U - 1);
      consume(kv[u]);
    }
  }
  for (; e < e1; e += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (e + u + U - 1 < e1) issue(kv[(u + U - 1) % U], e + u + U - 1);
      if (e + u < e1) consume(kv[u]);
    }
  }
  if (acc == kSentinel) sink[blockIdx.x] = acc;
}


// Wave w of the grid reads its equal share of entries [0, nstatic), then claims
// chunks c = 0, 1, ... of [nstatic, n) (entries nstatic + c chunk ...) from
// counter[0].  The entries of the current chunk and of the next one (chunks hold at
// least U entries, shares at least U or none) are in two lanes-wide registers, so
// the ring's look-ahead of U - 1 entries always finds its entry.  Every wave makes
// exactly one claim past the last chunk; the wave whose claim is the last of all
// (nchunks + waves - 1) resets the counter to zero for the next launch.
template <int U>
__global__ __attribute__((amdgpu_flat_work_group_size(64, 512))) void tile_gather_balanced_kernel(
    const char* __restrict__ k, const char* __restrict__ v, const int64_t* __restrict__ off, int64_t n,
    int64_t nstatic, int chunk, uint32_t* counter, int tile_bytes, uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
  const int64_t w = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  int64_t sp = w * nstatic / waves;
  const int64_t s1 = (w + 1) * nstatic / waves;
  const uint32_t nch = (uint32_t)((n - nstatic) / chunk);
  const int per = tile_bytes / 1024;
  uint32_t pend = 0;
  bool claimed = false, more = true;
  // The next span of entries: up to 64 of the static share (never leaving fewer than
  // U behind), else the chunk of the pending claim.  Lanes hold the span's offsets.
  auto next_span = [&](int64_t& o, int& len) {
    int64_t base = 0;
    int cnt = 0;
    if (sp < s1) {
      const int64_t rem = s1 - sp;
      cnt = rem <= 64 ? (int)rem : (rem - 64 < U ? (int)(rem - U) : 64);
      base = sp;
      sp += cnt;
      if (sp >= s1 && !claimed) {   // the share's last span: claim the first chunk
        if (lane == 0) pend = atomicAdd(counter, 1u);
        claimed = true;
      }
    } else if (more) {
      if (!claimed) {
        if (lane == 0) pend = atomicAdd(counter, 1u);
        claimed = true;
      }
      const uint32_t c = __builtin_amdgcn_readfirstlane(pend);
      if (c < nch) {
        base = nstatic + (int64_t)c * chunk;
        cnt = chunk;
        if (lane == 0) pend = atomicAdd(counter, 1u);
      } else {
        more = false;
        if (c == nch + (uint32_t)waves - 1 && lane == 0) atomicExch(counter, 0u);
      }
    }
    o = lane < cnt ? off[base + lane] : 0;
    len = cnt;
  };
  uint32_t acc = 0;
  u32x4 kv[U][2][4];
  auto issue = [&](u32x4 (&t)[2][4], int64_t o) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t b = o + (int64_t)c * 1024 + lane * 16;
      t[0][c] = c < per ? __builtin_nontemporal_load((const u32x4*)(k + b)) : u32x4{0, 0, 0, 0};
      t[1][c] = c < per ? __builtin_nontemporal_load((const u32x4*)(v + b)) : u32x4{0, 0, 0, 0};
    }
  };
  auto consume = [&](const u32x4 (&t)[2][4]) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc ^= fold(t[0][c]) ^ fold(t[1][c]);
  };
  int64_t co, no;
  int cl, nl;
  next_span(co, cl);
  next_span(no, nl);
  int64_t vb = 0;   // stream index of the current span's first entry
  auto off_at = [&](int64_t j) -> int64_t {
    const int l = (int)(j - vb);
    const int64_t x = l < cl ? co : no;
    const int ll = l < cl ? l : l - cl;
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, ll);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)x >> 32), ll);
    return (int64_t)(((uint64_t)hi << 32) | lo);
  };
#pragma unroll
  for (int u = 0; u < U - 1; ++u)
    if (u < cl + nl) issue(kv[u], off_at(u));
  bool done = cl == 0;
  int64_t j = 0;
  while (!done) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (!done) {
        const int64_t ji = j + u + U - 1;
        if (ji < vb + cl + nl) issue(kv[(u + U - 1) % U], off_at(ji));
        consume(kv[u]);
        if (j + u + 1 == vb + cl) {   // the current span is consumed: move on
          vb += cl;
          co = no;
          cl = nl;
          if (cl == 0) done = true; else next_span(no, nl);
        }
      }
    }
    j += U;
  }
  // Here every wave has made exactly one claim past the last chunk (next_span
  // returns an empty span only then).
  if (acc == kSentinel) sink[blockIdx.x] = acc;
}

template <int U>
int launch_stream(const void* buf, uint64_t n16, uint32_t* sink, int blocks, int threads, hipStream_t st) {
  hipLaunchKernelGGL((stream_read_kernel<U>), dim3(blocks), dim3(threads), 0, st, (const u32x4*)buf, n16, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

template <int U>
int launch_gather(const void* k, const void* v, const int64_t* off, int64_t n, int tile_bytes, uint32_t* sink,
                  int blocks, int threads, hipStream_t st) {
  hipLaunchKernelGGL((tile_gather_kernel<U>), dim3(blocks), dim3(threads), 0, st, (const char*)k, (const char*)v,
                     off, n, tile_bytes, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

bool shape_ok(int blocks, int threads) {
  // at most 512 threads: each wave may then use up to 256 registers (the rings)
  return blocks >= 1 && blocks <= (1 << 20) && threads >= 64 && threads <= 512 && threads % 64 == 0;
}

}  // namespace

extern "C" {

int hbm_probe_stream_read(const void* buf, uint64_t bytes, uint32_t* sink, int blocks, int threads, int unroll,
                          void* stream) {
  if (!buf || !sink || bytes % 16 || !shape_ok(blocks, threads)) return -1;
  const hipStream_t st = (hipStream_t)stream;
  const uint64_t n16 = bytes / 16;
  switch (unroll) {
    case 1: return launch_stream<1>(buf, n16, sink, blocks, threads, st);
    case 2: return launch_stream<2>(buf, n16, sink, blocks, threads, st);
    case 4: return launch_stream<4>(buf, n16, sink, blocks, threads, st);
    case 8: return launch_stream<8>(buf, n16, sink, blocks, threads, st);
    case 16: return launch_stream<16>(buf, n16, sink, blocks, threads, st);
  }
  return -1;
}

int hbm_probe_tile_gather(const void* k_pool, const void* v_pool, const int64_t* tile_offsets, int64_t ntiles,
                          int tile_bytes, uint32_t* sink, int blocks, int threads, int depth, void* stream) {
  if (!k_pool || !v_pool || !sink || ntiles < 0 || (ntiles > 0 && !tile_offsets)) return -1;
  if (tile_bytes < 1024 || tile_bytes > 4096 || tile_bytes % 1024 || !shape_ok(blocks, threads)) return -1;
  const hipStream_t st = (hipStream_t)stream;
  switch (depth) {
    case 1: return launch_gather<1>(k_pool, v_pool, tile_offsets, ntiles, tile_bytes, sink, blocks, threads, st);
    case 2: return launch_gather<2>(k_pool, v_pool, tile_offsets, ntiles, tile_bytes, sink, blocks, threads, st);
    case 3: return launch_gather<3>(k_pool, v_pool, tile_offsets, ntiles, tile_bytes, sink, blocks, threads, st);
    case 4: return launch_gather<4>(k_pool, v_pool, tile_offsets, ntiles, tile_bytes, sink, blocks, threads, st);
  }
  return -1;
}

int hbm_probe_tile_gather_balanced(const void* k_pool, const void* v_pool, const int64_t* tile_offsets, int64_t ntiles,
                                   int64_t nstatic, int chunk, uint32_t* counter, int tile_bytes, uint32_t* sink,
                                   int blocks, int threads, int depth, void* stream) {
  if (!k_pool || !v_pool || !sink || !counter || ntiles < 0 || (ntiles > 0 && !tile_offsets)) return -1;
  if (tile_bytes < 1024 || tile_bytes > 4096 || tile_bytes % 1024 || !shape_ok(blocks, threads)) return -1;
  if (depth < 2 || depth > 4 || chunk < depth || chunk > 64) return -1;
  if (nstatic < 0 || nstatic > ntiles || (ntiles - nstatic) % chunk) return -1;
  const int64_t waves = (int64_t)blocks * (threads / 64);
  if (nstatic > 0 && nstatic / waves < depth) return -1;
  const hipStream_t st = (hipStream_t)stream;
#define RLDA_BAL(U)                                                                                               \
  hipLaunchKernelGGL((tile_gather_balanced_kernel<U>), dim3(blocks), dim3(threads), 0, st, (const char*)k_pool, \
                     (const char*)v_pool, tile_offsets, ntiles, nstatic, chunk, counter, tile_bytes, sink)
  switch (depth) {
    case 2: RLDA_BAL(2); break;
    case 3: RLDA_BAL(3); break;
    case 4: RLDA_BAL(4); break;
  }
#undef RLDA_BAL
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

}  // extern "C"
