// Block-wide and single-pass device-wide exclusive scans (device side).
//
// The device-wide scan is a decoupled look-back scan (Merrill & Garland,
// "Single-pass parallel prefix scan with decoupled look-back", NVIDIA
// technical report NVR-2016-002): every tile publishes its aggregate at
// once, then walks back over its predecessors until it meets one that has
// published an inclusive prefix.  Tiles are numbered in the order in which
// workgroups start (an atomic ticket), so a tile only ever waits on tiles
// that are already running, and every tile publishes its aggregate before
// it waits: every wait ends.  The wait is still bounded (kLookbackSpins
// sleeps); a tile that runs out reports it, publishes a wrong prefix (so
// its successors still finish) and goes on.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gmb {

constexpr uint64_t kTileAggregate = 1ull << 62;
constexpr uint64_t kTilePrefix = 2ull << 62;
constexpr int kLookbackSpins = 1 << 22;

__device__ __forceinline__ int32_t wave_inclusive_scan(int32_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

__device__ __forceinline__ void publish_tile(uint64_t* tiles, int tile, uint64_t word) {
  __hip_atomic_store(&tiles[tile], word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive scans of NV values per thread over a block of BLOCK threads;
// `smem` holds NV * BLOCK/64 ints.  Every thread of the block must call it.
template <int BLOCK, int NV>
__device__ __forceinline__ void block_exclusive_scan_multi(const int32_t (&x)[NV], int32_t (&excl)[NV],
                                                           int32_t (&total)[NV], int32_t* smem) {
  constexpr int W = BLOCK / 64;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int32_t inc[NV];
#pragma unroll
  for (int a = 0; a < NV; ++a) inc[a] = wave_inclusive_scan(x[a]);
  if (lane == 63) {
#pragma unroll
    for (int a = 0; a < NV; ++a) smem[a * W + wave] = inc[a];
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < NV; ++a) {
    int32_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const int32_t s = smem[a * W + w];
      before += (w < wave) ? s : 0;
      all += s;
    }
    excl[a] = before + inc[a] - x[a];
    total[a] = all;
  }
  __syncthreads();
}

// Decoupled look-back over NV independent scans at once (array a of the
// look-back words starts at tiles + a * stride).  Called by the whole first
// wave of a tile.  Publishes the tile's aggregates, resolves the exclusive
// prefixes from the predecessors 64 at a time (lane i reads tile - 1 - i; a
// predecessor that has published nothing yet is re-read until it has),
// publishes the inclusive prefixes and returns the exclusive ones to every
// lane.  Values are non-negative and below 2^31.  Returns false if the wait
// ran out.
template <int NV>
__device__ bool tile_lookback_multi(uint64_t* tiles, int64_t stride, int tile,
                                    const int32_t (&aggregate)[NV], int32_t (&exclusive)[NV]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int a = 0; a < NV; ++a) exclusive[a] = 0;
  if (tile == 0) {
    if (lane == 0) {
#pragma unroll
      for (int a = 0; a < NV; ++a)
        publish_tile(tiles + a * stride, 0, kTilePrefix | static_cast<uint32_t>(aggregate[a]));
    }
    return true;
  }
  if (lane == 0) {
#pragma unroll
    for (int a = 0; a < NV; ++a)
      publish_tile(tiles + a * stride, tile, kTileAggregate | static_cast<uint32_t>(aggregate[a]));
  }
  bool done[NV];
#pragma unroll
  for (int a = 0; a < NV; ++a) done[a] = false;
  int spins = 0;
  bool ok = true;
  for (int base = tile - 1; ok; base -= 64) {
    const int t = base - lane;
    uint64_t w[NV];
#pragma unroll
    for (int a = 0; a < NV; ++a)
      w[a] = t >= 0 ? __hip_atomic_load(&tiles[a * stride + t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                    : kTilePrefix;

    for (;;) {
      bool pending = false;
#pragma unroll
      for (int a = 0; a < NV; ++a) pending |= !done[a] && (w[a] >> 62) == 0;
      if (!__any(pending)) break;
      if (++spins > kLookbackSpins) {
        ok = false;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      // re-read the whole window of every open scan (a word only ever moves
      // from nothing to aggregate to prefix, so re-reading is harmless)
#pragma unroll
      for (int a = 0; a < NV; ++a)
        if (!done[a] && t >= 0)
          w[a] = __hip_atomic_load(&tiles[a * stride + t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (!ok) break;
    bool all_done = true;
#pragma unroll
    for (int a = 0; a < NV; ++a) {
      if (done[a]) continue;
      const uint64_t prefixes = __ballot((w[a] >> 62) == 2);
      // lanes up to and including the nearest published prefix contribute
      const int stop = prefixes ? __ffsll(static_cast<long long>(prefixes)) - 1 : 63;
      int32_t v = lane <= stop ? static_cast<int32_t>(static_cast<uint32_t>(w[a])) : 0;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
      exclusive[a] += v;
      if (prefixes) done[a] = true;
      else all_done = false;
    }
    if (all_done) break;
  }
  if (lane == 0) {
#pragma unroll
    for (int a = 0; a < NV; ++a)
      publish_tile(tiles + a * stride, tile, kTilePrefix | static_cast<uint32_t>(exclusive[a] + aggregate[a]));
  }
  return ok;
}

// Claims the next tile number for this workgroup (thread 0 takes a ticket,
// the block reads it from LDS).
__device__ __forceinline__ int claim_tile(uint32_t* counter, int* s_tile) {
  if (threadIdx.x == 0) *s_tile = static_cast<int>(atomicAdd(counter, 1u));
  __syncthreads();
  return *s_tile;
}

}  // namespace gmb
