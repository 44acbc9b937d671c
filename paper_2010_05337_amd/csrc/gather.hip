// Feature-row gather on gfx950: out[i, :] = feats[ids[i], :] (the trainer's
// pull of the mini-batch's vertex features from the key-value store,
// DistDGL Section III-C, here a local copy in HBM).
//
// A group of G lanes copies one row with the widest access the row's
// alignment allows (16-byte loads for 400-byte fp32x100 and 256-byte
// bf16x128 rows); every group keeps U rows in flight before it stores, so
// each wave has U independent row reads outstanding.
#include "common.hpp"
#include "kernels.hpp"

#ifndef GMB_GATHER_MAX_BLOCKS
#define GMB_GATHER_MAX_BLOCKS 8192
#endif

namespace gmb {

namespace {

template <typename V>
__device__ __forceinline__ void opaque_vec(V& x) {
  static_assert(sizeof(V) % 4 == 0 || sizeof(V) == 2, "element size");
  if constexpr (sizeof(V) == 16) {
    asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
  } else if constexpr (sizeof(V) == 8) {
    asm volatile("" : "+v"(x.x), "+v"(x.y));
  } else {
    asm volatile("" : "+v"(x));
  }
}

// Every load is unconditional from a clamped address (row 0 for a lane
// without a row, an out-of-range id reads row 0 and is zeroed after the
// whole batch has been issued): a load under a divergent branch makes the
// compiler drain every outstanding load before the next one.
template <typename V, int G, int U>
__global__ __launch_bounds__(256) void k_gather(const int32_t* __restrict__ ids, const int32_t* n_dev,
                                                int64_t n_cap, const V* __restrict__ feats,
                                                int64_t num_nodes, int cpr, V* __restrict__ out,
                                                uint32_t* status) {
  int64_t n = n_cap;
  if (n_dev) {
    const int32_t m = load_size(n_dev);
    n = m < 0 ? 0 : (m < n_cap ? m : n_cap);
  }
  constexpr int kGroups = 256 / G;
  const int lane = threadIdx.x & (G - 1);
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kGroups;
  bool bad = false;
  for (int64_t row = static_cast<int64_t>(blockIdx.x) * kGroups + threadIdx.x / G; row < n;
       row += stride * U) {
    int32_t id[U];
    bool in[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t r = row + u * stride;
      id[u] = ids[r < n ? r : 0];
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t r = row + u * stride;
      const bool ok = valid_vertex(id[u], num_nodes);
      bad |= (r < n) & !ok;
      in[u] = (r < n) & ok;
      id[u] = in[u] ? id[u] : 0;
    }
    for (int c = lane; c < cpr; c += G) {
      V val[U];
#pragma unroll
      for (int u = 0; u < U; ++u) val[u] = feats[static_cast<int64_t>(id[u]) * cpr + c];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        opaque_vec(val[u]);
        const int64_t r = row + u * stride;
        if (r < n) out[r * cpr + c] = in[u] ? val[u] : V{};
      }
    }
  }
  if (bad) raise_status(status, GMB_STATUS_ERANGE);
}

template <typename V>
hipError_t dispatch(const int32_t* ids, const int32_t* n_dev, int64_t n_cap, const void* feats,
                    int64_t num_nodes, int cpr, void* out, uint32_t* status, hipStream_t s) {
  constexpr int U = 4;
  int G = 64;
  if (cpr <= 4) G = 4;
  else if (cpr <= 8) G = 8;
  else if (cpr <= 16) G = 16;
  else if (cpr <= 32) G = 32;
  const int64_t rows_per_block = (256 / G) * U;
  int64_t blocks = (n_cap + rows_per_block - 1) / rows_per_block;
  if (blocks > GMB_GATHER_MAX_BLOCKS) blocks = GMB_GATHER_MAX_BLOCKS;
  if (blocks < 1) blocks = 1;
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  const V* f = static_cast<const V*>(feats);
  V* o = static_cast<V*>(out);
  switch (G) {
    case 4: hipLaunchKernelGGL((k_gather<V, 4, U>), grid, block, 0, s, ids, n_dev, n_cap, f, num_nodes, cpr, o, status); break;
    case 8: hipLaunchKernelGGL((k_gather<V, 8, U>), grid, block, 0, s, ids, n_dev, n_cap, f, num_nodes, cpr, o, status); break;
    case 16: hipLaunchKernelGGL((k_gather<V, 16, U>), grid, block, 0, s, ids, n_dev, n_cap, f, num_nodes, cpr, o, status); break;
    case 32: hipLaunchKernelGGL((k_gather<V, 32, U>), grid, block, 0, s, ids, n_dev, n_cap, f, num_nodes, cpr, o, status); break;
    default: hipLaunchKernelGGL((k_gather<V, 64, U>), grid, block, 0, s, ids, n_dev, n_cap, f, num_nodes, cpr, o, status); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gather(const int32_t* ids, const int32_t* n_dev, int64_t n_cap, const void* feats,
                         int64_t num_nodes, int64_t row_bytes, void* out, uint32_t* status,
                         hipStream_t s) {
  const uintptr_t align = reinterpret_cast<uintptr_t>(feats) | reinterpret_cast<uintptr_t>(out);
  if (row_bytes % 16 == 0 && align % 16 == 0)
    return dispatch<uint4>(ids, n_dev, n_cap, feats, num_nodes, static_cast<int>(row_bytes / 16), out, status, s);
  if (row_bytes % 8 == 0 && align % 8 == 0)
    return dispatch<uint2>(ids, n_dev, n_cap, feats, num_nodes, static_cast<int>(row_bytes / 8), out, status, s);
  if (row_bytes % 4 == 0 && align % 4 == 0)
    return dispatch<uint32_t>(ids, n_dev, n_cap, feats, num_nodes, static_cast<int>(row_bytes / 4), out, status, s);
  return dispatch<uint16_t>(ids, n_dev, n_cap, feats, num_nodes, static_cast<int>(row_bytes / 2), out, status, s);
}

}  // namespace gmb
