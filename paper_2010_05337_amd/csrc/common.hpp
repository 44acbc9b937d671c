// Shared device helpers of the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gmb.h"
#include "kernels.hpp"

namespace gmb {

constexpr int kWave = 64;

// Dedup-table encoding (one uint32 per vertex):
//   kEmpty             vertex not seen in this call
//   < kEdgeTag         the vertex's local id (its position in src_ids)
//   kEdgeTag | e       the vertex is new in the current hop and e is the
//                      smallest edge position that sampled it
constexpr uint32_t kEmpty = 0xFFFFFFFFu;
constexpr uint32_t kEdgeTag = 0x80000000u;

struct CsrView {
  const void* indptr;
  const int32_t* indices;
  int64_t num_nodes;
  int wide;   // 1: int64 row offsets
};

__device__ __forceinline__ void row_range(const CsrView& g, int32_t v, int64_t& begin, int64_t& end) {
  if (g.wide) {
    const int64_t* p = static_cast<const int64_t*>(g.indptr);
    begin = p[v];
    end = p[v + 1];
  } else {
    const int32_t* p = static_cast<const int32_t*>(g.indptr);
    begin = p[v];
    end = p[v + 1];
  }
}

// The same with the row-offset width known at compile time (no branch
// between the reads of a batch).
template <bool WIDE>
__device__ __forceinline__ void row_range_t(const CsrView& g, int32_t v, int64_t& begin, int64_t& end) {
  if constexpr (WIDE) {
    const int64_t* p = static_cast<const int64_t*>(g.indptr);
    begin = p[v];
    end = p[v + 1];
  } else {
    const int32_t* p = static_cast<const int32_t*>(g.indptr);
    begin = p[v];
    end = p[v + 1];
  }
}

__device__ __forceinline__ bool valid_vertex(int32_t v, int64_t n) {
  return v >= 0 && static_cast<int64_t>(v) < n;
}

__device__ __forceinline__ void raise_status(uint32_t* status, uint32_t bit) {
  if (status) atomicOr(status, bit);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ int32_t load_size(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace gmb
