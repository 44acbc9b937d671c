// Host-side launchers of the gfx950 kernels (one translation unit per
// kernel family); called by the C ABI in api.cpp.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gmb {

// Indices of the per-block device size words.
constexpr int kNDst = 0, kNSrc = 1, kNnz = 2;

struct CsrArgs {
  const void* indptr;
  const int32_t* indices;
  int64_t num_nodes;
  int wide;
};

// Device pointers and host-known bounds of one sampling hop.
struct HopArgs {
  int32_t* sizes;        // this block's {n_dst, n_src, nnz, 0}
  int32_t* next_sizes;   // the next hop's size words (nullptr after the last hop)
  int32_t* indptr;       // [cap_dst + 1]
  int32_t* nbr;          // [cap_nnz]
  int32_t* local;        // [cap_nnz]
  uint64_t* count_tiles; // look-back words of the degree scan
  uint32_t* count_ticket;
  uint64_t* flag_tiles;  // look-back words of the new-vertex scan
  uint32_t* flag_ticket;
  int64_t cap_dst, cap_nnz, cap_src;
  int fanout;
  int layer;
};

constexpr int kScanBlock = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanBlock * kScanItems;

inline int64_t scan_tiles(int64_t n) { return n <= 0 ? 1 : (n + kScanTile - 1) / kScanTile; }

// sample.hip
hipError_t launch_state_init(uint32_t* table, uint32_t* status, int64_t num_nodes, hipStream_t s);
hipError_t launch_prep(const int32_t* seeds, int32_t num_seeds, int32_t* ids, uint32_t* table,
                       int64_t num_nodes, uint32_t* status, uint64_t* zero_words, int64_t num_zero,
                       int32_t* all_sizes, int32_t num_size_words, int32_t first_ndst_word,
                       hipStream_t s);
hipError_t launch_count_scan(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* status,
                             hipStream_t s);
hipError_t launch_sample(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* table,
                         uint32_t* status, uint32_t k0, uint32_t k1, hipStream_t s);
hipError_t launch_assign(const HopArgs& h, int32_t* ids, uint32_t* table, int64_t num_nodes,
                         hipStream_t s);
hipError_t launch_local(const HopArgs* hops, int num_hops, const int32_t* ids, int32_t num_seeds,
                        const uint32_t* table, int64_t num_nodes, uint32_t* status, hipStream_t s);
hipError_t launch_cleanup(const int32_t* ids, const int32_t* final_sizes, int64_t cap_src,
                          uint32_t* table, int64_t num_nodes, hipStream_t s);

// gather.hip
hipError_t launch_gather(const int32_t* ids, const int32_t* n_dev, int64_t n_cap, const void* feats,
                         int64_t num_nodes, int64_t row_bytes, void* out, uint32_t* status,
                         hipStream_t s);

// sage.hip
hipError_t launch_mean_aggregate(const int32_t* sizes, const int32_t* indptr, const int32_t* local,
                                 const void* h, int d, int bf16, void* agg, int64_t cap_dst,
                                 hipStream_t s);
hipError_t launch_sage_linear(const int32_t* sizes, const void* h_self, const void* agg,
                              const void* w_self, const void* w_neigh, const float* bias, int d_in,
                              int d_out, int bf16, int relu, int out_f32, void* out,
                              int64_t cap_rows, hipStream_t s);

}  // namespace gmb
