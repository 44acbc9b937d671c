// Host-side launchers of the gfx950 kernels (one translation unit per
// kernel family); called by the C ABI in api.cpp.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gmb.h"

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
  int32_t* indptr;       // [cap_dst + 1]
  int32_t* nbr;          // [cap_nnz]
  int32_t* local;        // [cap_nnz]
  uint64_t* tiles;       // look-back words of this hop's relabel scan
  uint32_t* ticket;
  int64_t tile_stride;   // words per scanned value (= routers)
  int items;             // relabel scan items per thread
  int64_t cap_dst, cap_nnz, cap_src;
  int fanout;
  int layer;
};

constexpr int kScanBlock = 256;
// Items per thread of a relabel tile (kScanBlock threads): 2, 4, 8 or 16.
// Small hops take small tiles so that their random reads spread over many
// CUs; large hops take large tiles, which cuts tickets and look-back.
inline int64_t scan_tiles(int64_t n, int items) {
  const int64_t tile = static_cast<int64_t>(kScanBlock) * items;
  return n <= 0 ? 1 : (n + tile - 1) / tile;
}
inline int scan_items_for(int64_t cap_nnz) {
  for (int items = 16; items > 2; items /= 2)
    if (scan_tiles(cap_nnz, items) >= 128) return items;
  return 2;
}

// Local ids that a hop's relabel left deferred (entries -(e0 + 1): copy the
// local id of edge e0); the next kernel on the stream resolves them.  The
// edge count is sizes[kNnz]; cap (>= 1) bounds it and every read of local.
// Nothing to resolve: any local array of cap entries and an edge count of 0.
struct DeferredArgs {
  int32_t* local;
  const int32_t* sizes;
  int64_t cap;
};

// Relabel arguments of a table hop `hop` (k_assign).  Value v >= 1 of its
// scan belongs to hop hop + v: indptr[v], fanout[v].
struct AssignArgs {
  const int32_t* nbr;
  int32_t* local;
  int32_t* sizes;
  int32_t* next_sizes;   // nullptr after the last hop
  uint64_t* tiles;
  int64_t tile_stride;
  uint32_t* ticket;
  int32_t* totals;
  int hop;
  int32_t* indptr[GMB_MAX_LAYERS];
  int32_t fanout[GMB_MAX_LAYERS];
};

// Dedup by owners (sample.hip): a router takes `span` destinations, whose
// edges fit one relabel tile (span * fanout <= kScanBlock * items), and
// routes them with the destinations themselves (at most kMaxRouteEntries
// pairs); an owner's LDS hash table has kOwnerSlots slots.
constexpr int kMaxRouters = 2048;
constexpr int kMaxOwners = 4096;
constexpr int kMaxRouteEntries = 8192;
constexpr int kMaxSpan = 1024;
constexpr int kOwnerSlots = 8192;
// pairs per owner the plan aims at, at full capacity (half the table)
constexpr int64_t kOwnerPairs = 4096;
// compute units of the MI355X (gfx950); an owner's LDS table takes most of
// a CU's LDS, so one owner workgroup runs per CU at a time
constexpr int kComputeUnits = 256;

// Sampling arguments of one hop (fan-out f, model layer `layer`); the
// first hop also checks the seeds (check_seeds).  fix: the previous hop's
// deferred local ids, resolved by the same grid.
struct SampleArgs {
  const int32_t* ids;
  const int32_t* sizes;
  const int32_t* indptr;   // the hop's block row offsets
  int32_t* nbr;
  uint32_t* status;
  int fanout, layer;
  uint32_t k0, k1;
  int check_seeds;
  DeferredArgs fix;
};

// Router arguments of one hop (k_route).
struct RouteArgs {
  const int32_t* sizes;    // the hop's size words (n_dst)
  const int32_t* indptr;   // the hop's block row offsets [n_dst + 1]
  const int32_t* ids;      // the destinations: ids[0 .. n_dst)
  const int32_t* nbr;      // the hop's sampled vertices [nnz]
  uint2* pairs;            // [cap_dst + cap_nnz] (key, value)
  int32_t* off;            // [(owners + 1) * routers], owner-major
  int32_t* rs;             // [routers] region start of each router
  int64_t num_nodes;
  int32_t span, routers, owners;
};

// Owner arguments of one hop (k_owner).
struct OwnerArgs {
  const uint2* pairs;
  const int32_t* off;
  const int32_t* rs;
  int32_t* res;            // [cap_dst + cap_nnz] answers, at the pairs' positions
  uint32_t* table;         // the state's per-vertex table (overflow only)
  uint32_t* status;
  int32_t routers, owners;
  int32_t max_slots;       // LDS table size limit, a power of two in 64 .. kOwnerSlots
};

// Relabel arguments of hop `hop` (k_rank).  Value v >= 1 of its scan
// belongs to hop hop + v: indptr[v], fanout[v].
struct RankArgs {
  const uint2* pairs;
  const int32_t* res;
  const int32_t* indptr0;  // this hop's block row offsets (router ranges)
  int32_t* local;
  int32_t* sizes;
  int32_t* next_sizes;     // nullptr after the last hop
  uint64_t* tiles;
  int64_t tile_stride;
  uint32_t* ticket;
  int32_t* totals;
  int hop;
  int32_t span;
  int32_t* indptr[GMB_MAX_LAYERS];
  int32_t fanout[GMB_MAX_LAYERS];
};

// Arguments of the seed kernel (segment 0: the seeds).  Per hop v:
// indptr[v] its block row offsets, fanout[v] its fan-out.  totals[v] is
// hop v's edge count over the segments placed so far (GMB_MAX_LAYERS
// words after the size words, cleared with them).
struct SeedArgs {
  const int32_t* seeds;
  int32_t num_seeds;
  int32_t first_sizes;   // offset of hop 0's size words in `sizes`
  int32_t* ids;
  uint64_t* zero;
  int64_t num_zero;
  int32_t* sizes;        // every size word, then the totals
  int32_t num_size_words;
  int32_t* totals;
  int32_t* indptr[GMB_MAX_LAYERS];
  int32_t fanout[GMB_MAX_LAYERS];
};

// One block's arrays and bounds, for the consistency check (k_validate).
struct ValidateArgs {
  const int32_t* indptr;
  const int32_t* local;
  const int32_t* nbr;
  const int32_t* ids;
  const int32_t* sizes;
  int64_t cap_dst, cap_src, cap_nnz;
  int fanout;
};

// sample.hip
hipError_t launch_state_init(uint32_t* table, uint32_t* status, int64_t num_nodes, hipStream_t s);
hipError_t launch_seed_scan(const SeedArgs& a, int num_values, const CsrArgs& g, hipStream_t s);
// Table hops (fan-outs up to 64): sampling with the first-edge atomics on
// the state's table, then the relabel scan.
hipError_t launch_sample_table(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* table,
                               uint32_t* status, uint32_t k0, uint32_t k1, int first_hop, const DeferredArgs& fix,
                               hipStream_t s);
hipError_t launch_assign(const AssignArgs& a, int num_values, const CsrArgs& g, int64_t cap_nnz, int items,
                         int32_t* ids, uint32_t* table, uint32_t* status, hipStream_t s);
// Owner hops with fan-outs above 64: sampling alone (then launch_route).
hipError_t launch_sample(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* status, uint32_t k0,
                         uint32_t k1, int first_hop, const DeferredArgs& fix, hipStream_t s);
hipError_t launch_route(const RouteArgs& a, hipStream_t s);
// Sampling and routing in one launch (fan-outs up to 64); otherwise
// launch_sample then launch_route.
hipError_t launch_sample_route(const CsrArgs& g, const SampleArgs& sa, const RouteArgs& ra, hipStream_t s);
hipError_t launch_owner(const OwnerArgs& a, hipStream_t s);
hipError_t launch_rank(const RankArgs& a, int num_values, const CsrArgs& g, int routers, int items, int32_t* ids,
                       uint32_t* status, hipStream_t s);
// The last hop's deferred local ids; with clear_sizes, also the table
// slots of ids[0 .. clear_sizes[kNSrc]) (the vertices the table hops
// recorded) back to empty.
// Checks one block's invariants (sizes within the capacities, row offsets
// from 0 to nnz with at most `fanout` edges per row, every local id below
// n_src and naming the edge's sampled vertex, every sampled vertex in the
// graph) and sets GMB_STATUS_INVALID in *status on a violation.
hipError_t launch_validate(const ValidateArgs& b, int64_t num_nodes, uint32_t* status, hipStream_t s);
hipError_t launch_fix(const DeferredArgs& fix, const int32_t* ids, const int32_t* clear_sizes, int64_t clear_cap,
                      uint32_t* table, int64_t num_nodes, hipStream_t s);

// gather.hip
hipError_t launch_gather(const int32_t* ids, const int32_t* n_dev, int64_t n_cap, const void* feats,
                         int64_t num_nodes, int64_t row_bytes, void* out, uint32_t* status,
                         hipStream_t s);

// sage.hip.  The mean reads rows H[ids[e]] with ids in [0, max_id)
// (others are read as row 0).
hipError_t launch_mean_aggregate(const int32_t* sizes, const int32_t* indptr, const int32_t* local,
                                 const void* h, int d, int bf16, void* agg, int64_t cap_dst,
                                 int fanout, int64_t max_id, hipStream_t s);
hipError_t launch_sage_linear(const int32_t* sizes, const void* h_self, const void* agg,
                              const void* w_self, const void* w_neigh, const float* bias, int d_in,
                              int d_out, int bf16, int relu, int out_f32, void* out,
                              int64_t cap_rows, hipStream_t s);

// sage_bwd.hip: the training step
struct SgdArgs {
  int count;
  float* w[3 * GMB_MAX_LAYERS];
  const float* g[3 * GMB_MAX_LAYERS];
  int64_t n[3 * GMB_MAX_LAYERS];
  // after the update, optionally: the new value rounded to bf16 (RNE) into
  // lo[t], and/or copied into mirror[t] (the bf16 model's matrices and
  // biases, kept beside fp32 master weights)
  uint16_t* lo[3 * GMB_MAX_LAYERS];
  float* mirror[3 * GMB_MAX_LAYERS];
};

// bf16 -> fp32 copies for the training step of a bf16 model: segment t is
// rows x cols elements, rows = *rows_dev[t] clamped to cap_rows[t] when
// rows_dev[t] is given, else cap_rows[t].
constexpr int kMaxWiden = 4 * GMB_MAX_LAYERS + 2;
struct WidenArgs {
  int count;
  const uint16_t* src[kMaxWiden];
  float* dst[kMaxWiden];
  const int32_t* rows_dev[kMaxWiden];
  int64_t cap_rows[kMaxWiden];
  int64_t cols[kMaxWiden];
};
hipError_t launch_xent(const float* logits, const int32_t* labels, int n, int C, int ldz, float* dz,
                       float* loss_rows, int32_t* clear, int64_t clear_n, hipStream_t s);
int wgrad_ldp(int d_out);
int wgrad_parts(int64_t cap_rows, int d_in, int d_out);
// The weight gradient's second step: the partial tiles summed into the
// gradients in a fixed order, `blocks` workgroups (the last one sums the
// loss terms loss_rows[0 .. n_loss) into *loss when loss is not NULL).
struct ReduceArgs {
  const float* partial;
  int parts, d_in, d_out, ldp;
  float* d_self;
  float* d_neigh;
  float* d_bias;
  const float* loss_rows;
  int n_loss;
  float* loss;
  int blocks;
};
// The weight gradient's products: a parts x ytiles x ztiles grid of
// workgroups writing partial tiles (vec: 16-byte loads of H and M).
struct WgradArgs {
  const int32_t* sizes;
  const float* H;
  const float* M;
  int d_in;
  const float* dZ;
  int ldz, ldp;
  float* partial;
  int parts, ytiles, ztiles;
  int vec;
};
// Launches the weight gradient's products and its reduction, or, for
// `defer` and `fold` when given, describes them instead, for later launches
// to run as extra workgroups of their grids (launch_mean_backward: the
// products beside the transpose scan, the reduction beside the fill).
hipError_t launch_wgrad(const int32_t* sizes, const float* H, const float* M, int d_in, const float* dZ, int ldz,
                        int d_out, int64_t cap_rows, float* partial, float* d_self, float* d_neigh,
                        float* d_bias, const float* loss_rows, int n_loss, float* loss, WgradArgs* defer,
                        ReduceArgs* fold, hipStream_t s);
hipError_t launch_dgrad(const int32_t* sizes, const float* dZ, int ldz, int d_out, const float* ws,
                        const float* wn, int d_in, float* dH, float* dM, int64_t cap_rows,
                        const int32_t* indptr, const int32_t* local, int64_t cap_nnz, int32_t fanout, int32_t* cnt,
                        hipStream_t s);
// look-back tiles of the transpose scan over cap_src sources; its state
// (the tile ticket, the long-row count, then 2 words per tile) must start
// zeroed; long_rows holds cap_src ints
int64_t csc_scan_tiles(int64_t cap_src);
// With table != NULL the pull applies table[ids[u]] -= lr * g instead of
// writing the masked gradient into dH (out unused).
// With `defer` (from launch_wgrad) the transpose scan's grid also runs the
// weight gradient's products, with `fold` the fill's grid its reduction.
hipError_t launch_mean_backward(const int32_t* sizes, const int32_t* indptr, const int32_t* local,
                                int64_t cap_nnz, int32_t fanout, const float* dM, const float* out, int d, float* dH,
                                int64_t cap_dst, int64_t cap_src, int32_t* cnt, int32_t* off, int32_t* pos,
                                uint32_t* scan_state, int2* csc, int32_t* long_rows, float* table, const int32_t* ids,
                                int64_t num_nodes, float lr, const WgradArgs* defer, const ReduceArgs* fold,
                                hipStream_t s);
hipError_t launch_sgd(const SgdArgs& a, float lr, hipStream_t s);
hipError_t launch_widen(const WidenArgs& a, hipStream_t s);
// every array of `a` (w[t], n[t]; g unused) and *scalar (if not NULL) to 0
hipError_t launch_zero(const SgdArgs& a, float* scalar, hipStream_t s);

}  // namespace gmb
