// Mini-batch construction on gfx950: recursive fan-out neighbour sampling
// with per-hop dedup and relabel into bipartite blocks (DistDGL, Section
// II-B: pick at most K neighbours of every target, repeat once per layer;
// the sampled graph is the mini-batch's computation graph, Fig. 1(b)).
//
// One hop, for destinations dst = ids[0 : n_dst] (device-resident count):
//   k_count_scan  k_p = min(deg(dst[p]), fanout), exclusive scan -> block
//                 row offsets and nnz (single-pass look-back scan)
//   k_sample      Floyd's algorithm per destination, one lane per draw,
//                 Philox-keyed draws; sampled slots sorted by rank; the
//                 sampled global ids are written in slot order and each
//                 vertex's first edge position is recorded by atomicMin in
//                 the dedup table
//   k_assign      scan of the "first occurrence" flags: new vertex number
//                 n_dst + rank, appended to ids and stored in the table
// After the last hop:
//   k_local       every edge's local id = table[global id] (all hops)
//   k_cleanup     table entries of every vertex of the batch back to empty
//
// ids[] is shared by all hops: the sources of a block are its destinations
// followed by its new vertices, which are exactly the next hop's
// destinations, so every hop only appends.  A vertex keeps the same local
// id in every block, and the table maps it to that id for the whole call.
#include "common.hpp"
#include "kernels.hpp"
#include "philox.hpp"
#include "scan.hpp"

namespace gmb {

namespace {

__device__ __forceinline__ CsrView view(const CsrArgs& a) {
  return CsrView{a.indptr, a.indices, a.num_nodes, a.wide};
}

// Items [base, base + 8) of a scan tile.  Full groups are two 16-byte loads
// (base is a multiple of 8 and the arrays are 256-byte aligned); the group
// holding the end of the data reads element-wise, and entries at or past n
// are left as they came (the caller ignores them).
__device__ __forceinline__ void load_items(const int32_t* a, int64_t base, int64_t n,
                                           int32_t (&v)[kScanItems]) {
  static_assert(kScanItems == 8, "two int4 loads per thread");
  if (base + kScanItems <= n) {
    const int4 x = *reinterpret_cast<const int4*>(a + base);
    const int4 y = *reinterpret_cast<const int4*>(a + base + 4);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
  } else {
#pragma unroll
    for (int q = 0; q < kScanItems; ++q) v[q] = base + q < n ? a[base + q] : 0;
  }
}

__global__ __launch_bounds__(256) void k_state_init(uint32_t* table, uint32_t* status, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
    table[i] = kEmpty;
  if (blockIdx.x == 0 && threadIdx.x == 0) *status = 0;
}

// Seeds -> ids[0:B] and their table slots; clears the look-back words and
// the size words.  all_sizes holds 4 words per layer; the first hop is the
// last layer.
__global__ __launch_bounds__(256) void k_prep(const int32_t* seeds, int32_t num_seeds, int32_t* ids,
                                              uint32_t* table, int64_t num_nodes, uint32_t* status,
                                              uint64_t* zero, int64_t num_zero, int32_t* all_sizes,
                                              int32_t num_size_words, int32_t first_ndst_word) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < num_zero) zero[i] = 0;
  if (i < num_size_words) all_sizes[i] = (i == first_ndst_word) ? num_seeds : 0;
  if (i < num_seeds) {
    const int32_t s = seeds[i];
    ids[i] = s;
    if (valid_vertex(s, num_nodes))
      atomicMin(&table[s], static_cast<uint32_t>(i));
    else
      raise_status(status, GMB_STATUS_ERANGE);
  }
}

__global__ __launch_bounds__(kScanBlock) void k_count_scan(CsrArgs ga, const int32_t* ids,
                                                           int32_t* sizes, int32_t* blk_indptr,
                                                           uint64_t* tiles, uint32_t* ticket,
                                                           int fanout, uint32_t* status) {
  __shared__ int s_tile;
  __shared__ int32_t s_excl;
  __shared__ int32_t s_wave[kScanBlock / 64];
  const CsrView g = view(ga);
  const int32_t n = load_size(&sizes[kNDst]);
  const int num_tiles = n <= 0 ? 1 : (n + kScanTile - 1) / kScanTile;
  const int tile = claim_tile(ticket, &s_tile);
  if (tile >= num_tiles) return;

  const int64_t base = static_cast<int64_t>(tile) * kScanTile + threadIdx.x * kScanItems;
  // Eight consecutive ids per thread, then all sixteen row-offset reads at
  // once from clamped vertices.
  int32_t v[kScanItems];
  load_items(ids, base, n, v);
  int64_t rb[kScanItems], re[kScanItems];
  bool bad = false;
#pragma unroll
  for (int q = 0; q < kScanItems; ++q) {
    const bool live = base + q < n;
    const bool ok = valid_vertex(v[q], g.num_nodes);
    bad |= live & !ok;
    v[q] = (live & ok) ? v[q] : -1;
    row_range(g, v[q] < 0 ? 0 : v[q], rb[q], re[q]);
  }
  if (bad) raise_status(status, GMB_STATUS_ERANGE);
  int32_t k[kScanItems];
  int32_t sum = 0;
#pragma unroll
  for (int q = 0; q < kScanItems; ++q) {
    const int64_t d = v[q] < 0 ? 0 : re[q] - rb[q];
    k[q] = static_cast<int32_t>(d < 0 ? 0 : (d < fanout ? d : fanout));
    sum += k[q];
  }
  int32_t total;
  const int32_t thread_excl = block_exclusive_scan<kScanBlock>(sum, total, s_wave);
  if (threadIdx.x < 64) {
    const int32_t ex = tile_lookback_wave(tiles, tile, total);
    if (threadIdx.x == 0) s_excl = ex;
  }
  __syncthreads();
  int32_t run = s_excl + thread_excl;
#pragma unroll
  for (int q = 0; q < kScanItems; ++q) {
    const int64_t p = base + q;
    if (p < n) blk_indptr[p] = run;
    run += k[q];
  }
  if (tile == num_tiles - 1 && threadIdx.x == 0) {
    const int32_t nnz = s_excl + total;
    blk_indptr[n < 0 ? 0 : n] = nnz;
    sizes[kNnz] = nnz;
  }
}

__device__ __forceinline__ void emit_edge(int32_t pos, int32_t u, int32_t* nbr, uint32_t* table,
                                          int64_t num_nodes, uint32_t* status) {
  nbr[pos] = u;
  if (valid_vertex(u, num_nodes)) {
    const uint32_t tag = kEdgeTag | static_cast<uint32_t>(pos);
    // Entries only decrease during the kernel, so a stale read that is
    // already <= tag proves the atomic would not change anything.
    if (table[u] > tag) atomicMin(&table[u], tag);
  } else {
    raise_status(status, GMB_STATUS_ERANGE);
  }
}

// G lanes per destination (G >= fanout, G a power of two <= 64): lane i
// draws t_i uniform in [0, j_i], j_i = d - f + i; Floyd's rule is then
// resolved in draw order with one group-wide vote per step (x_s = t_s
// unless an earlier lane already holds t_s, then x_s = j_s), and every lane
// finds the rank of its slot among the group's.
template <int G>
__global__ __launch_bounds__(256) void k_sample(CsrArgs ga, const int32_t* ids, const int32_t* sizes,
                                                const int32_t* blk_indptr, int32_t* nbr,
                                                uint32_t* table, uint32_t* status, int fanout,
                                                int layer, uint32_t k0, uint32_t k1) {
  const CsrView g = view(ga);
  const int64_t p = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / G;
  const int lane = threadIdx.x & (G - 1);
  const int32_t n_dst = load_size(&sizes[kNDst]);
  if (p >= n_dst) return;
  const int32_t v = ids[p];
  if (!valid_vertex(v, g.num_nodes)) return;   // the degree scan gave it k = 0
  int64_t begin, end;
  row_range(g, v, begin, end);
  const int64_t d = end - begin;
  const int32_t off = blk_indptr[p];

  int32_t pos = -1, u = 0;
  if (d <= fanout) {
    if (lane < d) {
      pos = off + lane;
      u = g.indices[begin + lane];
    }
  } else {
    const uint32_t f = static_cast<uint32_t>(fanout);
    uint32_t j = 0, t = 0;
    if (static_cast<uint32_t>(lane) < f) {
      j = static_cast<uint32_t>(d - fanout) + lane;
      t = draw_below(k0, k1, static_cast<uint32_t>(v), static_cast<uint32_t>(layer), lane, j + 1);
    }
    uint32_t x = t;
    const int group_base = (threadIdx.x & 63) & ~(G - 1);
    const uint64_t group_mask = (G == 64) ? ~0ull : ((1ull << G) - 1);
    for (uint32_t s = 1; s < f; ++s) {
      const uint32_t ts = __shfl(t, s, G);
      const bool hit = static_cast<uint32_t>(lane) < s && x == ts;
      const uint64_t votes = (__ballot(hit) >> group_base) & group_mask;
      if (static_cast<uint32_t>(lane) == s && votes != 0) x = j;
    }
    uint32_t rank = 0;
    for (uint32_t s = 0; s < f; ++s) rank += (__shfl(x, s, G) < x) ? 1u : 0u;
    if (static_cast<uint32_t>(lane) < f) {
      pos = off + static_cast<int32_t>(rank);
      u = g.indices[begin + x];
    }
  }
  if (pos >= 0) emit_edge(pos, u, nbr, table, g.num_nodes, status);
}

// Fan-outs above 64: one thread per destination; the block's output row
// holds the chosen slots while Floyd runs, is sorted in place, then mapped
// to vertex ids.
__global__ __launch_bounds__(256) void k_sample_wide(CsrArgs ga, const int32_t* ids,
                                                     const int32_t* sizes, const int32_t* blk_indptr,
                                                     int32_t* nbr, uint32_t* table, uint32_t* status,
                                                     int fanout, int layer, uint32_t k0, uint32_t k1) {
  const CsrView g = view(ga);
  const int64_t p = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int32_t n_dst = load_size(&sizes[kNDst]);
  if (p >= n_dst) return;
  const int32_t v = ids[p];
  if (!valid_vertex(v, g.num_nodes)) return;
  int64_t begin, end;
  row_range(g, v, begin, end);
  const int64_t d = end - begin;
  const int32_t off = blk_indptr[p];
  if (d <= fanout) {
    for (int64_t s = 0; s < d; ++s) emit_edge(off + static_cast<int32_t>(s), g.indices[begin + s], nbr, table, g.num_nodes, status);
    return;
  }
  const uint32_t f = static_cast<uint32_t>(fanout);
  int32_t* row = nbr + off;
  for (uint32_t i = 0; i < f; ++i) {
    const uint32_t j = static_cast<uint32_t>(d - fanout) + i;
    const uint32_t t = draw_below(k0, k1, static_cast<uint32_t>(v), static_cast<uint32_t>(layer), i, j + 1);
    bool present = false;
    for (uint32_t q = 0; q < i; ++q) present |= (static_cast<uint32_t>(row[q]) == t);
    row[i] = static_cast<int32_t>(present ? j : t);
  }
  for (uint32_t i = 1; i < f; ++i) {
    const int32_t key = row[i];
    int32_t q = static_cast<int32_t>(i) - 1;
    while (q >= 0 && row[q] > key) {
      row[q + 1] = row[q];
      --q;
    }
    row[q + 1] = key;
  }
  for (uint32_t i = 0; i < f; ++i) {
    const int32_t slot = row[i];
    emit_edge(off + static_cast<int32_t>(i), g.indices[begin + slot], nbr, table, g.num_nodes, status);
  }
}

// Edge e is the first occurrence of its vertex u when the table holds
// (tag | e).  Those edges are numbered by a scan; the vertex becomes source
// n_dst + rank of the block, is appended to ids and gets its local id in
// the table.  Other tiles may read table[u] while it is rewritten: they see
// either the tag of another edge or the local id, never their own tag, so
// their flag is 0 either way.
__global__ __launch_bounds__(kScanBlock) void k_assign(const int32_t* nbr, int32_t* sizes,
                                                       int32_t* next_sizes, int32_t* ids,
                                                       uint32_t* table, int64_t num_nodes,
                                                       uint64_t* tiles, uint32_t* ticket) {
  __shared__ int s_tile;
  __shared__ int32_t s_excl;
  __shared__ int32_t s_wave[kScanBlock / 64];
  const int32_t n = load_size(&sizes[kNnz]);
  const int32_t n_dst = load_size(&sizes[kNDst]);
  const int num_tiles = n <= 0 ? 1 : (n + kScanTile - 1) / kScanTile;
  const int tile = claim_tile(ticket, &s_tile);
  if (tile >= num_tiles) return;

  const int64_t base = static_cast<int64_t>(tile) * kScanTile + threadIdx.x * kScanItems;
  int32_t u[kScanItems];
  load_items(nbr, base, n, u);
  uint32_t t[kScanItems];
#pragma unroll
  for (int q = 0; q < kScanItems; ++q) {
    const bool ok = (base + q < n) & valid_vertex(u[q], num_nodes);
    u[q] = ok ? u[q] : -1;
    t[q] = table[u[q] < 0 ? 0 : u[q]];
  }
  uint32_t flags = 0;
  int32_t sum = 0;
#pragma unroll
  for (int q = 0; q < kScanItems; ++q) {
    if (u[q] >= 0 && t[q] == (kEdgeTag | static_cast<uint32_t>(base + q))) {
      flags |= 1u << q;
      ++sum;
    }
  }
  int32_t total;
  const int32_t thread_excl = block_exclusive_scan<kScanBlock>(sum, total, s_wave);
  if (threadIdx.x < 64) {
    const int32_t ex = tile_lookback_wave(tiles, tile, total);
    if (threadIdx.x == 0) s_excl = ex;
  }
  __syncthreads();
  int32_t r = n_dst + s_excl + thread_excl;
#pragma unroll
  for (int q = 0; q < kScanItems; ++q) {
    if (flags & (1u << q)) {
      ids[r] = u[q];
      table[u[q]] = static_cast<uint32_t>(r);
      ++r;
    }
  }
  if (tile == num_tiles - 1 && threadIdx.x == 0) {
    const int32_t n_src = n_dst + s_excl + total;
    sizes[kNSrc] = n_src;
    if (next_sizes) next_sizes[kNDst] = n_src;
  }
}

struct LocalSeg {
  const int32_t* nbr;
  int32_t* local;
  const int32_t* sizes;
  int64_t first_block;
};

struct LocalArgs {
  LocalSeg seg[GMB_MAX_LAYERS];
  int num_seg;
  int64_t seed_first_block;
};

// local[e] = table[nbr[e]] for the edges of every hop; the blocks past the
// edge segments check that each seed owns its table slot (a duplicated
// seed does not).
__global__ __launch_bounds__(256) void k_local(LocalArgs a, const int32_t* ids, int32_t num_seeds,
                                               const uint32_t* table, int64_t num_nodes,
                                               uint32_t* status) {
  const int64_t b = blockIdx.x;
  if (b >= a.seed_first_block) {
    const int64_t p = (b - a.seed_first_block) * blockDim.x + threadIdx.x;
    if (p < num_seeds) {
      const int32_t s = ids[p];
      if (valid_vertex(s, num_nodes) && table[s] != static_cast<uint32_t>(p))
        raise_status(status, GMB_STATUS_EDUP);
    }
    return;
  }
  int k = 0;
  while (k + 1 < a.num_seg && b >= a.seg[k + 1].first_block) ++k;
  const LocalSeg& s = a.seg[k];
  const int64_t e = (b - s.first_block) * blockDim.x + threadIdx.x;
  const int32_t n = load_size(&s.sizes[kNnz]);
  if (e >= n) return;
  const int32_t u = s.nbr[e];
  s.local[e] = valid_vertex(u, num_nodes) ? static_cast<int32_t>(table[u]) : -1;
}

__global__ __launch_bounds__(256) void k_cleanup(const int32_t* ids, const int32_t* final_sizes,
                                                 uint32_t* table, int64_t num_nodes) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int32_t n = load_size(&final_sizes[kNSrc]);
  if (i >= n) return;
  const int32_t u = ids[i];
  if (valid_vertex(u, num_nodes)) table[u] = kEmpty;
}

inline unsigned grid_for(int64_t threads, int block = 256) {
  int64_t g = (threads + block - 1) / block;
  return static_cast<unsigned>(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_state_init(uint32_t* table, uint32_t* status, int64_t num_nodes, hipStream_t s) {
  int64_t blocks = (num_nodes + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_state_init, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, table, status,
                     num_nodes);
  return hipGetLastError();
}

hipError_t launch_prep(const int32_t* seeds, int32_t num_seeds, int32_t* ids, uint32_t* table,
                       int64_t num_nodes, uint32_t* status, uint64_t* zero_words, int64_t num_zero,
                       int32_t* all_sizes, int32_t num_size_words, int32_t first_ndst_word,
                       hipStream_t s) {
  int64_t n = num_zero;
  if (num_seeds > n) n = num_seeds;
  if (num_size_words > n) n = num_size_words;
  hipLaunchKernelGGL(k_prep, dim3(grid_for(n)), dim3(256), 0, s, seeds, num_seeds, ids, table,
                     num_nodes, status, zero_words, num_zero, all_sizes, num_size_words,
                     first_ndst_word);
  return hipGetLastError();
}

hipError_t launch_count_scan(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* status,
                             hipStream_t s) {
  const unsigned grid = static_cast<unsigned>(scan_tiles(h.cap_dst));
  hipLaunchKernelGGL(k_count_scan, dim3(grid), dim3(kScanBlock), 0, s, g, ids, h.sizes, h.indptr,
                     h.count_tiles, h.count_ticket, h.fanout, status);
  return hipGetLastError();
}

hipError_t launch_sample(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* table,
                         uint32_t* status, uint32_t k0, uint32_t k1, hipStream_t s) {
  const int f = h.fanout;
#define GMB_LAUNCH_SAMPLE(G)                                                                       \
  hipLaunchKernelGGL(k_sample<G>, dim3(grid_for(h.cap_dst * (G))), dim3(256), 0, s, g, ids, h.sizes, \
                     h.indptr, h.nbr, table, status, f, h.layer, k0, k1)
  if (f <= 8) GMB_LAUNCH_SAMPLE(8);
  else if (f <= 16) GMB_LAUNCH_SAMPLE(16);
  else if (f <= 32) GMB_LAUNCH_SAMPLE(32);
  else if (f <= 64) GMB_LAUNCH_SAMPLE(64);
  else
    hipLaunchKernelGGL(k_sample_wide, dim3(grid_for(h.cap_dst)), dim3(256), 0, s, g, ids, h.sizes,
                       h.indptr, h.nbr, table, status, f, h.layer, k0, k1);
#undef GMB_LAUNCH_SAMPLE
  return hipGetLastError();
}

hipError_t launch_assign(const HopArgs& h, int32_t* ids, uint32_t* table, int64_t num_nodes,
                         hipStream_t s) {
  const unsigned grid = static_cast<unsigned>(scan_tiles(h.cap_nnz));
  hipLaunchKernelGGL(k_assign, dim3(grid), dim3(kScanBlock), 0, s, h.nbr, h.sizes, h.next_sizes, ids,
                     table, num_nodes, h.flag_tiles, h.flag_ticket);
  return hipGetLastError();
}

hipError_t launch_local(const HopArgs* hops, int num_hops, const int32_t* ids, int32_t num_seeds,
                        const uint32_t* table, int64_t num_nodes, uint32_t* status, hipStream_t s) {
  LocalArgs a{};
  int64_t blocks = 0;
  for (int i = 0; i < num_hops; ++i) {
    a.seg[i].nbr = hops[i].nbr;
    a.seg[i].local = hops[i].local;
    a.seg[i].sizes = hops[i].sizes;
    a.seg[i].first_block = blocks;
    blocks += (hops[i].cap_nnz + 255) / 256;
  }
  a.num_seg = num_hops;
  a.seed_first_block = blocks;
  blocks += (num_seeds + 255) / 256;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_local, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, a, ids, num_seeds,
                     table, num_nodes, status);
  return hipGetLastError();
}

hipError_t launch_cleanup(const int32_t* ids, const int32_t* final_sizes, int64_t cap_src,
                          uint32_t* table, int64_t num_nodes, hipStream_t s) {
  hipLaunchKernelGGL(k_cleanup, dim3(grid_for(cap_src)), dim3(256), 0, s, ids, final_sizes, table,
                     num_nodes);
  return hipGetLastError();
}

}  // namespace gmb
