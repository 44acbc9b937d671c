// Mini-batch construction on gfx950: recursive fan-out neighbour sampling
// with per-hop dedup and relabel into bipartite blocks (DistDGL, Section
// II-B: pick at most K neighbours of every target, repeat once per layer;
// the sampled graph is the mini-batch's computation graph, Fig. 1(b)).
//
// ids[] is shared by all hops: the sources of a block are its destinations
// followed by its new vertices, which are exactly the next hop's
// destinations, so every hop only appends, and a vertex keeps the same
// local id (its position in ids) in every block.  The positions come in
// segments: segment 0 = the seeds, segment j >= 1 = the vertices new in hop
// j - 1; hop h's destinations are segments 0..h.
//
// A vertex's clamped degree k_h = min(deg, fanout of hop h) is computed for
// every later hop h as soon as the vertex gets its position, and scanned
// within its segment; hop h's block row offsets are then the segment's
// offsets plus the totals of the earlier segments.  So no hop needs a
// degree pass of its own:
//   k_seed_scan   (one workgroup) seeds -> ids; degree scans of segment 0
//                 for all hops; clears the look-back words; the first
//                 hop's sampling writes the seeds' table slots
//   k_sample(h)   Floyd's algorithm per destination, one lane per draw,
//                 Philox-keyed draws; sampled slots ranked in the group and
//                 written in slot order; each vertex's first edge position
//                 recorded by atomicMin in the dedup table
//   k_assign(h)   scan of the "first occurrence" flags (new vertex number
//                 n_dst + rank) together with the degree scans of the new
//                 vertices for the later hops; writes every edge's local id
//   k_cleanup     the table back to empty (the whole table when that is
//                 cheaper, else the slots of the batch's vertices); the
//                 last hop's deferred local ids
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"
#include "philox.hpp"
#include "scan.hpp"

namespace gmb {

namespace {

__device__ __forceinline__ CsrView view(const CsrArgs& a) {
  return CsrView{a.indptr, a.indices, a.num_nodes, a.wide};
}

__device__ __forceinline__ int32_t clamp_degree(int64_t d, int fanout) {
  return static_cast<int32_t>(d < 0 ? 0 : (d < fanout ? d : fanout));
}

// Items [base, base + ITEMS) of a scan tile.  Full groups are 8- or
// 16-byte loads (base is a multiple of ITEMS and the arrays are 256-byte
// aligned); the group holding the end of the data reads element-wise, and
// entries at or past n are left as 0 (the caller ignores them).
template <int ITEMS>
__device__ __forceinline__ void load_items(const int32_t* a, int64_t base, int64_t n, int32_t (&v)[ITEMS]) {
  if (base + ITEMS <= n) {
    if constexpr (ITEMS % 4 == 0) {
#pragma unroll
      for (int c = 0; c < ITEMS / 4; ++c) {
        const int4 x = *reinterpret_cast<const int4*>(a + base + 4 * c);
        v[4 * c] = x.x; v[4 * c + 1] = x.y; v[4 * c + 2] = x.z; v[4 * c + 3] = x.w;
      }
    } else {
      static_assert(ITEMS == 2, "2, 4, 8 or 16 items");
      const int2 x = *reinterpret_cast<const int2*>(a + base);
      v[0] = x.x; v[1] = x.y;
    }
  } else {
#pragma unroll
    for (int q = 0; q < ITEMS; ++q) v[q] = base + q < n ? a[base + q] : 0;
  }
}

__global__ __launch_bounds__(256) void k_state_init(uint32_t* table, uint32_t* status, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
    table[i] = kEmpty;
  if (blockIdx.x == 0 && threadIdx.x == 0) *status = 0;
}

// One workgroup.  Seeds -> ids[0:B]; segment 0's degree scans for every
// hop; clears the look-back words and the size words.  (The seeds' table
// slots are written by the first hop's sampling kernel.)
constexpr int kSeedItems = 4;
// one workgroup: 1024 threads while the register budget allows (NV <= 4)
template <int NV>
constexpr int seed_block() { return NV <= 4 ? 1024 : 512; }

// Every store of this kernel follows its reads: on gfx9 the same counter
// tracks outstanding loads and stores, so a store issued before a load
// would add its own latency to the wait for that load.
template <int NV, bool WIDE, int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_seed_scan(SeedArgs a, CsrArgs ga) {
  __shared__ int32_t s_wave[NV * (BLOCK / 64)];
  const CsrView g = view(ga);
  const int tid = threadIdx.x;
  const int32_t B = a.num_seeds;
  int32_t running[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) running[v] = 0;
  // each thread takes kSeedItems consecutive seeds: one batch of reads (the
  // seeds, then their row offsets), the degree scans, then the stores:
  // block row offsets and ids (the seeds' table slots are written by the
  // first hop's sampling, spread over its workgroups)
  for (int32_t base = 0; base < B; base += BLOCK * kSeedItems) {
    int32_t sd[kSeedItems];
#pragma unroll
    for (int q = 0; q < kSeedItems; ++q) {
      const int32_t p = base + tid * kSeedItems + q;
      sd[q] = a.seeds[p < B ? p : B - 1];
    }
    int32_t deg[kSeedItems];
#pragma unroll
    for (int q = 0; q < kSeedItems; ++q) {
      const int32_t p = base + tid * kSeedItems + q;
      const bool ok = p < B && valid_vertex(sd[q], g.num_nodes);
      int64_t b, e;
      row_range_t<WIDE>(g, ok ? sd[q] : 0, b, e);
      deg[q] = ok ? static_cast<int32_t>(e - b) : 0;
    }
    int32_t sum[NV], excl[NV], total[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      sum[v] = 0;
#pragma unroll
      for (int q = 0; q < kSeedItems; ++q) sum[v] += clamp_degree(deg[q], a.fanout[v]);
    }
    block_exclusive_scan_multi<BLOCK, NV>(sum, excl, total, s_wave);
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      int32_t run = running[v] + excl[v];
#pragma unroll
      for (int q = 0; q < kSeedItems; ++q) {
        const int32_t p = base + tid * kSeedItems + q;
        if (p < B) a.indptr[v][p] = run;
        run += clamp_degree(deg[q], a.fanout[v]);
      }
      running[v] += total[v];
    }
#pragma unroll
    for (int q = 0; q < kSeedItems; ++q) {
      const int32_t p = base + tid * kSeedItems + q;
      if (p < B) a.ids[p] = sd[q];
    }
  }
  // look-back words and tickets of the relabel scans, size words
  for (int64_t i = tid; i < a.num_zero; i += BLOCK) a.zero[i] = 0;
  for (int i = tid; i < a.num_size_words; i += BLOCK) a.sizes[i] = 0;
  __syncthreads();
  if (tid == 0) {
#pragma unroll
    for (int v = 0; v < NV; ++v) a.totals[v] = running[v];   // segment 0's edges of hop v
    // hop 0 has one segment: its sizes are known now
    a.sizes[a.first_sizes + kNDst] = B;
    a.sizes[a.first_sizes + kNnz] = running[0];
    a.indptr[0][B] = running[0];
  }
}

// Emits edge `pos` (sampled vertex u) and records it in the dedup table.
// With GMB_EMIT_PREREAD the table is read first: entries only decrease
// during the kernel, so a read that is already <= the edge's tag proves the
// atomic would change nothing and it is skipped.
#ifndef GMB_EMIT_PREREAD
#define GMB_EMIT_PREREAD 1
#endif
__device__ __forceinline__ void emit_edge(int32_t pos, int32_t u, int32_t* nbr, uint32_t* table,
                                          int64_t num_nodes, uint32_t* status) {
  // the table read goes out before the store (one counter tracks both)
  const bool ok = valid_vertex(u, num_nodes);
  const uint32_t tag = kEdgeTag | static_cast<uint32_t>(pos);
  const uint32_t seen = GMB_EMIT_PREREAD ? table[ok ? u : 0] : kEmpty;
  nbr[pos] = u;
  if (ok) {
    if (seen > tag) atomicMin(&table[u], tag);
  } else {
    raise_status(status, GMB_STATUS_ERANGE);
  }
}

// Deferred local ids of the previous hop (written by its relabel as
// -(e0 + 1), e0 = the vertex's first edge, in an earlier tile): edge e
// takes the local id of edge e0, final since that relabel ended.  One edge
// per thread.  The reads are unconditional (clamped indices; the first hop
// passes an edge count of 0) so that they overlap with the caller's.
struct DeferredItem {
  int32_t n, x, y;
};

// First read: the edge count and the edge's entry.
__device__ __forceinline__ DeferredItem deferred_read(const DeferredArgs& fix, int64_t e) {
  DeferredItem it;
  it.n = load_size(&fix.sizes[kNnz]);
  it.x = fix.local[e < fix.cap ? e : fix.cap - 1];
  it.y = 0;
  return it;
}

// Second read: the entry of the first occurrence (entry 0 when nothing is
// deferred).
__device__ __forceinline__ void deferred_fetch(const DeferredArgs& fix, DeferredItem& it) {
  const int32_t e0 = it.x < 0 ? -(it.x + 1) : 0;
  it.y = fix.local[e0 < it.n ? e0 : 0];
}

__device__ __forceinline__ void deferred_store(const DeferredArgs& fix, int64_t e, const DeferredItem& it) {
  if (e < it.n && it.x < 0) fix.local[e] = it.y;
}

// G lanes per destination (G >= fanout, G a power of two <= 64): lane i
// draws t_i uniform in [0, j_i], j_i = d - f + i; Floyd's rule is then
// resolved in draw order with one group-wide vote per step (x_s = t_s
// unless an earlier lane already holds t_s, then x_s = j_s), and every lane
// finds the rank of its slot among the group's.  The grid also covers the
// previous hop's edges for the deferred local ids.
template <int G, bool WIDE>
__global__ __launch_bounds__(256) void k_sample(CsrArgs ga, const int32_t* ids, const int32_t* sizes,
                                                const int32_t* blk_indptr, int64_t cap_dst,
                                                int32_t* nbr, uint32_t* table, uint32_t* status,
                                                int fanout, int layer, uint32_t k0, uint32_t k1,
                                                int check_seeds, DeferredArgs fix) {
  const CsrView g = view(ga);
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t p = tid / G;
  const int lane = threadIdx.x & (G - 1);
  // the first reads do not depend on each other: a position past the
  // capacity reads the last one and is dropped below
  const int64_t pc = p < cap_dst ? p : cap_dst - 1;
  const int32_t n_dst = load_size(&sizes[kNDst]);
  const int32_t v = ids[pc];
  const int32_t off = blk_indptr[pc];
  DeferredItem it = deferred_read(fix, tid);
  // second round, again independent reads: the deferred edge's source
  // entry, the seed's table slot (first hop) and the row of v
  const bool valid = valid_vertex(v, g.num_nodes);
  const int32_t vc = valid ? v : 0;
  deferred_fetch(fix, it);
  int64_t begin, end;
  row_range_t<WIDE>(g, vc, begin, end);
  deferred_store(fix, tid, it);
  if (p >= n_dst) return;
  // first hop: the seed's table slot is its position, lowered with
  // atomicMin: the edges emitted meanwhile lower slots to tags >= 2^31
  // only, so the slot ends at p whatever the order, and a seed listed
  // twice finds its other copy's position there (checked at the end, so
  // that the wait for the old value does not hold up the sampling)
  uint32_t seed_old = kEmpty;
  if (check_seeds && lane == 0) {
    if (valid) seed_old = atomicMin(&table[v], static_cast<uint32_t>(p));
    else raise_status(status, GMB_STATUS_ERANGE);
  }
  if (!valid) return;   // an invalid vertex's clamped degree was 0
  const int64_t d = end - begin;

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
  if (seed_old < kEdgeTag) raise_status(status, GMB_STATUS_EDUP);
}

// Fan-outs above 64: one thread per destination; the block's output row
// holds the chosen slots while Floyd runs, is sorted in place, then mapped
// to vertex ids.
__global__ __launch_bounds__(256) void k_sample_wide(CsrArgs ga, const int32_t* ids,
                                                     const int32_t* sizes, const int32_t* blk_indptr,
                                                     int32_t* nbr, uint32_t* table, uint32_t* status,
                                                     int fanout, int layer, uint32_t k0, uint32_t k1,
                                                     int check_seeds, DeferredArgs fix) {
  const CsrView g = view(ga);
  const int64_t p = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  {
    DeferredItem it = deferred_read(fix, p);
    deferred_fetch(fix, it);
    deferred_store(fix, p, it);
  }
  const int32_t n_dst = load_size(&sizes[kNDst]);
  if (p >= n_dst) return;
  const int32_t v = ids[p];
  if (check_seeds) {   // the seed's table slot and the repeat check (see k_sample)
    if (!valid_vertex(v, g.num_nodes)) raise_status(status, GMB_STATUS_ERANGE);
    else if (atomicMin(&table[v], static_cast<uint32_t>(p)) < kEdgeTag) raise_status(status, GMB_STATUS_EDUP);
  }
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

// Hop h's relabel.  Edge e is the first occurrence of its vertex u when the
// table holds (tag | e); those edges are numbered by a scan, the vertex
// becomes source n_dst + rank, is appended to ids and gets its local id in
// the table.  Value 0 of the scan counts them; value v >= 1 carries the
// new vertices' clamped degrees for hop h + v, which become those hops'
// block row offsets.  Every edge's local id is written here, or deferred:
// a vertex seen before this hop has it in the table; a repeat of a vertex
// that is new in this hop takes it from LDS when the first occurrence is in
// the same tile, else it stores -(e0 + 1) (e0 = the first occurrence) and
// the next kernel on the stream copies local[e0].  Other tiles may read
// table[u] while it is rewritten: they see either a tag or the local id,
// never their own tag, so their flag is 0 either way, and either one gives
// them the right local id; so the table store needs no ordering within
// this kernel.  After the last hop no kernel reads a new vertex's slot
// (the cleanup reads only the seeds' slots), so the last hop leaves its
// new vertices' tags in place: its repeats then always take the LDS or the
// deferred route, and the cleanup resets the slots as it does the others.
template <int NV, bool WIDE, int ITEMS>
__global__ __launch_bounds__(kScanBlock) void k_assign(AssignArgs a, CsrArgs ga, int32_t* ids,
                                                       uint32_t* table, uint32_t* status) {
  __shared__ int s_tile;
  __shared__ int32_t s_excl[NV];
  __shared__ int32_t s_wave[NV * (kScanBlock / 64)];
  __shared__ int32_t s_pos[(kScanBlock * ITEMS)];
  const CsrView g = view(ga);
  // row offsets of hop h + v start after the edges of segments 0..h
  // (final before this kernel; read early, used after the look-back)
  int32_t basev[NV];
#pragma unroll
  for (int v = 1; v < NV; ++v) basev[v] = a.totals[a.hop + v];
  const int32_t n = load_size(&a.sizes[kNnz]);
  const int32_t n_dst = load_size(&a.sizes[kNDst]);
  const int tile = claim_tile(a.ticket, &s_tile);
  const int num_tiles = n <= 0 ? 1 : (n + (kScanBlock * ITEMS) - 1) / (kScanBlock * ITEMS);
  if (tile >= num_tiles) return;

  const int64_t tile_base = static_cast<int64_t>(tile) * (kScanBlock * ITEMS);
  const int64_t base = tile_base + threadIdx.x * ITEMS;
  int32_t u[ITEMS];
  load_items<ITEMS>(a.nbr, base, n, u);
  // table entries and (for the later hops) the degrees of every item, in
  // one round of reads; an invalid item reads vertex 0 and is dropped
  uint32_t t[ITEMS];
  int32_t deg[ITEMS];
#pragma unroll
  for (int q = 0; q < ITEMS; ++q) {
    const bool ok = (base + q < n) & valid_vertex(u[q], g.num_nodes);
    u[q] = ok ? u[q] : -1;
    const int32_t uc = u[q] < 0 ? 0 : u[q];
    t[q] = table[uc];
    deg[q] = 0;
    if constexpr (NV > 1) {
      int64_t b, e;
      row_range_t<WIDE>(g, uc, b, e);
      deg[q] = static_cast<int32_t>(e - b);
    }
  }
  uint32_t flags = 0;
#pragma unroll
  for (int q = 0; q < ITEMS; ++q)
    if (u[q] >= 0 && t[q] == (kEdgeTag | static_cast<uint32_t>(base + q))) flags |= 1u << q;
  int32_t sum[NV], thr[NV], total[NV], excl[NV];
  sum[0] = __popc(flags);
#pragma unroll
  for (int v = 1; v < NV; ++v) {
    sum[v] = 0;
#pragma unroll
    for (int q = 0; q < ITEMS; ++q) sum[v] += ((flags >> q) & 1u) ? clamp_degree(deg[q], a.fanout[v]) : 0;
  }
  block_exclusive_scan_multi<kScanBlock, NV>(sum, thr, total, s_wave);
  if (threadIdx.x < 64) {
    int32_t ex[NV];
    const bool ok = tile_lookback_multi<NV>(a.tiles, a.tile_stride, tile, total, ex);
    if (threadIdx.x == 0) {
      if (!ok) raise_status(status, GMB_STATUS_INTERNAL);
#pragma unroll
      for (int v = 0; v < NV; ++v) s_excl[v] = ex[v];
    }
  }
  __syncthreads();
#pragma unroll
  for (int v = 0; v < NV; ++v) excl[v] = s_excl[v];

  // new vertices: position, ids, table, local id, later hops' row offsets
  int32_t r = n_dst + excl[0] + thr[0];
  int32_t run[NV];
#pragma unroll
  for (int v = 1; v < NV; ++v) run[v] = basev[v] + excl[v] + thr[v];
#pragma unroll
  for (int q = 0; q < ITEMS; ++q) {
    if ((flags >> q) & 1u) {
      ids[r] = u[q];
      a.local[base + q] = r;
      if (a.next_sizes) table[u[q]] = static_cast<uint32_t>(r);   // read by the later hops
      s_pos[threadIdx.x * ITEMS + q] = r;
#pragma unroll
      for (int v = 1; v < NV; ++v) {
        a.indptr[v][r] = run[v];
        run[v] += clamp_degree(deg[q], a.fanout[v]);
      }
      ++r;
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < ITEMS; ++q) {
    if (base + q >= n || ((flags >> q) & 1u)) continue;
    int32_t loc = 0;   // an invalid vertex (reported by the sampling) gets 0
    if (u[q] >= 0) {
      if (t[q] < kEdgeTag) {
        loc = static_cast<int32_t>(t[q]);
      } else {
        const int64_t e0 = t[q] & ~kEdgeTag;
        loc = e0 >= tile_base ? s_pos[e0 - tile_base] : -static_cast<int32_t>(e0) - 1;
      }
    }
    a.local[base + q] = loc;
  }
  if (tile == num_tiles - 1 && threadIdx.x == 0) {
    const int32_t n_src = n_dst + excl[0] + total[0];
    a.sizes[kNSrc] = n_src;
    if (a.next_sizes) {
      a.next_sizes[kNDst] = n_src;
      if constexpr (NV > 1) {
        // this hop's new vertices are segment h + 1
#pragma unroll
        for (int v = 1; v < NV; ++v) a.totals[a.hop + v] = basev[v] + excl[v] + total[v];
        // the next hop's destinations are complete: its edge count is known
        const int32_t nnz = basev[1] + excl[1] + total[1];
        a.next_sizes[kNnz] = nnz;
        a.indptr[1][n_src] = nnz;
      }
    }
  }
}

// Resolves the last hop's deferred local ids (the table is not read for
// those) and clears the table: if `whole`, every slot, thread i storing
// slots 4i..4i+3 with one 16-byte store (the table is 16-byte aligned) and
// the first threads the num_nodes % 4 slots past the last full group; else
// the slots of the batch's vertices, one random store each.
__global__ __launch_bounds__(256) void k_cleanup(const int32_t* ids, int64_t cap_src, const int32_t* final_sizes,
                                                 uint32_t* table, int64_t num_nodes, int whole, DeferredArgs fix) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  DeferredItem it = deferred_read(fix, i);
  if (whole) {
    deferred_fetch(fix, it);
    deferred_store(fix, i, it);
    const int64_t full = num_nodes >> 2;
    if (i < full) reinterpret_cast<uint4*>(table)[i] = make_uint4(kEmpty, kEmpty, kEmpty, kEmpty);
    if (i < (num_nodes & 3)) table[(full << 2) + i] = kEmpty;
    return;
  }
  const int32_t n = load_size(&final_sizes[kNSrc]);
  const int32_t u = ids[i < cap_src ? i : cap_src - 1];
  const bool ok = i < n && valid_vertex(u, num_nodes);
  deferred_fetch(fix, it);
  deferred_store(fix, i, it);
  if (ok) table[u] = kEmpty;
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

hipError_t launch_seed_scan(const SeedArgs& a, int num_values, const CsrArgs& g, hipStream_t s) {
#define GMB_SEED(V)                                                                          \
  if (g.wide)                                                                                \
    hipLaunchKernelGGL((k_seed_scan<V, true, seed_block<V>()>), dim3(1), dim3(seed_block<V>()), \
                       0, s, a, g);                                                           \
  else                                                                                       \
    hipLaunchKernelGGL((k_seed_scan<V, false, seed_block<V>()>), dim3(1), dim3(seed_block<V>()), \
                       0, s, a, g)
  switch (num_values) {
    case 1: { GMB_SEED(1); } break;
    case 2: { GMB_SEED(2); } break;
    case 3: { GMB_SEED(3); } break;
    case 4: { GMB_SEED(4); } break;
    case 5: { GMB_SEED(5); } break;
    case 6: { GMB_SEED(6); } break;
    case 7: { GMB_SEED(7); } break;
    case 8: { GMB_SEED(8); } break;
    default: return hipErrorInvalidValue;
  }
#undef GMB_SEED
  return hipGetLastError();
}

hipError_t launch_sample(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* table,
                         uint32_t* status, uint32_t k0, uint32_t k1, int first_hop,
                         const DeferredArgs& fix, hipStream_t s) {
  const int f = h.fanout;
  const int64_t cap_dst = h.cap_dst < 1 ? 1 : h.cap_dst;   // ids and indptr hold >= 1 entry
  auto threads = [&](int64_t per_dst) { return std::max(h.cap_dst * per_dst, fix.cap); };
#define GMB_LAUNCH_SAMPLE(G)                                                                     \
  if (g.wide)                                                                                     \
    hipLaunchKernelGGL((k_sample<G, true>), dim3(grid_for(threads(G))), dim3(256), 0, s, g, ids,  \
                       h.sizes, h.indptr, cap_dst, h.nbr, table, status, f, h.layer, k0, k1,      \
                       first_hop, fix);                                                           \
  else                                                                                            \
    hipLaunchKernelGGL((k_sample<G, false>), dim3(grid_for(threads(G))), dim3(256), 0, s, g, ids, \
                       h.sizes, h.indptr, cap_dst, h.nbr, table, status, f, h.layer, k0, k1,      \
                       first_hop, fix)
  if (f <= 8) {
    GMB_LAUNCH_SAMPLE(8);
  } else if (f <= 16) {
    GMB_LAUNCH_SAMPLE(16);
  } else if (f <= 32) {
    GMB_LAUNCH_SAMPLE(32);
  } else if (f <= 64) {
    GMB_LAUNCH_SAMPLE(64);
  } else
    hipLaunchKernelGGL(k_sample_wide, dim3(grid_for(threads(1))), dim3(256), 0, s, g, ids, h.sizes,
                       h.indptr, h.nbr, table, status, f, h.layer, k0, k1, first_hop, fix);
#undef GMB_LAUNCH_SAMPLE
  return hipGetLastError();
}

hipError_t launch_assign(const AssignArgs& a, int num_values, const CsrArgs& g, int64_t cap_nnz,
                         int items, int32_t* ids, uint32_t* table, uint32_t* status, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>(scan_tiles(cap_nnz, items));
#define GMB_ASSIGN_I(V, W, I) \
  hipLaunchKernelGGL((k_assign<V, W, I>), dim3(grid), dim3(kScanBlock), 0, s, a, g, ids, table, status)
#define GMB_ASSIGN_W(V, W)                       \
  switch (items) {                               \
    case 2: GMB_ASSIGN_I(V, W, 2); break;        \
    case 4: GMB_ASSIGN_I(V, W, 4); break;        \
    case 8: GMB_ASSIGN_I(V, W, 8); break;        \
    case 16: GMB_ASSIGN_I(V, W, 16); break;      \
    default: return hipErrorInvalidValue;        \
  }
#define GMB_ASSIGN(V)         \
  if (g.wide) {               \
    GMB_ASSIGN_W(V, true)     \
  } else {                    \
    GMB_ASSIGN_W(V, false)    \
  }
  switch (num_values) {
    case 1: { GMB_ASSIGN(1); } break;
    case 2: { GMB_ASSIGN(2); } break;
    case 3: { GMB_ASSIGN(3); } break;
    case 4: { GMB_ASSIGN(4); } break;
    case 5: { GMB_ASSIGN(5); } break;
    case 6: { GMB_ASSIGN(6); } break;
    case 7: { GMB_ASSIGN(7); } break;
    case 8: { GMB_ASSIGN(8); } break;
    default: return hipErrorInvalidValue;
  }
#undef GMB_ASSIGN
#undef GMB_ASSIGN_W
#undef GMB_ASSIGN_I
  return hipGetLastError();
}

hipError_t launch_cleanup(const int32_t* ids, const int32_t* final_sizes, int64_t cap_src, uint32_t* table,
                          int64_t num_nodes, const DeferredArgs& fix, hipStream_t s) {
  // the whole table in 16-byte stores costs about as much HBM time as
  // eight random 4-byte stores per slot it covers; clear it whole when it
  // has no more than eight slots per possible source of the batch
  const bool whole = num_nodes <= 8 * std::max<int64_t>(cap_src, 1);
  const int64_t threads = std::max(whole ? std::max<int64_t>(num_nodes / 4, 4) : cap_src, fix.cap);
  hipLaunchKernelGGL(k_cleanup, dim3(grid_for(threads)), dim3(256), 0, s, ids, std::max<int64_t>(cap_src, 1),
                     final_sizes, table, num_nodes, whole ? 1 : 0, fix);
  return hipGetLastError();
}

}  // namespace gmb
