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
// degree pass of its own.
//
// Dedup, two ways.  The hops before the last are small (a few thousand to
// a few tens of thousands of edges); they dedup through a per-vertex table
// in the sampler state: each sampled edge lowers its vertex's slot to its
// own position (atomicMin), and the relabel scan numbers the edges that
// still find their own position there.  The last hop holds almost all the
// edges, and a table touched once per edge costs a 128-byte line per 4-byte
// access from every XCD's L2 (and a memory-side atomic per new vertex).
// So its edges (and its destinations, the vertices known so far) are routed
// to "owner" workgroups by a hash of the vertex id; an owner sees every
// occurrence of its vertices, so a hash table in its LDS finds, per vertex,
// its local id if it is known, else its first edge (atomicMin on the edge
// position in LDS).  The answer goes back to the edge's slot, and the
// relabel scan numbers the first occurrences in edge order.  The kernels,
// per call:
//   k_seed_scan   (one workgroup) seeds -> ids; degree scans of segment 0
//                 for all hops; clears the look-back words
//   table hops (all but the last, fan-outs up to 64):
//   k_sample_table(h)  Floyd's algorithm per destination, one lane per
//                 draw, Philox-keyed draws; sampled slots ranked in the
//                 group and written in slot order; each vertex's first
//                 edge recorded by atomicMin in the table (the first hop
//                 also records the seeds' positions)
//   k_assign(h)   scan of the "first occurrence" flags (new vertex number
//                 n_dst + rank) together with the degree scans of the new
//                 vertices for the later hops; every edge's local id
//   owner hops (the last, and any hop after one with a fan-out above 64):
//   k_sample_route(h)  "routers": each takes a span of destinations (a
//                 contiguous range of edges), samples them as above and
//                 writes its edges and its destinations, grouped by owner,
//                 into its own region of the pair array, with the group
//                 offsets (fan-outs above 64: k_sample_wide_wave, a wave
//                 per destination, or k_sample_wide above 256, then k_route)
//   k_owner(h)    one workgroup per owner: gathers its pairs from every
//                 router's region, dedups them in an LDS hash table and
//                 writes each edge's answer (known local id, first
//                 occurrence, or repeat of edge e0) into the edge's slot
//   k_rank(h)     per router, in router order: the answers back in edge
//                 order (LDS), the scan of the first occurrences with the
//                 degree scans for the later hops; every edge's local id
//   k_fix         the last hop's deferred local ids (a repeat whose first
//                 occurrence lies in an earlier tile or router is written
//                 as -(e0 + 1); the next kernel copies local[e0]), and the
//                 table slots the table hops recorded back to empty
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

// Owner of a vertex (multiplicative hash scaled to [0, owners)) and its
// first slot in a power-of-two LDS table (another multiplier, top bits).
__device__ __forceinline__ uint32_t owner_of(uint32_t key, uint32_t owners) {
  return static_cast<uint32_t>((static_cast<uint64_t>(key * 0x9E3779B1u) * owners) >> 32);
}
__device__ __forceinline__ uint32_t slot_of(uint32_t key, int shift) {
  return (key * 0x85EBCA77u) >> shift;
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

// The state: the status word, the vertex count (int64 at byte 8, for
// clearing the table again after a failed call), the table.
__global__ __launch_bounds__(256) void k_state_init(uint32_t* table, uint32_t* status, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
    table[i] = kEmpty;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    *status = 0;
    *reinterpret_cast<int64_t*>(status + 2) = n;
  }
}

// One workgroup.  Seeds -> ids[0:B]; segment 0's degree scans for every
// hop; clears the look-back words and the size words.
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
  // block row offsets and ids
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

// Deferred local ids of the previous hop (written by its relabel as
// -(e0 + 1), e0 = the vertex's first edge, in an earlier router's range):
// edge e takes the local id of edge e0, final since that relabel ended.
// One edge per thread.  The reads are unconditional (clamped indices; the
// first hop passes an edge count of 0) so that they overlap with the
// caller's.
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

// Emits edge `pos` (sampled vertex u) and records it in the dedup table.
// With GMB_EMIT_PREREAD the table is read first: entries only decrease
// during the kernel, so a read that is already <= the edge's tag proves the
// atomic would change nothing and it is skipped.
#ifndef GMB_EMIT_PREREAD
#define GMB_EMIT_PREREAD 1
#endif
__device__ __forceinline__ void emit_edge_table(int32_t pos, int32_t u, int32_t* nbr, uint32_t* table,
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

// Writes edge `pos` (sampled vertex u); an id outside the graph (a broken
// CSR) is reported and routed as "no vertex" (local id 0).
__device__ __forceinline__ void emit_edge(int32_t pos, int32_t u, int32_t* nbr, int64_t num_nodes,
                                          uint32_t* status) {
  nbr[pos] = u;
  if (!valid_vertex(u, num_nodes)) raise_status(status, GMB_STATUS_ERANGE);
}

// Sampling of a hop whose dedup runs through the state's per-vertex table
// (the small hops before the last: few edges, so few table lines).
// G lanes per destination (G >= fanout, G a power of two <= 64): lane i
// draws t_i uniform in [0, j_i], j_i = d - f + i; Floyd's rule is then
// resolved in draw order with one group-wide vote per step (x_s = t_s
// unless an earlier lane already holds t_s, then x_s = j_s), and every lane
// finds the rank of its slot among the group's.  The grid also covers the
// previous hop's edges for the deferred local ids.
template <int G, bool WIDE>
__global__ __launch_bounds__(256) void k_sample_table(CsrArgs ga, const int32_t* ids, const int32_t* sizes,
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
  if (pos >= 0) emit_edge_table(pos, u, nbr, table, g.num_nodes, status);
  if (seed_old < kEdgeTag) raise_status(status, GMB_STATUS_EDUP);
}

// Fan-outs from 65 to 64 I: one wave per destination (grid-stride), I
// draws per lane (draw q on lane q % 64, slot q / 64).  Floyd's rule is
// resolved in draw order: draw q keeps its value unless a draw r < q holds
// it (one ballot over the values held so far), else it takes j_q = d - f + q;
// each value's rank (the count of smaller values) is its place in the row,
// which is so written in slot order.  The same draws and the same rule as
// the one-thread form below, hence the same rows.  The deferred local ids
// of the previous hop are copied by the grid's threads (grid-stride).
template <int I>
__global__ __launch_bounds__(256) void k_sample_wide_wave(CsrArgs ga, const int32_t* ids, const int32_t* sizes,
                                                          const int32_t* blk_indptr, int32_t* nbr, uint32_t* status,
                                                          int fanout, int layer, uint32_t k0, uint32_t k1,
                                                          int check_seeds, DeferredArgs fix) {
  const CsrView g = view(ga);
  const int64_t gid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t nthreads = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t e = gid; e < fix.cap; e += nthreads) {
    DeferredItem it = deferred_read(fix, e);
    deferred_fetch(fix, it);
    deferred_store(fix, e, it);
  }
  const int32_t n_dst = load_size(&sizes[kNDst]);
  const int lane = threadIdx.x & 63;
  const uint32_t f = static_cast<uint32_t>(fanout);
  for (int64_t p = gid / 64; p < n_dst; p += nthreads / 64) {   // uniform per wave
    const int32_t v = ids[p];
    if (!valid_vertex(v, g.num_nodes)) {
      if (check_seeds && lane == 0) raise_status(status, GMB_STATUS_ERANGE);
      continue;
    }
    int64_t begin, end;
    row_range(g, v, begin, end);
    const int64_t d = end - begin;
    const int32_t off = blk_indptr[p];
    if (d <= fanout) {
      for (int64_t s = lane; s < d; s += 64)
        emit_edge(off + static_cast<int32_t>(s), g.indices[begin + s], nbr, g.num_nodes, status);
      continue;
    }
    const uint32_t base = static_cast<uint32_t>(d - fanout);
    uint32_t t[I], x[I];
#pragma unroll
    for (int i = 0; i < I; ++i) {
      const uint32_t q = static_cast<uint32_t>(lane + 64 * i);
      t[i] = q < f ? draw_below(k0, k1, static_cast<uint32_t>(v), static_cast<uint32_t>(layer), q, base + q + 1) : 0u;
      x[i] = t[i];
    }
    for (uint32_t q = 1; q < f; ++q) {
      const int qi = static_cast<int>(q >> 6), ql = static_cast<int>(q & 63);
      uint32_t mine = t[0];
#pragma unroll
      for (int i = 1; i < I; ++i) mine = i == qi ? t[i] : mine;
      const uint32_t tq = __shfl(mine, ql, 64);
      bool hit = false;
#pragma unroll
      for (int i = 0; i < I; ++i) hit |= (static_cast<uint32_t>(lane + 64 * i) < q) & (x[i] == tq);
      if (__ballot(hit) != 0 && lane == ql) {   // the ballot is uniform
#pragma unroll
        for (int i = 0; i < I; ++i)
          if (i == qi) x[i] = base + q;
      }
    }
    uint32_t rank[I];
#pragma unroll
    for (int i = 0; i < I; ++i) rank[i] = 0;
    for (uint32_t q = 0; q < f; ++q) {
      const int qi = static_cast<int>(q >> 6), ql = static_cast<int>(q & 63);
      uint32_t mine = x[0];
#pragma unroll
      for (int i = 1; i < I; ++i) mine = i == qi ? x[i] : mine;
      const uint32_t xq = __shfl(mine, ql, 64);
#pragma unroll
      for (int i = 0; i < I; ++i) rank[i] += xq < x[i] ? 1u : 0u;
    }
#pragma unroll
    for (int i = 0; i < I; ++i) {
      const uint32_t q = static_cast<uint32_t>(lane + 64 * i);
      if (q < f) emit_edge(off + static_cast<int32_t>(rank[i]), g.indices[begin + x[i]], nbr, g.num_nodes, status);
    }
  }
}

// Fan-outs above 64 I_max (256): one thread per destination; the block's output row
// holds the chosen slots while Floyd runs, is sorted in place, then mapped
// to vertex ids.
__global__ __launch_bounds__(256) void k_sample_wide(CsrArgs ga, const int32_t* ids, const int32_t* sizes,
                                                     const int32_t* blk_indptr, int32_t* nbr, uint32_t* status,
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
  if (!valid_vertex(v, g.num_nodes)) {
    if (check_seeds) raise_status(status, GMB_STATUS_ERANGE);
    return;
  }
  int64_t begin, end;
  row_range(g, v, begin, end);
  const int64_t d = end - begin;
  const int32_t off = blk_indptr[p];
  if (d <= fanout) {
    for (int64_t s = 0; s < d; ++s) emit_edge(off + static_cast<int32_t>(s), g.indices[begin + s], nbr, g.num_nodes, status);
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
    emit_edge(off + static_cast<int32_t>(i), g.indices[begin + slot], nbr, g.num_nodes, status);
  }
}

// Relabel of a table hop.  Edge e is the first occurrence of its vertex u
// when the table holds (tag | e); those edges are numbered by a scan, the
// vertex becomes source n_dst + rank, is appended to ids and gets its local
// id in the table (read by the later hops).  Value 0 of the scan counts
// them; value v >= 1 carries the new vertices' clamped degrees for hop
// h + v, which become those hops' block row offsets.  Every edge's local
// id is written here, or deferred: a vertex seen before this hop has it in
// the table; a repeat of a vertex that is new in this hop takes it from LDS
// when the first occurrence is in the same tile, else it stores -(e0 + 1)
// (e0 = the first occurrence) and the next kernel on the stream copies
// local[e0].  Other tiles may read table[u] while it is rewritten: they see
// either a tag or the local id, never their own tag, so their flag is 0
// either way, and either one gives them the right local id; so the table
// store needs no ordering within this kernel.
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
      table[u[q]] = static_cast<uint32_t>(r);   // read by the later hops
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

// The destinations [p0, p1) of router w (span destinations each; the last
// routers may be empty) and their edges [e0, e1).
struct RouterRange {
  int32_t p0, p1, e0, e1;
};
__device__ __forceinline__ RouterRange router_range(int w, int32_t span, int32_t n_dst, const int32_t* indptr) {
  RouterRange r;
  const int64_t a = static_cast<int64_t>(w) * span;
  r.p0 = static_cast<int32_t>(a < n_dst ? a : n_dst);
  r.p1 = static_cast<int32_t>(a + span < n_dst ? a + span : n_dst);
  r.e0 = indptr[r.p0];
  r.e1 = indptr[r.p1];
  return r;
}

// Exclusive scan of s[0 .. n) in place over one block of BLOCK threads
// (each thread a run of consecutive entries); returns the total.  Every
// thread of the block must call it.
template <int BLOCK>
__device__ int32_t block_scan_inplace(int32_t* s, int n, int32_t* s_wave) {
  const int per = (n + BLOCK - 1) / BLOCK;
  const int lo = threadIdx.x * per;
  int32_t sum[1] = {0}, excl[1], total[1];
  for (int i = lo; i < lo + per && i < n; ++i) sum[0] += s[i];
  block_exclusive_scan_multi<BLOCK, 1>(sum, excl, total, s_wave);
  int32_t run = excl[0];
  for (int i = lo; i < lo + per && i < n; ++i) {
    const int32_t x = s[i];
    s[i] = run;
    run += x;
  }
  __syncthreads();
  return total[0];
}

// Router w: its edges (key = sampled vertex, value = kEdgeTag | edge) and
// its destinations (key = vertex, value = local id = position), grouped by
// owner, into pairs[region .. region + count), region = e0 + p0 (the
// regions of the routers tile [0, nnz + n_dst) in order).  off[b * W + w]
// is where owner b's group starts within the region (b = owners: the
// region's length); rs[w] the region.  An id outside the graph is routed
// as key -1 to owner 0, which answers it with local id 0.  Each thread
// takes kRouteItems entries with one batch of reads; their ranks within
// their group come from LDS atomics and stay in registers.
constexpr int kRouteBlock = 1024;
constexpr int kRouteItems = kMaxRouteEntries / kRouteBlock;
__global__ __launch_bounds__(kRouteBlock) void k_route(RouteArgs a) {
  __shared__ int32_t s_hist[kMaxOwners + 1];
  __shared__ int32_t s_wave[kRouteBlock / 64];
  const int w = blockIdx.x;
  const int P = a.owners;
  const int32_t n_dst = load_size(&a.sizes[kNDst]);
  const RouterRange r = router_range(w, a.span, n_dst, a.indptr);
  const int32_t E = r.e1 - r.e0;
  const int32_t M = E + (r.p1 - r.p0);   // <= kMaxRouteEntries (host-checked span and fan-out)
  int32_t key[kRouteItems];
#pragma unroll
  for (int k = 0; k < kRouteItems; ++k) {
    const int32_t i = threadIdx.x + k * kRouteBlock;
    const int32_t* src = i < E ? a.nbr + (r.e0 + i) : a.ids + (i < M ? r.p0 + (i - E) : 0);
    key[k] = *src;
  }
  for (int b = threadIdx.x; b <= P; b += kRouteBlock) s_hist[b] = 0;
  __syncthreads();
  uint32_t bucket[kRouteItems];
  int32_t rank[kRouteItems];
#pragma unroll
  for (int k = 0; k < kRouteItems; ++k) {
    const int32_t i = threadIdx.x + k * kRouteBlock;
    const bool ok = valid_vertex(key[k], a.num_nodes);
    bucket[k] = ok ? owner_of(static_cast<uint32_t>(key[k]), P) : 0u;
    if (!ok) key[k] = -1;
    rank[k] = i < M ? atomicAdd(&s_hist[bucket[k]], 1) : 0;
  }
  __syncthreads();
  block_scan_inplace<kRouteBlock>(s_hist, P + 1, s_wave);
  const int64_t region = static_cast<int64_t>(r.e0) + r.p0;
  for (int b = threadIdx.x; b <= P; b += kRouteBlock) a.off[static_cast<int64_t>(b) * a.routers + w] = s_hist[b];
  if (threadIdx.x == 0) a.rs[w] = static_cast<int32_t>(region);
#pragma unroll
  for (int k = 0; k < kRouteItems; ++k) {
    const int32_t i = threadIdx.x + k * kRouteBlock;
    if (i >= M) continue;
    const uint32_t val = i < E ? (kEdgeTag | static_cast<uint32_t>(r.e0 + i)) : static_cast<uint32_t>(r.p0 + (i - E));
    a.pairs[region + s_hist[bucket[k]] + rank[k]] = make_uint2(static_cast<uint32_t>(key[k]), val);
  }
}

// Floyd's rule for one group of G lanes whose lane i < f holds its draw
// t_i in [0, j_i], j_i = base + i: in draw order, x_s = t_s unless an
// earlier x already equals t_s, then x_s = j_s.  On return x is lane i's
// slot x_i and rank the number of slots below it (its position in the
// sorted row).  Groups of up to 16 lanes broadcast all draws once and
// resolve the rule in registers (no dependent cross-lane steps); wider
// groups resolve it with one group vote per step.
template <int G>
__device__ __forceinline__ void floyd_resolve(uint32_t& x, uint32_t& rank, uint32_t base, uint32_t f, int lane,
                                              int group_base, uint64_t group_mask) {
  if constexpr (G <= 16) {
    uint32_t t[G], xs[G];
#pragma unroll
    for (int q = 0; q < G; ++q) t[q] = __shfl(x, q, G);
#pragma unroll
    for (int q = 0; q < G; ++q) {
      bool hit = false;
#pragma unroll
      for (int r = 0; r < q; ++r) hit |= xs[r] == t[q];
      xs[q] = hit ? base + q : t[q];
    }
    uint32_t mine = 0;
#pragma unroll
    for (int q = 0; q < G; ++q) mine = q == lane ? xs[q] : mine;
    rank = 0;
#pragma unroll
    for (int q = 0; q < G; ++q) rank += (static_cast<uint32_t>(q) < f && xs[q] < mine) ? 1u : 0u;
    x = mine;
  } else {
    const uint32_t t0 = x, j = base + lane;
    for (uint32_t q = 1; q < f; ++q) {
      const uint32_t tq = __shfl(t0, q, G);
      const bool hit = static_cast<uint32_t>(lane) < q && x == tq;
      const uint64_t votes = (__ballot(hit) >> group_base) & group_mask;
      if (static_cast<uint32_t>(lane) == q && votes != 0) x = j;
    }
    rank = 0;
    for (uint32_t q = 0; q < f; ++q) rank += (__shfl(x, q, G) < x) ? 1u : 0u;
  }
}

// Sampling and routing in one kernel, for fan-outs up to 64 (G lanes per
// destination as in k_sample): router w first resolves its share of the
// previous hop's deferred local ids, loads its span of destinations (id,
// block row offset, CSR row) into LDS with one batch of reads, samples
// them in rounds of kRouteBlock / G destinations (all rounds' draws first,
// then all their neighbour reads in one batch), writes the sampled ids and
// keeps them in LDS, and routes them with the destinations as k_route does.
constexpr int kSampleRounds = 8;   // span * G < 2 * (edges per tile) <= 8192 lanes
template <int G, bool WIDE>
__global__ __launch_bounds__(kRouteBlock) void k_sample_route(CsrArgs ga, SampleArgs a, RouteArgs ra) {
  __shared__ int32_t s_v[kMaxSpan];
  __shared__ int32_t s_off[kMaxSpan];
  __shared__ int32_t s_deg[kMaxSpan];
  __shared__ int64_t s_beg[kMaxSpan];
  __shared__ int32_t s_key[kMaxRouteEntries];
  __shared__ int32_t s_hist[kMaxOwners + 1];
  __shared__ int32_t s_wave[kRouteBlock / 64];
  const CsrView g = view(ga);
  const int w = blockIdx.x;
  const int tid = threadIdx.x;
  // the previous hop's deferred local ids (grid-stride; none on the first hop)
  {
    const int32_t n_prev = load_size(&a.fix.sizes[kNnz]);
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kRouteBlock;
    for (int64_t e = static_cast<int64_t>(w) * kRouteBlock + tid; e < n_prev; e += stride) {
      DeferredItem it = deferred_read(a.fix, e);
      deferred_fetch(a.fix, it);
      deferred_store(a.fix, e, it);
    }
  }
  const int32_t n_dst = load_size(&a.sizes[kNDst]);
  const RouterRange r = router_range(w, ra.span, n_dst, a.indptr);
  const int32_t E = r.e1 - r.e0;
  const int32_t K = r.p1 - r.p0;   // <= span <= kMaxSpan
  for (int t = tid; t < K; t += kRouteBlock) {
    const int32_t v = a.ids[r.p0 + t];
    const int32_t off = a.indptr[r.p0 + t];
    const bool valid = valid_vertex(v, g.num_nodes);
    int64_t b, e;
    row_range_t<WIDE>(g, valid ? v : 0, b, e);
    if (!valid && a.check_seeds) raise_status(a.status, GMB_STATUS_ERANGE);
    s_v[t] = v;
    s_off[t] = off;
    s_beg[t] = b;
    s_deg[t] = valid ? static_cast<int32_t>(e - b) : 0;
    s_key[E + t] = v;
  }
  __syncthreads();
  // draws: lane task q = tid + k * kRouteBlock is lane q % G of destination q / G
  const int lane = tid & (G - 1);
  const int group_base = (tid & 63) & ~(G - 1);
  const uint64_t group_mask = (G == 64) ? ~0ull : ((1ull << G) - 1);
  const uint32_t f = static_cast<uint32_t>(a.fanout);
  int32_t pos[kSampleRounds];
  int64_t slot[kSampleRounds];
#pragma unroll
  for (int k = 0; k < kSampleRounds; ++k) {
    pos[k] = -1;
    slot[k] = 0;
    const int32_t t = (tid + k * kRouteBlock) / G;
    if (k * kRouteBlock >= K * G || t >= K) continue;   // the first test is uniform
    const int32_t d = s_deg[t];
    if (d <= a.fanout) {
      if (lane < d) {
        pos[k] = s_off[t] + lane;
        slot[k] = s_beg[t] + lane;
      }
    } else {
      uint32_t x = 0, rank = 0;
      if (static_cast<uint32_t>(lane) < f)
        x = draw_below(a.k0, a.k1, static_cast<uint32_t>(s_v[t]), static_cast<uint32_t>(a.layer), lane,
                       static_cast<uint32_t>(d) - f + lane + 1);
      floyd_resolve<G>(x, rank, static_cast<uint32_t>(d) - f, f, lane, group_base, group_mask);
      if (static_cast<uint32_t>(lane) < f) {
        pos[k] = s_off[t] + static_cast<int32_t>(rank);
        slot[k] = s_beg[t] + x;
      }
    }
  }
  int32_t u[kSampleRounds];
#pragma unroll
  for (int k = 0; k < kSampleRounds; ++k) u[k] = g.indices[pos[k] >= 0 ? slot[k] : 0];
#pragma unroll
  for (int k = 0; k < kSampleRounds; ++k) {
    if (pos[k] < 0) continue;
    a.nbr[pos[k]] = u[k];
    s_key[pos[k] - r.e0] = u[k];
    if (!valid_vertex(u[k], g.num_nodes)) raise_status(a.status, GMB_STATUS_ERANGE);
  }
  // routing (see k_route), the keys from LDS
  const int P = ra.owners;
  const int32_t M = E + K;
  for (int b = tid; b <= P; b += kRouteBlock) s_hist[b] = 0;
  __syncthreads();
  int32_t key[kRouteItems];
  uint32_t bucket[kRouteItems];
  int32_t rank[kRouteItems];
#pragma unroll
  for (int k = 0; k < kRouteItems; ++k) {
    const int32_t i = tid + k * kRouteBlock;
    key[k] = i < M ? s_key[i] : -1;
    const bool ok = valid_vertex(key[k], ra.num_nodes);
    bucket[k] = ok ? owner_of(static_cast<uint32_t>(key[k]), P) : 0u;
    if (!ok) key[k] = -1;
    rank[k] = i < M ? atomicAdd(&s_hist[bucket[k]], 1) : 0;
  }
  __syncthreads();
  block_scan_inplace<kRouteBlock>(s_hist, P + 1, s_wave);
  const int64_t region = static_cast<int64_t>(r.e0) + r.p0;
  for (int b = tid; b <= P; b += kRouteBlock) ra.off[static_cast<int64_t>(b) * ra.routers + w] = s_hist[b];
  if (tid == 0) ra.rs[w] = static_cast<int32_t>(region);
#pragma unroll
  for (int k = 0; k < kRouteItems; ++k) {
    const int32_t i = tid + k * kRouteBlock;
    if (i >= M) continue;
    const uint32_t val = i < E ? (kEdgeTag | static_cast<uint32_t>(r.e0 + i)) : static_cast<uint32_t>(r.p0 + (i - E));
    ra.pairs[region + s_hist[bucket[k]] + rank[k]] = make_uint2(static_cast<uint32_t>(key[k]), val);
  }
}

// Owner b.  Its pairs are group b of every router's region; s_seg holds
// the running count over routers, s_start the group's address.  Each
// vertex key keeps in LDS the minimum of its values: a known vertex's local
// id (< kEdgeTag) wins over any edge, else the smallest edge position.
// Answer per edge: its known local id, kFirstOccurrence if it is the
// vertex's first edge, else -(e0 + 1) with e0 the first edge.  Two
// destinations with the same id (a repeated seed) are reported (EDUP).
// The pairs are read in chunks of kOwnerBlock * kOwnerItems, each thread
// issuing its reads as one batch, once to insert and once to answer (the
// second time from the L2).  If the table overflows (more distinct keys
// than slots, possible only when the owner's pair count exceeds its
// table), the owner redoes its pairs through the per-vertex table of the
// sampler state: atomicMin, a barrier, the read-back, and the slots reset;
// only this owner ever touches those slots, so the state stays clear.
constexpr int kOwnerBlock = 1024;
constexpr int kOwnerItems = 4;
constexpr int32_t kFirstOccurrence = INT32_MIN;
constexpr int32_t kEmptyKey = INT32_MIN;

__device__ __forceinline__ int32_t owner_answer(uint32_t best, uint32_t val) {
  if (best < kEdgeTag) return static_cast<int32_t>(best);
  if (best == val) return kFirstOccurrence;
  return -static_cast<int32_t>(best & ~kEdgeTag) - 1;
}

__global__ __launch_bounds__(kOwnerBlock) void k_owner(OwnerArgs a) {
  __shared__ int32_t s_seg[kMaxRouters + 1];
  __shared__ int32_t s_start[kMaxRouters];
  __shared__ int32_t s_key[kOwnerSlots];
  __shared__ uint32_t s_val[kOwnerSlots];
  constexpr int kChunk = kOwnerBlock * kOwnerItems;
  __shared__ uint2 s_pair[kChunk];   // the first chunk's pairs and positions, kept for the answers
  __shared__ int32_t s_at[kChunk];
  __shared__ int32_t s_wave[kOwnerBlock / 64];
  __shared__ int s_overflow;
  constexpr int kRouterItems = kMaxRouters / kOwnerBlock;
  const int b = blockIdx.x;
  const int W = a.routers;
  const int64_t row = static_cast<int64_t>(b) * W;
  {
    int32_t lo[kRouterItems], hi[kRouterItems], rs[kRouterItems];
#pragma unroll
    for (int k = 0; k < kRouterItems; ++k) {
      const int w = threadIdx.x + k * kOwnerBlock;
      const int wc = w < W ? w : 0;
      lo[k] = a.off[row + wc];
      hi[k] = a.off[row + W + wc];
      rs[k] = a.rs[wc];
    }
#pragma unroll
    for (int k = 0; k < kRouterItems; ++k) {
      const int w = threadIdx.x + k * kOwnerBlock;
      if (w < W) {
        s_seg[w] = hi[k] - lo[k];
        s_start[w] = rs[k] + lo[k];
      }
    }
  }
  if (threadIdx.x == 0) s_overflow = 0;
  __syncthreads();
  const int32_t M = block_scan_inplace<kOwnerBlock>(s_seg, W, s_wave);
  if (threadIdx.x == 0) s_seg[W] = M;
  // table size: a power of two >= 2 M (load <= 1/2), 64 .. kOwnerSlots
  int logc = 6;
  while ((1 << logc) < 2 * static_cast<int64_t>(M) && (1 << logc) < a.max_slots) ++logc;
  const int C = 1 << logc, shift = 32 - logc;
  for (int i = threadIdx.x; i < C; i += kOwnerBlock) {
    s_key[i] = kEmptyKey;
    s_val[i] = kEmpty;
  }
  __syncthreads();
  // pair i of this owner: router w with s_seg[w] <= i < s_seg[w + 1]
  auto pair_index = [&](int32_t i) -> int64_t {
    int lo = 0, hi = W;   // s_seg[lo] <= i < s_seg[hi]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_seg[mid] <= i) lo = mid;
      else hi = mid;
    }
    return static_cast<int64_t>(s_start[lo]) + (i - s_seg[lo]);
  };
  for (int32_t base = 0; base < M; base += kChunk) {
    uint2 pr[kOwnerItems];
    int64_t at[kOwnerItems];
#pragma unroll
    for (int k = 0; k < kOwnerItems; ++k) {
      const int32_t i = base + threadIdx.x + k * kOwnerBlock;
      at[k] = i < M ? pair_index(i) : 0;
      pr[k] = a.pairs[at[k]];
    }
#pragma unroll
    for (int k = 0; k < kOwnerItems; ++k) {
      const int32_t i = base + threadIdx.x + k * kOwnerBlock;
      if (base == 0) {
        s_pair[i] = pr[k];
        s_at[i] = static_cast<int32_t>(at[k]);
      }
      const int32_t key = static_cast<int32_t>(pr[k].x);
      if (i >= M || key < 0) continue;
      uint32_t h = slot_of(pr[k].x, shift);
      for (int probes = 0;; ++probes) {
        int32_t cur = s_key[h];
        if (cur == kEmptyKey) {
          cur = atomicCAS(&s_key[h], kEmptyKey, key);
          if (cur == kEmptyKey) cur = key;
        }
        if (cur == key) {
          const uint32_t old = atomicMin(&s_val[h], pr[k].y);
          if (pr[k].y < kEdgeTag && old < kEdgeTag && old != pr[k].y) raise_status(a.status, GMB_STATUS_EDUP);
          break;
        }
        if (probes + 1 >= C) {
          s_overflow = 1;
          break;
        }
        h = (h + 1) & (C - 1);
      }
    }
  }
  __syncthreads();
  if (!s_overflow) {
    for (int32_t base = 0; base < M; base += kChunk) {
      uint2 pr[kOwnerItems];
      int64_t at[kOwnerItems];
#pragma unroll
      for (int k = 0; k < kOwnerItems; ++k) {
        const int32_t i = base + threadIdx.x + k * kOwnerBlock;
        if (base == 0) {   // the first chunk from LDS
          at[k] = s_at[i];
          pr[k] = s_pair[i];
        } else {
          at[k] = i < M ? pair_index(i) : 0;
          pr[k] = a.pairs[at[k]];
        }
      }
#pragma unroll
      for (int k = 0; k < kOwnerItems; ++k) {
        const int32_t i = base + threadIdx.x + k * kOwnerBlock;
        if (i >= M || !(pr[k].y & kEdgeTag)) continue;
        int32_t ans = 0;   // an id outside the graph: local id 0
        if (static_cast<int32_t>(pr[k].x) >= 0) {
          uint32_t h = slot_of(pr[k].x, shift);
          for (int probes = 0; probes < C; ++probes, h = (h + 1) & (C - 1)) {
            if (s_key[h] == static_cast<int32_t>(pr[k].x)) {
              ans = owner_answer(s_val[h], pr[k].y);
              break;
            }
          }
        }
        a.res[at[k]] = ans;
      }
    }
    return;
  }
  // overflow: the same through the state's per-vertex table
  for (int32_t i = threadIdx.x; i < M; i += kOwnerBlock) {
    const uint2 pr = a.pairs[pair_index(i)];
    if (static_cast<int32_t>(pr.x) < 0) continue;
    const uint32_t old = atomicMin(&a.table[pr.x], pr.y);
    if (pr.y < kEdgeTag && old < kEdgeTag && old != pr.y) raise_status(a.status, GMB_STATUS_EDUP);
  }
  __threadfence();
  __syncthreads();
  for (int32_t i = threadIdx.x; i < M; i += kOwnerBlock) {
    const int64_t at = pair_index(i);
    const uint2 pr = a.pairs[at];
    if (!(pr.y & kEdgeTag)) continue;
    int32_t ans = 0;
    if (static_cast<int32_t>(pr.x) >= 0)
      ans = owner_answer(__hip_atomic_load(&a.table[pr.x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), pr.y);
    a.res[at] = ans;
  }
  __threadfence();
  __syncthreads();
  for (int32_t i = threadIdx.x; i < M; i += kOwnerBlock) {
    const uint2 pr = a.pairs[pair_index(i)];
    if (static_cast<int32_t>(pr.x) >= 0) a.table[pr.x] = kEmpty;
  }
}

// Hop h's relabel, one workgroup per router, routers taken in ticket order
// (the scan order).  The router's edges come back from its region with the
// owners' answers and are laid out in edge order in LDS; a first
// occurrence becomes source n_dst + rank and is appended to ids; value 0
// of the scan counts them, value v >= 1 carries the new vertices' clamped
// degrees for hop h + v, which become those hops' block row offsets.  A
// repeat of a vertex new in this hop takes the local id from LDS when the
// first occurrence is in the same router's range, else it keeps the
// answer -(e0 + 1) and the next kernel on the stream copies local[e0].
template <int NV, bool WIDE, int ITEMS>
__global__ __launch_bounds__(kScanBlock) void k_rank(RankArgs a, CsrArgs ga, int32_t* ids, uint32_t* status) {
  constexpr int T = kScanBlock * ITEMS;
  __shared__ int s_tile;
  __shared__ int32_t s_excl[NV];
  __shared__ int32_t s_wave[NV * (kScanBlock / 64)];
  // edge j of the router at slot(j): one pad word after every ITEMS
  // entries, so that a thread's ITEMS consecutive entries start ITEMS + 1
  // words after its neighbour's (an odd stride: no two lanes of a wave on
  // one bank)
  auto slot = [](int32_t j) { return j + j / ITEMS; };
  __shared__ int32_t s_key[T + T / ITEMS];
  __shared__ int32_t s_res[T + T / ITEMS];   // the answers; then the new vertices' local ids
  const CsrView g = view(ga);
  int32_t basev[NV];
#pragma unroll
  for (int v = 1; v < NV; ++v) basev[v] = a.totals[a.hop + v];
  const int32_t n_dst = load_size(&a.sizes[kNDst]);
  const int tile = claim_tile(a.ticket, &s_tile);
  const int num_tiles = gridDim.x;
  const RouterRange r = router_range(tile, a.span, n_dst, a.indptr0);
  const int32_t E = r.e1 - r.e0;            // <= T (host-checked span)
  const int32_t M = E + (r.p1 - r.p0);
  const int64_t region = static_cast<int64_t>(r.e0) + r.p0;
  {
    // the region (at most 2 T entries: the edges and the destinations) in
    // one batch of reads per thread
    uint2 pr[2 * ITEMS];
    int32_t an[2 * ITEMS];
#pragma unroll
    for (int k = 0; k < 2 * ITEMS; ++k) {
      const int32_t i = threadIdx.x + k * kScanBlock;
      const int64_t at = i < M ? region + i : 0;
      pr[k] = a.pairs[at];
      an[k] = a.res[at];
    }
#pragma unroll
    for (int k = 0; k < 2 * ITEMS; ++k) {
      const int32_t i = threadIdx.x + k * kScanBlock;
      const int32_t j = static_cast<int32_t>(pr[k].y & ~kEdgeTag) - r.e0;
      if (i < M && (pr[k].y & kEdgeTag) && j >= 0 && j < E) {
        s_key[slot(j)] = static_cast<int32_t>(pr[k].x);
        s_res[slot(j)] = an[k];
      }
    }
  }
  __syncthreads();
  const int base = threadIdx.x * ITEMS;
  int32_t u[ITEMS], ans[ITEMS];
#pragma unroll
  for (int q = 0; q < ITEMS; ++q) {
    const bool in = base + q < E;
    u[q] = in ? s_key[slot(base + q)] : -1;
    ans[q] = in ? s_res[slot(base + q)] : 0;
  }
  uint32_t flags = 0;
#pragma unroll
  for (int q = 0; q < ITEMS; ++q)
    if (ans[q] == kFirstOccurrence) flags |= 1u << q;
  // the new vertices' degrees for the later hops, in one round of reads
  // (other items read vertex 0's row: one line for all of them)
  int32_t deg[ITEMS];
#pragma unroll
  for (int q = 0; q < ITEMS; ++q) {
    deg[q] = 0;
    if constexpr (NV > 1) {
      int64_t b, e;
      row_range_t<WIDE>(g, ((flags >> q) & 1u) ? u[q] : 0, b, e);
      deg[q] = static_cast<int32_t>(e - b);
    }
  }
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

  // new vertices: position, ids, local id, later hops' row offsets
  int32_t rk = n_dst + excl[0] + thr[0];
  int32_t run[NV];
#pragma unroll
  for (int v = 1; v < NV; ++v) run[v] = basev[v] + excl[v] + thr[v];
#pragma unroll
  for (int q = 0; q < ITEMS; ++q) {
    if ((flags >> q) & 1u) {
      ids[rk] = u[q];
      a.local[r.e0 + base + q] = rk;
      s_res[slot(base + q)] = rk;
#pragma unroll
      for (int v = 1; v < NV; ++v) {
        a.indptr[v][rk] = run[v];
        run[v] += clamp_degree(deg[q], a.fanout[v]);
      }
      ++rk;
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < ITEMS; ++q) {
    if (base + q >= E || ((flags >> q) & 1u)) continue;
    int32_t loc = ans[q];   // a known vertex's local id
    if (loc < 0) {
      const int32_t e0 = -(loc + 1);   // the first occurrence, earlier than this edge
      if (e0 >= r.e0 && e0 < r.e1) loc = s_res[slot(e0 - r.e0)];
    }
    a.local[r.e0 + base + q] = loc;
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

// The last hop's deferred local ids, and (clear_sizes != NULL) the table
// slots of the vertices the table hops recorded back to empty: they are
// ids[0 .. n), n = the last table hop's source count.
__global__ __launch_bounds__(256) void k_fix(DeferredArgs fix, const int32_t* ids, const int32_t* clear_sizes,
                                             int64_t clear_cap, uint32_t* table, int64_t num_nodes) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  DeferredItem it = deferred_read(fix, i);
  int32_t u = -1, n = 0;
  if (clear_sizes) {
    n = load_size(&clear_sizes[kNSrc]);
    u = ids[i < clear_cap ? i : clear_cap - 1];
  }
  deferred_fetch(fix, it);
  deferred_store(fix, i, it);
  if (i < n && valid_vertex(u, num_nodes)) table[u] = kEmpty;
}

// The consistency check of one block (see launch_validate).  Every read is
// bounded by the capacities, whatever the size words hold.
__global__ __launch_bounds__(256) void k_validate(ValidateArgs b, int64_t num_nodes, uint32_t* status) {
  const int32_t n_dst = load_size(&b.sizes[kNDst]);
  const int32_t n_src = load_size(&b.sizes[kNSrc]);
  const int32_t nnz = load_size(&b.sizes[kNnz]);
  const bool sizes_ok = n_dst >= 0 && n_dst <= b.cap_dst && n_src >= n_dst && n_src <= b.cap_src && nnz >= 0 &&
                        nnz <= b.cap_nnz;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (!sizes_ok) {
    if (i == 0) raise_status(status, GMB_STATUS_INVALID);
    return;
  }
  bool bad = false;
  if (i <= n_dst) {
    const int32_t a = b.indptr[i];
    if (i == 0) bad |= a != 0;
    if (i == n_dst) bad |= a != nnz;
    if (i < n_dst) {
      const int32_t c = b.indptr[i + 1];
      bad |= c < a || c - a > b.fanout;
    }
  }
  if (i < nnz) {
    const int32_t l = b.local[i];
    const int32_t u = b.nbr[i];
    bad |= !valid_vertex(u, num_nodes);
    if (l < 0 || l >= n_src) bad = true;
    else bad |= b.ids[l] != u;
  }
  if (bad) raise_status(status, GMB_STATUS_INVALID);
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

hipError_t launch_sample_table(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* table,
                               uint32_t* status, uint32_t k0, uint32_t k1, int first_hop, const DeferredArgs& fix,
                               hipStream_t s) {
  const int f = h.fanout;
  if (f > 64) return hipErrorInvalidValue;
  const int64_t cap_dst = h.cap_dst < 1 ? 1 : h.cap_dst;   // ids and indptr hold >= 1 entry
  auto threads = [&](int64_t per_dst) { return std::max(h.cap_dst * per_dst, fix.cap); };
#define GMB_LAUNCH_SAMPLE(G)                                                                             \
  if (g.wide)                                                                                             \
    hipLaunchKernelGGL((k_sample_table<G, true>), dim3(grid_for(threads(G))), dim3(256), 0, s, g, ids,    \
                       h.sizes, h.indptr, cap_dst, h.nbr, table, status, f, h.layer, k0, k1, first_hop, fix); \
  else                                                                                                    \
    hipLaunchKernelGGL((k_sample_table<G, false>), dim3(grid_for(threads(G))), dim3(256), 0, s, g, ids,   \
                       h.sizes, h.indptr, cap_dst, h.nbr, table, status, f, h.layer, k0, k1, first_hop, fix)
  if (f <= 8) {
    GMB_LAUNCH_SAMPLE(8);
  } else if (f <= 16) {
    GMB_LAUNCH_SAMPLE(16);
  } else if (f <= 32) {
    GMB_LAUNCH_SAMPLE(32);
  } else {
    GMB_LAUNCH_SAMPLE(64);
  }
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

hipError_t launch_sample(const CsrArgs& g, const int32_t* ids, const HopArgs& h, uint32_t* status, uint32_t k0,
                         uint32_t k1, int first_hop, const DeferredArgs& fix, hipStream_t s) {
  if (h.fanout <= 256) {
    // a wave per destination (grid-stride over the destinations and the
    // deferred ids, at most 16384 workgroups)
    const int64_t threads = std::max<int64_t>(64 * std::max<int64_t>(h.cap_dst, 1), fix.cap);
    const unsigned grid = std::min<unsigned>(grid_for(threads), 16384u);
    if (h.fanout <= 128)
      hipLaunchKernelGGL(k_sample_wide_wave<2>, dim3(grid), dim3(256), 0, s, g, ids, h.sizes, h.indptr, h.nbr,
                         status, h.fanout, h.layer, k0, k1, first_hop, fix);
    else
      hipLaunchKernelGGL(k_sample_wide_wave<4>, dim3(grid), dim3(256), 0, s, g, ids, h.sizes, h.indptr, h.nbr,
                         status, h.fanout, h.layer, k0, k1, first_hop, fix);
    return hipGetLastError();
  }
  auto threads = std::max(h.cap_dst, fix.cap);
  hipLaunchKernelGGL(k_sample_wide, dim3(grid_for(threads)), dim3(256), 0, s, g, ids, h.sizes, h.indptr, h.nbr,
                     status, h.fanout, h.layer, k0, k1, first_hop, fix);
  return hipGetLastError();
}

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
  if (a.routers < 1 || a.routers > kMaxRouters || a.owners < 1 || a.owners > kMaxOwners)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_route, dim3(static_cast<unsigned>(a.routers)), dim3(kRouteBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sample_route(const CsrArgs& g, const SampleArgs& sa, const RouteArgs& ra, hipStream_t s) {
  if (ra.routers < 1 || ra.routers > kMaxRouters || ra.owners < 1 || ra.owners > kMaxOwners ||
      ra.span < 1 || ra.span > kMaxSpan || sa.fanout < 1 || sa.fanout > 64)
    return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(ra.routers)), block(kRouteBlock);
#define GMB_LAUNCH_SR(G)                                                                         \
  if (g.wide)                                                                                     \
    hipLaunchKernelGGL((k_sample_route<G, true>), grid, block, 0, s, g, sa, ra);                  \
  else                                                                                            \
    hipLaunchKernelGGL((k_sample_route<G, false>), grid, block, 0, s, g, sa, ra)
  if (sa.fanout <= 8) {
    GMB_LAUNCH_SR(8);
  } else if (sa.fanout <= 16) {
    GMB_LAUNCH_SR(16);
  } else if (sa.fanout <= 32) {
    GMB_LAUNCH_SR(32);
  } else {
    GMB_LAUNCH_SR(64);
  }
#undef GMB_LAUNCH_SR
  return hipGetLastError();
}

hipError_t launch_owner(const OwnerArgs& a, hipStream_t s) {
  if (a.routers < 1 || a.routers > kMaxRouters || a.owners < 1 || a.owners > kMaxOwners || a.max_slots < 64 ||
      a.max_slots > kOwnerSlots || (a.max_slots & (a.max_slots - 1)))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_owner, dim3(static_cast<unsigned>(a.owners)), dim3(kOwnerBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rank(const RankArgs& a, int num_values, const CsrArgs& g, int routers, int items, int32_t* ids,
                       uint32_t* status, hipStream_t s) {
  if (routers < 1 || routers > kMaxRouters) return hipErrorInvalidValue;
  const unsigned grid = static_cast<unsigned>(routers);
#define GMB_RANK_I(V, W, I) \
  hipLaunchKernelGGL((k_rank<V, W, I>), dim3(grid), dim3(kScanBlock), 0, s, a, g, ids, status)
#define GMB_RANK_W(V, W)                       \
  switch (items) {                             \
    case 2: GMB_RANK_I(V, W, 2); break;        \
    case 4: GMB_RANK_I(V, W, 4); break;        \
    case 8: GMB_RANK_I(V, W, 8); break;        \
    case 16: GMB_RANK_I(V, W, 16); break;      \
    default: return hipErrorInvalidValue;      \
  }
#define GMB_RANK(V)         \
  if (g.wide) {             \
    GMB_RANK_W(V, true)     \
  } else {                  \
    GMB_RANK_W(V, false)    \
  }
  switch (num_values) {
    case 1: { GMB_RANK(1); } break;
    case 2: { GMB_RANK(2); } break;
    case 3: { GMB_RANK(3); } break;
    case 4: { GMB_RANK(4); } break;
    case 5: { GMB_RANK(5); } break;
    case 6: { GMB_RANK(6); } break;
    case 7: { GMB_RANK(7); } break;
    case 8: { GMB_RANK(8); } break;
    default: return hipErrorInvalidValue;
  }
#undef GMB_RANK
#undef GMB_RANK_W
#undef GMB_RANK_I
  return hipGetLastError();
}

hipError_t launch_validate(const ValidateArgs& b, int64_t num_nodes, uint32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(k_validate, dim3(grid_for(std::max(b.cap_dst + 1, b.cap_nnz))), dim3(256), 0, s, b, num_nodes,
                     status);
  return hipGetLastError();
}

hipError_t launch_fix(const DeferredArgs& fix, const int32_t* ids, const int32_t* clear_sizes, int64_t clear_cap,
                      uint32_t* table, int64_t num_nodes, hipStream_t s) {
  const int64_t cap = std::max<int64_t>(clear_cap, 1);
  hipLaunchKernelGGL(k_fix, dim3(grid_for(std::max(fix.cap, clear_sizes ? cap : 0))), dim3(256), 0, s, fix, ids,
                     clear_sizes, cap, table, num_nodes);
  return hipGetLastError();
}

}  // namespace gmb
