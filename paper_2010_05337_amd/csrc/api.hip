// C ABI of the mini-batch GNN hot path (declared in include/gmb.h):
// argument validation, workspace planning and kernel launches.  No C++
// exception crosses the ABI; every entry point returns a gmb_status.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>

#include "gmb.h"
#include "kernels.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  return GMB_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(GMB_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
constexpr int64_t kMaxInt32 = 0x7FFFFFFF;
constexpr size_t kStateHeader = 256;
// largest fan-out: one destination's edges must fit one relabel tile
constexpr int kMaxFanout = gmb::kScanBlock * 16;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// ---- sampling workspace plan -------------------------------------------

struct HopPlan {
  int layer;
  int fanout;
  int64_t cap_dst, cap_nnz, cap_src;
  size_t off_indptr, off_nbr, off_local;
  int64_t tiles_word, ticket_word, tile_stride;
  int items;
  bool table;                      // dedup through the state's per-vertex table (small hops)
  int32_t span, routers, owners;   // else by owners: destinations per router, routers, owners
};

struct SamplePlan {
  int num_layers;
  HopPlan hop[GMB_MAX_LAYERS];
  // the blocks (outputs), relative to the output buffer
  size_t off_ids, off_sizes;
  int64_t cap_ids;
  size_t out_total;
  // scratch, relative to the scratch buffer: the look-back words and
  // tickets of the relabel scans (cleared by the seed kernel), the running
  // edge count of every hop, and the dedup's pairs, answers, owner offsets
  // and router regions (one set, reused by every hop)
  size_t off_zero, off_totals, off_pairs, off_res, off_owner, off_rs;
  int64_t num_zero_words;
  size_t scratch_total;
  // one workspace holding both: the outputs, then the scratch
  size_t total;
};

constexpr int kTotalsWords = GMB_MAX_LAYERS;

// Fills the plan; returns GMB_OK or an argument error (message set).
int plan_sampling(int32_t num_seeds, const int32_t* fanouts, int32_t num_layers, int64_t num_nodes,
                  SamplePlan* plan) {
  if (num_layers < 1 || num_layers > GMB_MAX_LAYERS)
    return fail(GMB_EINVAL, "num_layers=%d outside 1..%d", num_layers, GMB_MAX_LAYERS);
  if (!fanouts) return fail(GMB_EINVAL, "fanouts is NULL");
  if (num_nodes < 1 || num_nodes > kMaxInt32)
    return fail(GMB_EINVAL, "num_nodes=%lld outside 1..2^31-1", static_cast<long long>(num_nodes));
  if (num_seeds < 0) return fail(GMB_EINVAL, "num_seeds=%d < 0", num_seeds);
  if (num_seeds > num_nodes)
    return fail(GMB_EINVAL, "num_seeds=%d exceeds num_nodes (seeds must be distinct)", num_seeds);
  for (int l = 0; l < num_layers; ++l)
    if (fanouts[l] < 1 || fanouts[l] > kMaxFanout)
      return fail(GMB_EINVAL, "fanouts[%d]=%d outside 1..%d", l, fanouts[l], kMaxFanout);

  SamplePlan p{};
  p.num_layers = num_layers;
  int64_t cap_dst = num_seeds;
  int64_t zero_words = 0;
  for (int h = 0; h < num_layers; ++h) {
    HopPlan& hp = p.hop[h];
    hp.layer = num_layers - 1 - h;
    hp.fanout = fanouts[hp.layer];
    hp.cap_dst = cap_dst;
    hp.cap_nnz = cap_dst * static_cast<int64_t>(hp.fanout);
    hp.cap_src = cap_dst + std::min<int64_t>(hp.cap_nnz, num_nodes);
    // every position (edge, source) and every edge tag must fit in 31 bits
    if (hp.cap_nnz >= kMaxInt32 || hp.cap_src >= kMaxInt32 || hp.cap_nnz + hp.cap_dst >= kMaxInt32)
      return fail(GMB_EINVAL, "hop %d: capacity %lld edges / %lld sources exceeds 2^31-1", h,
                  static_cast<long long>(hp.cap_nnz), static_cast<long long>(hp.cap_src));
    // The hops before the last dedup through the per-vertex table while
    // their fan-outs allow the group sampler (few edges, few table lines);
    // the last hop, and every hop after one that cannot, by owners.  The
    // relabel scan of hop h carries 1 + (later hops) values.
    hp.items = gmb::scan_items_for(hp.cap_nnz);
    hp.table = h + 1 < num_layers && hp.fanout <= 64 && (h == 0 || p.hop[h - 1].table);
    if (hp.table) {
      hp.tile_stride = gmb::scan_tiles(hp.cap_nnz, hp.items);
    } else {
      // a relabel tile is one router: `span` destinations whose edges fit it
      while (gmb::kScanBlock * hp.items < hp.fanout) hp.items *= 2;
      hp.span = std::min(gmb::kMaxSpan, std::max(1, gmb::kScanBlock * hp.items / hp.fanout));
      const int64_t routers = std::max<int64_t>(1, (hp.cap_dst + hp.span - 1) / hp.span);
      if (routers > gmb::kMaxRouters)
        return fail(GMB_EINVAL, "hop %d: %lld destinations need %lld routers, above %d", h,
                    static_cast<long long>(hp.cap_dst), static_cast<long long>(routers), gmb::kMaxRouters);
      hp.routers = static_cast<int32_t>(routers);
      const int64_t pairs = hp.cap_nnz + hp.cap_dst;
      int64_t owners = std::max<int64_t>(1, (pairs + gmb::kOwnerPairs - 1) / gmb::kOwnerPairs);
      // one owner per CU at a time: a count just past a multiple of the CU
      // count would run its last owners as a wave of their own, doubling
      // the kernel; take the multiple below while each owner's share at full
      // capacity still fits three quarters of its table
      if (owners > gmb::kComputeUnits) {
        const int64_t lower = (owners - 1) / gmb::kComputeUnits * gmb::kComputeUnits;
        if ((pairs + lower - 1) / lower <= gmb::kOwnerSlots * 3 / 4) owners = lower;
      }
      hp.owners = static_cast<int32_t>(std::min<int64_t>(gmb::kMaxOwners, owners));
      hp.tile_stride = hp.routers;
    }
    hp.tiles_word = zero_words;
    zero_words += hp.tile_stride * (num_layers - h);
    hp.ticket_word = zero_words++;
    cap_dst = hp.cap_src;
  }
  p.cap_ids = p.hop[num_layers - 1].cap_src;
  size_t off = 0;
  p.off_ids = off;
  off = align_up(off + sizeof(int32_t) * std::max<int64_t>(p.cap_ids, 1));
  p.off_sizes = off;
  off = align_up(off + sizeof(int32_t) * 4 * num_layers);
  for (int h = 0; h < num_layers; ++h) {
    HopPlan& hp = p.hop[h];
    hp.off_indptr = off;
    off = align_up(off + sizeof(int32_t) * (hp.cap_dst + 1));
    hp.off_nbr = off;
    off = align_up(off + sizeof(int32_t) * std::max<int64_t>(hp.cap_nnz, 1));
    hp.off_local = off;
    off = align_up(off + sizeof(int32_t) * std::max<int64_t>(hp.cap_nnz, 1));
  }
  p.out_total = off;
  off = 0;
  p.off_zero = off;
  p.num_zero_words = zero_words;
  off = align_up(off + sizeof(uint64_t) * zero_words);
  p.off_totals = off;
  off = align_up(off + sizeof(int32_t) * kTotalsWords);
  int64_t pairs = 1, owner_words = 1, routers = 1;
  for (int h = 0; h < num_layers; ++h) {
    const HopPlan& hp = p.hop[h];
    if (hp.table) continue;
    pairs = std::max(pairs, hp.cap_nnz + hp.cap_dst);
    owner_words = std::max(owner_words, static_cast<int64_t>(hp.owners + 1) * hp.routers);
    routers = std::max<int64_t>(routers, hp.routers);
  }
  p.off_pairs = off;
  off = align_up(off + 8 * static_cast<size_t>(pairs));
  p.off_res = off;
  off = align_up(off + 4 * static_cast<size_t>(pairs));
  p.off_owner = off;
  off = align_up(off + 4 * static_cast<size_t>(owner_words));
  p.off_rs = off;
  off = align_up(off + 4 * static_cast<size_t>(routers));
  p.scratch_total = off;
  p.total = p.out_total + p.scratch_total;
  *plan = p;
  return GMB_OK;
}

// Host-side checks shared by the sampling entry points (the buffers for the
// blocks and the scratch are checked by each).
int check_sampling(const gmb_csr* csr, const int32_t* seeds, int32_t num_seeds, const int32_t* fanouts,
                   int32_t num_layers, void* state, size_t state_bytes, SamplePlan* p) {
  if (!csr) return fail(GMB_EINVAL, "csr is NULL");
  if (!csr->indptr || (!csr->indices && csr->num_edges > 0))
    return fail(GMB_EINVAL, "csr has a NULL array");
  if (csr->indptr_bits != 32 && csr->indptr_bits != 64)
    return fail(GMB_EINVAL, "indptr_bits=%d (32 or 64)", csr->indptr_bits);
  if (csr->num_edges < 0 || (csr->indptr_bits == 32 && csr->num_edges > kMaxInt32))
    return fail(GMB_EINVAL, "num_edges=%lld does not fit the row-offset type", static_cast<long long>(csr->num_edges));
  if (num_seeds > 0 && !seeds) return fail(GMB_EINVAL, "seeds is NULL");
  int st = plan_sampling(num_seeds, fanouts, num_layers, csr->num_nodes, p);
  if (st != GMB_OK) return st;
  if (!state) return fail(GMB_EINVAL, "state is NULL");
  if (reinterpret_cast<uintptr_t>(state) % kAlign) return fail(GMB_EINVAL, "state must be 256-byte aligned");
  const size_t need = kStateHeader + align_up(sizeof(uint32_t) * static_cast<size_t>(csr->num_nodes));
  if (state_bytes < need) return fail(GMB_ENOSPC, "state holds %zu bytes, %zu needed", state_bytes, need);
  return GMB_OK;
}

// The owners' LDS table size limit: kOwnerSlots, or a smaller power of two
// from the environment variable GMB_OWNER_TABLE_SLOTS (64 .. kOwnerSlots), a
// test hook that makes owners overflow into the state table so that path
// runs on small inputs.
int32_t owner_slots() {
  const char* v = std::getenv("GMB_OWNER_TABLE_SLOTS");
  if (!v) return gmb::kOwnerSlots;
  const long x = std::strtol(v, nullptr, 10);
  int32_t slots = 64;
  while (slots < x && slots < gmb::kOwnerSlots) slots *= 2;
  return slots;
}

int enqueue_validation(const gmb_csr* csr, const gmb_blocks* b, uint32_t* status, hipStream_t s);
bool validate_every_call();

// Enqueues the sampling kernels: the blocks go to `outb` (plan offsets
// off_ids, off_sizes and the hops'), the scratch words to `scr`.
int run_sampling(const gmb_csr* csr, const int32_t* seeds, int32_t num_seeds, int32_t num_layers, uint64_t seed,
                 void* state, const SamplePlan& p, char* outb, char* scr, gmb_blocks* out, hipStream_t s) {
  int32_t* ids = reinterpret_cast<int32_t*>(outb + p.off_ids);
  int32_t* sizes = reinterpret_cast<int32_t*>(outb + p.off_sizes);
  uint64_t* zero = reinterpret_cast<uint64_t*>(scr + p.off_zero);
  int32_t* totals = reinterpret_cast<int32_t*>(scr + p.off_totals);
  uint32_t* status = static_cast<uint32_t*>(state);
  uint32_t* table = reinterpret_cast<uint32_t*>(static_cast<char*>(state) + kStateHeader);

  gmb::CsrArgs g{csr->indptr, csr->indices, csr->num_nodes, csr->indptr_bits == 64 ? 1 : 0};
  gmb::HopArgs hops[GMB_MAX_LAYERS];
  gmb_blocks res{};
  res.num_layers = num_layers;
  res.num_seeds = num_seeds;
  for (int h = 0; h < num_layers; ++h) {
    const HopPlan& hp = p.hop[h];
    gmb::HopArgs& a = hops[h];
    a.sizes = sizes + 4 * hp.layer;
    a.indptr = reinterpret_cast<int32_t*>(outb + hp.off_indptr);
    a.nbr = reinterpret_cast<int32_t*>(outb + hp.off_nbr);
    a.local = reinterpret_cast<int32_t*>(outb + hp.off_local);
    a.tiles = zero + hp.tiles_word;
    a.ticket = reinterpret_cast<uint32_t*>(zero + hp.ticket_word);
    a.tile_stride = hp.tile_stride;
    a.cap_dst = hp.cap_dst;
    a.cap_nnz = hp.cap_nnz;
    a.cap_src = hp.cap_src;
    a.fanout = hp.fanout;
    a.layer = hp.layer;
    gmb_block& bk = res.blk[hp.layer];
    bk.indptr = a.indptr;
    bk.indices = a.local;
    bk.nbr = a.nbr;
    bk.src_ids = ids;
    bk.sizes = a.sizes;
    bk.cap_dst = hp.cap_dst;
    bk.cap_src = hp.cap_src;
    bk.cap_nnz = hp.cap_nnz;
    bk.fanout = hp.fanout;
    bk.layer = hp.layer;
  }

  gmb::SeedArgs sa{};
  sa.seeds = seeds;
  sa.num_seeds = num_seeds;
  sa.first_sizes = 4 * p.hop[0].layer;
  sa.ids = ids;
  sa.zero = zero;
  sa.num_zero = p.num_zero_words;
  sa.sizes = sizes;
  sa.num_size_words = 4 * num_layers;
  sa.totals = totals;
  for (int h = 0; h < num_layers; ++h) {
    sa.indptr[h] = hops[h].indptr;
    sa.fanout[h] = hops[h].fanout;
  }
  const uint32_t k0 = static_cast<uint32_t>(seed), k1 = static_cast<uint32_t>(seed >> 32);
  hipError_t e = gmb::launch_seed_scan(sa, num_layers, g, s);
  if (e != hipSuccess) return hip_fail(e, "seed launch");
  uint2* pairs = reinterpret_cast<uint2*>(scr + p.off_pairs);
  int32_t* answers = reinterpret_cast<int32_t*>(scr + p.off_res);
  int32_t* owner_off = reinterpret_cast<int32_t*>(scr + p.off_owner);
  int32_t* region = reinterpret_cast<int32_t*>(scr + p.off_rs);
  for (int h = 0; h < num_layers; ++h) {
    const HopPlan& hp = p.hop[h];
    // the first hop has nothing deferred: word 3 of a block's sizes is 0
    gmb::DeferredArgs fix{hops[0].local, hops[0].sizes + 3 - gmb::kNnz, 1};
    if (h > 0) fix = gmb::DeferredArgs{hops[h - 1].local, hops[h - 1].sizes, std::max<int64_t>(hops[h - 1].cap_nnz, 1)};
    if (hp.table) {
      e = gmb::launch_sample_table(g, ids, hops[h], table, status, k0, k1, h == 0 ? 1 : 0, fix, s);
      if (e != hipSuccess) return hip_fail(e, "sample launch");
      gmb::AssignArgs aa{};
      aa.nbr = hops[h].nbr;
      aa.local = hops[h].local;
      aa.sizes = hops[h].sizes;
      aa.next_sizes = (h + 1 < num_layers) ? hops[h + 1].sizes : nullptr;
      aa.tiles = hops[h].tiles;
      aa.tile_stride = hops[h].tile_stride;
      aa.ticket = hops[h].ticket;
      aa.totals = totals;
      aa.hop = h;
      for (int v = 1; h + v < num_layers; ++v) {
        aa.indptr[v] = hops[h + v].indptr;
        aa.fanout[v] = hops[h + v].fanout;
      }
      e = gmb::launch_assign(aa, num_layers - h, g, hops[h].cap_nnz, hp.items, ids, table, status, s);
      if (e != hipSuccess) return hip_fail(e, "relabel launch");
      continue;
    }
    gmb::RouteArgs ra{hops[h].sizes, hops[h].indptr, ids, hops[h].nbr, pairs, owner_off, region,
                      csr->num_nodes, hp.span, hp.routers, hp.owners};
    if (hp.fanout <= 64) {
      gmb::SampleArgs sa{ids, hops[h].sizes, hops[h].indptr, hops[h].nbr, status, hp.fanout, hp.layer, k0, k1,
                         h == 0 ? 1 : 0, fix};
      e = gmb::launch_sample_route(g, sa, ra, s);
      if (e != hipSuccess) return hip_fail(e, "sample launch");
    } else {
      e = gmb::launch_sample(g, ids, hops[h], status, k0, k1, h == 0 ? 1 : 0, fix, s);
      if (e != hipSuccess) return hip_fail(e, "sample launch");
      e = gmb::launch_route(ra, s);
      if (e != hipSuccess) return hip_fail(e, "route launch");
    }
    gmb::OwnerArgs oa{pairs, owner_off, region, answers, table, status, hp.routers, hp.owners, owner_slots()};
    e = gmb::launch_owner(oa, s);
    if (e != hipSuccess) return hip_fail(e, "owner launch");
    gmb::RankArgs rk{};
    rk.pairs = pairs;
    rk.res = answers;
    rk.indptr0 = hops[h].indptr;
    rk.local = hops[h].local;
    rk.sizes = hops[h].sizes;
    rk.next_sizes = (h + 1 < num_layers) ? hops[h + 1].sizes : nullptr;
    rk.tiles = hops[h].tiles;
    rk.tile_stride = hops[h].tile_stride;
    rk.ticket = hops[h].ticket;
    rk.totals = totals;
    rk.hop = h;
    rk.span = hp.span;
    for (int v = 1; h + v < num_layers; ++v) {
      rk.indptr[v] = hops[h + v].indptr;
      rk.fanout[v] = hops[h + v].fanout;
    }
    e = gmb::launch_rank(rk, num_layers - h, g, hp.routers, hp.items, ids, status, s);
    if (e != hipSuccess) return hip_fail(e, "relabel launch");
  }
  // the last hop's deferred ids; the slots the table hops recorded (their
  // sources: the seeds and the vertices they added) back to empty
  int table_hops = 0;
  while (table_hops < num_layers && p.hop[table_hops].table) ++table_hops;
  const gmb::HopArgs& last = hops[num_layers - 1];
  const int32_t* clear = table_hops ? hops[table_hops - 1].sizes : nullptr;
  const int64_t clear_cap = table_hops ? hops[table_hops - 1].cap_src : 0;
  e = gmb::launch_fix(gmb::DeferredArgs{last.local, last.sizes, std::max<int64_t>(last.cap_nnz, 1)}, ids, clear,
                      clear_cap, table, csr->num_nodes, s);
  if (e != hipSuccess) return hip_fail(e, "deferred-id launch");
  *out = res;
  if (validate_every_call()) return enqueue_validation(csr, out, status, s);
  return ok();
}

// Enqueues the consistency check of every block (gmb_validate_blocks).
int enqueue_validation(const gmb_csr* csr, const gmb_blocks* b, uint32_t* status, hipStream_t s) {
  for (int l = 0; l < b->num_layers; ++l) {
    const gmb_block& k = b->blk[l];
    gmb::ValidateArgs v{k.indptr, k.indices, k.nbr, k.src_ids, k.sizes, k.cap_dst, k.cap_src, k.cap_nnz, k.fanout};
    hipError_t e = gmb::launch_validate(v, csr->num_nodes, status, s);
    if (e != hipSuccess) return hip_fail(e, "validation launch");
  }
  return GMB_OK;
}

// GMB_VALIDATE=1 in the environment: every sampling call checks its blocks.
bool validate_every_call() {
  const char* v = std::getenv("GMB_VALIDATE");
  return v && v[0] == '1';
}

// The scratch of gmb_sample_blocks_noalloc: a fixed array in device memory
// that every GPU the library runs on holds once, until the process ends.
// Host code never uses the name itself (on the host it is only a stand-in
// for the symbol): it uses the address hipGetSymbolAddress returns for the
// current device, taken once per device.
constexpr size_t kNoAllocScratchBytes = GMB_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
char* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`.
int noalloc_scratch(char** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(GMB_EDEVICE, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || reinterpret_cast<uintptr_t>(p) % kAlign) return fail(GMB_EDEVICE, "scratch symbol has no aligned device address");
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *ptr = g_scratch_ptr[dev];
  return GMB_OK;
}

// ---- forward workspace plan --------------------------------------------

struct ForwardPlan {
  size_t off_agg[GMB_MAX_LAYERS];      // every layer's mean (kept for the backward)
  size_t off_hidden[GMB_MAX_LAYERS];
  size_t total;
};

int check_blocks(const gmb_blocks* b) {
  if (!b) return fail(GMB_EINVAL, "blocks is NULL");
  if (b->num_layers < 1 || b->num_layers > GMB_MAX_LAYERS)
    return fail(GMB_EINVAL, "blocks->num_layers=%d outside 1..%d", b->num_layers, GMB_MAX_LAYERS);
  for (int l = 0; l < b->num_layers; ++l) {
    const gmb_block& k = b->blk[l];
    if (!k.indptr || !k.indices || !k.src_ids || !k.sizes)
      return fail(GMB_EINVAL, "block %d has a NULL array", l);
    if (k.cap_dst < 0 || k.cap_src < k.cap_dst || k.cap_nnz < 0)
      return fail(GMB_EINVAL, "block %d has inconsistent capacities", l);
  }
  return GMB_OK;
}

int plan_forward(const gmb_blocks* b, const gmb_sage_weights* w, ForwardPlan* plan) {
  int st = check_blocks(b);
  if (st != GMB_OK) return st;
  if (!w) return fail(GMB_EINVAL, "weights is NULL");
  if (w->num_layers != b->num_layers)
    return fail(GMB_EINVAL, "weights have %d layers, blocks %d", w->num_layers, b->num_layers);
  if (w->dtype != GMB_F32 && w->dtype != GMB_BF16) return fail(GMB_EINVAL, "dtype=%d unknown", w->dtype);
  for (int l = 0; l <= w->num_layers; ++l)
    if (w->dims[l] < 1 || w->dims[l] > 65536) return fail(GMB_EINVAL, "dims[%d]=%d outside 1..65536", l, w->dims[l]);
  for (int l = 0; l < w->num_layers; ++l)
    if (!w->w_self[l] || !w->w_neigh[l] || !w->bias[l]) return fail(GMB_EINVAL, "layer %d weight is NULL", l);
  for (int l = 1; l < b->num_layers; ++l)
    if (b->blk[l].cap_src != b->blk[l - 1].cap_dst)
      return fail(GMB_EINVAL, "block %d sources (cap %lld) are not block %d destinations (cap %lld)", l,
                  static_cast<long long>(b->blk[l].cap_src), l - 1,
                  static_cast<long long>(b->blk[l - 1].cap_dst));
  const size_t es = w->dtype == GMB_BF16 ? 2 : 4;
  ForwardPlan p{};
  size_t off = 0;
  for (int l = 0; l < w->num_layers; ++l) {
    p.off_agg[l] = off;
    off = align_up(off + static_cast<size_t>(std::max<int64_t>(b->blk[l].cap_dst, 1)) * w->dims[l] * es);
  }
  for (int l = 0; l + 1 < w->num_layers; ++l) {
    p.off_hidden[l] = off;
    off = align_up(off + static_cast<size_t>(std::max<int64_t>(b->blk[l].cap_dst, 1)) * w->dims[l + 1] * es);
  }
  p.total = off;
  *plan = p;
  return GMB_OK;
}

int check_forward(const gmb_blocks* blocks, const gmb_sage_weights* weights, const float* logits, const void* ws,
                  size_t ws_bytes, ForwardPlan* p) {
  int st = plan_forward(blocks, weights, p);
  if (st != GMB_OK) return st;
  if (!logits && blocks->num_seeds > 0) return fail(GMB_EINVAL, "logits is NULL");
  if (!ws) return fail(GMB_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign) return fail(GMB_EINVAL, "workspace is not 256-byte aligned");
  if (ws_bytes < p->total) return fail(GMB_ENOSPC, "workspace holds %zu bytes, %zu needed", ws_bytes, p->total);
  return GMB_OK;
}

// The layers in order.  Layer 0's linear reads its destination rows from
// x_self; its mean reads the rows mean_rows[mean_ids[e]] (the gathered
// input and the local ids, or the feature table and the global ids).
int run_forward(const gmb_blocks* blocks, const void* x_self, const int32_t* mean_ids, const void* mean_rows,
                int64_t mean_max_id, const gmb_sage_weights* weights, float* logits, const ForwardPlan& p,
                void* ws, hipStream_t s) {
  const int L = weights->num_layers;
  const int bf16 = weights->dtype == GMB_BF16;
  char* base = static_cast<char*>(ws);
  const void* h_in = x_self;
  for (int l = 0; l < L; ++l) {
    const gmb_block& bk = blocks->blk[l];
    void* agg = base + p.off_agg[l];
    const int d_in = weights->dims[l], d_out = weights->dims[l + 1];
    const bool last = (l == L - 1);
    void* h_out = last ? static_cast<void*>(logits) : static_cast<void*>(base + p.off_hidden[l]);
    const int32_t* ids = l == 0 ? mean_ids : bk.indices;
    const void* rows = l == 0 ? mean_rows : h_in;
    const int64_t max_id = l == 0 ? mean_max_id : std::max<int64_t>(bk.cap_src, 1);
    hipError_t e = gmb::launch_mean_aggregate(bk.sizes, bk.indptr, ids, rows, d_in, bf16, agg, bk.cap_dst,
                                              bk.fanout, max_id, s);
    if (e != hipSuccess) return hip_fail(e, "mean-aggregation launch");
    e = gmb::launch_sage_linear(bk.sizes, h_in, agg, weights->w_self[l], weights->w_neigh[l],
                                weights->bias[l], d_in, d_out, bf16, last ? 0 : 1,
                                (last || !bf16) ? 1 : 0, h_out, bk.cap_dst, s);
    if (e != hipSuccess) return hip_fail(e, "linear launch");
    h_in = h_out;
  }
  return ok();
}

}  // namespace

extern "C" {

int32_t gmb_abi_version(void) { return GMB_ABI_VERSION; }

const char* gmb_last_error(void) { return g_last_error.c_str(); }

size_t gmb_sampler_state_bytes(int64_t num_nodes) {
  if (num_nodes < 1 || num_nodes > kMaxInt32) return 0;
  return kStateHeader + align_up(sizeof(uint32_t) * static_cast<size_t>(num_nodes));
}

uint32_t* gmb_state_status_word(void* state) { return static_cast<uint32_t*>(state); }

int gmb_sampler_state_init(void* state, size_t state_bytes, int64_t num_nodes, void* stream) {
  const size_t need = gmb_sampler_state_bytes(num_nodes);
  if (need == 0) return fail(GMB_EINVAL, "num_nodes=%lld outside 1..2^31-1", static_cast<long long>(num_nodes));
  if (!state) return fail(GMB_EINVAL, "state is NULL");
  if (reinterpret_cast<uintptr_t>(state) % kAlign) return fail(GMB_EINVAL, "state is not 256-byte aligned");
  if (state_bytes < need) return fail(GMB_ENOSPC, "state holds %zu bytes, %zu needed", state_bytes, need);
  uint32_t* status = static_cast<uint32_t*>(state);
  uint32_t* table = reinterpret_cast<uint32_t*>(static_cast<char*>(state) + kStateHeader);
  hipError_t e = gmb::launch_state_init(table, status, num_nodes, as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "state init launch");
  return ok();
}

int gmb_read_status(void* state, void* stream) {
  if (!state) return fail(GMB_EINVAL, "state is NULL");
  // the status word and (at byte 8) the vertex count written by the init
  uint32_t head[4] = {0, 0, 0, 0};
  hipError_t e = hipStreamSynchronize(as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "stream synchronize");
  e = hipMemcpy(head, state, sizeof head, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "status read");
  const uint32_t word = head[0];
  if (word != 0) {
    e = hipMemset(state, 0, sizeof word);
    if (e != hipSuccess) return hip_fail(e, "status clear");
  }
  if (word & GMB_STATUS_INTERNAL) {
    // the relabel numbered some vertices wrongly, so the call's cleanup may
    // have missed table slots: clear the whole table again
    int64_t n = 0;
    std::memcpy(&n, head + 2, sizeof n);
    if (n >= 1 && n <= kMaxInt32) {
      uint32_t* table = reinterpret_cast<uint32_t*>(static_cast<char*>(state) + kStateHeader);
      e = gmb::launch_state_init(table, static_cast<uint32_t*>(state), n, as_stream(stream));
      if (e == hipSuccess) e = hipStreamSynchronize(as_stream(stream));
      if (e != hipSuccess) return hip_fail(e, "state re-init");
    }
  }
  if (word & GMB_STATUS_ERANGE) return fail(GMB_ERANGE, "a vertex id outside [0, num_nodes) was found on the device");
  if (word & GMB_STATUS_EDUP) return fail(GMB_EDUP, "the seed list holds a vertex more than once");
  if (word & GMB_STATUS_INTERNAL)
    return fail(GMB_EDEVICE, "a bounded wait in the relabel scan ran out: the blocks of that call are wrong "
                             "(the sampler state has been cleared again)");
  if (word & GMB_STATUS_INVALID) return fail(GMB_EDEVICE, "gmb_validate_blocks found an inconsistent block");
  return ok();
}

size_t gmb_sample_workspace_bytes(int32_t num_seeds, const int32_t* fanouts, int32_t num_layers,
                                  int64_t num_nodes) {
  SamplePlan p;
  if (plan_sampling(num_seeds, fanouts, num_layers, num_nodes, &p) != GMB_OK) return 0;
  return p.total;
}

int gmb_sample_blocks(const gmb_csr* csr, const int32_t* seeds, int32_t num_seeds,
                      const int32_t* fanouts, int32_t num_layers, uint64_t seed, void* state,
                      size_t state_bytes, void* ws, size_t ws_bytes, gmb_blocks* out, void* stream) {
  SamplePlan p;
  int st = check_sampling(csr, seeds, num_seeds, fanouts, num_layers, state, state_bytes, &p);
  if (st != GMB_OK) return st;
  if (!ws) return fail(GMB_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign) return fail(GMB_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < p.total) return fail(GMB_ENOSPC, "workspace holds %zu bytes, %zu needed", ws_bytes, p.total);
  char* base = static_cast<char*>(ws);
  return run_sampling(csr, seeds, num_seeds, num_layers, seed, state, p, base, base + p.out_total, out,
                      as_stream(stream));
}

int gmb_sample_blocks_noalloc(const gmb_csr* csr, const int32_t* seeds, int32_t num_seeds, const int32_t* fanouts,
                              int32_t num_layers, uint64_t seed, void* state, size_t state_bytes, void* out_buf,
                              size_t out_bytes, gmb_blocks* out, void* stream) {
  SamplePlan p;
  int st = check_sampling(csr, seeds, num_seeds, fanouts, num_layers, state, state_bytes, &p);
  if (st != GMB_OK) return st;
  if (!out_buf) return fail(GMB_EINVAL, "output buffer is NULL");
  if (reinterpret_cast<uintptr_t>(out_buf) % kAlign) return fail(GMB_EINVAL, "output buffer must be 256-byte aligned");
  if (out_bytes < p.out_total)
    return fail(GMB_ENOSPC, "output buffer holds %zu bytes, %zu needed", out_bytes, p.out_total);
  if (p.scratch_total > kNoAllocScratchBytes)
    return fail(GMB_ENOSPC, "these shapes need %zu bytes of scratch, above the fixed %zu of the no-allocation entry point",
                p.scratch_total, kNoAllocScratchBytes);
  char* scratch_ptr = nullptr;
  st = noalloc_scratch(&scratch_ptr);
  if (st != GMB_OK) return st;
  return run_sampling(csr, seeds, num_seeds, num_layers, seed, state, p, static_cast<char*>(out_buf), scratch_ptr,
                      out, as_stream(stream));
}

int gmb_validate_blocks(const gmb_csr* csr, const gmb_blocks* blocks, void* state, void* stream) {
  if (!csr) return fail(GMB_EINVAL, "csr is NULL");
  if (csr->num_nodes < 1 || csr->num_nodes > kMaxInt32)
    return fail(GMB_EINVAL, "num_nodes=%lld outside 1..2^31-1", static_cast<long long>(csr->num_nodes));
  int st = check_blocks(blocks);
  if (st != GMB_OK) return st;
  if (!state) return fail(GMB_EINVAL, "state is NULL");
  return enqueue_validation(csr, blocks, static_cast<uint32_t*>(state), as_stream(stream));
}

int gmb_read_sizes(const gmb_blocks* blocks, int64_t* sizes, void* stream) {
  int st = check_blocks(blocks);
  if (st != GMB_OK) return st;
  if (!sizes) return fail(GMB_EINVAL, "sizes is NULL");
  hipError_t e = hipStreamSynchronize(as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "stream synchronize");
  for (int l = 0; l < blocks->num_layers; ++l) {
    int32_t w[4];
    e = hipMemcpy(w, blocks->blk[l].sizes, sizeof w, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "size read");
    sizes[3 * l + 0] = w[gmb::kNDst];
    sizes[3 * l + 1] = w[gmb::kNSrc];
    sizes[3 * l + 2] = w[gmb::kNnz];
  }
  return ok();
}

int gmb_gather_features(const int32_t* ids, const int32_t* n_dev, int64_t n_cap, const void* feats,
                        int64_t num_nodes, int32_t dim, int32_t dtype, void* out, uint32_t* status,
                        void* stream) {
  if (n_cap < 0) return fail(GMB_EINVAL, "n_cap=%lld < 0", static_cast<long long>(n_cap));
  if (dim < 1) return fail(GMB_EINVAL, "dim=%d < 1", dim);
  if (dtype != GMB_F32 && dtype != GMB_BF16) return fail(GMB_EINVAL, "dtype=%d unknown", dtype);
  if (num_nodes < 1 || num_nodes > kMaxInt32)
    return fail(GMB_EINVAL, "num_nodes=%lld outside 1..2^31-1", static_cast<long long>(num_nodes));
  if (n_cap == 0) return ok();
  if (!ids || !feats || !out) return fail(GMB_EINVAL, "a NULL array");
  const int64_t row_bytes = static_cast<int64_t>(dim) * (dtype == GMB_BF16 ? 2 : 4);
  hipError_t e = gmb::launch_gather(ids, n_dev, n_cap, feats, num_nodes, row_bytes, out, status,
                                    as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "gather launch");
  return ok();
}

size_t gmb_forward_workspace_bytes(const gmb_blocks* blocks, const gmb_sage_weights* weights) {
  ForwardPlan p;
  if (plan_forward(blocks, weights, &p) != GMB_OK) return 0;
  return p.total;
}

int64_t gmb_forward_hidden_offset(const gmb_blocks* blocks, const gmb_sage_weights* weights, int32_t layer) {
  ForwardPlan p;
  if (plan_forward(blocks, weights, &p) != GMB_OK) return -1;
  if (layer < 0 || layer + 1 >= weights->num_layers) return -1;
  return static_cast<int64_t>(p.off_hidden[layer]);
}

int gmb_sage_forward(const gmb_blocks* blocks, const void* x, const gmb_sage_weights* weights,
                     float* logits, void* ws, size_t ws_bytes, void* stream) {
  ForwardPlan p;
  int st = check_forward(blocks, weights, logits, ws, ws_bytes, &p);
  if (st != GMB_OK) return st;
  if (blocks->num_seeds == 0) return ok();   // an empty batch: no rows anywhere
  if (!x) return fail(GMB_EINVAL, "x is NULL");
  const gmb_block& b0 = blocks->blk[0];
  return run_forward(blocks, x, b0.indices, x, std::max<int64_t>(b0.cap_src, 1), weights, logits, p, ws,
                     as_stream(stream));
}

int gmb_sage_forward_fused(const gmb_blocks* blocks, const void* feats, int64_t num_nodes, void* x_dst,
                           const gmb_sage_weights* weights, float* logits, void* ws, size_t ws_bytes,
                           uint32_t* status, void* stream) {
  ForwardPlan p;
  int st = check_forward(blocks, weights, logits, ws, ws_bytes, &p);
  if (st != GMB_OK) return st;
  if (!feats) return fail(GMB_EINVAL, "feats is NULL");
  if (num_nodes < 1 || num_nodes > kMaxInt32)
    return fail(GMB_EINVAL, "num_nodes=%lld outside 1..2^31-1", static_cast<long long>(num_nodes));
  if (blocks->num_seeds == 0) return ok();   // an empty batch: no rows anywhere
  if (!x_dst) return fail(GMB_EINVAL, "x_dst is NULL");
  const hipStream_t s = as_stream(stream);
  const gmb_block& b0 = blocks->blk[0];
  const int64_t row_bytes = static_cast<int64_t>(weights->dims[0]) * (weights->dtype == GMB_BF16 ? 2 : 4);
  // block 0's destinations are the first n_dst source ids
  hipError_t e = gmb::launch_gather(b0.src_ids, b0.sizes + gmb::kNDst, b0.cap_dst, feats, num_nodes, row_bytes,
                                    x_dst, status, s);
  if (e != hipSuccess) return hip_fail(e, "gather launch");
  return run_forward(blocks, x_dst, b0.nbr, feats, num_nodes, weights, logits, p, ws, s);
}

}  // extern "C"

// ---- training step ------------------------------------------------------

namespace {

struct BackwardPlan {
  int ldz[GMB_MAX_LAYERS];   // row stride of dZ of layer l (floats, multiple of 4)
  size_t off_a, off_b, off_dm, off_part, off_lossrows;
  size_t off_cnt, off_off, off_pos, off_csc, off_long;   // the transpose of a block
  int64_t cnt_len;                             // ints of the edge counters
  int64_t scan_len;                            // ints of one layer's scan state
  int64_t clear_len;                           // ints cleared at the start (counters + scan states)
  size_t total;
  // bf16 models: fp32 copies of what the backward reads (the forward
  // workspace laid out for fp32, block 0's destination rows of x, the
  // matrices), after the fp32 backward's own workspace
  size_t off_shadow, off_x32, off_w32[GMB_MAX_LAYERS][2];
  size_t fp32_total;
};

// embed: layer 0's inputs are learnable vertex embeddings, so the backward
// also runs layer 0's input gradient and its transpose (the rows it needs:
// layer 0's destinations for the self part and the mean's gradient).
int plan_backward_f32(const gmb_blocks* b, const gmb_sage_weights* w, BackwardPlan* plan, bool embed);

// The fp32 weights struct of a bf16 model's training step: the same dims
// and biases, the matrices at the fp32 copies of the plan in `ws`.
gmb_sage_weights widened_weights(const gmb_sage_weights* w, const BackwardPlan& p, char* ws) {
  gmb_sage_weights w32 = *w;
  w32.dtype = GMB_F32;
  for (int l = 0; l < w->num_layers; ++l) {
    w32.w_self[l] = ws + p.off_w32[l][0];
    w32.w_neigh[l] = ws + p.off_w32[l][1];
  }
  return w32;
}

int plan_backward(const gmb_blocks* b, const gmb_sage_weights* w, BackwardPlan* plan, bool embed) {
  if (!w) return fail(GMB_EINVAL, "weights is NULL");
  if (w->dtype != GMB_BF16) return plan_backward_f32(b, w, plan, embed);
  if (embed) return fail(GMB_EINVAL, "learnable embeddings are fp32 only");
  // the fp32 backward on fp32 copies, then room for the copies
  gmb_sage_weights w32 = *w;
  w32.dtype = GMB_F32;
  BackwardPlan p;
  int st = plan_backward_f32(b, &w32, &p, false);
  if (st != GMB_OK) return st;
  ForwardPlan fp32;
  plan_forward(b, &w32, &fp32);
  size_t off = p.total;
  p.fp32_total = p.total;
  p.off_shadow = off;
  off = align_up(off + fp32.total);
  p.off_x32 = off;
  off = align_up(off + 4 * static_cast<size_t>(std::max<int64_t>(b->blk[0].cap_dst, 1)) * w->dims[0]);
  for (int l = 0; l < w->num_layers; ++l)
    for (int k = 0; k < 2; ++k) {
      p.off_w32[l][k] = off;
      off = align_up(off + 4 * static_cast<size_t>(w->dims[l]) * w->dims[l + 1]);
    }
  p.total = off;
  *plan = p;
  return GMB_OK;
}

int plan_backward_f32(const gmb_blocks* b, const gmb_sage_weights* w, BackwardPlan* plan, bool embed) {
  ForwardPlan fp;
  int st = plan_forward(b, w, &fp);
  if (st != GMB_OK) return st;
  if (w->dtype != GMB_F32) return fail(GMB_EINVAL, "the training step is fp32 only");
  const int L = w->num_layers;
  const int first = embed ? 0 : 1;   // the lowest layer whose input gradient runs
  for (int l = first; l < L; ++l)
    if (w->dims[l] % 4) return fail(GMB_EINVAL, "dims[%d]=%d is not a multiple of 4", l, w->dims[l]);
  for (int l = first; l < L; ++l)
    if (w->dims[l + 1] > 640) return fail(GMB_EINVAL, "dims[%d]=%d above 640 (input-gradient kernel)", l + 1, w->dims[l + 1]);
  BackwardPlan p{};
  size_t buf = 0, dm = 0, part = 0, src = 1, nnz = 1;
  for (int l = 0; l < L; ++l) {
    const int d_in = w->dims[l], d_out = w->dims[l + 1];
    const gmb_block& k = b->blk[l];
    p.ldz[l] = (l == L - 1) ? (d_out + 3) / 4 * 4 : d_out;
    buf = std::max(buf, static_cast<size_t>(std::max<int64_t>(k.cap_dst, 1)) * p.ldz[l]);
    if (l > 0) buf = std::max(buf, static_cast<size_t>(std::max<int64_t>(k.cap_src, 1)) * d_in);
    if (l == 0 && embed) buf = std::max(buf, static_cast<size_t>(std::max<int64_t>(k.cap_dst, 1)) * d_in);
    if (l >= first) {
      dm = std::max(dm, static_cast<size_t>(std::max<int64_t>(k.cap_dst, 1)) * d_in);
      src = std::max(src, static_cast<size_t>(k.cap_src));
      nnz = std::max(nnz, static_cast<size_t>(k.cap_nnz));
    }
    const size_t parts = gmb::wgrad_parts(std::max<int64_t>(k.cap_dst, 1), d_in, d_out);
    part = std::max(part, parts * (2 * static_cast<size_t>(d_in) + 1) * gmb::wgrad_ldp(d_out));
  }
  size_t off = 0;
  p.off_a = off;
  off = align_up(off + 4 * buf);
  p.off_b = off;
  off = align_up(off + 4 * buf);
  p.off_dm = off;
  off = align_up(off + 4 * std::max<size_t>(dm, 1));
  p.off_part = off;
  off = align_up(off + 4 * part);
  p.off_lossrows = off;
  off = align_up(off + 4 * static_cast<size_t>(std::max(b->num_seeds, 1)));
  p.cnt_len = static_cast<int64_t>((src + 1) / 2 * 2);
  p.scan_len = 2 + 2 * gmb::csc_scan_tiles(static_cast<int64_t>(src));
  p.clear_len = p.cnt_len + static_cast<int64_t>(std::max(L - first, 0)) * p.scan_len;
  p.off_cnt = off;
  off = align_up(off + 4 * static_cast<size_t>(p.clear_len));
  p.off_off = off;
  off = align_up(off + 4 * (src + 1));
  p.off_pos = off;
  off = align_up(off + 4 * src);
  p.off_csc = off;
  off = align_up(off + 8 * nnz);
  p.off_long = off;
  off = align_up(off + 4 * src);
  p.total = off;
  *plan = p;
  return GMB_OK;
}

int check_grads(const gmb_sage_grads* g, const gmb_sage_weights* w) {
  if (!g) return fail(GMB_EINVAL, "grads is NULL");
  if (g->num_layers != w->num_layers)
    return fail(GMB_EINVAL, "grads have %d layers, weights %d", g->num_layers, w->num_layers);
  for (int l = 0; l < w->num_layers; ++l)
    if (!g->d_self[l] || !g->d_neigh[l] || !g->d_bias[l]) return fail(GMB_EINVAL, "layer %d gradient is NULL", l);
  return GMB_OK;
}

// Transpose scans over at most this many sources take the weight
// gradient's products into their launch (a larger scan's own workgroups
// would hold the CUs while the products wait behind them: measured slower
// on the 1.06M-source scan of layer 0 with learnable embeddings, whose
// products take the part-product kernel of their own launch).
constexpr int64_t kFoldScanSources = 262144;

// The backward from the loss down; with table != NULL layer 0's input
// gradient is applied to the embedding rows of block 0's sources.
int run_backward(const gmb_blocks* blocks, const void* x, const gmb_sage_weights* weights, const float* logits,
                 const int32_t* labels, const void* fwd_ws, size_t fwd_ws_bytes, const gmb_sage_grads* grads,
                 float* loss, void* ws, size_t ws_bytes, float* table, int64_t num_nodes, float emb_lr,
                 void* stream) {
  const bool embed = table != nullptr;
  BackwardPlan p;
  int st = plan_backward(blocks, weights, &p, embed);
  if (st != GMB_OK) return st;
  ForwardPlan fp;
  plan_forward(blocks, weights, &fp);
  st = check_grads(grads, weights);
  if (st != GMB_OK) return st;
  if (!fwd_ws || fwd_ws_bytes < fp.total) return fail(GMB_ENOSPC, "forward workspace missing or too small");
  if (!ws) return fail(GMB_EINVAL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign || reinterpret_cast<uintptr_t>(fwd_ws) % kAlign)
    return fail(GMB_EINVAL, "workspaces must be 256-byte aligned");
  if (ws_bytes < p.total) return fail(GMB_ENOSPC, "workspace holds %zu bytes, %zu needed", ws_bytes, p.total);
  const hipStream_t s = as_stream(stream);
  const int L = weights->num_layers;
  if (weights->dtype == GMB_BF16 && blocks->num_seeds > 0) {
    // a bf16 model: widen what the backward reads to fp32 (block 0's
    // destination rows of x, every layer's mean and hidden output in the
    // fp32 layout, the matrices), then the fp32 backward on the copies
    if (!x) return fail(GMB_EINVAL, "x is NULL");
    char* base = static_cast<char*>(ws);
    const gmb_sage_weights w32 = widened_weights(weights, p, base);
    ForwardPlan f32;
    plan_forward(blocks, &w32, &f32);
    const char* fsrc = static_cast<const char*>(fwd_ws);
    gmb::WidenArgs wa{};
    auto add = [&](const void* src, void* dst, const int32_t* rows_dev, int64_t cap_rows, int64_t cols) {
      wa.src[wa.count] = static_cast<const uint16_t*>(src);
      wa.dst[wa.count] = static_cast<float*>(dst);
      wa.rows_dev[wa.count] = rows_dev;
      wa.cap_rows[wa.count] = cap_rows;
      wa.cols[wa.count++] = cols;
    };
    const gmb_block& b0 = blocks->blk[0];
    add(x, base + p.off_x32, b0.sizes + gmb::kNDst, std::max<int64_t>(b0.cap_dst, 1), weights->dims[0]);
    for (int l = 0; l < L; ++l) {
      const gmb_block& bk = blocks->blk[l];
      add(fsrc + fp.off_agg[l], base + p.off_shadow + f32.off_agg[l], bk.sizes + gmb::kNDst,
          std::max<int64_t>(bk.cap_dst, 1), weights->dims[l]);
      if (l + 1 < L)
        add(fsrc + fp.off_hidden[l], base + p.off_shadow + f32.off_hidden[l], bk.sizes + gmb::kNDst,
            std::max<int64_t>(bk.cap_dst, 1), weights->dims[l + 1]);
      add(weights->w_self[l], base + p.off_w32[l][0], nullptr, weights->dims[l], weights->dims[l + 1]);
      add(weights->w_neigh[l], base + p.off_w32[l][1], nullptr, weights->dims[l], weights->dims[l + 1]);
    }
    hipError_t e = gmb::launch_widen(wa, s);
    if (e != hipSuccess) return hip_fail(e, "widen launch");
    return run_backward(blocks, base + p.off_x32, &w32, logits, labels, base + p.off_shadow, f32.total, grads, loss,
                        ws, p.fp32_total, nullptr, 0, 0.f, stream);
  }
  if (blocks->num_seeds == 0) {
    // an empty batch: the mean over no seeds is taken as 0, so are the
    // gradients, and no embedding row changes
    gmb::SgdArgs z{};
    for (int l = 0; l < L; ++l) {
      const int64_t n = static_cast<int64_t>(weights->dims[l]) * weights->dims[l + 1];
      z.w[z.count] = grads->d_self[l];
      z.n[z.count++] = n;
      z.w[z.count] = grads->d_neigh[l];
      z.n[z.count++] = n;
      z.w[z.count] = grads->d_bias[l];
      z.n[z.count++] = weights->dims[l + 1];
    }
    hipError_t e = gmb::launch_zero(z, loss, s);
    if (e != hipSuccess) return hip_fail(e, "zero-fill launch");
    return ok();
  }
  if (!x || !logits || !labels) return fail(GMB_EINVAL, "x, logits or labels is NULL");
  char* base = static_cast<char*>(ws);
  const char* fbase = static_cast<const char*>(fwd_ws);
  float* cur = reinterpret_cast<float*>(base + p.off_a);
  float* other = reinterpret_cast<float*>(base + p.off_b);
  float* dM = reinterpret_cast<float*>(base + p.off_dm);
  float* part = reinterpret_cast<float*>(base + p.off_part);
  int32_t* cnt = reinterpret_cast<int32_t*>(base + p.off_cnt);
  int32_t* offs = reinterpret_cast<int32_t*>(base + p.off_off);
  int32_t* pos = reinterpret_cast<int32_t*>(base + p.off_pos);
  int2* csc = reinterpret_cast<int2*>(base + p.off_csc);
  int32_t* long_rows = reinterpret_cast<int32_t*>(base + p.off_long);
  float* loss_rows = reinterpret_cast<float*>(base + p.off_lossrows);
  hipError_t e = gmb::launch_xent(logits, labels, blocks->num_seeds, weights->dims[L], p.ldz[L - 1], cur,
                                  loss_rows, cnt, p.clear_len, s);
  if (e != hipSuccess) return hip_fail(e, "loss launch");
  for (int l = L - 1; l >= 0; --l) {
    const gmb_block& bk = blocks->blk[l];
    const int d_in = weights->dims[l], d_out = weights->dims[l + 1];
    const float* h_in = l == 0 ? static_cast<const float*>(x)
                               : reinterpret_cast<const float*>(fbase + fp.off_hidden[l - 1]);
    const float* m = reinterpret_cast<const float*>(fbase + fp.off_agg[l]);
    // the last layer's reduction also sums the loss.  On a layer whose
    // input gradient runs, the weight gradient's reduction rides in the
    // transpose fill's launch, and, while the transpose scan is small
    // enough not to hold the CUs back, its products in the scan's
    // (described here, launched by launch_mean_backward after the input
    // gradient)
    const bool top = l == L - 1;
    const bool below = l > 0 || embed;
    const bool beside_scan = below && bk.cap_src <= kFoldScanSources;
    gmb::WgradArgs defer{};
    gmb::ReduceArgs fold{};
    e = gmb::launch_wgrad(bk.sizes, h_in, m, d_in, cur, p.ldz[l], d_out, std::max<int64_t>(bk.cap_dst, 1), part,
                          grads->d_self[l], grads->d_neigh[l], grads->d_bias[l], top ? loss_rows : nullptr,
                          blocks->num_seeds, top ? loss : nullptr, beside_scan ? &defer : nullptr,
                          below ? &fold : nullptr, s);
    if (e != hipSuccess) return hip_fail(e, "weight-gradient launch");
    if (!below) break;
    // dZ [W_self; W_neigh]^T: dH_self into `other`, dM; the block's
    // in-edge counts per source on the way
    e = gmb::launch_dgrad(bk.sizes, cur, p.ldz[l], d_out, static_cast<const float*>(weights->w_self[l]),
                          static_cast<const float*>(weights->w_neigh[l]), d_in, other, dM, bk.cap_dst, bk.indptr,
                          bk.indices, bk.cap_nnz, bk.fanout, cnt, s);
    if (e != hipSuccess) return hip_fail(e, "input-gradient launch");
    // the mean's backward through the block's transpose, the ReLU of the
    // layer below on the way out: `other` becomes that layer's dZ; on layer
    // 0 (learnable embeddings) the input gradient goes into the table rows
    uint32_t* scan_state = reinterpret_cast<uint32_t*>(cnt + p.cnt_len + (embed ? l : l - 1) * p.scan_len);
    e = gmb::launch_mean_backward(bk.sizes, bk.indptr, bk.indices, bk.cap_nnz, bk.fanout, dM,
                                  l == 0 ? nullptr : h_in, d_in, other, bk.cap_dst, bk.cap_src, cnt, offs, pos,
                                  scan_state, csc, long_rows, l == 0 ? table : nullptr, bk.src_ids, num_nodes,
                                  emb_lr, beside_scan ? &defer : nullptr, &fold, s);
    if (e != hipSuccess) return hip_fail(e, "mean-backward launch");
    std::swap(cur, other);
  }
  return ok();
}

}  // namespace

extern "C" {

size_t gmb_backward_workspace_bytes(const gmb_blocks* blocks, const gmb_sage_weights* weights) {
  BackwardPlan p;
  if (plan_backward(blocks, weights, &p, false) != GMB_OK) return 0;
  return p.total;
}

size_t gmb_backward_embedding_workspace_bytes(const gmb_blocks* blocks, const gmb_sage_weights* weights) {
  BackwardPlan p;
  if (plan_backward(blocks, weights, &p, true) != GMB_OK) return 0;
  return p.total;
}

int gmb_sage_backward(const gmb_blocks* blocks, const void* x, const gmb_sage_weights* weights,
                      const float* logits, const int32_t* labels, const void* fwd_ws, size_t fwd_ws_bytes,
                      const gmb_sage_grads* grads, float* loss, void* ws, size_t ws_bytes, void* stream) {
  return run_backward(blocks, x, weights, logits, labels, fwd_ws, fwd_ws_bytes, grads, loss, ws, ws_bytes, nullptr,
                      0, 0.f, stream);
}

int gmb_sage_backward_embedding(const gmb_blocks* blocks, const void* x, const gmb_sage_weights* weights,
                                const float* logits, const int32_t* labels, const void* fwd_ws, size_t fwd_ws_bytes,
                                const gmb_sage_grads* grads, float* loss, void* ws, size_t ws_bytes, float* table,
                                int64_t num_nodes, float emb_lr, void* stream) {
  if (!table) return fail(GMB_EINVAL, "table is NULL");
  if (num_nodes < 1 || num_nodes > kMaxInt32)
    return fail(GMB_EINVAL, "num_nodes=%lld outside 1..2^31-1", static_cast<long long>(num_nodes));
  if (reinterpret_cast<uintptr_t>(table) % 16) return fail(GMB_EINVAL, "table must be 16-byte aligned");
  return run_backward(blocks, x, weights, logits, labels, fwd_ws, fwd_ws_bytes, grads, loss, ws, ws_bytes, table,
                      num_nodes, emb_lr, stream);
}

int gmb_sgd_update(const gmb_sage_weights* weights, const gmb_sage_grads* grads, float lr, void* stream) {
  if (!weights) return fail(GMB_EINVAL, "weights is NULL");
  if (weights->dtype != GMB_F32) return fail(GMB_EINVAL, "the update is fp32 only");
  if (weights->num_layers < 1 || weights->num_layers > GMB_MAX_LAYERS)
    return fail(GMB_EINVAL, "num_layers=%d outside 1..%d", weights->num_layers, GMB_MAX_LAYERS);
  int st = check_grads(grads, weights);
  if (st != GMB_OK) return st;
  gmb::SgdArgs a{};
  for (int l = 0; l < weights->num_layers; ++l) {
    const int64_t n = static_cast<int64_t>(weights->dims[l]) * weights->dims[l + 1];
    if (!weights->w_self[l] || !weights->w_neigh[l] || !weights->bias[l]) return fail(GMB_EINVAL, "layer %d weight is NULL", l);
    a.w[a.count] = static_cast<float*>(const_cast<void*>(weights->w_self[l]));
    a.g[a.count] = grads->d_self[l];
    a.n[a.count++] = n;
    a.w[a.count] = static_cast<float*>(const_cast<void*>(weights->w_neigh[l]));
    a.g[a.count] = grads->d_neigh[l];
    a.n[a.count++] = n;
    a.w[a.count] = const_cast<float*>(weights->bias[l]);
    a.g[a.count] = grads->d_bias[l];
    a.n[a.count++] = weights->dims[l + 1];
  }
  hipError_t e = gmb::launch_sgd(a, lr, as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "update launch");
  return ok();
}

int gmb_sgd_update_bf16(const gmb_sage_weights* weights, const gmb_sage_weights* master, const gmb_sage_grads* grads,
                        float lr, void* stream) {
  if (!weights || !master) return fail(GMB_EINVAL, "weights or master is NULL");
  if (weights->dtype != GMB_BF16 || master->dtype != GMB_F32)
    return fail(GMB_EINVAL, "weights must be bf16 and master fp32");
  if (weights->num_layers != master->num_layers || weights->num_layers < 1 || weights->num_layers > GMB_MAX_LAYERS)
    return fail(GMB_EINVAL, "weights and master differ in layers (or none)");
  for (int l = 0; l <= weights->num_layers; ++l)
    if (weights->dims[l] != master->dims[l]) return fail(GMB_EINVAL, "dims[%d] differ", l);
  int st = check_grads(grads, weights);
  if (st != GMB_OK) return st;
  gmb::SgdArgs a{};
  for (int l = 0; l < weights->num_layers; ++l) {
    if (!weights->w_self[l] || !weights->w_neigh[l] || !weights->bias[l] || !master->w_self[l] ||
        !master->w_neigh[l] || !master->bias[l])
      return fail(GMB_EINVAL, "layer %d weight is NULL", l);
    const int64_t n = static_cast<int64_t>(weights->dims[l]) * weights->dims[l + 1];
    const void* lo[2] = {weights->w_self[l], weights->w_neigh[l]};
    const void* hi[2] = {master->w_self[l], master->w_neigh[l]};
    float* const g[2] = {grads->d_self[l], grads->d_neigh[l]};
    for (int k = 0; k < 2; ++k) {
      a.w[a.count] = static_cast<float*>(const_cast<void*>(hi[k]));
      a.g[a.count] = g[k];
      a.lo[a.count] = static_cast<uint16_t*>(const_cast<void*>(lo[k]));
      a.n[a.count++] = n;
    }
    a.w[a.count] = const_cast<float*>(master->bias[l]);
    a.g[a.count] = grads->d_bias[l];
    a.mirror[a.count] = weights->bias[l] == master->bias[l] ? nullptr : const_cast<float*>(weights->bias[l]);
    a.n[a.count++] = weights->dims[l + 1];
  }
  hipError_t e = gmb::launch_sgd(a, lr, as_stream(stream));
  if (e != hipSuccess) return hip_fail(e, "update launch");
  return ok();
}

}  // extern "C"
