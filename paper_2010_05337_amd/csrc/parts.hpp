// The part-product GEMM of the SAGE layers: fp32 operands on the bf16
// matrix cores of gfx950 through an exact three-way cut (below), a
// weight slab resident in LDS, persistent over row tiles.  Shared by the
// forward linear (sage.hip) and the input gradient of the backward
// (sage_bwd.hip) through an operation policy that says how A rows are read,
// what B holds and where the results go.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace gmb {
namespace parts {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ void opaque(float& x) { asm volatile("" : "+v"(x)); }

__device__ __forceinline__ const float* pick_ptr(bool c, const float* a, const float* b) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return reinterpret_cast<const float*>(c ? x : y);
}

// fp32 on the bf16 matrix cores.  Every fp32 value x is cut exactly into
// three bf16 parts by truncation, x = x0 + x1 + x2: x0 keeps the top 8 bits
// of the significand, x1 the next 8, x2 the last 8, so |x1| < 2^-7 |x| and
// |x2| < 2^-15 |x|.  A product a b is taken as the six part products of
// weight at least 2^-16 |a b| (a0 b0, a0 b1, a1 b0, a0 b2, a1 b1, a2 b0);
// what is left out (a1 b2, a2 b1, a2 b2) is below 2^-21 |a b|, and every
// part product is exact in fp32, summed with fp32 accumulation: a relative
// error of the order of fp32's own rounding.  Per 32 k that is six
// v_mfma_f32_16x16x32_bf16 against eight v_mfma_f32_16x16x4f32, at a
// quarter of the matrix-core cycles each; the cost is the cutting of A
// (about 44 VALU instructions per lane, 32 k and 16 rows), and on gfx950 a
// VALU instruction takes the SIMD's issue for about as long as a fifth of
// such a product, also beside it.  Values whose parts carry no more than 8
// (or 16) bits give the exact products.
//
// Layout, for C = A B with K rows of B and N columns (the policy gives A,
// B and where C goes): lane l (q = l / 16) of a wave supplies
// A[l % 16][32c + 8q .. +7] and B[32c + 8q .. +7][l % 16] of chunk c to
// v_mfma_f32_16x16x32_bf16 and holds C[4q + r][l % 16].  The slab holds the
// three parts of the workgroup's BN = 16 J columns of B for all K rows in
// operand order, Bp[p][(c * 4 + q) * BN + n][s] = part p of B[32c + 8q +
// s][n] (zero past K and past N): one 16-byte LDS read per lane, plane and
// column subtile.  A is read as fp32, two 16-byte global reads per lane and
// chunk, and cut into parts one chunk ahead of its products.  SPLIT = 1:
// wave w of WAVES owns R row fragments of 16 rows (16 WAVES R rows per
// tile) and reuses each B fragment R times; SPLIT > 1 (layers with few
// rows): the waves share the tile's R fragments, wave w takes the chunks c
// = w (mod WAVES), partial sums meet in LDS and are added in wave order.
// Persistent over row tiles, the next tile's A reads issued as soon as each
// chunk is cut; loads are unconditional from clamped addresses (a row past
// the end reads the last row and is not stored; k past K reads valid values
// that meet zero rows of the slab; a load under a divergent branch would
// make the compiler drain every outstanding load first).
__device__ __forceinline__ void split3(float x, uint32_t& p0, uint32_t& p1, uint32_t& p2) {
  const uint32_t t0 = __float_as_uint(x) & 0xFFFF0000u;
  const float r1 = x - __uint_as_float(t0);
  const uint32_t t1 = __float_as_uint(r1) & 0xFFFF0000u;
  const float r2 = r1 - __uint_as_float(t1);
  p0 = t0;
  p1 = t1;
  p2 = __float_as_uint(r2);   // at most 8 significant bits: its low half is zero
}

// Eight fp32 values -> their three parts as bf16x8 operands (element s in
// half s % 2 of word s / 2).
__device__ __forceinline__ void split8(const float4& lo, const float4& hi, bf16x8 (&part)[3]) {
  const float x[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
  uint32_t w[3][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t a0, a1, a2, b0, b1, b2;
    split3(x[2 * i], a0, a1, a2);
    split3(x[2 * i + 1], b0, b1, b2);
    w[0][i] = (a0 >> 16) | (b0 & 0xFFFF0000u);
    w[1][i] = (a1 >> 16) | (b1 & 0xFFFF0000u);
    w[2][i] = (a2 >> 16) | (b2 & 0xFFFF0000u);
  }
#pragma unroll
  for (int p = 0; p < 3; ++p) part[p] = __builtin_bit_cast(bf16x8, make_uint4(w[p][0], w[p][1], w[p][2], w[p][3]));
}

constexpr int parts_lds_bytes(int nch, int j, int r, int split, int waves) {
  return 3 * nch * 4 * 16 * j * 8 * 2 + (split > 1 ? waves * r * j * 64 * 16 : 16);
}


// The forward linear: A = [h_v | mean] (two arrays of K = d_in columns,
// row stride d_in), B = [W_self; W_neigh] (2 d_in x d_out, row-major),
// out = act(A B + b) with row stride d_out.
struct LinearOp {
  const float* Hs;
  const float* Ag;
  const float* Ws;
  const float* Wn;
  const float* bias_v;
  int K, N, relu;
  float* out;
  int quad_b;   // N % 4 == 0 and 16-byte aligned matrices: the slab takes load_b8x4
  static constexpr bool kQuadCapable = true;
  static constexpr bool kEarlyA = true;   // the first tile's A loads overlap the slab's
  __host__ __device__ int k2() const { return 2 * K; }
  __host__ __device__ int n() const { return N; }
  __host__ __device__ int64_t ldo() const { return N; }
  __device__ void a_rows(int64_t row, const float*& p0, const float*& p1) const {
    p0 = Hs + row * K;
    p1 = Ag + row * K;
  }
  // A[row][k .. k + 3]: from h_v (k < d_in) or the mean (d_in % 4 == 0, so
  // four k never straddle the two); k past 2 d_in reads the row's first
  // values, which meet zero rows of B
  __device__ float4 load_a4(const float* p0, const float* p1, int k) const {
    const int K2 = 2 * K;
    const int kk = k >= K2 ? 0 : (k < K ? k : k - K);
    return *reinterpret_cast<const float4*>(pick_ptr((k >= K) & (k < K2), p1, p0) + kk);
  }
  // B[k0 .. k0 + 7][gn]: eight loads, coalesced over gn; in[s] false where
  // the entry lies outside B (its load reads W_self[0][0])
  __device__ void load_b8(bool item, int k0, int gn, float (&w)[8], bool (&in)[8]) const {
#pragma unroll
    for (int s8 = 0; s8 < 8; ++s8) {
      const int k = k0 + s8;
      in[s8] = item & (k < 2 * K) & (gn < N);
      const int kr = in[s8] ? (k < K ? k : k - K) : 0;
      w[s8] = pick_ptr(in[s8] & (k >= K), Wn, Ws)[static_cast<int64_t>(kr) * N + (in[s8] ? gn : 0)];
    }
  }
  // B[k0 .. k0 + 7][gn .. gn + 3] (quad_b set, gn % 4 == 0): eight 16-byte
  // loads, one per row, w[j][s] = B[k0 + s][gn + j]; in[s] false where row
  // k0 + s lies outside B or the quad past N (its load reads W_self's first
  // values).  K N < 2^31, so an element offset fits in 32 bits.
  __device__ void load_b8x4(bool item, int k0, int gn, float (&w)[4][8], bool (&in)[8]) const {
    const bool cols = item & (gn < N);
    const uint32_t gc = cols ? static_cast<uint32_t>(gn) : 0u;
#pragma unroll
    for (int s8 = 0; s8 < 8; ++s8) {
      const int k = k0 + s8;
      in[s8] = cols & (k < 2 * K);
      const bool hi = in[s8] & (k >= K);
      const uint32_t kr = in[s8] ? static_cast<uint32_t>(hi ? k - K : k) : 0u;
      const float4 x = *reinterpret_cast<const float4*>(pick_ptr(hi, Wn, Ws) + (kr * static_cast<uint32_t>(N) + gc));
      w[0][s8] = x.x; w[1][s8] = x.y; w[2][s8] = x.z; w[3][s8] = x.w;
    }
  }
  __device__ float bias(int col) const { return bias_v[col < N ? col : N - 1]; }
  __device__ float act(float z) const { return relu ? (z > 0.f ? z : 0.f) : z; }
  __device__ float* out_at(int64_t row, int col) const { return out + row * N + col; }
};

// The input gradient: A = dZ (d_out columns, row stride ldz), B = [W_self;
// W_neigh]^T (B[k][nn] = W[nn][k], 2 d_in columns), the result's columns
// nn < d_in to dH and the others to dM (row stride d_in each).
struct DgradOp {
  static constexpr bool kQuadCapable = false;   // its eight k are one contiguous run already
  static constexpr bool kEarlyA = false;        // (the largest tiling has no registers to spare for it)
  const float* dZ;
  const float* Ws;
  const float* Wn;
  int ldz, d_out, d_in;
  float* dH;
  float* dM;
  __host__ __device__ int k2() const { return d_out; }
  __host__ __device__ int n() const { return 2 * d_in; }
  __host__ __device__ int64_t ldo() const { return d_in; }
  __device__ void a_rows(int64_t row, const float*& p0, const float*& p1) const {
    p0 = dZ + row * ldz;
    p1 = p0;
  }
  // dZ[row][k .. k + 3] (d_out % 4 == 0); k past d_out reads the row's
  // first values, which meet zero rows of B
  __device__ float4 load_a4(const float* p0, const float*, int k) const {
    return *reinterpret_cast<const float4*>(p0 + (k < d_out ? k : 0));
  }
  // B[k0 .. k0 + 7][nn] = W[nn][k0 .. k0 + 7]: two 16-byte loads of the
  // weight row (d_out % 4 == 0 and 16-byte aligned rows, checked by the
  // launcher); a group of four k past d_out is zero
  __device__ void load_b8(bool item, int k0, int nn, float (&w)[8], bool (&in)[8]) const {
    const bool row_in = item & (nn < 2 * d_in);
    const float* wr = row_in ? (nn < d_in ? Ws + static_cast<int64_t>(nn) * d_out
                                          : Wn + static_cast<int64_t>(nn - d_in) * d_out)
                             : Ws;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k = k0 + 4 * h;
      const bool ok = row_in & (k < d_out);
      const float4 x = *reinterpret_cast<const float4*>(wr + (ok ? k : 0));
      w[4 * h] = x.x; w[4 * h + 1] = x.y; w[4 * h + 2] = x.z; w[4 * h + 3] = x.w;
#pragma unroll
      for (int t = 0; t < 4; ++t) in[4 * h + t] = ok;
    }
  }
  __device__ float bias(int) const { return 0.f; }
  __device__ float act(float z) const { return z; }
  __device__ float* out_at(int64_t row, int col) const {
    return col < d_in ? dH + row * d_in + col : dM + row * d_in + (col - d_in);
  }
};

template <class Op, int NCH, int J, int R, int SPLIT, int WAVES>
__device__ __forceinline__ void parts_gemm(const Op& op, int32_t M) {
  constexpr int BN = 16 * J;
  constexpr int THREADS = 64 * WAVES;
  constexpr int ROWS = SPLIT > 1 ? 16 * R : 16 * WAVES * R;
  constexpr int MYCH = SPLIT > 1 ? (NCH + WAVES - 1) / WAVES : NCH;
  constexpr int PLANE = NCH * 4 * BN * 8;   // uint16 per plane
  constexpr int ENTRIES = R * J * 64;       // split K: output entries of four rows per tile
  constexpr int PER_THREAD = SPLIT > 1 ? (ENTRIES + THREADS - 1) / THREADS : 1;
  __shared__ __attribute__((aligned(16))) uint16_t Bp[3 * PLANE];
  __shared__ __attribute__((aligned(16))) float Red[SPLIT > 1 ? WAVES * ENTRIES * 4 : 4];
  const int row_tiles = (M + ROWS - 1) / ROWS;
  if (static_cast<int>(blockIdx.x) >= row_tiles) return;
  const int n0 = blockIdx.y * BN;
  const int N = op.n();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, r16 = lane & 15;
  // first row of fragment f of row tile rt (SPLIT = 1: wave w owns
  // fragments w R .. w R + R - 1; split K: every wave takes all R)
  auto frag_row0 = [&](int rt, int f) { return rt * ROWS + (SPLIT > 1 ? f : wave * R + f) * 16; };
  auto frag_rows = [&](int rt, int f, const float*& hrow, const float*& grow) {
    const int row = frag_row0(rt, f) + r16;
    op.a_rows(row < M ? row : M - 1, hrow, grow);   // a row past the end reads row M-1
  };
  auto load4 = [&](const float* hrow, const float* grow, int k) -> float4 { return op.load_a4(hrow, grow, k); };
  auto chunk_of = [&](int i) { return SPLIT > 1 ? wave + WAVES * i : i; };
  float4 a[R][MYCH][2];
  const float* hr[R];
  const float* gr[R];
  // the first tile's A values, issued between the slab's loads and their
  // use, so that the two round trips overlap
  auto issue_first_a = [&]() {
#pragma unroll
    for (int f = 0; f < R; ++f) {
      frag_rows(blockIdx.x, f, hr[f], gr[f]);
#pragma unroll
      for (int i = 0; i < MYCH; ++i) {
        const int k = chunk_of(i) * 32 + 8 * q;
        a[f][i][0] = load4(hr[f], gr[f], k);
        a[f][i][1] = load4(hr[f], gr[f], k + 4);
      }
    }
  };
  // slab fill: item (c, q, n) reads B[32c + 8q .. +7][n0 + n] (the
  // policy's eight loads), cuts them into parts and writes one 16-byte word
  // per plane; where the policy can (the forward's row-major matrices with N
  // % 4 == 0), an item takes four adjacent columns with eight 16-byte loads
  // instead (a quarter of the load instructions and their address work).  A
  // thread issues the loads of all its items before the first use (one
  // round trip to the L2 instead of one per item), and with kEarlyA the
  // first tile's A loads go out behind them
  bool quad = false;
  if constexpr (Op::kQuadCapable) quad = op.quad_b != 0;
  if (quad) {
    // four adjacent columns per item: eight 16-byte loads, four words per plane
    if constexpr (Op::kQuadCapable) {
      constexpr int kQuads = NCH * 4 * BN / 4, kPer = (kQuads + THREADS - 1) / THREADS;
      float w[kPer][4][8];
      bool in[kPer][8];
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int it = threadIdx.x + THREADS * u;
        const int n4 = it % (BN / 4), cq = it / (BN / 4);
        op.load_b8x4(it < kQuads, cq * 8, n0 + 4 * n4, w[u], in[u]);
      }
      if constexpr (Op::kEarlyA) issue_first_a();
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int it = threadIdx.x + THREADS * u;
        if (it >= kQuads) continue;
        const int n4 = it % (BN / 4), cq = it / (BN / 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
          for (int s8 = 0; s8 < 8; ++s8) {
            opaque(w[u][j][s8]);
            w[u][j][s8] = in[u][s8] ? w[u][j][s8] : 0.f;
          }
          bf16x8 part[3];
          split8(make_float4(w[u][j][0], w[u][j][1], w[u][j][2], w[u][j][3]),
                 make_float4(w[u][j][4], w[u][j][5], w[u][j][6], w[u][j][7]), part);
#pragma unroll
          for (int p = 0; p < 3; ++p)
            *reinterpret_cast<bf16x8*>(&Bp[p * PLANE + (cq * BN + 4 * n4 + j) * 8]) = part[p];
        }
      }
    }
  } else {
    constexpr int kItems = NCH * 4 * BN, kPer = (kItems + THREADS - 1) / THREADS;
    float w[kPer][8];
    bool in[kPer][8];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int it = threadIdx.x + THREADS * u;
      const int n = it % BN, cq = it / BN;
      op.load_b8(it < kItems, cq * 8, n0 + n, w[u], in[u]);
    }
    if constexpr (Op::kEarlyA) issue_first_a();
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int it = threadIdx.x + THREADS * u;
      if (it >= kItems) continue;
      const int n = it % BN, cq = it / BN;
#pragma unroll
      for (int s8 = 0; s8 < 8; ++s8) {
        opaque(w[u][s8]);
        w[u][s8] = in[u][s8] ? w[u][s8] : 0.f;
      }
      bf16x8 part[3];
      split8(make_float4(w[u][0], w[u][1], w[u][2], w[u][3]), make_float4(w[u][4], w[u][5], w[u][6], w[u][7]), part);
#pragma unroll
      for (int p = 0; p < 3; ++p) *reinterpret_cast<bf16x8*>(&Bp[p * PLANE + (cq * BN + n) * 8]) = part[p];
    }
  }
  __syncthreads();
  if constexpr (!Op::kEarlyA) issue_first_a();
  // bias of this lane's columns n0 + 16 j + lane % 16 (fixed over the tiles;
  // with split K the thread's stored entries have the same lane % 16)
  float bv[J];
#pragma unroll
  for (int j = 0; j < J; ++j) bv[j] = op.bias(n0 + j * 16 + r16);
  // A tile's results are stored in the middle of the next tile (and after
  // the last one): stores and loads share one counter on gfx9, and with
  // stores pending the next wait on a prefetched A value is a wait for
  // everything, so stores issued at the end of a tile would stall the start
  // of the next one for a whole write round trip.
  floatx4 held[SPLIT > 1 ? PER_THREAD : R][SPLIT > 1 ? 1 : J];
  int held_rt = -1;
  const int64_t ld = op.ldo();
  auto store4 = [&](int row0, int col, const floatx4& v, float b) {
    if (col >= N) return;
    float* o = op.out_at(row0, col);
    const bool full = row0 + 4 <= M;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (full || row0 + r < M) o[static_cast<int64_t>(r) * ld] = op.act(v[r] + b);
  };
  auto store_held = [&]() {
    if (held_rt < 0) return;
    if constexpr (SPLIT > 1) {
#pragma unroll
      for (int u = 0; u < PER_THREAD; ++u) {
        const int e = threadIdx.x + THREADS * u;
        if (e < ENTRIES) {
          const int f = e / (J * 64), j = (e / 64) % J, l = e % 64;
          store4(frag_row0(held_rt, f) + 4 * (l >> 4), n0 + j * 16 + (l & 15), held[u][0], bv[j]);
        }
      }
    } else {
#pragma unroll
      for (int f = 0; f < R; ++f) {
        const int row0 = frag_row0(held_rt, f) + 4 * q;
        if (row0 + 4 <= M && n0 + BN <= N) {   // inside the matrix: no per-element checks
#pragma unroll
          for (int j = 0; j < J; ++j) {
            float* o = op.out_at(row0, n0 + j * 16 + r16);
#pragma unroll
            for (int r = 0; r < 4; ++r) o[static_cast<int64_t>(r) * ld] = op.act(held[f][j][r] + bv[j]);
          }
        } else {
#pragma unroll
          for (int j = 0; j < J; ++j) store4(row0, n0 + j * 16 + r16, held[f][j], bv[j]);
        }
      }
    }
  };
  for (int rt = blockIdx.x; rt < row_tiles; rt += gridDim.x) {
#pragma unroll
    for (int f = 0; f < R; ++f) frag_rows(rt + gridDim.x, f, hr[f], gr[f]);
    floatx4 acc[R][J];
#pragma unroll
    for (int f = 0; f < R; ++f)
#pragma unroll
      for (int j = 0; j < J; ++j) acc[f][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    auto load_b = [&](int i, bf16x8 (&b)[3][J]) {
      const int c = chunk_of(i);
      const int cc = c < NCH ? c : NCH - 1;
#pragma unroll
      for (int p = 0; p < 3; ++p)
#pragma unroll
        for (int j = 0; j < J; ++j)
          b[p][j] = *reinterpret_cast<const bf16x8*>(&Bp[p * PLANE + ((cc * 4 + q) * BN + j * 16 + r16) * 8]);
    };
    // B fragments double-buffered with one wave per SIMD (chunk i + 1's LDS
    // reads issued before chunk i's products); with two waves per SIMD the
    // other wave covers the LDS latency and one buffer saves the registers
    constexpr bool kDoubleB = WAVES == 4;
    bf16x8 b0[3][J], b1[kDoubleB ? 3 : 1][kDoubleB ? J : 1];
    if (kDoubleB) load_b(0, b0);
    // A parts one chunk ahead: chunk i + 1 is cut while chunk i's products
    // run (independent work, interleaved below so that the VALU instructions
    // issue between the matrix-core ones)
    bf16x8 p0[R][3], p1[R][3];
#pragma unroll
    for (int f = 0; f < R; ++f) split8(a[f][0][0], a[f][0][1], p0[f]);
#pragma unroll
    for (int f = 0; f < R; ++f) {
      const int k = chunk_of(0) * 32 + 8 * q;
      a[f][0][0] = load4(hr[f], gr[f], k);
      a[f][0][1] = load4(hr[f], gr[f], k + 4);
    }
#pragma unroll
    for (int i = 0; i < MYCH; ++i) {
      bf16x8 (&pc)[R][3] = (i & 1) ? p1 : p0;
      bf16x8 (&pn)[R][3] = (i & 1) ? p0 : p1;
      bf16x8 (*bcp)[J];
      if constexpr (kDoubleB) {
        bf16x8 (&bn)[3][J] = (i & 1) ? b0 : b1;
        if (i + 1 < MYCH) load_b(i + 1, bn);
        bcp = (i & 1) ? b1 : b0;
      } else {
        load_b(i, b0);
        bcp = b0;
      }
      bf16x8 (&bc)[3][J] = *reinterpret_cast<bf16x8 (*)[3][J]>(bcp);
      __builtin_amdgcn_sched_barrier(0);
      if (i + 1 < MYCH) {
#pragma unroll
        for (int f = 0; f < R; ++f) split8(a[f][i + 1][0], a[f][i + 1][1], pn[f]);
      }
      if (chunk_of(i) < NCH) {   // uniform: depends on the wave index only
#pragma unroll
        for (int f = 0; f < R; ++f) {
          const bf16x8 (&ap)[3] = pc[f];
          // the smallest part products first
#pragma unroll
          for (int j = 0; j < J; ++j) acc[f][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[0], bc[2][j], acc[f][j], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < J; ++j) acc[f][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[1], bc[1][j], acc[f][j], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < J; ++j) acc[f][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[2], bc[0][j], acc[f][j], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < J; ++j) acc[f][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[0], bc[1][j], acc[f][j], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < J; ++j) acc[f][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[1], bc[0][j], acc[f][j], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < J; ++j) acc[f][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[0], bc[0][j], acc[f][j], 0, 0, 0);
        }
      }
      // one product, then two VALU instructions of the next chunk's cut
#pragma unroll
      for (int m = 0; m < 6 * R * J; ++m) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
      }
      // the A values of chunk i + 1 are cut: its registers take the next
      // tile's chunk i + 1 (chunk 0 was reloaded before the loop)
      if (i + 1 < MYCH) {
#pragma unroll
        for (int f = 0; f < R; ++f) {
          const int k = chunk_of(i + 1) * 32 + 8 * q;
          a[f][i + 1][0] = load4(hr[f], gr[f], k);
          a[f][i + 1][1] = load4(hr[f], gr[f], k + 4);
        }
      }
      if (i == MYCH / 2) store_held();
    }
    if constexpr (SPLIT > 1) {
      // partials of the waves -> LDS; thread t then holds the entries
      // e = t + THREADS u, each the sum of the partials in wave order
#pragma unroll
      for (int f = 0; f < R; ++f)
#pragma unroll
        for (int j = 0; j < J; ++j)
          *reinterpret_cast<floatx4*>(&Red[((wave * R + f) * J + j) * 64 * 4 + lane * 4]) = acc[f][j];
      __syncthreads();
#pragma unroll
      for (int u = 0; u < PER_THREAD; ++u) {
        const int e = threadIdx.x + THREADS * u;
        if (e < ENTRIES) {
          floatx4 sum = *reinterpret_cast<const floatx4*>(&Red[e * 4]);
#pragma unroll
          for (int w = 1; w < WAVES; ++w) sum += *reinterpret_cast<const floatx4*>(&Red[(w * ENTRIES + e) * 4]);
          held[u][0] = sum;
        }
      }
      __syncthreads();
    } else {
#pragma unroll
      for (int f = 0; f < R; ++f)
#pragma unroll
        for (int j = 0; j < J; ++j) held[f][j] = acc[f][j];
    }
    held_rt = rt;
  }
  store_held();
}


// Grid of a part-product launch: row tiles of the persistent grid, column tiles.
template <int J, int R, int SPLIT, int WAVES>
inline dim3 parts_grid(int64_t cap_rows, int N) {
  constexpr int BN = 16 * J;
  constexpr int ROWS = SPLIT > 1 ? 16 * R : 16 * WAVES * R;
  const int col_tiles = (N + BN - 1) / BN;
  int64_t rows = (cap_rows + ROWS - 1) / ROWS;
  // one workgroup per CU (the LDS holds one slab), the grid covering the chip once
  const int64_t want = (256 + col_tiles - 1) / col_tiles;
  if (rows > want) rows = want;
  if (rows < 1) rows = 1;
  return dim3(static_cast<unsigned>(rows), col_tiles);
}

}  // namespace parts
}  // namespace gmb
