// Training step of the GraphSAGE-mean model on gfx950: the loss, the
// backward through the layers of Eq. (1) (DistDGL Section II-A; the
// trainer's iteration of Section III-E), and the SGD update.  fp32.
//
//   k_xent         softmax cross-entropy per target row (one wave per row):
//                  dZ = (softmax(z) - e_y) / B, and the row's loss term; also
//                  clears the per-source edge counters of the transposes
//   k_wgrad_parts  [dW_self; dW_neigh] = [H | M]^T dZ and db = sum of dZ rows
//                  on the bf16 matrix cores through the exact three-way cut
//                  of the operands (parts.hpp), the rows of the block as the
//                  reduction dimension; a workgroup owns a 64 x 64 tile of
//                  the output and a range of rows, its eight waves (two per
//                  SIMD) split the rows and are summed through LDS, and every
//                  workgroup writes its partial sums (no atomics: the same
//                  result on every run).  The same products in fp32
//                  (v_mfma_f32_16x16x4_f32, wgrad_block) ride in the
//                  transpose scan's launch on the layers with an input
//                  gradient
//   k_wgrad_reduce sums the partials in a fixed order into the gradients;
//                  on the last layer one more workgroup sums the loss terms
//                  into the mean loss (fixed order).  On a layer whose input
//                  gradient runs, the reduction's workgroups ride at the end
//                  of that layer's k_csc_fill grid, and (for a small scan)
//                  the products' at the end of its k_csc_scan grid, instead of
//                  launches of their own (the input gradient then goes
//                  first)
//   k_dgrad        [dH_self | dM] = dZ [W_self; W_neigh]^T: the weights'
//                  transpose for 64 output columns resident in LDS in MFMA
//                  operand order, 64-row tiles, persistent over row tiles;
//                  also counts every source's in-edges in the block
//   k_csc_scan     exclusive scan of the counts: the transpose's row offsets
//   k_csc_fill     the transpose's entries (v, 1/k_v), one per block edge
//   k_pull_mean    dH[u] = relu'(below) * (dH_self[u] + sum over the block
//                  edges (v <- u) of dM[v] / k_v), one pass per source row:
//                  the mean's backward as a gather over the transpose, with
//                  the ReLU of the layer below applied on the way out
//   k_pull_update  on layer 0 with learnable vertex embeddings: the same
//                  sum applied at once as the sparse SGD step of the rows
//                  (both end their grids with workgroups that take the
//                  sources with long transpose lists, hubs, one each)
//   k_sgd          W -= lr dW over every parameter array
//   k_zero         the gradients and the loss of an empty batch
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"
#include "parts.hpp"
#include "scan.hpp"

namespace gmb {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// ---- loss ---------------------------------------------------------------

// Row v of z [n, C] (row stride C): dz row (stride ldz, columns C..ldz-1
// written as 0) and the row's loss term log(sum exp z) - z_y.  A label
// outside [0, C) is a data error: its row gets the softmax as gradient and
// no loss term (every access stays in bounds).  The grid also clears
// clear[0 .. clear_n).
__global__ __launch_bounds__(256) void k_xent(const float* __restrict__ z, const int32_t* __restrict__ y,
                                              int n, int C, int ldz, float* __restrict__ dz,
                                              float* __restrict__ loss_rows, int32_t* __restrict__ clear,
                                              int64_t clear_n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < clear_n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    clear[i] = 0;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const float* zr = z + static_cast<int64_t>(row) * C;
  float mx = -INFINITY;
  for (int c = lane; c < C; c += 64) mx = fmaxf(mx, zr[c]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  float sum = 0.f;
  for (int c = lane; c < C; c += 64) sum += expf(zr[c] - mx);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
  const float lse = mx + logf(sum);
  const int32_t label = y[row];
  const bool valid = label >= 0 && label < C;
  const float inv_n = 1.f / static_cast<float>(n);
  float* dr = dz + static_cast<int64_t>(row) * ldz;
  for (int c = lane; c < ldz; c += 64) {
    float g = 0.f;
    if (c < C) g = (expf(zr[c] - lse) - ((valid && c == label) ? 1.f : 0.f)) * inv_n;
    dr[c] = g;
  }
  if (lane == 0) loss_rows[row] = valid ? lse - zr[label] : 0.f;
}

// The mean loss by one workgroup of 256 threads, in a fixed order.  It runs
// as an extra workgroup of the last layer's weight-gradient reduction (the
// launch after the loss kernel's), which saves a launch of its own.
__device__ void loss_sum_block(const float* __restrict__ rows, int n, float* __restrict__ loss) {
  __shared__ float part[256];
  float s = 0.f;
  for (int i = threadIdx.x; i < n; i += 256) s += rows[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss = n > 0 ? part[0] / static_cast<float>(n) : 0.f;
}

// ---- weight gradient ------------------------------------------------------

// Workgroup (p, y, z) owns 64 rows of [dW_self; dW_neigh] -- columns
// [64 z', 64 z' + 64) of H (z < TI = ceil(d_in / 64), z' = z) or of M
// (z' = z - TI), the output rows d_in + those -- and output columns
// [64 y, 64 y + 64), over the block rows [p R, (p + 1) R) (R: the n_dst rows
// split over the gridDim.x ranges); wave w takes the
// 16-row steps w, w + 4, ... of that range.  Lane (q, c) = (l / 16, l % 16)
// owns the four columns 64 z' + 4c + t of its array and o = 64 y + 4c + j of
// dZ, and reads each as one 16-byte load (VEC; else four scalar loads).
// MFMA (t, j) multiplies A[m][k] = X[row k][64 z' + 4m + t] by
// B[k][n] = dZ[row k][64 y + 4n + j] over four rows, so its accumulator
// register r of lane (q, c) holds the sum for column 64 z' + 16q + 4r + t of
// X and column 64 y + 4c + j of dZ.  Rows at or past the end of the range
// read its last row and their dZ is zeroed before the product (the columns
// past the arrays' ends feed only outputs that are never written).  The
// four waves' sums meet in LDS in a fixed order; workgroup p writes its
// partial to partial[p][i][o] (row stride ldp = d_out rounded up to 4; row
// 2 d_in: the column sums of dZ, written by the z = 0 workgroups).  Every
// array of this kernel has fewer than 2^32 bytes (checked by the launcher),
// so loads take a uniform base and a 32-bit byte offset.
constexpr int kWgradRed = 2 * 64 * 64;   // LDS floats of the cross-wave sum
#ifndef GMB_WGRAD_DEPTH
#define GMB_WGRAD_DEPTH 3
#endif
constexpr int kWgradDepth = GMB_WGRAD_DEPTH;   // row steps in flight per wave (loads depth - 1 ahead)

// Workgroup (bx, by, bz) of a weight-gradient grid with gx row ranges.
template <bool VEC>
__device__ __forceinline__ void wgrad_block(const int32_t* __restrict__ sizes, const float* __restrict__ H,
                                            const float* __restrict__ M, int d_in, const float* __restrict__ dZ,
                                            int ldz, int ldp, float* __restrict__ partial, int bx, int by, int bz,
                                            int gx) {
  __shared__ float red[kWgradRed];
  __shared__ float red_db[4][64];
  const int32_t n = load_size(&sizes[kNDst]);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, c16 = lane & 15;
  const int p = bx;
  const int K2 = 2 * d_in;
  const int TI = (d_in + 63) / 64;
  const bool from_m = bz >= TI;
  const int zc = from_m ? bz - TI : bz;
  const char* X = reinterpret_cast<const char*>(from_m ? M : H);   // uniform per workgroup
  const char* Zb = reinterpret_cast<const char*>(dZ);
  const int cb = zc * 64 + 4 * c16;           // this lane's first column of X
  const int ob = by * 64 + 4 * c16;   // this lane's first column of dZ
  const uint32_t xrow = static_cast<uint32_t>(d_in) * 4u, zrow = static_cast<uint32_t>(ldz) * 4u;
  const uint32_t ocol = static_cast<uint32_t>(ob < ldz ? ob : 0) * 4u;
  uint32_t xcol[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) xcol[t] = static_cast<uint32_t>(VEC ? (cb < d_in ? cb : 0) : (cb + t < d_in ? cb + t : 0)) * 4u;
  // the block's actual rows split evenly over the gx ranges (16-row
  // granules); every range writes its partial, empty or not
  const int rows_per_part = ((n + gx - 1) / gx + 15) / 16 * 16;
  const int r0 = min(p * rows_per_part, n);
  const int r1 = min(r0 + rows_per_part, n);
  floatx4 acc[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[t][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  float dbs[4] = {0.f, 0.f, 0.f, 0.f};

  auto load = [&](int k0, float4 (&xa)[4], float4 (&zb)[4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int row = k0 + 4 * s + q;
      const uint32_t rc = static_cast<uint32_t>(row < r1 ? row : r1 - 1);
      if (VEC) {
        xa[s] = *reinterpret_cast<const float4*>(X + (rc * xrow + xcol[0]));
      } else {
        xa[s] = make_float4(*reinterpret_cast<const float*>(X + (rc * xrow + xcol[0])),
                            *reinterpret_cast<const float*>(X + (rc * xrow + xcol[1])),
                            *reinterpret_cast<const float*>(X + (rc * xrow + xcol[2])),
                            *reinterpret_cast<const float*>(X + (rc * xrow + xcol[3])));
      }
      zb[s] = *reinterpret_cast<const float4*>(Zb + (rc * zrow + ocol));
    }
  };
  auto compute = [&](int k0, const float4 (&xa)[4], const float4 (&zb)[4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bool in = k0 + 4 * s + q < r1;
      const float a[4] = {xa[s].x, xa[s].y, xa[s].z, xa[s].w};
      const float b[4] = {in ? zb[s].x : 0.f, in ? zb[s].y : 0.f, in ? zb[s].z : 0.f, in ? zb[s].w : 0.f};
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[t][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t], b[j], acc[t][j], 0, 0, 0);
#pragma unroll
      for (int j = 0; j < 4; ++j) dbs[j] += b[j];
    }
  };

  // loads run kWgradDepth - 1 steps ahead of the products.  The body is
  // unrolled kWgradDepth times so that every buffer keeps its registers (a
  // copy between buffers would wait for the load); the step count is
  // rounded up to a multiple of the depth, the extra steps read the range's
  // last row and add zero, and no branch surrounds a product, so the
  // accumulators stay in place
  int k0 = r0 + 16 * wave;
  const int nsteps = __builtin_amdgcn_readfirstlane(k0 < r1 ? (r1 - k0 + 63) / 64 : 0);
  constexpr int D = kWgradDepth;
  float4 xs[D][4], zs[D][4];
  if (nsteps > 0) {
#pragma unroll
    for (int b = 0; b + 1 < D; ++b) load(k0 + 64 * b, xs[b], zs[b]);
  }
  for (int it = 0; it < nsteps; it += D) {
#pragma unroll
    for (int b = 0; b < D; ++b) {
      load(k0 + 64 * (b + D - 1), xs[(b + D - 1) % D], zs[(b + D - 1) % D]);
      __builtin_amdgcn_sched_barrier(0);
      compute(k0 + 64 * b, xs[b], zs[b]);
    }
    k0 += 64 * D;
  }
  // column sums of dZ: over the lane's rows, then over q
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    dbs[j] += __shfl_xor(dbs[j], 16, 64);
    dbs[j] += __shfl_xor(dbs[j], 32, 64);
  }
  // waves 2, 3 -> LDS; waves 0, 1 add; wave 1 -> LDS; wave 0 adds:
  // ((w0 + w2) + (w1 + w3)), the same order on every run
  auto put = [&](int slot) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[(slot * 64 + (t * 16 + j * 4 + r)) * 64 + lane] = acc[t][j][r];
  };
  auto add = [&](int slot) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[t][j][r] += red[(slot * 64 + (t * 16 + j * 4 + r)) * 64 + lane];
  };
  if (wave >= 2) put(wave - 2);
  if (q == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) red_db[wave][4 * c16 + j] = dbs[j];
  }
  __syncthreads();
  if (wave < 2) add(wave);
  __syncthreads();
  if (wave == 1) put(0);
  __syncthreads();
  if (wave != 0) return;
  add(0);
  float* part = partial + static_cast<int64_t>(p) * (K2 + 1) * ldp;
  if (ob < ldp) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = zc * 64 + 16 * q + 4 * r + t;
        if (c < d_in)
          *reinterpret_cast<float4*>(part + static_cast<int64_t>(from_m ? d_in + c : c) * ldp + ob) =
              make_float4(acc[t][0][r], acc[t][1][r], acc[t][2][r], acc[t][3][r]);
      }
    if (bz == 0 && q == 0) {
      float v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        v[j] = (red_db[0][4 * c16 + j] + red_db[2][4 * c16 + j]) + (red_db[1][4 * c16 + j] + red_db[3][4 * c16 + j]);
      *reinterpret_cast<float4*>(part + static_cast<int64_t>(K2) * ldp + ob) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// The same gradient on the bf16 matrix cores through the exact three-way
// cut of the operands (parts.hpp: six part products, fp32 accumulation),
// for the layers whose weight gradient has a launch of its own: the same
// workgroups (p, y, z), 64 x 64 tiles, row ranges, partials and reduction
// as above.  The block rows are the reduction dimension: per 32-row chunk,
// lane (g, i) = (l / 16, l % 16) supplies A[i][8g .. +7] = X[row 8g .. +7]
// [64 z' + 16 b + i] and B[8g .. +7][i] = dZ[row 8g .. +7][64 y + 16 b' + i]
// of v_mfma_f32_16x16x32_bf16 for the four column blocks b, b' of the tile
// (eight 4-byte loads per column: the sixteen lanes of a row read 64
// consecutive bytes), cuts them in registers and holds C[4g + r][i] of the
// 4 x 4 blocks.  Wave w of W takes the chunks w, w + W, ... of the range;
// rows past the range read its last row and their dZ is zeroed (also in
// the bias sums); columns past the arrays read column 0 and feed only
// outputs that are never written.  The W waves' tiles meet in LDS and are
// added in wave order.  The cut costs about as many VALU issue cycles as
// the products take on the matrix core, and a wave does not overlap the
// two by itself: two waves per SIMD (W = 8, the loads of a chunk issued
// just before its products) measured 35 us on the 100 -> 256 layer of a
// 39k-row block, against 46 us for four waves with the next chunk's loads
// in flight (depth 2; depth 3 and 4: 50 us) and 47 us for the fp32 products.
#ifndef GMB_WGRAD_PARTS_DEPTH
#define GMB_WGRAD_PARTS_DEPTH 1
#endif
#ifndef GMB_WGRAD_PARTS_WAVES
#define GMB_WGRAD_PARTS_WAVES 8
#endif
constexpr int kWgradPartsDepth = GMB_WGRAD_PARTS_DEPTH;   // chunks in flight per wave
constexpr int kWgradPartsWaves = GMB_WGRAD_PARTS_WAVES;   // waves per workgroup, two per SIMD at 8

__global__ __launch_bounds__(64 * kWgradPartsWaves)
__attribute__((amdgpu_waves_per_eu(kWgradPartsWaves / 4, kWgradPartsWaves / 4)))
void k_wgrad_parts(const int32_t* __restrict__ sizes, const float* __restrict__ H, const float* __restrict__ M,
                   int d_in, const float* __restrict__ dZ, int ldz, int ldp, float* __restrict__ partial) {
  using parts::bf16x8;
  constexpr int W = kWgradPartsWaves;
  constexpr int kPad = 68;   // LDS row stride of the waves' tiles
  __shared__ __attribute__((aligned(16))) float red[W][64 * kPad];
  __shared__ float red_db[W][64];
  const int32_t n = load_size(&sizes[kNDst]);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, li = lane & 15;
  const int p = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
  const int K2 = 2 * d_in;
  const int TI = (d_in + 63) / 64;
  const bool from_m = bz >= TI;
  const int zc = from_m ? bz - TI : bz;
  const char* X = reinterpret_cast<const char*>(from_m ? M : H);   // uniform per workgroup
  const char* Zb = reinterpret_cast<const char*>(dZ);
  const uint32_t xrow = static_cast<uint32_t>(d_in) * 4u, zrow = static_cast<uint32_t>(ldz) * 4u;
  uint32_t xo[4], zo[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int c = zc * 64 + 16 * b + li, o = by * 64 + 16 * b + li;
    xo[b] = static_cast<uint32_t>(c < d_in ? c : 0) * 4u;
    zo[b] = static_cast<uint32_t>(o < ldz ? o : 0) * 4u;
  }
  const int gx = gridDim.x;
  const int rows_per_part = ((n + gx - 1) / gx + 15) / 16 * 16;
  const int r0 = min(p * rows_per_part, n);
  const int r1 = min(r0 + rows_per_part, n);
  floatx4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};
  float dbs[4] = {0.f, 0.f, 0.f, 0.f};

  auto load = [&](int k0, float (&xa)[4][8], float (&zb)[4][8]) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int row = k0 + 8 * g + e;
      const uint32_t rc = static_cast<uint32_t>(row < r1 ? row : r1 - 1);
      const uint32_t xr = rc * xrow, zr = rc * zrow;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        xa[b][e] = *reinterpret_cast<const float*>(X + (xr + xo[b]));
        zb[b][e] = *reinterpret_cast<const float*>(Zb + (zr + zo[b]));
      }
    }
  };
  auto compute = [&](int k0, float (&xa)[4][8], float (&zb)[4][8]) {
    if (k0 + 32 > r1) {   // uniform: the range's last chunk of this wave
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (k0 + 8 * g + e >= r1) {
#pragma unroll
          for (int b = 0; b < 4; ++b) zb[b][e] = 0.f;
        }
    }
    if (bz == 0) {   // uniform: the bias sums ride on the first column tile
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e) dbs[b] += zb[b][e];
    }
    bf16x8 bp[4][3];
#pragma unroll
    for (int b = 0; b < 4; ++b)
      parts::split8(make_float4(zb[b][0], zb[b][1], zb[b][2], zb[b][3]),
                    make_float4(zb[b][4], zb[b][5], zb[b][6], zb[b][7]), bp[b]);
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      bf16x8 ap[3];
      parts::split8(make_float4(xa[a][0], xa[a][1], xa[a][2], xa[a][3]),
                    make_float4(xa[a][4], xa[a][5], xa[a][6], xa[a][7]), ap);
      // the smallest part products first
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[0], bp[b][2], acc[a][b], 0, 0, 0);
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[1], bp[b][1], acc[a][b], 0, 0, 0);
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[2], bp[b][0], acc[a][b], 0, 0, 0);
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[0], bp[b][1], acc[a][b], 0, 0, 0);
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[1], bp[b][0], acc[a][b], 0, 0, 0);
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[0], bp[b][0], acc[a][b], 0, 0, 0);
    }
  };

  // loads run D - 1 chunks ahead of the products; the body is unrolled D
  // times so that every buffer keeps its registers, the chunk count is
  // rounded up to a multiple of D and a chunk past the range adds zero
  constexpr int D = kWgradPartsDepth, STRIDE = 32 * W;
  int k0 = r0 + 32 * wave;
  const int nsteps = __builtin_amdgcn_readfirstlane(k0 < r1 ? (r1 - k0 + STRIDE - 1) / STRIDE : 0);
  float xs[D][4][8], zs[D][4][8];
  if (nsteps > 0) {
#pragma unroll
    for (int b = 0; b + 1 < D; ++b) load(k0 + STRIDE * b, xs[b], zs[b]);
  }
  for (int it = 0; it < nsteps; it += D) {
#pragma unroll
    for (int b = 0; b < D; ++b) {
      load(k0 + STRIDE * (b + D - 1), xs[(b + D - 1) % D], zs[(b + D - 1) % D]);
      __builtin_amdgcn_sched_barrier(0);
      compute(k0 + STRIDE * b, xs[b], zs[b]);
      __builtin_amdgcn_sched_barrier(0);
    }
    k0 += STRIDE * D;
  }
  // the bias sums over the lane's rows, then over g
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    dbs[b] += __shfl_xor(dbs[b], 16, 64);
    dbs[b] += __shfl_xor(dbs[b], 32, 64);
  }
  float* mine = red[wave];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) mine[(16 * a + 4 * g + r) * kPad + 16 * b + li] = acc[a][b][r];
  if (g == 0) {
#pragma unroll
    for (int b = 0; b < 4; ++b) red_db[wave][16 * b + li] = dbs[b];
  }
  __syncthreads();
  // thread t of the 64 W: tile row t / W, the 64 / W columns from
  // (64 / W) (t % W); the waves' sums added in wave order
  constexpr int kPer = 64 / W;
  float* part = partial + static_cast<int64_t>(p) * (K2 + 1) * ldp;
  const int m = threadIdx.x / W, n0 = kPer * (threadIdx.x % W);
  const int c = zc * 64 + m;
  if (c < d_in) {
    float* dst = part + static_cast<int64_t>(from_m ? d_in + c : c) * ldp;
#pragma unroll
    for (int s4 = 0; s4 < kPer / 4; ++s4) {
      const int o = by * 64 + n0 + 4 * s4;
      if (o >= ldp) break;
      float4 v = *reinterpret_cast<const float4*>(&red[0][m * kPad + n0 + 4 * s4]);
#pragma unroll
      for (int w = 1; w < W; ++w) {
        const float4 x = *reinterpret_cast<const float4*>(&red[w][m * kPad + n0 + 4 * s4]);
        v.x += x.x; v.y += x.y; v.z += x.z; v.w += x.w;
      }
      *reinterpret_cast<float4*>(dst + o) = v;
    }
  }
  if (bz == 0 && threadIdx.x < 16) {
    const int o = by * 64 + 4 * threadIdx.x;
    if (o < ldp) {
      float v[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int cc = 4 * threadIdx.x + j;
        v[j] = red_db[0][cc];
#pragma unroll
        for (int w = 1; w < W; ++w) v[j] += red_db[w][cc];
      }
      *reinterpret_cast<float4*>(part + static_cast<int64_t>(K2) * ldp + o) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// One float4 of output per thread group of four: group g sums the parts
// p = g, g + 4, ... in ascending order, the four groups meet in LDS in a
// fixed order.  Rows i < 2 d_in go to dW_self / dW_neigh, row 2 d_in to db.
// Workgroup `block` of the reduction of `r` (block r.blocks - 1 sums the
// loss when r.loss is set).
__device__ void wgrad_reduce_block(const ReduceArgs& r, int block) {
  if (r.loss && block == r.blocks - 1) {   // the appended workgroup (uniform)
    loss_sum_block(r.loss_rows, r.n_loss, r.loss);
    return;
  }
  __shared__ float4 red[3][64];
  const int d_in = r.d_in, d_out = r.d_out, ldp = r.ldp, parts = r.parts;
  const int K2 = 2 * d_in;
  const int per_row = ldp / 4;
  const int64_t total = static_cast<int64_t>(K2 + 1) * per_row;
  const int64_t idx = static_cast<int64_t>(block) * 64 + (threadIdx.x & 63);
  const int g = threadIdx.x >> 6;
  const bool live = idx < total;
  const int64_t stride = static_cast<int64_t>(K2 + 1) * ldp;
  const float* src = r.partial + (live ? idx * 4 : 0);
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
  int p = g;
  for (; p + 4 < parts; p += 8) {
    const float4 x = *reinterpret_cast<const float4*>(src + p * stride);
    const float4 y = *reinterpret_cast<const float4*>(src + (p + 4) * stride);
    a.x += x.x; a.y += x.y; a.z += x.z; a.w += x.w;
    b.x += y.x; b.y += y.y; b.z += y.z; b.w += y.w;
  }
  if (p < parts) {
    const float4 x = *reinterpret_cast<const float4*>(src + p * stride);
    a.x += x.x; a.y += x.y; a.z += x.z; a.w += x.w;
  }
  a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
  if (g > 0) red[g - 1][threadIdx.x & 63] = a;
  __syncthreads();
  if (g != 0 || !live) return;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const float4 x = red[k][threadIdx.x];
    a.x += x.x; a.y += x.y; a.z += x.z; a.w += x.w;
  }
  const int i = static_cast<int>(idx / per_row);
  const int o = static_cast<int>(idx % per_row) * 4;
  float* dst = i < d_in ? r.d_self + static_cast<int64_t>(i) * d_out
                        : (i < K2 ? r.d_neigh + static_cast<int64_t>(i - d_in) * d_out : r.d_bias);
  const float v[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (o + j < d_out) dst[o + j] = v[j];
}

__global__ __launch_bounds__(256) void k_wgrad_reduce(ReduceArgs r) { wgrad_reduce_block(r, blockIdx.x); }

// ---- input gradient -------------------------------------------------------

// The block's edges as slots (v, j), j < fanout (a sampled row holds at
// most fanout edges): slot (v, j) is edge indptr[v] + j if that is below
// indptr[v+1] and cap_nnz; sources outside [0, n_src) are skipped (only
// after a data error).  The count and the fill below enumerate the same
// slots, so every source's places in the transpose are filled exactly once.
struct EdgeView {
  const int32_t* indptr;
  const int32_t* local;
  int64_t cap_nnz;
  int32_t fanout;
};

__device__ __forceinline__ void edge_range(const EdgeView& ev, int64_t v, int32_t& b, int32_t& e) {
  b = ev.indptr[v];
  e = ev.indptr[v + 1];
  b = b < 0 ? 0 : (b > ev.cap_nnz ? static_cast<int32_t>(ev.cap_nnz) : b);
  e = e < b ? b : (e > ev.cap_nnz ? static_cast<int32_t>(ev.cap_nnz) : e);
}

// Calls f(v, u, k_v) for every slot of the block that holds an edge, slot
// t = v * fanout + j over a grid-stride loop starting at t0.
template <typename F>
__device__ __forceinline__ void for_each_edge_slot(const EdgeView& ev, int32_t n_dst, int32_t n_src, int64_t t0,
                                                   int64_t stride, F&& f) {
  if (ev.fanout < 1) return;
  const int64_t total = static_cast<int64_t>(n_dst) * ev.fanout;
  for (int64_t t = t0; t < total; t += stride) {
    const int64_t v = t / ev.fanout;
    const int32_t j = static_cast<int32_t>(t - v * ev.fanout);
    int32_t b, e;
    edge_range(ev, v, b, e);
    if (b + j >= e) continue;
    const int32_t u = ev.local[b + j];
    if (u < 0 || u >= n_src) continue;
    f(v, u, e - b);
  }
}

// out = dZ [W_self; W_neigh]^T over the block's n_dst rows: K = d_out (in
// NCH chunks of 16), output column nn < d_in goes to dH, d_in <= nn < 2 d_in
// to dM (both with row stride d_in).  The slab holds B[k][nn] = W[nn][k]
// for the workgroup's 64 columns in operand order (as the forward's slab
// kernel), filled with 16-byte loads and stores when d_out % 4 == 0 (VEC);
// lane l (q = l/16) of a wave reads B[16c + 4q .. +3][nn] with one 16-byte
// LDS read and A = dZ[row][16c + 4q .. +3] (ldz % 4 == 0, zero past d_out)
// with one 16-byte global read.  Afterwards every thread of the grid
// counts in-edges of the block's sources into cnt (grid-stride over the
// edge slots).
template <int NCH, bool VEC>
__global__ __launch_bounds__(256) void k_dgrad(const int32_t* __restrict__ sizes, const float* __restrict__ dZ,
                                               int ldz, int d_out, const float* __restrict__ Ws,
                                               const float* __restrict__ Wn, int d_in,
                                               float* __restrict__ dH, float* __restrict__ dM, EdgeView ev,
                                               int32_t* __restrict__ cnt) {
  constexpr int BN = 64;
  // float4 stride of the slab rows (c, q): one float4 of padding where it
  // fits, so that the fill's stores (consecutive lanes in consecutive rows)
  // spread over all banks
  constexpr int RS = NCH <= 32 ? BN + 1 : BN;
  __shared__ __attribute__((aligned(16))) float Bp[NCH * 4 * RS * 4];
  const int32_t M = load_size(&sizes[kNDst]);
  const int row_tiles = (M + 63) / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, r16 = lane & 15;
  const int n0 = blockIdx.y * BN;
  const int K2 = 2 * d_in;
  if (static_cast<int>(blockIdx.x) < row_tiles) {
    // A of the first row tile: dZ[row][16c + 4q .. +3], issued before the
    // slab fill so that the two latencies overlap
    // (all loads issued first, then one opaque step over the values so that
    // the selects cannot become branched loads, then the selects: one wait)
    auto issue_a = [&](int rt, float4 (&a)[NCH]) {
      const int row = rt * 64 + wave * 16 + r16;
      const float* zr = dZ + static_cast<int64_t>(row < M ? row : M - 1) * ldz;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int k = 16 * c + 4 * q;
        a[c] = *reinterpret_cast<const float4*>(zr + (k < ldz ? k : 0));
      }
    };
    auto finish_a = [&](float4 (&a)[NCH]) {
#pragma unroll
      for (int c = 0; c < NCH; ++c) asm volatile("" : "+v"(a[c].x), "+v"(a[c].y), "+v"(a[c].z), "+v"(a[c].w));
#pragma unroll
      for (int c = 0; c < NCH; ++c)
        if (16 * c + 4 * q >= ldz) a[c] = make_float4(0.f, 0.f, 0.f, 0.f);
    };
    float4 a[NCH];
    issue_a(blockIdx.x, a);
    if (VEC) {
      // item (nn, k4): W[n0 + nn][4 k4 .. 4 k4 + 3], k4 fastest; all of a
      // thread's loads in flight at once
      constexpr int kPer = BN * NCH * 4 / 256;
      constexpr int kBatch = kPer % 16 == 0 ? 16 : (kPer % 8 == 0 ? 8 : kPer);
      static_assert(kPer % kBatch == 0, "the fill batches must tile the slab exactly");
      for (int u0 = 0; u0 < kPer; u0 += kBatch) {
        float4 v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int idx = (u0 + u) * 256 + threadIdx.x;
          const int nn = idx / (NCH * 4), k4 = idx % (NCH * 4);
          const int gn = n0 + nn;
          const bool in = gn < K2 && 4 * k4 < d_out;
          const float* w = gn < d_in ? Ws + static_cast<int64_t>(gn) * d_out
                                     : Wn + static_cast<int64_t>(in ? gn - d_in : 0) * d_out;
          v[u] = *reinterpret_cast<const float4*>(w + (in ? 4 * k4 : 0));
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) asm volatile("" : "+v"(v[u].x), "+v"(v[u].y), "+v"(v[u].z), "+v"(v[u].w));
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int idx = (u0 + u) * 256 + threadIdx.x;
          const int nn = idx / (NCH * 4), k4 = idx % (NCH * 4);
          const bool in = n0 + nn < K2 && 4 * k4 < d_out;
          *reinterpret_cast<float4*>(&Bp[(k4 * RS + nn) * 4]) = in ? v[u] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
    } else {
      // item (nn, k) with k fastest, so a weight row is read contiguously
      constexpr int kItems = BN * NCH * 16;
      for (int base = 0; base < kItems; base += 256 * 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int idx = base + u * 256 + threadIdx.x;
          const int nn = idx / (NCH * 16), k = idx % (NCH * 16);
          const int gn = n0 + nn;
          const bool in = idx < kItems && gn < K2 && k < d_out;
          const float* w = gn < d_in ? Ws + static_cast<int64_t>(gn) * d_out
                                     : Wn + static_cast<int64_t>(in ? gn - d_in : 0) * d_out;
          v[u] = w[in ? k : 0];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) asm volatile("" : "+v"(v[u]));
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int idx = base + u * 256 + threadIdx.x;
          if (idx >= kItems) continue;
          const int nn = idx / (NCH * 16), k = idx % (NCH * 16);
          const bool in = n0 + nn < K2 && k < d_out;
          Bp[((k >> 2) * RS + nn) * 4 + (k & 3)] = in ? v[u] : 0.f;
        }
      }
    }
    finish_a(a);
    __syncthreads();
    for (int rt = blockIdx.x;;) {
      floatx4 acc[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        float4 b[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = *reinterpret_cast<const float4*>(&Bp[((c * 4 + q) * RS + j * 16 + r16) * 4]);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[c].x, b[j].x, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[c].y, b[j].y, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[c].z, b[j].z, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[c].w, b[j].w, acc[j], 0, 0, 0);
      }
      const int orow0 = rt * 64 + wave * 16 + 4 * q;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int nn = n0 + j * 16 + r16;
        if (nn >= K2) continue;
        float* dst = nn < d_in ? dH + nn : dM + (nn - d_in);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (orow0 + r < M) dst[static_cast<int64_t>(orow0 + r) * d_in] = acc[j][r];
      }
      rt += gridDim.x;
      if (rt >= row_tiles) break;
      issue_a(rt, a);
      finish_a(a);
    }
  }
  // the block's in-edge count per source, for the transpose (the next
  // kernel on the stream reads it)
  for_each_edge_slot(ev, M, load_size(&sizes[kNSrc]),
                     (static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x) * blockDim.x + threadIdx.x,
                     static_cast<int64_t>(gridDim.x) * gridDim.y * blockDim.x,
                     [&](int64_t, int32_t u, int32_t) { atomicAdd(&cnt[u], 1); });
}

// The same product on the bf16 matrix cores through the exact three-way
// cut of the operands (parts.hpp), for d_out % 4 == 0 and d_out <= 512: A =
// dZ, B = the weights' transpose in the slab; then the in-edge count, as
// above.  The workgroups past the product's row tiles go straight to the
// count.
template <int NCH, int J, int R, int SPLIT, int WAVES>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(WAVES / 4, WAVES / 4)))
void k_dgrad_parts(const int32_t* __restrict__ sizes, parts::DgradOp op, EdgeView ev, int32_t* __restrict__ cnt) {
  const int32_t M = load_size(&sizes[kNDst]);
  parts::parts_gemm<parts::DgradOp, NCH, J, R, SPLIT, WAVES>(op, M);
  for_each_edge_slot(ev, M, load_size(&sizes[kNSrc]),
                     (static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x) * blockDim.x + threadIdx.x,
                     static_cast<int64_t>(gridDim.x) * gridDim.y * blockDim.x,
                     [&](int64_t, int32_t u, int32_t) { atomicAdd(&cnt[u], 1); });
}

template <int NCH, int J, int R, int SPLIT, int WAVES>
void launch_dgrad_parts(const int32_t* sizes, const parts::DgradOp& op, int64_t cap_rows, const EdgeView& ev,
                        int32_t* cnt, hipStream_t s) {
  static_assert(parts::parts_lds_bytes(NCH, J, R, SPLIT, WAVES) <= 160 * 1024, "slab exceeds the LDS");
  hipLaunchKernelGGL((k_dgrad_parts<NCH, J, R, SPLIT, WAVES>), (parts::parts_grid<J, R, SPLIT, WAVES>(cap_rows, op.n())),
                     dim3(64 * WAVES), 0, s, sizes, op, ev, cnt);
}

// Tiling as the forward's part-product launches: eight waves per
// workgroup; many rows: a wave's own 16 rows of a 64-column slab (K up to
// 256); fewer: split K over the eight waves.  False where the shape has no
// part-product tiling (the fp32-instruction kernel takes it).
template <int NCH>
bool dgrad_parts_for(const int32_t* sizes, const parts::DgradOp& op, int64_t cap_rows, const EdgeView& ev,
                     int32_t* cnt, hipStream_t s) {
  const int N = op.n();
  const int64_t big_tiles = ((cap_rows + 127) / 128) * ((N + 63) / 64);
  if (big_tiles >= 2 * 256) {
    if constexpr (NCH <= 8) {
      launch_dgrad_parts<NCH, 4, 1, 1, 8>(sizes, op, cap_rows, ev, cnt, s);
      return true;
    }
    return false;
  }
  if (cap_rows * N > (int64_t{1} << 18)) {
    // 64 columns a workgroup where the slab allows it: twice the workgroups
    // per column tile, half the row tiles each walks
    if constexpr (NCH <= 8)
      launch_dgrad_parts<NCH, 4, 1, 4, 8>(sizes, op, cap_rows, ev, cnt, s);
    else
      launch_dgrad_parts<NCH, 2, 1, 4, 8>(sizes, op, cap_rows, ev, cnt, s);
  } else
    launch_dgrad_parts<NCH, 1, 1, 4, 8>(sizes, op, cap_rows, ev, cnt, s);
  return true;
}

// ---- mean backward: the block's transpose -----------------------------------

// off[u] = sum of cnt[0 .. u), off[n_src] = the total, pos[u] = off[u]
// (the fill's cursors), cnt cleared for the next layer, and the sources
// with more than kLongList entries listed in long_rows[0 .. *n_long).  Tiles of 1024
// counts (four per thread), numbered by an atomic ticket, joined by the
// decoupled look-back (both the ticket and the look-back words start at 0).
// If the look-back's bounded wait runs out (it does not when every tile
// runs), the offsets come out wrong but the fill and the pull stay in
// bounds.
// Counts per scan workgroup (256 threads, kScanTile / 1024 int4 each):
// 4096 measured no faster than 1024 on the 342k sources of a products2m
// block's bottom layer (13 against 14 us; the hidden layer's fused scan 1 us
// slower), once workgroups past the tiles leave without a ticket.
#ifndef GMB_SCAN_TILE
#define GMB_SCAN_TILE 1024
#endif
constexpr int kScanTile = GMB_SCAN_TILE;
constexpr int kScanVec = kScanTile / 1024;
constexpr int kLongList = 16;   // transpose lists longer than this take a workgroup each

// The embedding update's groups: lanes per row, rows per group, entries per
// row read in the first batch (tuning macros, -D at build time).
#ifndef GMB_PULL_UPDATE_G
#define GMB_PULL_UPDATE_G 32
#endif
#ifndef GMB_PULL_UPDATE_R
#define GMB_PULL_UPDATE_R 4
#endif
#ifndef GMB_PULL_UPDATE_E
#define GMB_PULL_UPDATE_E 1
#endif

// WG = 0: the scan alone (its own small register and LDS footprint);
// 1, 2: workgroups past the scan's run the same layer's weight-gradient
// products (16-byte or scalar loads of H and M), independent of the scan:
// one launch for both; the scan's workgroups come first, so its tiles
// start before the products fill the CUs.
constexpr int wg_occupancy(int wg) { return wg == 0 ? 8 : (kWgradDepth <= 4 ? 2 : 1); }

template <int WG>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(wg_occupancy(WG), wg_occupancy(WG))))
void k_csc_scan(const int32_t* __restrict__ sizes, int32_t* __restrict__ cnt, int32_t* __restrict__ off,
                int32_t* __restrict__ pos, uint32_t* __restrict__ ticket, uint64_t* __restrict__ words,
                uint32_t* __restrict__ n_long, int32_t* __restrict__ long_rows, int scan_blocks, WgradArgs wg) {
  if constexpr (WG != 0) {
    if (static_cast<int>(blockIdx.x) >= scan_blocks) {
      const int w = blockIdx.x - scan_blocks;
      wgrad_block<WG == 1>(wg.sizes, wg.H, wg.M, wg.d_in, wg.dZ, wg.ldz, wg.ldp, wg.partial, w % wg.parts,
                           (w / wg.parts) % wg.ytiles, w / (wg.parts * wg.ytiles), wg.parts);
      return;
    }
  }
  __shared__ int s_tile;
  __shared__ int32_t s_excl;
  __shared__ int32_t smem[4];
  const int32_t n = load_size(&sizes[kNSrc]);
  const int ntiles = (n + kScanTile - 1) / kScanTile;
  // the grid is sized by the capacity: a workgroup past the tiles leaves
  // without a ticket (the first ntiles workgroups take tickets 0 ..
  // ntiles - 1, in the order in which they start)
  if (static_cast<int>(blockIdx.x) >= ntiles) {
    if (blockIdx.x == 0 && threadIdx.x == 0) off[0] = 0;
    return;
  }
  const int tile = claim_tile(ticket, &s_tile);
  // thread t holds the counts i0 + j, j < 4 kScanVec, of the tile
  const int32_t i0 = tile * kScanTile + 4 * kScanVec * static_cast<int32_t>(threadIdx.x);
  constexpr int C = 4 * kScanVec;
  int32_t c[C];
#pragma unroll
  for (int v = 0; v < kScanVec; ++v) {
    const int32_t a = i0 + 4 * v;
    if (a + 3 < n) {
      const int4 x = *reinterpret_cast<const int4*>(cnt + a);
      c[4 * v] = x.x; c[4 * v + 1] = x.y; c[4 * v + 2] = x.z; c[4 * v + 3] = x.w;
      *reinterpret_cast<int4*>(cnt + a) = make_int4(0, 0, 0, 0);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[4 * v + j] = a + j < n ? cnt[a + j] : 0;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (a + j < n) cnt[a + j] = 0;
    }
  }
  int32_t sum = 0;
#pragma unroll
  for (int j = 0; j < C; ++j) sum += c[j];
  const int32_t x[1] = {sum};
  int32_t excl[1], total[1];
  block_exclusive_scan_multi<256, 1>(x, excl, total, smem);
  if (threadIdx.x < 64) {
    const int32_t agg[1] = {total[0]};
    int32_t ex[1];
    tile_lookback_multi<1>(words, 0, tile, agg, ex);
    if (threadIdx.x == 0) s_excl = ex[0];
  }
  __syncthreads();
  int32_t o = s_excl + excl[0];
#pragma unroll
  for (int v = 0; v < kScanVec; ++v) {
    const int32_t a = i0 + 4 * v;
    int32_t e[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      e[j] = o;
      o += c[4 * v + j];
    }
    if (a + 3 < n) {
      *reinterpret_cast<int4*>(off + a) = make_int4(e[0], e[1], e[2], e[3]);
      *reinterpret_cast<int4*>(pos + a) = make_int4(e[0], e[1], e[2], e[3]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (a + j < n) {
          off[a + j] = e[j];
          pos[a + j] = e[j];
        }
    }
  }
  if (tile == ntiles - 1 && threadIdx.x == 0) off[n] = s_excl + total[0];
  // sources with long lists (hubs) go to the list the workgroup-per-row
  // kernel takes (the per-row kernels skip them); after the look-back, so
  // that the successors' waits do not include it; one atomic per wave and
  // item, the lanes' places from the ballot
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < C; ++j) {
    const uint64_t mask = __ballot(c[j] > kLongList);
    if (!mask) continue;   // uniform
    const int leader = __ffsll(static_cast<long long>(mask)) - 1;
    uint32_t base = 0;
    if (lane == leader) base = atomicAdd(n_long, static_cast<uint32_t>(__popcll(mask)));
    base = __shfl(base, leader, 64);
    if (c[j] > kLongList) long_rows[base + __popcll(mask & ((1ull << lane) - 1ull))] = i0 + j;
  }
}

// Thread per edge slot: the edge (v <- u) takes the next place of u and
// stores (v, 1/k_v) there.
// Workgroups past fill_blocks run the same layer's weight-gradient
// reduction (it only needs the products of the launch before).
__global__ __launch_bounds__(256) void k_csc_fill(const int32_t* __restrict__ sizes, EdgeView ev,
                                                  int32_t* __restrict__ pos, const int32_t* __restrict__ off,
                                                  int2* __restrict__ csc, int fill_blocks, ReduceArgs fold) {
  if (static_cast<int>(blockIdx.x) >= fill_blocks) {
    wgrad_reduce_block(fold, blockIdx.x - fill_blocks);
    return;
  }
  for_each_edge_slot(ev, load_size(&sizes[kNDst]), load_size(&sizes[kNSrc]),
                     static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x,
                     static_cast<int64_t>(fill_blocks) * blockDim.x, [&](int64_t v, int32_t u, int32_t k) {
                       const int32_t slot = atomicAdd(&pos[u], 1);
                       if (slot < off[u + 1] && slot < ev.cap_nnz)
                         csc[slot] = make_int2(static_cast<int32_t>(v), __float_as_int(1.f / static_cast<float>(k)));
                     });
}

// The sources with long transpose lists, one workgroup per row (the n_wg
// workgroups that the row kernels append to their grids stride over the
// list; wg is this one's index among them): the eight 32-lane groups take the entries
// j = g, g + 8, ... four at a time (one round of entry reads, then one of
// dM rows), lane c covers the float4 columns c, c + 32, ...; the groups'
// sums meet in LDS in a fixed order, then the row is finished as in
// k_pull_mean (UPDATE = false: masked by the layer below's output, written
// to dH) or k_pull_update (UPDATE = true: applied to the table row).
template <bool UPDATE>
__device__ void pull_long_rows(int wg, int n_wg, const int32_t* __restrict__ sizes,
                               const uint32_t* __restrict__ n_long, const int32_t* __restrict__ long_rows,
                               const int32_t* __restrict__ off, const int2* __restrict__ csc, int64_t cap_nnz,
                               const float* __restrict__ dM, const float* __restrict__ out, int d,
                               float* __restrict__ dH, float* __restrict__ table, const int32_t* __restrict__ ids,
                               int64_t num_nodes, float lr) {
  constexpr int kGroups = 8, E = 4;
  __shared__ float4 part[kGroups - 1][32];
  const int32_t n_dst = load_size(&sizes[kNDst]);
  const int32_t n_src = load_size(&sizes[kNSrc]);
  const int32_t nl = static_cast<int32_t>(__hip_atomic_load(n_long, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  const int grp = threadIdx.x >> 5, lane = threadIdx.x & 31;
  const int chunks = d / 4;
  for (int32_t li = wg; li < nl; li += n_wg) {
    const int32_t u = long_rows[li];
    if (u < 0 || u >= n_src) continue;   // uniform over the workgroup
    int32_t s0 = off[u], s1 = off[u + 1];
    s0 = s0 < 0 ? 0 : s0;
    s1 = s1 > cap_nnz ? static_cast<int32_t>(cap_nnz) : s1;
    const int32_t cnt = s1 > s0 ? s1 - s0 : 0;
    int64_t trow = 0;
    bool live = true;
    if (UPDATE) {
      const int32_t id = ids[u];
      live = id >= 0 && id < num_nodes;
      trow = live ? id : 0;
    }
    for (int c0 = lane; c0 < chunks + 31 - (chunks - 1) % 32; c0 += 32) {   // whole passes
      const int c = c0 < chunks ? c0 : chunks - 1;
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int32_t base = grp; base < cnt; base += kGroups * E) {
        int2 e[E];
#pragma unroll
        for (int j = 0; j < E; ++j) {
          const int32_t k = base + j * kGroups;
          e[j] = csc[k < cnt ? s0 + k : s0];
        }
        float4 g[E];
        float w[E];
#pragma unroll
        for (int j = 0; j < E; ++j) {
          const bool ok = base + j * kGroups < cnt && e[j].x >= 0 && e[j].x < n_dst;
          w[j] = ok ? __int_as_float(e[j].y) : 0.f;
          g[j] = *reinterpret_cast<const float4*>(dM + static_cast<int64_t>(ok ? e[j].x : 0) * d + 4 * c);
        }
#pragma unroll
        for (int j = 0; j < E; ++j) {
          acc.x += w[j] * g[j].x; acc.y += w[j] * g[j].y; acc.z += w[j] * g[j].z; acc.w += w[j] * g[j].w;
        }
      }
      if (grp > 0) part[grp - 1][lane] = acc;
      __syncthreads();
      if (grp == 0) {
#pragma unroll
        for (int k = 0; k < kGroups - 1; ++k) {
          const float4 x = part[k][lane];
          acc.x += x.x; acc.y += x.y; acc.z += x.z; acc.w += x.w;
        }
        const int64_t at = static_cast<int64_t>(u) * d + 4 * c;
        if (u < n_dst) {
          const float4 x = *reinterpret_cast<const float4*>(dH + at);
          acc.x += x.x; acc.y += x.y; acc.z += x.z; acc.w += x.w;
        }
        if (c0 < chunks) {
          if (UPDATE) {
            if (live) {
              float4* t = reinterpret_cast<float4*>(table + trow * d + 4 * c);
              float4 v = *t;
              v.x -= lr * acc.x; v.y -= lr * acc.y; v.z -= lr * acc.z; v.w -= lr * acc.w;
              *t = v;
            }
          } else {
            const float4 o = *reinterpret_cast<const float4*>(out + at);
            acc.x = o.x > 0.f ? acc.x : 0.f;
            acc.y = o.y > 0.f ? acc.y : 0.f;
            acc.z = o.z > 0.f ? acc.z : 0.f;
            acc.w = o.w > 0.f ? acc.w : 0.f;
            *reinterpret_cast<float4*>(dH + at) = acc;
          }
        }
      }
      __syncthreads();
    }
  }
}

// G lanes per source row u, lane c covers columns 4c, 4c + G, ... (d % 4 ==
// 0): g = (u < n_dst ? dH[u] : 0) + sum over u's transpose entries (v, w) of
// w * dM[v].  UPDATE = false: dH[u] = (out[u] > 0) * g (out: the layer
// below's output).  UPDATE = true (layer 0 with learnable vertex
// embeddings): table[ids[u]] -= lr * g, a plain read-modify-write (the rows
// of one mini-batch are distinct; mini-batches in flight together update
// without locks, as Hogwild does); an id outside [0, num_nodes) skips the
// row (only after a data error).
template <int G>
__global__ __launch_bounds__(256) void k_pull_mean(const int32_t* __restrict__ sizes,
                                                   const int32_t* __restrict__ off, const int2* __restrict__ csc,
                                                   int64_t cap_nnz, const float* __restrict__ dM,
                                                   const float* __restrict__ out, int d, float* __restrict__ dH,
                                                   int row_blocks, const uint32_t* __restrict__ n_long,
                                                   const int32_t* __restrict__ long_rows) {
  if (static_cast<int>(blockIdx.x) >= row_blocks) {   // the long lists
    pull_long_rows<false>(blockIdx.x - row_blocks, gridDim.x - row_blocks, sizes, n_long, long_rows, off, csc,
                          cap_nnz, dM, out, d, dH, nullptr, nullptr, 0, 0.f);
    return;
  }
  const int32_t n_dst = load_size(&sizes[kNDst]);
  const int32_t n_src = load_size(&sizes[kNSrc]);
  const int64_t u = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / G;
  const int lane = threadIdx.x & (G - 1);
  if (u >= n_src) return;
  int32_t s0 = off[u], s1 = off[u + 1];
  if (s1 - s0 > kLongList) return;   // a long list: the appended workgroups take it
  s0 = s0 < 0 ? 0 : s0;
  s1 = s1 > cap_nnz ? static_cast<int32_t>(cap_nnz) : s1;
  const bool self = u < n_dst;
  const int chunks = d / 4;
  for (int c = lane; c < chunks; c += G) {
    const int64_t at = u * d + 4 * c;
    // the layer below's output does not depend on the gradient: read first
    const float4 o = *reinterpret_cast<const float4*>(out + at);
    float4 acc = self ? *reinterpret_cast<const float4*>(dH + at) : make_float4(0.f, 0.f, 0.f, 0.f);
    // four entries per round of reads (the sum still runs in entry order)
    for (int32_t s = s0; s < s1; s += 4) {
      int2 x[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = s + q < s1 ? csc[s + q] : make_int2(-1, 0);
      float4 g[4];
      float w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bool ok = x[q].x >= 0 && x[q].x < n_dst;
        w[q] = ok ? __int_as_float(x[q].y) : 0.f;
        g[q] = ok ? *reinterpret_cast<const float4*>(dM + static_cast<int64_t>(x[q].x) * d + 4 * c)
                  : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (s + q >= s1) break;
        acc.x += w[q] * g[q].x; acc.y += w[q] * g[q].y; acc.z += w[q] * g[q].z; acc.w += w[q] * g[q].w;
      }
    }
    acc.x = o.x > 0.f ? acc.x : 0.f;
    acc.y = o.y > 0.f ? acc.y : 0.f;
    acc.z = o.z > 0.f ? acc.z : 0.f;
    acc.w = o.w > 0.f ? acc.w : 0.f;
    *reinterpret_cast<float4*>(dH + at) = acc;
  }
}

// Layer 0 with learnable vertex embeddings: table[ids[u]] -= lr * g_u with
// g_u = (u < n_dst ? dH[u] : 0) + sum over u's transpose entries (v, w) of
// w * dM[v], as a plain read-modify-write (the rows of one mini-batch are
// distinct; mini-batches in flight together update without locks, as
// Hogwild does; an id outside [0, num_nodes) skips its row).  Each row
// takes dependent rounds of reads (offsets and ids; table row, self part
// and the first E entries; the entries' dM rows; then the rest of a longer
// list, four entries per round), and every round is issued for the R rows
// of a G-lane group at once.  What bounds the kernel is the rate of its
// scattered 400-byte row accesses (table rows and dM rows), not the
// rounds' latency: one round fewer per row measured no faster.  Lane c
// covers the float4 columns c, c + G, ...
template <int G, int R, int E>
__global__ __launch_bounds__(256) void k_pull_update(const int32_t* __restrict__ sizes,
                                                     const int32_t* __restrict__ off,
                                                     const int2* __restrict__ csc, int64_t cap_nnz,
                                                     const float* __restrict__ dM, float* __restrict__ dH,
                                                     int d, float* __restrict__ table,
                                                     const int32_t* __restrict__ ids, int64_t num_nodes, float lr,
                                                     int row_blocks, const uint32_t* __restrict__ n_long,
                                                     const int32_t* __restrict__ long_rows) {
  if (static_cast<int>(blockIdx.x) >= row_blocks) {   // the long lists
    pull_long_rows<true>(blockIdx.x - row_blocks, gridDim.x - row_blocks, sizes, n_long, long_rows, off, csc,
                         cap_nnz, dM, nullptr, d, dH, table, ids, num_nodes, lr);
    return;
  }
  const int32_t n_dst = load_size(&sizes[kNDst]);
  const int32_t n_src = load_size(&sizes[kNSrc]);
  const int64_t group = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / G;
  const int lane = threadIdx.x & (G - 1);
  const int64_t u0 = group * R;
  if (u0 >= n_src) return;
  // first reads: the rows' offsets and table ids
  int32_t s0[R], cnt[R], trow[R];
  bool live[R], self[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t u = u0 + r;
    const int64_t uc = u < n_src ? u : u0;
    int32_t a = off[uc], b = off[uc + 1];
    const int32_t id = ids[uc];
    const bool long_list = b - a > kLongList;   // the appended workgroups take it
    a = a < 0 ? 0 : a;
    b = b > cap_nnz ? static_cast<int32_t>(cap_nnz) : b;
    s0[r] = a;
    cnt[r] = b > a && !long_list ? b - a : 0;
    live[r] = u < n_src && id >= 0 && id < num_nodes && !long_list;
    trow[r] = live[r] ? id : 0;
    self[r] = u < n_dst;
  }
  const int chunks = d / 4;
  for (int c0 = lane; c0 < chunks + G - 1 - (chunks - 1) % G; c0 += G) {   // whole passes of the group
    const int c = c0 < chunks ? c0 : chunks - 1;
    // second reads: table rows, self parts, the first E entries of every row
    float4 keep[R], acc[R];
    int2 e[R][E];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      keep[r] = *reinterpret_cast<const float4*>(table + static_cast<int64_t>(trow[r]) * d + 4 * c);
      acc[r] = *reinterpret_cast<const float4*>(dH + (self[r] ? u0 + r : 0) * d + 4 * c);
#pragma unroll
      for (int j = 0; j < E; ++j) e[r][j] = csc[j < cnt[r] ? s0[r] + j : 0];
    }
    // third reads: the entries' dM rows
    float4 g[R][E];
    float w[R][E];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int j = 0; j < E; ++j) {
        const bool ok = j < cnt[r] && e[r][j].x >= 0 && e[r][j].x < n_dst;
        w[r][j] = ok ? __int_as_float(e[r][j].y) : 0.f;
        g[r][j] = *reinterpret_cast<const float4*>(dM + static_cast<int64_t>(ok ? e[r][j].x : 0) * d + 4 * c);
      }
    // (the table rows and self parts are used unconditionally from here, so
    // the compiler cannot turn their reads into branched ones; the step
    // comes after the dM reads are issued so that all of them overlap)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      asm volatile("" : "+v"(keep[r].x), "+v"(keep[r].y), "+v"(keep[r].z), "+v"(keep[r].w));
      asm volatile("" : "+v"(acc[r].x), "+v"(acc[r].y), "+v"(acc[r].z), "+v"(acc[r].w));
      if (!self[r]) acc[r] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int j = 0; j < E; ++j) {
        acc[r].x += w[r][j] * g[r][j].x;
        acc[r].y += w[r][j] * g[r][j].y;
        acc[r].z += w[r][j] * g[r][j].z;
        acc[r].w += w[r][j] * g[r][j].w;
      }
    // the rest of the longer lists, four entries per round of reads (the
    // sum still runs in entry order)
#pragma unroll
    for (int r = 0; r < R; ++r)
      for (int32_t j = E; j < cnt[r]; j += 4) {
        int2 x[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) x[q] = j + q < cnt[r] ? csc[s0[r] + j + q] : make_int2(-1, 0);
        float4 gx[4];
        float wx[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const bool ok = x[q].x >= 0 && x[q].x < n_dst;
          wx[q] = ok ? __int_as_float(x[q].y) : 0.f;
          gx[q] = ok ? *reinterpret_cast<const float4*>(dM + static_cast<int64_t>(x[q].x) * d + 4 * c)
                     : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (j + q >= cnt[r]) break;
          acc[r].x += wx[q] * gx[q].x; acc[r].y += wx[q] * gx[q].y;
          acc[r].z += wx[q] * gx[q].z; acc[r].w += wx[q] * gx[q].w;
        }
      }
    if (c0 >= chunks) continue;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (!live[r]) continue;
      float4 v = keep[r];
      v.x -= lr * acc[r].x; v.y -= lr * acc[r].y; v.z -= lr * acc[r].z; v.w -= lr * acc[r].w;
      *reinterpret_cast<float4*>(table + static_cast<int64_t>(trow[r]) * d + 4 * c) = v;
    }
  }
}

// ---- SGD ------------------------------------------------------------------

// Every listed array set to zero, and *scalar too when given (the
// gradients and the loss of an empty batch).
__global__ __launch_bounds__(256) void k_zero(SgdArgs a, float* scalar) {
  if (scalar && blockIdx.x == 0 && threadIdx.x == 0) *scalar = 0.f;
  for (int t = 0; t < a.count; ++t) {
    float* w = a.w[t];
    const int64_t n = a.n[t];
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
      w[i] = 0.f;
  }
}

__global__ __launch_bounds__(256) void k_sgd(SgdArgs a, float lr) {
  for (int t = 0; t < a.count; ++t) {
    float* w = a.w[t];
    const float* g = a.g[t];
    uint16_t* lo = a.lo[t];
    float* mirror = a.mirror[t];
    const int64_t n = a.n[t];
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
      const float v = w[i] - lr * g[i];
      w[i] = v;
      if (lo) lo[i] = f32_to_bf16(v);
      if (mirror) mirror[i] = v;
    }
  }
}

// bf16 -> fp32, eight elements per step where a segment allows it.
__global__ __launch_bounds__(256) void k_widen(WidenArgs a) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  for (int t = 0; t < a.count; ++t) {
    int64_t rows = a.cap_rows[t];
    if (a.rows_dev[t]) {
      const int64_t r = load_size(a.rows_dev[t]);
      rows = r < 0 ? 0 : (r < rows ? r : rows);
    }
    const int64_t n = rows * a.cols[t];
    const uint16_t* src = a.src[t];
    float* dst = a.dst[t];
    const int64_t n8 = n / 8;
    for (int64_t i = tid; i < n8; i += stride) {
      const uint4 x = *reinterpret_cast<const uint4*>(src + 8 * i);
      const uint32_t w[4] = {x.x, x.y, x.z, x.w};
      float4 lo, hi;
      lo.x = bf16_to_f32(static_cast<uint16_t>(w[0])); lo.y = bf16_to_f32(static_cast<uint16_t>(w[0] >> 16));
      lo.z = bf16_to_f32(static_cast<uint16_t>(w[1])); lo.w = bf16_to_f32(static_cast<uint16_t>(w[1] >> 16));
      hi.x = bf16_to_f32(static_cast<uint16_t>(w[2])); hi.y = bf16_to_f32(static_cast<uint16_t>(w[2] >> 16));
      hi.z = bf16_to_f32(static_cast<uint16_t>(w[3])); hi.w = bf16_to_f32(static_cast<uint16_t>(w[3] >> 16));
      *reinterpret_cast<float4*>(dst + 8 * i) = lo;
      *reinterpret_cast<float4*>(dst + 8 * i + 4) = hi;
    }
    for (int64_t i = 8 * n8 + tid; i < n; i += stride) dst[i] = bf16_to_f32(src[i]);
  }
}

inline unsigned grid_of(int64_t threads, int64_t cap = 65535) {
  int64_t g = (threads + 255) / 256;
  if (g > cap) g = cap;
  return static_cast<unsigned>(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_xent(const float* logits, const int32_t* labels, int n, int C, int ldz, float* dz,
                       float* loss_rows, int32_t* clear, int64_t clear_n, hipStream_t s) {
  const unsigned g = static_cast<unsigned>(std::max(1, (n + 3) / 4));
  hipLaunchKernelGGL(k_xent, dim3(g), dim3(256), 0, s, logits, labels, n, C, ldz, dz, loss_rows, clear, clear_n);
  return hipGetLastError();
}

int wgrad_ldp(int d_out) { return (d_out + 3) / 4 * 4; }

// Row ranges of the weight gradient: about 256 workgroups over all tiles
// (one per CU: with 512, twice the partial tiles to write and reduce, the
// training iteration measured 1.3% slower; 384 was slower still),
// at least 64 rows each, a multiple of 8 when above 8 so that the tiles of
// one row range (workgroup ids p + k * parts) share an XCD and its L2.
int wgrad_parts(int64_t cap_rows, int d_in, int d_out) {
  const int tiles = ((wgrad_ldp(d_out) + 63) / 64) * (2 * ((d_in + 63) / 64));
  int parts = (256 + tiles - 1) / tiles;
  const int64_t by_rows = (cap_rows + 63) / 64;
  if (parts > by_rows) parts = static_cast<int>(by_rows);
  if (parts > 8) parts = parts / 8 * 8;
  return parts < 1 ? 1 : parts;
}

hipError_t launch_wgrad(const int32_t* sizes, const float* H, const float* M, int d_in, const float* dZ, int ldz,
                        int d_out, int64_t cap_rows, float* partial, float* d_self, float* d_neigh,
                        float* d_bias, const float* loss_rows, int n_loss, float* loss, WgradArgs* defer,
                        ReduceArgs* fold, hipStream_t s) {
  const int parts = wgrad_parts(cap_rows, d_in, d_out);
  const int ldp = wgrad_ldp(d_out);
  const dim3 grid(parts, (ldp + 63) / 64, 2 * ((d_in + 63) / 64));
  if (static_cast<uint64_t>(std::max<int64_t>(cap_rows, 1)) * std::max(d_in, ldz) * 4 >= (1ull << 32))
    return hipErrorInvalidValue;
  const bool vec = d_in % 4 == 0 && reinterpret_cast<uintptr_t>(H) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(M) % 16 == 0;
  const int64_t outs = static_cast<int64_t>(2 * d_in + 1) * (ldp / 4);
  const ReduceArgs r{partial, parts, d_in, d_out, ldp, d_self, d_neigh, d_bias, loss_rows, n_loss, loss,
                     static_cast<int>((outs + 63) / 64) + (loss ? 1 : 0)};
  if (defer) {
    *defer = WgradArgs{sizes, H, M, d_in, dZ, ldz, ldp, partial, parts, static_cast<int>(grid.y),
                       static_cast<int>(grid.z), vec ? 1 : 0};
  } else {
    hipLaunchKernelGGL(k_wgrad_parts, grid, dim3(64 * kWgradPartsWaves), 0, s, sizes, H, M, d_in, dZ, ldz, ldp,
                       partial);
  }
  if (fold)
    *fold = r;
  else
    hipLaunchKernelGGL(k_wgrad_reduce, dim3(static_cast<unsigned>(r.blocks)), dim3(256), 0, s, r);
  return hipGetLastError();
}

hipError_t launch_dgrad(const int32_t* sizes, const float* dZ, int ldz, int d_out, const float* ws,
                        const float* wn, int d_in, float* dH, float* dM, int64_t cap_rows,
                        const int32_t* indptr, const int32_t* local, int64_t cap_nnz, int32_t fanout, int32_t* cnt,
                        hipStream_t s) {
  const EdgeView ev0{indptr, local, cap_nnz, fanout};
  const uintptr_t align = reinterpret_cast<uintptr_t>(dZ) | reinterpret_cast<uintptr_t>(ws) |
                          reinterpret_cast<uintptr_t>(wn);
  const int nch32 = (d_out + 31) / 32;
  if (d_out % 4 == 0 && ldz % 4 == 0 && align % 16 == 0 && nch32 <= 16) {
    const parts::DgradOp op{dZ, ws, wn, ldz, d_out, d_in, dH, dM};
    bool done;
#define GMB_DPARTS(C) done = dgrad_parts_for<C>(sizes, op, cap_rows, ev0, cnt, s)
    if (nch32 <= 2) GMB_DPARTS(2);
    else if (nch32 <= 4) GMB_DPARTS(4);
    else if (nch32 <= 8) GMB_DPARTS(8);
    else GMB_DPARTS(16);
#undef GMB_DPARTS
    if (done) return hipGetLastError();
  }
  const int nch = (d_out + 15) / 16;
  const int col_tiles = (2 * d_in + 63) / 64;
  int64_t rows = (cap_rows + 63) / 64;
  const int64_t want = (512 + col_tiles - 1) / col_tiles;
  if (rows > want) rows = want;
  if (rows < 1) rows = 1;
  const dim3 grid(static_cast<unsigned>(rows), col_tiles);
  const EdgeView ev{indptr, local, cap_nnz, fanout};
  const bool vec = d_out % 4 == 0 && reinterpret_cast<uintptr_t>(ws) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(wn) % 16 == 0;
#define GMB_DGRAD(C)                                                                                          \
  do {                                                                                                        \
    if (vec)                                                                                                  \
      hipLaunchKernelGGL((k_dgrad<C, true>), grid, dim3(256), 0, s, sizes, dZ, ldz, d_out, ws, wn, d_in, dH, dM, \
                         ev, cnt);                                                                            \
    else                                                                                                      \
      hipLaunchKernelGGL((k_dgrad<C, false>), grid, dim3(256), 0, s, sizes, dZ, ldz, d_out, ws, wn, d_in, dH,    \
                         dM, ev, cnt);                                                                        \
  } while (0)
  if (nch <= 4) GMB_DGRAD(4);
  else if (nch <= 8) GMB_DGRAD(8);
  else if (nch <= 16) GMB_DGRAD(16);
  else if (nch <= 32) GMB_DGRAD(32);
  else if (nch <= 40) GMB_DGRAD(40);
  else return hipErrorInvalidValue;
#undef GMB_DGRAD
  return hipGetLastError();
}

int64_t csc_scan_tiles(int64_t cap_src) { return std::max<int64_t>(1, (cap_src + kScanTile - 1) / kScanTile); }

constexpr int kLongGrid = 512;   // workgroups appended for the long lists (grid-stride over them)

hipError_t launch_mean_backward(const int32_t* sizes, const int32_t* indptr, const int32_t* local,
                                int64_t cap_nnz, int32_t fanout, const float* dM, const float* out, int d, float* dH,
                                int64_t cap_dst, int64_t cap_src, int32_t* cnt, int32_t* off, int32_t* pos,
                                uint32_t* scan_state, int2* csc, int32_t* long_rows, float* table, const int32_t* ids,
                                int64_t num_nodes, float lr, const WgradArgs* defer, const ReduceArgs* fold,
                                hipStream_t s) {
  const EdgeView ev{indptr, local, cap_nnz, fanout};
  // scan_state: [0] the tile ticket, [1] the long-row count, then the
  // look-back words
  const int scan_blocks = static_cast<int>(csc_scan_tiles(cap_src));
  const WgradArgs no_wg{};
  const int wg_blocks = defer ? defer->parts * defer->ytiles * defer->ztiles : 0;
  const dim3 scan_grid(static_cast<unsigned>(scan_blocks + wg_blocks));
  uint64_t* words = reinterpret_cast<uint64_t*>(scan_state + 2);
  if (!defer)
    hipLaunchKernelGGL(k_csc_scan<0>, scan_grid, dim3(256), 0, s, sizes, cnt, off, pos, scan_state, words,
                       scan_state + 1, long_rows, scan_blocks, no_wg);
  else if (defer->vec)
    hipLaunchKernelGGL(k_csc_scan<1>, scan_grid, dim3(256), 0, s, sizes, cnt, off, pos, scan_state, words,
                       scan_state + 1, long_rows, scan_blocks, *defer);
  else
    hipLaunchKernelGGL(k_csc_scan<2>, scan_grid, dim3(256), 0, s, sizes, cnt, off, pos, scan_state, words,
                       scan_state + 1, long_rows, scan_blocks, *defer);
  const int64_t slots = std::max<int64_t>(cap_dst, 1) * std::max(fanout, 1);
  const int fill_blocks = static_cast<int>(grid_of(slots, 1 << 16));
  const ReduceArgs no_red{};
  hipLaunchKernelGGL(k_csc_fill, dim3(static_cast<unsigned>(fill_blocks + (fold ? fold->blocks : 0))), dim3(256), 0,
                     s, sizes, ev, pos, off, csc, fill_blocks, fold ? *fold : no_red);
  const int chunks = d / 4;
  // each grid ends with kLongGrid workgroups for the long lists
  if (table) {
    constexpr int kG = GMB_PULL_UPDATE_G, kR = GMB_PULL_UPDATE_R, kE = GMB_PULL_UPDATE_E;
    const unsigned rows = grid_of((std::max<int64_t>(cap_src, 1) + kR - 1) / kR * kG, 1 << 30);
    hipLaunchKernelGGL((k_pull_update<kG, kR, kE>), dim3(rows + kLongGrid), dim3(256), 0, s, sizes, off, csc,
                       cap_nnz, dM, dH, d, table, ids, num_nodes, lr, static_cast<int>(rows), scan_state + 1,
                       long_rows);
    return hipGetLastError();
  }
  int G = 64;
  if (chunks <= 4) G = 4;
  else if (chunks <= 8) G = 8;
  else if (chunks <= 16) G = 16;
  else if (chunks <= 32) G = 32;
  const unsigned rows = grid_of(std::max<int64_t>(cap_src, 1) * G, 1 << 30);
#define GMB_PULL(GG)                                                                                     \
  hipLaunchKernelGGL((k_pull_mean<GG>), dim3(rows + kLongGrid), dim3(256), 0, s, sizes, off, csc, cap_nnz, dM, \
                     out, d, dH, static_cast<int>(rows), scan_state + 1, long_rows)
  switch (G) {
    case 4: GMB_PULL(4); break;
    case 8: GMB_PULL(8); break;
    case 16: GMB_PULL(16); break;
    case 32: GMB_PULL(32); break;
    default: GMB_PULL(64); break;
  }
#undef GMB_PULL
  return hipGetLastError();
}

hipError_t launch_zero(const SgdArgs& a, float* scalar, hipStream_t s) {
  int64_t most = 1;
  for (int t = 0; t < a.count; ++t) most = std::max(most, a.n[t]);
  hipLaunchKernelGGL(k_zero, dim3(grid_of(most, 1024)), dim3(256), 0, s, a, scalar);
  return hipGetLastError();
}

hipError_t launch_widen(const WidenArgs& a, hipStream_t s) {
  int64_t most = 1;
  for (int t = 0; t < a.count; ++t) most = std::max(most, a.cap_rows[t] * a.cols[t] / 8);
  hipLaunchKernelGGL(k_widen, dim3(grid_of(most, 4096)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sgd(const SgdArgs& a, float lr, hipStream_t s) {
  int64_t most = 1;
  for (int t = 0; t < a.count; ++t) most = std::max(most, a.n[t]);
  hipLaunchKernelGGL(k_sgd, dim3(grid_of(most, 1024)), dim3(256), 0, s, a, lr);
  return hipGetLastError();
}

}  // namespace gmb
