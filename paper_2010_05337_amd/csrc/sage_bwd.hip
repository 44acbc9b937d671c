// Training step of the GraphSAGE-mean model on gfx950: the loss, the
// backward through the layers of Eq. (1) (DistDGL Section II-A; the
// trainer's iteration of Section III-E), and the SGD update.  fp32.
//
//   k_xent         softmax cross-entropy per target row (one wave per row):
//                  dZ = (softmax(z) - e_y) / B, and the row's loss term
//   k_loss_sum     the mean loss, one workgroup, fixed order
//   k_wgrad        [dW_self; dW_neigh] = [H | M]^T dZ and db = sum of dZ rows:
//                  v_mfma_f32_16x16x4_f32 with the rows of the block as the
//                  reduction dimension, split over workgroups (each writes
//                  its partial sums; no atomics, so the result is the same
//                  on every run)
//   k_wgrad_reduce sums the partials in a fixed order into the gradients
//   k_dgrad        [dH_self | dM] = dZ [W_self; W_neigh]^T: the weights'
//                  transpose for 64 output columns resident in LDS in MFMA
//                  operand order, 64-row tiles, persistent over row tiles
//   k_scatter_mean dH[local[e]] += dM[v] / k_v over the block's edges
//                  (hardware fp32 atomic adds)
//   k_relu_mask    dZ of the layer below = dH where its output is > 0
//   k_sgd          W -= lr dW over every parameter array
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace gmb {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

// ---- loss ---------------------------------------------------------------

// Row v of z [n, C] (row stride ldz): dz row (stride ldz, columns C..ldz-1
// written as 0) and the row's loss term log(sum exp z) - z_y.  A label
// outside [0, C) is a data error: its row gets the softmax as gradient and
// no loss term (every access stays in bounds).
__global__ __launch_bounds__(256) void k_xent(const float* __restrict__ z, const int32_t* __restrict__ y,
                                              int n, int C, int ldz, float* __restrict__ dz,
                                              float* __restrict__ loss_rows) {
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

__global__ __launch_bounds__(256) void k_loss_sum(const float* __restrict__ rows, int n, float* __restrict__ loss) {
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

// Workgroup (p, y, z): rows [p R, (p + 1) R) of the block's destinations,
// output columns [64 y, 64 y + 64), rows i of [dW_self; dW_neigh] in the
// i-blocks 16 (4 z + w + 4 t) .. +15 of wave w, t < 4.  Lane l supplies
// A^T[i][k] = X[k][i] with i = i0 + l%16, k = k0 + l/16 (X = [H | M]) and
// B[k][o] = dZ[k][o0 + l%16]; the MFMA sums over four rows.  Rows at or past
// the end read row r0 and are zeroed; the partial of a workgroup with no
// rows is zero.  Wave 0 of the z = 0 workgroups also sums the dZ rows (db).
constexpr int kWgradIB = 4;   // i-blocks per wave

__global__ __launch_bounds__(256) void k_wgrad(const int32_t* __restrict__ sizes, const float* __restrict__ H,
                                               const float* __restrict__ M, int d_in,
                                               const float* __restrict__ dZ, int ldz, int d_out,
                                               int rows_per_part, int k2p, float* __restrict__ partial,
                                               float* __restrict__ partial_db) {
  const int32_t n = load_size(&sizes[kNDst]);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, c16 = lane & 15;
  const int p = blockIdx.x;
  const int o0 = blockIdx.y * 64;
  const int ib0 = blockIdx.z * 16 + wave;   // i-blocks ib0 + 4 t
  const int K2 = 2 * d_in;
  const int r0 = p * rows_per_part;
  const int r1 = min(r0 + rows_per_part, n);
  floatx4 acc[kWgradIB][4];
#pragma unroll
  for (int t = 0; t < kWgradIB; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[t][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  float dbs[4] = {0.f, 0.f, 0.f, 0.f};
  // per lane: the columns it reads, clamped into the arrays
  int icol[kWgradIB];
  bool iok[kWgradIB], from_m[kWgradIB];
#pragma unroll
  for (int t = 0; t < kWgradIB; ++t) {
    const int i = (ib0 + 4 * t) * 16 + c16;
    iok[t] = i < K2;
    from_m[t] = i >= d_in;
    icol[t] = iok[t] ? (from_m[t] ? i - d_in : i) : 0;
  }
  int ocol[4];
  bool ook[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int o = o0 + j * 16 + c16;
    ook[j] = o < d_out;
    ocol[j] = ook[j] ? o : 0;
  }
  for (int k0 = r0; k0 < r1; k0 += 16) {
    float a[4][kWgradIB], b[4][4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int row = k0 + 4 * s + q;
      const int rc = row < r1 ? row : r0;
      const float* hr = H + static_cast<int64_t>(rc) * d_in;
      const float* mr = M + static_cast<int64_t>(rc) * d_in;
      const float* zr = dZ + static_cast<int64_t>(rc) * ldz;
#pragma unroll
      for (int t = 0; t < kWgradIB; ++t) a[s][t] = (from_m[t] ? mr : hr)[icol[t]];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[s][j] = zr[ocol[j]];
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bool in = k0 + 4 * s + q < r1;
#pragma unroll
      for (int t = 0; t < kWgradIB; ++t) a[s][t] = (in && iok[t]) ? a[s][t] : 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) b[s][j] = (in && ook[j]) ? b[s][j] : 0.f;
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int t = 0; t < kWgradIB; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[t][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s][t], b[s][j], acc[t][j], 0, 0, 0);
    if (wave == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) dbs[j] += b[0][j] + b[1][j] + b[2][j] + b[3][j];
    }
  }
  // partial[p][i][o], i < k2p
#pragma unroll
  for (int t = 0; t < kWgradIB; ++t) {
    const int ib = ib0 + 4 * t;
    if (ib * 16 >= k2p) continue;   // uniform per wave
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = o0 + j * 16 + c16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = ib * 16 + 4 * q + r;
        if (o < d_out) partial[(static_cast<int64_t>(p) * k2p + i) * d_out + o] = acc[t][j][r];
      }
    }
  }
  if (wave == 0 && blockIdx.z == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float v = dbs[j];
      v += __shfl_xor(v, 16, 64);
      v += __shfl_xor(v, 32, 64);
      const int o = o0 + j * 16 + c16;
      if (q == 0 && o < d_out) partial_db[static_cast<int64_t>(p) * d_out + o] = v;
    }
  }
}

__global__ __launch_bounds__(256) void k_wgrad_reduce(const float* __restrict__ partial,
                                                      const float* __restrict__ partial_db, int parts,
                                                      int k2p, int d_in, int d_out, float* __restrict__ d_self,
                                                      float* __restrict__ d_neigh, float* __restrict__ d_bias) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t nw = static_cast<int64_t>(2 * d_in) * d_out;
  if (idx < nw) {
    const int i = static_cast<int>(idx / d_out), o = static_cast<int>(idx % d_out);
    float s = 0.f;
    for (int p = 0; p < parts; ++p) s += partial[(static_cast<int64_t>(p) * k2p + i) * d_out + o];
    if (i < d_in) d_self[static_cast<int64_t>(i) * d_out + o] = s;
    else d_neigh[static_cast<int64_t>(i - d_in) * d_out + o] = s;
  } else if (idx < nw + d_out) {
    const int o = static_cast<int>(idx - nw);
    float s = 0.f;
    for (int p = 0; p < parts; ++p) s += partial_db[static_cast<int64_t>(p) * d_out + o];
    d_bias[o] = s;
  }
}

// ---- input gradient -------------------------------------------------------

// out = dZ [W_self; W_neigh]^T over the block's n_dst rows: K = d_out (in
// NCH chunks of 16), output column nn < d_in goes to dH, d_in <= nn < 2 d_in
// to dM (both with row stride d_in).  The slab holds B[k][nn] = W[nn][k]
// for the workgroup's 64 columns in operand order (as the forward's slab
// kernel); lane l (q = l/16) of a wave reads B[16c + 4q .. +3][nn] with one
// 16-byte LDS read and A = dZ[row][16c + 4q .. +3] (ldz % 4 == 0, zero past
// d_out) with one 16-byte global read.
template <int NCH>
__global__ __launch_bounds__(256) void k_dgrad(const int32_t* __restrict__ sizes, const float* __restrict__ dZ,
                                               int ldz, int d_out, const float* __restrict__ Ws,
                                               const float* __restrict__ Wn, int d_in,
                                               float* __restrict__ dH, float* __restrict__ dM) {
  constexpr int BN = 64;
  __shared__ __attribute__((aligned(16))) float Bp[NCH * 16 * BN];
  const int32_t M = load_size(&sizes[kNDst]);
  const int row_tiles = (M + 63) / 64;
  if (static_cast<int>(blockIdx.x) >= row_tiles) return;
  const int n0 = blockIdx.y * BN;
  const int K2 = 2 * d_in;
  // fill: item (nn, k) with k fastest, so a weight row is read contiguously
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
      float x = w[in ? k : 0];
      asm volatile("" : "+v"(x));
      v[u] = in ? x : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int idx = base + u * 256 + threadIdx.x;
      if (idx >= kItems) continue;
      const int nn = idx / (NCH * 16), k = idx % (NCH * 16);
      Bp[(((k >> 4) * 4 + ((k >> 2) & 3)) * BN + nn) * 4 + (k & 3)] = v[u];
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, r16 = lane & 15;
  for (int rt = blockIdx.x; rt < row_tiles; rt += gridDim.x) {
    const int row = rt * 64 + wave * 16 + r16;
    const float* zr = dZ + static_cast<int64_t>(row < M ? row : M - 1) * ldz;
    float4 a[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int k = 16 * c + 4 * q;
      float4 x = *reinterpret_cast<const float4*>(zr + (k < ldz ? k : 0));
      asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
      a[c] = k < ldz ? x : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    floatx4 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      float4 b[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = *reinterpret_cast<const float4*>(&Bp[(((c * 4 + q) * BN) + j * 16 + r16) * 4]);
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
  }
}

// ---- mean backward, ReLU, zero fill, SGD ----------------------------------

// rows [n_dst, n_src) of dH (row stride d) := 0
__global__ __launch_bounds__(256) void k_zero_tail(const int32_t* __restrict__ sizes, float* __restrict__ dH, int d) {
  const int64_t n_dst = load_size(&sizes[kNDst]), n_src = load_size(&sizes[kNSrc]);
  const int64_t total = (n_src - n_dst) * d;
  float* base = dH + n_dst * d;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    base[i] = 0.f;
}

// G lanes per destination row v; lane c covers columns 4c .. 4c+3 (d % 4 == 0)
template <int G>
__global__ __launch_bounds__(256) void k_scatter_mean(const int32_t* __restrict__ sizes,
                                                      const int32_t* __restrict__ indptr,
                                                      const int32_t* __restrict__ local,
                                                      const float* __restrict__ dM, int d,
                                                      float* __restrict__ dH) {
  const int32_t n_dst = load_size(&sizes[kNDst]);
  const int32_t n_src = load_size(&sizes[kNSrc]);
  const int64_t v = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / G;
  const int lane = threadIdx.x & (G - 1);
  if (v >= n_dst) return;
  const int32_t beg = indptr[v], end = indptr[v + 1];
  const int32_t k = end - beg;
  if (k <= 0) return;
  const float inv = 1.f / static_cast<float>(k);
  const int chunks = d / 4;
  for (int c = lane; c < chunks; c += G) {
    float4 g = *reinterpret_cast<const float4*>(dM + v * d + 4 * c);
    g.x *= inv; g.y *= inv; g.z *= inv; g.w *= inv;
    for (int32_t e = beg; e < end; ++e) {
      const int32_t u = local[e];
      if (u < 0 || u >= n_src) continue;   // only after a data error
      float* h = dH + static_cast<int64_t>(u) * d + 4 * c;
      unsafeAtomicAdd(h, g.x);
      unsafeAtomicAdd(h + 1, g.y);
      unsafeAtomicAdd(h + 2, g.z);
      unsafeAtomicAdd(h + 3, g.w);
    }
  }
}

// dH[i] := dH[i] if out[i] > 0 else 0, for the n_dst rows of the block that
// produced `out` (row stride d)
__global__ __launch_bounds__(256) void k_relu_mask(const int32_t* __restrict__ sizes, const float* __restrict__ out,
                                                   int d, float* __restrict__ dH) {
  const int64_t n = static_cast<int64_t>(load_size(&sizes[kNDst])) * d;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    dH[i] = out[i] > 0.f ? dH[i] : 0.f;
}

__global__ __launch_bounds__(256) void k_sgd(SgdArgs a, float lr) {
  for (int t = 0; t < a.count; ++t) {
    float* w = a.w[t];
    const float* g = a.g[t];
    const int64_t n = a.n[t];
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
      w[i] -= lr * g[i];
  }
}

inline unsigned grid_of(int64_t threads, int64_t cap = 65535) {
  int64_t g = (threads + 255) / 256;
  if (g > cap) g = cap;
  return static_cast<unsigned>(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_xent(const float* logits, const int32_t* labels, int n, int C, int ldz, float* dz,
                       float* loss_rows, float* loss, hipStream_t s) {
  if (n > 0)
    hipLaunchKernelGGL(k_xent, dim3((n + 3) / 4), dim3(256), 0, s, logits, labels, n, C, ldz, dz, loss_rows);
  if (loss) hipLaunchKernelGGL(k_loss_sum, dim3(1), dim3(256), 0, s, loss_rows, n, loss);
  return hipGetLastError();
}

int wgrad_parts(int64_t cap_rows, int d_in, int d_out) {
  const int col_tiles = (d_out + 63) / 64;
  const int zg = (2 * d_in + 255) / 256;
  int parts = static_cast<int>((1024 + col_tiles * zg - 1) / (col_tiles * zg));
  const int64_t by_rows = (cap_rows + 15) / 16;
  if (parts > by_rows) parts = static_cast<int>(by_rows);
  return parts < 1 ? 1 : parts;
}

int wgrad_rows_per_part(int64_t cap_rows, int parts) {
  int64_t r = (cap_rows + parts - 1) / parts;
  r = (r + 15) / 16 * 16;
  return static_cast<int>(r < 16 ? 16 : r);
}

int wgrad_k2p(int d_in) { return (2 * d_in + 15) / 16 * 16; }

hipError_t launch_wgrad(const int32_t* sizes, const float* H, const float* M, int d_in, const float* dZ, int ldz,
                        int d_out, int64_t cap_rows, float* partial, float* partial_db, float* d_self,
                        float* d_neigh, float* d_bias, hipStream_t s) {
  const int parts = wgrad_parts(cap_rows, d_in, d_out);
  const int rpp = wgrad_rows_per_part(cap_rows, parts);
  const int k2p = wgrad_k2p(d_in);
  const dim3 grid(parts, (d_out + 63) / 64, (2 * d_in + 255) / 256);
  hipLaunchKernelGGL(k_wgrad, grid, dim3(256), 0, s, sizes, H, M, d_in, dZ, ldz, d_out, rpp, k2p, partial,
                     partial_db);
  const int64_t outs = static_cast<int64_t>(2 * d_in) * d_out + d_out;
  hipLaunchKernelGGL(k_wgrad_reduce, dim3(grid_of(outs, 1 << 30)), dim3(256), 0, s, partial, partial_db, parts,
                     k2p, d_in, d_out, d_self, d_neigh, d_bias);
  return hipGetLastError();
}

hipError_t launch_dgrad(const int32_t* sizes, const float* dZ, int ldz, int d_out, const float* ws,
                        const float* wn, int d_in, float* dH, float* dM, int64_t cap_rows, hipStream_t s) {
  const int nch = (d_out + 15) / 16;
  const int col_tiles = (2 * d_in + 63) / 64;
  int64_t rows = (cap_rows + 63) / 64;
  const int64_t want = (512 + col_tiles - 1) / col_tiles;
  if (rows > want) rows = want;
  if (rows < 1) rows = 1;
  const dim3 grid(static_cast<unsigned>(rows), col_tiles);
#define GMB_DGRAD(C) hipLaunchKernelGGL(k_dgrad<C>, grid, dim3(256), 0, s, sizes, dZ, ldz, d_out, ws, wn, d_in, dH, dM)
  if (nch <= 4) GMB_DGRAD(4);
  else if (nch <= 8) GMB_DGRAD(8);
  else if (nch <= 16) GMB_DGRAD(16);
  else if (nch <= 32) GMB_DGRAD(32);
  else if (nch <= 40) GMB_DGRAD(40);
  else return hipErrorInvalidValue;
#undef GMB_DGRAD
  return hipGetLastError();
}

hipError_t launch_mean_backward(const int32_t* sizes, const int32_t* indptr, const int32_t* local, const float* dM,
                                int d, float* dH, int64_t cap_dst, int64_t cap_src, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_tail, dim3(grid_of((cap_src - 0) * d / 4 + 1, 8192)), dim3(256), 0, s, sizes, dH, d);
  const int chunks = d / 4;
  int G = 64;
  if (chunks <= 8) G = 8;
  else if (chunks <= 16) G = 16;
  else if (chunks <= 32) G = 32;
  const dim3 grid(grid_of(std::max<int64_t>(cap_dst, 1) * G, 1 << 30));
  switch (G) {
    case 8: hipLaunchKernelGGL(k_scatter_mean<8>, grid, dim3(256), 0, s, sizes, indptr, local, dM, d, dH); break;
    case 16: hipLaunchKernelGGL(k_scatter_mean<16>, grid, dim3(256), 0, s, sizes, indptr, local, dM, d, dH); break;
    case 32: hipLaunchKernelGGL(k_scatter_mean<32>, grid, dim3(256), 0, s, sizes, indptr, local, dM, d, dH); break;
    default: hipLaunchKernelGGL(k_scatter_mean<64>, grid, dim3(256), 0, s, sizes, indptr, local, dM, d, dH); break;
  }
  return hipGetLastError();
}

hipError_t launch_relu_mask(const int32_t* sizes, const float* out, int d, float* dH, int64_t cap_rows,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_relu_mask, dim3(grid_of(std::max<int64_t>(cap_rows, 1) * d / 4 + 1, 8192)), dim3(256), 0,
                     s, sizes, out, d, dH);
  return hipGetLastError();
}

hipError_t launch_sgd(const SgdArgs& a, float lr, hipStream_t s) {
  int64_t most = 1;
  for (int t = 0; t < a.count; ++t) most = std::max(most, a.n[t]);
  hipLaunchKernelGGL(k_sgd, dim3(grid_of(most, 1024)), dim3(256), 0, s, a, lr);
  return hipGetLastError();
}

}  // namespace gmb
