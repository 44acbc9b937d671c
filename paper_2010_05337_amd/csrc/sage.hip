// GraphSAGE-mean layer on gfx950 (DistDGL Section II-A, Eq. (1), with the
// message f = h_u, the aggregator = mean over the sampled in-neighbours and
// the update g = act(h_v W_self + m_v W_neigh + b); Section IV model).
//
//   k_mean    m_v = (1/k_v) sum_e H[ids[e]] (ids: the block's local ids into the
//             layer input, or for a layer 0 that reads the feature table,
//             the edges' global ids), fp32 accumulation; a group of
//             G lanes per destination row, 16-byte chunks of the feature
//             row per lane; the group reads the row's local ids in one
//             access and then up to U neighbour rows in one batch.
//   k_linear  out = act([H_dst | M] [W_self; W_neigh] + b): one GEMM with
//             K = 2 d_in on the matrix cores, the weights resident in LDS
//             (slab kernels): bf16 on v_mfma_f32_16x16x32_bf16 with fp32
//             accumulation; fp32 on the same instruction through an exact
//             three-way bf16 cut of both operands (k_linear_f32_parts), or
//             on v_mfma_f32_16x16x4_f32 where that is faster or the shape
//             does not fit (k_linear_f32_slab, k_linear_f32).
#include "common.hpp"
#include "kernels.hpp"
#include "parts.hpp"

namespace gmb {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// Makes a loaded value opaque to the optimiser, so that a later select on
// it cannot turn the load itself into a conditional (branched) load.
__device__ __forceinline__ void opaque(float& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void opaque(float4& x) {
  asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
}

// ---- mean aggregation -------------------------------------------------

// VEC elements per lane access, from fp32 or bf16 (uint16_t bits) rows.
template <int VEC>
__device__ __forceinline__ void load_chunk(const float* p, float (&v)[VEC]) {
  if constexpr (VEC == 4) {
    const float4 x = *reinterpret_cast<const float4*>(p);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) v[i] = p[i];
  }
}

template <int VEC>
__device__ __forceinline__ void load_chunk(const uint16_t* p, float (&v)[VEC]) {
  if constexpr (VEC == 8) {
    const uint4 x = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) v[i] = bf16_to_f32(p[i]);
  }
}

template <int VEC>
__device__ __forceinline__ void store_chunk(float* p, const float (&v)[VEC]) {
  if constexpr (VEC == 4) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) p[i] = v[i];
  }
}

template <int VEC>
__device__ __forceinline__ void store_chunk(uint16_t* p, const float (&v)[VEC]) {
  if constexpr (VEC == 8) {
    uint4 x;
    x.x = f32_to_bf16(v[0]) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
    x.y = f32_to_bf16(v[2]) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
    x.z = f32_to_bf16(v[4]) | (static_cast<uint32_t>(f32_to_bf16(v[5])) << 16);
    x.w = f32_to_bf16(v[6]) | (static_cast<uint32_t>(f32_to_bf16(v[7])) << 16);
    *reinterpret_cast<uint4*>(p) = x;
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) p[i] = f32_to_bf16(v[i]);
  }
}

template <typename T, int VEC, int G, int U>
__global__ __launch_bounds__(256) void k_mean(const int32_t* sizes, const int32_t* __restrict__ indptr,
                                              const int32_t* __restrict__ local,
                                              const T* __restrict__ H, int d, T* __restrict__ M,
                                              int64_t cap_rows, int64_t max_id) {
  const int64_t row = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) / G;
  const int lane = threadIdx.x & (G - 1);
  // independent first reads, the row offsets first (the compiler keeps
  // later reads behind the size word's atomic read); a row past the
  // capacity reads the last one
  const int64_t rc = row < cap_rows ? row : cap_rows - 1;
  const int32_t beg = indptr[rc], end = indptr[rc + 1];
  const int32_t n_dst = load_size(&sizes[kNDst]);
  if (row >= n_dst) return;   // the whole group leaves together
  const int32_t k = end - beg;
  const int chunks = d / VEC;
  const int passes = (chunks + G - 1) / G;
  for (int cc = 0; cc < passes; ++cc) {
    const int c = cc * G + lane;
    const int cl = c < chunks ? c : chunks - 1;
    float acc[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) acc[i] = 0.f;
    // the group reads G row ids at once (lane i: edge base + i), then
    // its rows U at a time (U >= the fan-out where possible, so one batch
    // per row) with every read unconditional; past the row's end a slot
    // re-reads the first id and is dropped.  An id outside [0, max_id)
    // only exists after a data error; it is read as row 0.
    for (int32_t base = 0; base < k; base += G) {
      const int32_t n_here = k - base < G ? k - base : G;
      int32_t mine = local[beg + base + (lane < n_here ? lane : 0)];
      mine = (mine < 0 || mine >= max_id) ? 0 : mine;
      for (int u0 = 0; u0 < n_here; u0 += U) {
        int32_t id[U];
#pragma unroll
        for (int u = 0; u < U; ++u) id[u] = __shfl(mine, u0 + u < n_here ? u0 + u : 0, G);
        float x[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u)
          load_chunk<VEC>(H + static_cast<int64_t>(id[u]) * d + cl * VEC, x[u]);
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const bool in = u0 + u < n_here;
#pragma unroll
          for (int i = 0; i < VEC; ++i) {
            float xv = x[u][i];
            opaque(xv);
            acc[i] += in ? xv : 0.f;
          }
        }
      }
    }
    if (k > 0) {
      const float kf = static_cast<float>(k);
#pragma unroll
      for (int i = 0; i < VEC; ++i) acc[i] = acc[i] / kf;
    }
    if (c < chunks) store_chunk<VEC>(M + row * d + c * VEC, acc);
  }
}

template <typename T, int VEC>
hipError_t mean_dispatch(const int32_t* sizes, const int32_t* indptr, const int32_t* local, const void* h,
                         int d, void* m, int64_t cap_dst, int fanout, int64_t max_id, hipStream_t s) {
  const int chunks = d / VEC;
  int G = 64;
  if (chunks <= 4) G = 4;
  else if (chunks <= 8) G = 8;
  else if (chunks <= 16) G = 16;
  else if (chunks <= 32) G = 32;
  // rows in flight per lane: the fan-out rounded up to 8, 16 or 32 (16 at
  // most for chunks wider than four values)
  const int U = fanout <= 8 ? 8 : (fanout <= 16 || VEC > 4 ? 16 : 32);
  int64_t blocks = (cap_dst * G + 255) / 256;
  if (blocks < 1) blocks = 1;
  const dim3 grid(static_cast<unsigned>(blocks)), block(256);
  const T* H = static_cast<const T*>(h);
  T* M = static_cast<T*>(m);
  const int64_t cap = cap_dst < 1 ? 1 : cap_dst;   // indptr holds cap_dst + 1 >= 1 entries
#define GMB_MEAN(GG, UU) \
  hipLaunchKernelGGL((k_mean<T, VEC, GG, UU>), grid, block, 0, s, sizes, indptr, local, H, d, M, cap, max_id)
#define GMB_MEAN_G(UU)                \
  switch (G) {                        \
    case 4: GMB_MEAN(4, UU); break;   \
    case 8: GMB_MEAN(8, UU); break;   \
    case 16: GMB_MEAN(16, UU); break; \
    case 32: GMB_MEAN(32, UU); break; \
    default: GMB_MEAN(64, UU); break; \
  }
  if (U == 8) {
    GMB_MEAN_G(8)
  } else if (U == 16) {
    GMB_MEAN_G(16)
  } else {
    GMB_MEAN_G(32)
  }
#undef GMB_MEAN_G
#undef GMB_MEAN
  return hipGetLastError();
}

// ---- linear layer on the matrix cores ---------------------------------

constexpr int kBM = 64, kBN = 64;

// fp32: v_mfma_f32_16x16x4_f32.  Lane l supplies A[l%16][l/16] and
// B[l/16][l%16] of a 16x4 by 4x16 step and holds C[4*(l/16)+r][l%16],
// r = 0..3.  Four waves tile the 64x64 output as 2x2 blocks of 32x32.
constexpr int kBK32 = 32;
constexpr int kAStride32 = kBK32 + 1;
constexpr int kBStride32 = kBN + 16;

__global__ __launch_bounds__(256) void k_linear_f32(const int32_t* sizes, const float* __restrict__ Hs,
                                                    const float* __restrict__ Ag,
                                                    const float* __restrict__ Ws,
                                                    const float* __restrict__ Wn,
                                                    const float* __restrict__ bias, int K, int N,
                                                    int relu, float* __restrict__ out) {
  __shared__ float As[kBM * kAStride32];
  __shared__ float Bs[kBK32 * kBStride32];
  const int32_t M = load_size(&sizes[kNDst]);
  const int m0 = blockIdx.x * kBM, n0 = blockIdx.y * kBN;
  if (m0 >= M) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
  const int K2 = 2 * K;
  floatx4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < K2; k0 += kBK32) {
#pragma unroll
    for (int q = 0; q < (kBM * kBK32) / 256; ++q) {
      const int idx = tid + 256 * q;
      const int r = idx / kBK32, c = idx % kBK32;
      const int gm = m0 + r, gk = k0 + c;
      float v = 0.f;
      if (gm < M && gk < K2) v = gk < K ? Hs[static_cast<int64_t>(gm) * K + gk] : Ag[static_cast<int64_t>(gm) * K + (gk - K)];
      As[r * kAStride32 + c] = v;
    }
#pragma unroll
    for (int q = 0; q < (kBK32 * kBN) / 256; ++q) {
      const int idx = tid + 256 * q;
      const int r = idx / kBN, c = idx % kBN;
      const int gk = k0 + r, gn = n0 + c;
      float v = 0.f;
      if (gk < K2 && gn < N) v = gk < K ? Ws[static_cast<int64_t>(gk) * N + gn] : Wn[static_cast<int64_t>(gk - K) * N + gn];
      Bs[r * kBStride32 + c] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kBK32; kk += 4) {
      float a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = As[(wm + i * 16 + (lane & 15)) * kAStride32 + kk + (lane >> 4)];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = Bs[(kk + (lane >> 4)) * kBStride32 + wn + j * 16 + (lane & 15)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn + j * 16 + (lane & 15);
      if (col >= N) continue;
      const float bv = bias[col];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + i * 16 + 4 * (lane >> 4) + r;
        if (row < M) {
          float z = acc[i][j][r] + bv;
          if (relu) z = z > 0.f ? z : 0.f;
          out[static_cast<int64_t>(row) * N + col] = z;
        }
      }
    }
}

// bf16: v_mfma_f32_16x16x32_bf16.  Lane l supplies A[l%16][8(l/16) .. +7]
// and B[8(l/16) .. +7][l%16] and holds C as in the fp32 case.  B is kept
// transposed in LDS so that a lane's eight k values are contiguous.
constexpr int kBK16 = 64;
constexpr int kAStride16 = kBK16 + 8;   // in bf16 elements; rows stay 16-byte aligned
constexpr int kBStride16 = kBK16 + 8;

__global__ __launch_bounds__(256) void k_linear_bf16(const int32_t* sizes, const uint16_t* __restrict__ Hs,
                                                     const uint16_t* __restrict__ Ag,
                                                     const uint16_t* __restrict__ Ws,
                                                     const uint16_t* __restrict__ Wn,
                                                     const float* __restrict__ bias, int K, int N,
                                                     int relu, int out_f32, void* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) uint16_t As[kBM * kAStride16];
  __shared__ __attribute__((aligned(16))) uint16_t Bt[kBN * kBStride16];
  const int32_t M = load_size(&sizes[kNDst]);
  const int m0 = blockIdx.x * kBM, n0 = blockIdx.y * kBN;
  if (m0 >= M) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
  const int K2 = 2 * K;
  floatx4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < K2; k0 += kBK16) {
#pragma unroll
    for (int q = 0; q < (kBM * kBK16) / 256; ++q) {
      const int idx = tid + 256 * q;
      const int r = idx / kBK16, c = idx % kBK16;
      const int gm = m0 + r, gk = k0 + c;
      uint16_t v = 0;
      if (gm < M && gk < K2) v = gk < K ? Hs[static_cast<int64_t>(gm) * K + gk] : Ag[static_cast<int64_t>(gm) * K + (gk - K)];
      As[r * kAStride16 + c] = v;
    }
#pragma unroll
    for (int q = 0; q < (kBK16 * kBN) / 256; ++q) {
      const int idx = tid + 256 * q;
      const int r = idx / kBN, c = idx % kBN;   // r: k within the tile, c: output column
      const int gk = k0 + r, gn = n0 + c;
      uint16_t v = 0;
      if (gk < K2 && gn < N) v = gk < K ? Ws[static_cast<int64_t>(gk) * N + gn] : Wn[static_cast<int64_t>(gk - K) * N + gn];
      Bt[c * kBStride16 + r] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kBK16; kk += 32) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(&As[(wm + i * 16 + (lane & 15)) * kAStride16 + kk + 8 * (lane >> 4)]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(&Bt[(wn + j * 16 + (lane & 15)) * kBStride16 + kk + 8 * (lane >> 4)]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn + j * 16 + (lane & 15);
      if (col >= N) continue;
      const float bv = bias[col];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + i * 16 + 4 * (lane >> 4) + r;
        if (row < M) {
          float z = acc[i][j][r] + bv;
          if (relu) z = z > 0.f ? z : 0.f;
          if (out_f32)
            static_cast<float*>(out)[static_cast<int64_t>(row) * N + col] = z;
          else
            static_cast<uint16_t*>(out)[static_cast<int64_t>(row) * N + col] = f32_to_bf16(z);
        }
      }
    }
}

// fp32 with the weight slab resident in LDS.  A workgroup owns 64 output
// columns and keeps those columns of [W_self; W_neigh] (all 2 d_in rows,
// zero-padded to NCH chunks of 16) in LDS for its whole life, walking over
// row tiles of 64 rows (persistent), so the weights are read once per
// workgroup.  The slab is stored in MFMA operand order: for chunk c of k,
// lane l (q = l/16) of a wave reads W[16c + 4q + s][col], s = 0..3, with one
// 16-byte LDS read and feeds the four values to four consecutive
// v_mfma_f32_16x16x4_f32 steps; its A operand is the matching float4
// A[row][16c + 4q .. +3], one 16-byte global read.  The MFMA sums over its
// four k slots, so any assignment of k to slots that A and B share gives
// the same product.  Each wave computes 16 rows x 64 columns; it issues
// all NCH A reads of its row tile before the first MFMA (at this LDS-bound
// occupancy registers are plentiful), then runs the 16 NCH MFMAs.
//
// Loads are unconditional from clamped addresses: rows past M read row
// M-1 and are never stored, k past 2 d_in reads the row's first elements
// and meets zero rows of the slab.  (A load under a divergent branch makes
// the compiler drain every outstanding load before the next one.)
__device__ __forceinline__ const float* pick(bool c, const float* a, const float* b) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return reinterpret_cast<const float*>(c ? x : y);
}

// NCH chunks of 16 k, J column subtiles of 16 (BN = 16 J columns per
// workgroup), SPLIT = 1: each wave owns 16 rows of a 64-row tile and all
// chunks; SPLIT = 4: the four waves share one 16-row tile, wave w takes the
// chunks c = w (mod 4), and the partial sums meet in LDS (for layers with
// few rows, where one wave per 16 rows would leave most SIMDs idle).
// LDS bytes of one slab workgroup and the workgroups per CU that LDS
// allows (at most 3: one to three waves per SIMD).
constexpr int slab_lds_bytes(int nch, int j, int split) {
  return nch * 16 * 16 * j * 4 + (split > 1 ? 4 * j * 64 * 16 : 16);
}
constexpr int slab_occupancy(int nch, int j, int split) {
  const int by_lds = (160 * 1024) / slab_lds_bytes(nch, j, split);
  return by_lds < 1 ? 1 : (by_lds > 3 ? 3 : by_lds);
}

template <int NCH, int J, int SPLIT>
__global__ __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(slab_occupancy(NCH, J, SPLIT), slab_occupancy(NCH, J, SPLIT))))
void k_linear_f32_slab(const int32_t* sizes,
                                                         const float* __restrict__ Hs,
                                                         const float* __restrict__ Ag,
                                                         const float* __restrict__ Ws,
                                                         const float* __restrict__ Wn,
                                                         const float* __restrict__ bias, int K,
                                                         int N, int relu, int vec4,
                                                         float* __restrict__ out) {
  constexpr int BN = 16 * J;
  constexpr int ROWS = SPLIT > 1 ? 16 : 64;
  constexpr int MYCH = SPLIT > 1 ? (NCH + 3) / 4 : NCH;
  __shared__ __attribute__((aligned(16))) float Bp[NCH * 16 * BN];
  __shared__ __attribute__((aligned(16))) float Red[SPLIT > 1 ? 4 * J * 64 * 4 : 4];
  const int32_t M = load_size(&sizes[kNDst]);
  const int row_tiles = (M + ROWS - 1) / ROWS;
  if (static_cast<int>(blockIdx.x) >= row_tiles) return;
  const int n0 = blockIdx.y * BN;
  const int K2 = 2 * K;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, r16 = lane & 15;
  // A fragment i of row tile rt (a tile past the end reads row M-1: every
  // load is unconditional)
  auto tile_rows = [&](int rt, const float*& hrow, const float*& grow) {
    const int row = SPLIT > 1 ? rt * 16 + r16 : rt * 64 + wave * 16 + r16;
    const int64_t arow = row < M ? row : M - 1;
    hrow = Hs + arow * K;
    grow = Ag + arow * K;
  };
  auto load_frag = [&](const float* hrow, const float* grow, int i) -> float4 {
    const int c = SPLIT > 1 ? wave + 4 * i : i;
    const int k = c * 16 + 4 * q;
    const int kk = k >= K2 ? 0 : (k < K ? k : k - K);
    return *reinterpret_cast<const float4*>(pick((k >= K) & (k < K2), grow, hrow) + kk);
  };
  auto slab_at = [&](int k, int n) -> float& {
    return Bp[((((k >> 4) * 4 + ((k >> 2) & 3)) * BN) + n) * 4 + (k & 3)];
  };
  // Slab fill: a batch of independent loads per thread, made opaque only
  // after the whole batch is issued, then the zero-padding select.
  if (vec4) {   // N % 4 == 0 and 16-byte aligned weights: float4 along n
    constexpr int per_row = BN / 4;
    constexpr int total = NCH * 16 * per_row;
    for (int base = 0; base < total; base += 256 * 8) {
      float4 v[8];
      bool in[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int idx = base + u * 256 + threadIdx.x;
        const int k = idx / per_row, n = (idx % per_row) * 4;
        in[u] = (idx < total) & (k < K2) & (n0 + n < N);
        const int kr = in[u] ? (k < K ? k : k - K) : 0;
        const float* src = pick(in[u] & (k >= K), Wn, Ws) + static_cast<int64_t>(kr) * N + (in[u] ? n0 + n : 0);
        v[u] = *reinterpret_cast<const float4*>(src);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        opaque(v[u]);
        const int idx = base + u * 256 + threadIdx.x;
        if (idx < total) {
          const int k = idx / per_row, n = (idx % per_row) * 4;
          const float4 x = in[u] ? v[u] : make_float4(0.f, 0.f, 0.f, 0.f);
          slab_at(k, n) = x.x;
          slab_at(k, n + 1) = x.y;
          slab_at(k, n + 2) = x.z;
          slab_at(k, n + 3) = x.w;
        }
      }
    }
  } else {
    constexpr int total = NCH * 16 * BN;
    for (int base = 0; base < total; base += 256 * 32) {
      float v[32];
      bool in[32];
#pragma unroll
      for (int u = 0; u < 32; ++u) {
        const int idx = base + u * 256 + threadIdx.x;
        const int k = idx / BN, n = idx % BN;
        in[u] = (idx < total) & (k < K2) & (n0 + n < N);
        const int kr = in[u] ? (k < K ? k : k - K) : 0;
        const float* src = pick(in[u] & (k >= K), Wn, Ws) + static_cast<int64_t>(kr) * N + (in[u] ? n0 + n : 0);
        v[u] = *src;
      }
#pragma unroll
      for (int u = 0; u < 32; ++u) {
        opaque(v[u]);
        const int idx = base + u * 256 + threadIdx.x;
        if (idx < total) slab_at(idx / BN, idx % BN) = in[u] ? v[u] : 0.f;
      }
    }
  }
  __syncthreads();
  // the first tile's A fragments (after the fill: both at once would not
  // fit the registers of three waves per SIMD)
  float4 a[MYCH];
  {
    const float *hrow, *grow;
    tile_rows(blockIdx.x, hrow, grow);
#pragma unroll
    for (int i = 0; i < MYCH; ++i) a[i] = load_frag(hrow, grow, i);
  }
  // bias of this thread's output columns (fixed over the row tiles); with
  // split K, thread t stores column block t / 64 (t < 64 J)
  float bv[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int col = n0 + (SPLIT > 1 ? ((threadIdx.x >> 6) % J) : j) * 16 + r16;
    bv[j] = bias[col < N ? col : N - 1];
  }
  // software pipeline over the workgroup's row tiles: as soon as chunk i's
  // MFMAs are issued, a[i] is reloaded with the next tile's fragment i, so
  // the next tile's reads are in flight during the rest of this tile
  // without a second set of registers
  for (int rt = blockIdx.x; rt < row_tiles; rt += gridDim.x) {
    const float *hnext, *gnext;
    tile_rows(rt + gridDim.x, hnext, gnext);
    floatx4 acc[J];
#pragma unroll
    for (int j = 0; j < J; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    // B fragments double-buffered: chunk i + 1's LDS reads are issued
    // before chunk i's MFMAs, so a wave never waits on LDS between chunks
    // (the waves of a SIMD run in step, so the other wave cannot cover it)
    auto load_b = [&](int i, float4 (&b)[J]) {
      const int c = SPLIT > 1 ? wave + 4 * i : i;
      const int cc = c < NCH ? c : NCH - 1;
#pragma unroll
      for (int j = 0; j < J; ++j)
        b[j] = *reinterpret_cast<const float4*>(&Bp[(((cc * 4 + q) * BN) + j * 16 + r16) * 4]);
    };
    float4 b0[J], b1[J];
    load_b(0, b0);
#pragma unroll
    for (int i = 0; i < MYCH; ++i) {
      const int c = SPLIT > 1 ? wave + 4 * i : i;
      float4 (&bc)[J] = (i & 1) ? b1 : b0;
      float4 (&bn)[J] = (i & 1) ? b0 : b1;
      if (i + 1 < MYCH) load_b(i + 1, bn);
      __builtin_amdgcn_sched_barrier(0);
      if (c < NCH) {   // uniform: depends on the wave index only
#pragma unroll
        for (int j = 0; j < J; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].x, bc[j].x, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < J; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].y, bc[j].y, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < J; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].z, bc[j].z, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < J; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].w, bc[j].w, acc[j], 0, 0, 0);
      }
      a[i] = load_frag(hnext, gnext, i);
    }
    if constexpr (SPLIT > 1) {
      // partials of the four waves -> LDS; thread t then owns output entry
      // (subtile j, lane l) = t and sums the four partials
#pragma unroll
      for (int j = 0; j < J; ++j)
        *reinterpret_cast<floatx4*>(&Red[((wave * J + j) * 64 + lane) * 4]) = acc[j];
      __syncthreads();
      if (threadIdx.x < J * 64) {
        const int j = threadIdx.x >> 6, l = threadIdx.x & 63;
        floatx4 sum = *reinterpret_cast<const floatx4*>(&Red[((0 * J + j) * 64 + l) * 4]);
#pragma unroll
        for (int w = 1; w < 4; ++w) sum += *reinterpret_cast<const floatx4*>(&Red[((w * J + j) * 64 + l) * 4]);
        const int col = n0 + j * 16 + (l & 15);
        const int row0 = rt * 16 + 4 * (l >> 4);
        float* o = out + static_cast<int64_t>(row0) * N + col;
        const bool full = row0 + 4 <= M && col < N;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float z = sum[r] + bv[0];
          if (relu) z = z > 0.f ? z : 0.f;
          if (full || (row0 + r < M && col < N)) o[static_cast<int64_t>(r) * N] = z;
        }
      }
      __syncthreads();
    } else {
      // one row pointer per accumulator row; a tile inside the matrix
      // stores without per-element checks (column offsets fold into the
      // store's immediate offset)
      const int row0 = rt * 64 + wave * 16 + 4 * q;
      float* o0 = out + static_cast<int64_t>(row0) * N + n0 + r16;
      const bool full = row0 + 4 <= M && n0 + BN <= N;
      if (full) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float* o = o0 + static_cast<int64_t>(r) * N;
#pragma unroll
          for (int j = 0; j < J; ++j) {
            float z = acc[j][r] + bv[j];
            if (relu) z = z > 0.f ? z : 0.f;
            o[j * 16] = z;
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < J; ++j) {
          const int col = n0 + j * 16 + r16;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float z = acc[j][r] + bv[j];
            if (relu) z = z > 0.f ? z : 0.f;
            if (row0 + r < M && col < N) o0[static_cast<int64_t>(r) * N + j * 16] = z;
          }
        }
      }
    }
  }
}

// Workgroups per CU of the persistent slab grids.  One: a second
// workgroup per CU barely shortens a kernel run alone (each workgroup
// fills its own slab from L2, and that part does not shrink), while the
// smaller grid leaves CUs, LDS and L2 bandwidth to the kernels other
// streams run beside it (four-stream inference: +2% seeds/s with fp32
// features, +1.5% with bf16).
#ifndef GMB_SLAB_BLOCKS_WIDE
#define GMB_SLAB_BLOCKS_WIDE 1
#endif
#ifndef GMB_SLAB_BLOCKS_SPLIT
#define GMB_SLAB_BLOCKS_SPLIT 1
#endif
#ifndef GMB_SLAB_BLOCKS_BF16
#define GMB_SLAB_BLOCKS_BF16 1
#endif
constexpr int kSlabBlocksWide = GMB_SLAB_BLOCKS_WIDE;    // fp32, one wave per 16 rows
constexpr int kSlabBlocksSplit = GMB_SLAB_BLOCKS_SPLIT;  // fp32, split-K tiles
constexpr int kSlabBlocksBf16 = GMB_SLAB_BLOCKS_BF16;    // bf16

template <int NCH, int J, int SPLIT>
void launch_slab(const int32_t* sizes, const float* hs, const float* ag, const float* ws, const float* wn,
                 const float* bias, int K, int N, int relu, float* out, int64_t cap_rows, hipStream_t s) {
  // The persistent grid holds kSlabBlocks{Wide,Split} workgroups per CU
  // (capped by LDS): every workgroup reloads the slab, so a smaller grid
  // reads the weights fewer times and leaves room for kernels of other
  // streams.
  constexpr int BN = 16 * J;
  constexpr int ROWS = SPLIT > 1 ? 16 : 64;
  constexpr int lds = NCH * 16 * BN * 4 + (SPLIT > 1 ? 4 * J * 64 * 16 : 0);
  constexpr int per_cu = (160 * 1024) / lds;
  const int col_tiles = (N + BN - 1) / BN;
  int64_t rows = (cap_rows + ROWS - 1) / ROWS;
  const int occ = SPLIT > 1 ? kSlabBlocksSplit : kSlabBlocksWide;
  const int blocks_per_cu = occ < per_cu ? occ : (per_cu < 1 ? 1 : per_cu);
  int64_t want = (256 * blocks_per_cu + col_tiles - 1) / col_tiles;
  if (rows > want) rows = want;
  if (rows < 1) rows = 1;
  const uintptr_t walign = reinterpret_cast<uintptr_t>(ws) | reinterpret_cast<uintptr_t>(wn);
  const int vec4 = (N % 4 == 0 && walign % 16 == 0) ? 1 : 0;
  hipLaunchKernelGGL((k_linear_f32_slab<NCH, J, SPLIT>), dim3(static_cast<unsigned>(rows), col_tiles),
                     dim3(256), 0, s, sizes, hs, ag, ws, wn, bias, K, N, relu, vec4, out);
}

// Picks the tiling: layers with enough 64-row tiles to fill the chip twice
// keep one wave per 16 rows and 64 columns; smaller layers split K over
// the waves and use 32-column tiles, which halves the slab.
template <int NCH>
void launch_slab_for(const int32_t* sizes, const float* hs, const float* ag, const float* ws,
                     const float* wn, const float* bias, int K, int N, int relu, float* out,
                     int64_t cap_rows, hipStream_t s) {
  const int64_t big_tiles = ((cap_rows + 63) / 64) * ((N + 63) / 64);
  if (big_tiles >= 2 * 256)
    launch_slab<NCH, 4, 1>(sizes, hs, ag, ws, wn, bias, K, N, relu, out, cap_rows, s);
  else
    launch_slab<NCH, 2, 4>(sizes, hs, ag, ws, wn, bias, K, N, relu, out, cap_rows, s);
}

template <int NCH, int J, int R, int SPLIT, int WAVES>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(WAVES / 4, WAVES / 4)))
void k_linear_f32_parts(const int32_t* sizes, parts::LinearOp op) {
  parts::parts_gemm<parts::LinearOp, NCH, J, R, SPLIT, WAVES>(op, load_size(&sizes[kNDst]));
}

template <int NCH, int J, int R, int SPLIT, int WAVES>
void launch_parts(const int32_t* sizes, const float* hs, const float* ag, const float* ws, const float* wn,
                  const float* bias, int K, int N, int relu, float* out, int64_t cap_rows, hipStream_t s) {
  static_assert(parts::parts_lds_bytes(NCH, J, R, SPLIT, WAVES) <= 160 * 1024, "slab exceeds the LDS");
  const bool quad = N % 4 == 0 && (reinterpret_cast<uintptr_t>(ws) | reinterpret_cast<uintptr_t>(wn)) % 16 == 0;
  const parts::LinearOp op{hs, ag, ws, wn, bias, K, N, relu, out, quad ? 1 : 0};
  hipLaunchKernelGGL((k_linear_f32_parts<NCH, J, R, SPLIT, WAVES>), (parts::parts_grid<J, R, SPLIT, WAVES>(cap_rows, N)),
                     dim3(64 * WAVES), 0, s, sizes, op);
}

// Tiling of the part-product kernel, from timings of the three layer shapes
// of the 3-layer model (39k x 200 -> 256, 4.6k x 512 -> 256, 1k x 512 -> 47):
// eight waves per workgroup (two per SIMD, one slab: each wave's cutting of
// its A values then runs beside the other wave's products, since one wave's
// VALU and matrix-core instructions barely overlap).  Layers with enough
// 128-row tiles to fill the chip twice give each wave its own 16 rows of a
// 64-column slab; smaller layers split K over the eight waves, on 16-row
// tiles of 32 columns when there are enough rows, else 16.  Returns false
// where the fp32 slab kernel is the faster choice (wide K on many rows:
// the eight-wave tiling would not fit its registers).
template <int NCH>
bool launch_parts_for(const int32_t* sizes, const float* hs, const float* ag, const float* ws,
                      const float* wn, const float* bias, int K, int N, int relu, float* out,
                      int64_t cap_rows, hipStream_t s) {
  const int64_t big_tiles = ((cap_rows + 127) / 128) * ((N + 63) / 64);
  if (big_tiles >= 2 * 256) {
    if constexpr (NCH <= 8) {
      launch_parts<NCH, 4, 1, 1, 8>(sizes, hs, ag, ws, wn, bias, K, N, relu, out, cap_rows, s);
      return true;
    }
    return false;
  }
  if (cap_rows * N > (int64_t{1} << 18))
    launch_parts<NCH, 2, 1, 4, 8>(sizes, hs, ag, ws, wn, bias, K, N, relu, out, cap_rows, s);
  else
    launch_parts<NCH, 1, 1, 4, 8>(sizes, hs, ag, ws, wn, bias, K, N, relu, out, cap_rows, s);
  return true;
}

// bf16 with the weight slab resident in LDS (same scheme as the fp32 slab
// kernel, on v_mfma_f32_16x16x32_bf16).  Lane l (q = l/16) supplies
// A[l%16][32c + 8q .. +7] and B[32c + 8q .. +7][l%16] of chunk c and holds
// C[4q + r][l%16].  The slab keeps the workgroup's BN = 16 J columns of
// [W_self; W_neigh] for all 2 d_in rows (zero past 2 d_in and past d_out)
// in operand order, Bp[((c * 4 + q) * BN + n) * 8 + s] = W[32c + 8q + s][n],
// so a lane reads its eight k values with one 16-byte LDS read; its A
// operand is one 16-byte global read (d_in % 8 == 0, so a group of eight k
// never straddles [h_v | mean]).  Each wave computes 16 rows x BN columns,
// the workgroup 64 rows, persistent over row tiles with the next tile's A
// reads issued as soon as each chunk's MFMAs are; fp32 accumulation, bias
// and ReLU, then fp32 or bf16 (round to nearest even) output.
template <int NCH, int J>
__global__ __launch_bounds__(256) void k_linear_bf16_slab(const int32_t* sizes,
                                                          const uint16_t* __restrict__ Hs,
                                                          const uint16_t* __restrict__ Ag,
                                                          const uint16_t* __restrict__ Ws,
                                                          const uint16_t* __restrict__ Wn,
                                                          const float* __restrict__ bias, int K, int N,
                                                          int relu, int out_f32, int wvec,
                                                          void* __restrict__ out) {
  constexpr int BN = 16 * J;
  __shared__ __attribute__((aligned(16))) uint16_t Bp[NCH * 4 * BN * 8];
  const int32_t M = load_size(&sizes[kNDst]);
  const int row_tiles = (M + 63) / 64;
  if (static_cast<int>(blockIdx.x) >= row_tiles) return;
  const int n0 = blockIdx.y * BN;
  const int K2 = 2 * K;
  // slab fill: thread item = (k, 8 consecutive columns); one 16-byte read
  // of a weight row when the row is vector-aligned and inside the matrix,
  // else element-wise with zero padding
  constexpr int kItems = NCH * 32 * (BN / 8);
  for (int base = 0; base < kItems; base += 256 * 4) {
    uint4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = base + u * 256 + threadIdx.x;
      const int k = idx / (BN / 8), n8 = idx % (BN / 8);
      const int gn = n0 + 8 * n8;
      const bool in_k = idx < kItems && k < K2;
      const uint16_t* row = (k < K ? Ws + static_cast<int64_t>(k) * N
                                   : Wn + static_cast<int64_t>(in_k ? k - K : 0) * N);
      // every read is unconditional (clamped column), zeros selected after
      if (wvec) {   // uniform: N % 8 == 0 and 16-byte aligned rows
        uint4 x = *reinterpret_cast<const uint4*>(row + (gn < N ? gn : 0));
        asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
        v[u] = (in_k && gn < N) ? x : make_uint4(0u, 0u, 0u, 0u);
      } else {
        uint32_t e[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) e[i] = row[gn + i < N ? gn + i : N - 1];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          asm volatile("" : "+v"(e[i]));
          e[i] = (in_k && gn + i < N) ? e[i] : 0u;
        }
        v[u] = make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16));
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = base + u * 256 + threadIdx.x;
      if (idx >= kItems) continue;
      const int k = idx / (BN / 8), n8 = idx % (BN / 8);
      const int c = k >> 5, q = (k >> 3) & 3, sl = k & 7;
      const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
      for (int i = 0; i < 8; ++i)
        Bp[((c * 4 + q) * BN + 8 * n8 + i) * 8 + sl] = static_cast<uint16_t>(w[i >> 1] >> (16 * (i & 1)));
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, r16 = lane & 15;
  auto tile_rows = [&](int rt, const uint16_t*& hrow, const uint16_t*& grow) {
    const int row = rt * 64 + wave * 16 + r16;
    const int64_t arow = row < M ? row : M - 1;
    hrow = Hs + arow * K;
    grow = Ag + arow * K;
  };
  auto load_frag = [&](const uint16_t* hrow, const uint16_t* grow, int c) -> bf16x8 {
    const int k = 32 * c + 8 * q;
    const bool in = k < K2;
    const uint16_t* p = (k < K ? hrow + k : grow + (in ? k - K : 0));
    uint4 x = *reinterpret_cast<const uint4*>(p);
    asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
    if (!in) x = make_uint4(0u, 0u, 0u, 0u);
    return __builtin_bit_cast(bf16x8, x);
  };
  bf16x8 a[NCH];
  {
    const uint16_t *hrow, *grow;
    tile_rows(blockIdx.x, hrow, grow);
#pragma unroll
    for (int c = 0; c < NCH; ++c) a[c] = load_frag(hrow, grow, c);
  }
  float bv[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int col = n0 + j * 16 + r16;
    bv[j] = bias[col < N ? col : N - 1];
  }
  for (int rt = blockIdx.x; rt < row_tiles; rt += gridDim.x) {
    const uint16_t *hnext, *gnext;
    tile_rows(rt + gridDim.x, hnext, gnext);
    floatx4 acc[J];
#pragma unroll
    for (int j = 0; j < J; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    auto load_b = [&](int c, bf16x8 (&b)[J]) {
#pragma unroll
      for (int j = 0; j < J; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(&Bp[((c * 4 + q) * BN + j * 16 + r16) * 8]);
    };
    bf16x8 b0[J], b1[J];
    load_b(0, b0);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      bf16x8 (&bc)[J] = (c & 1) ? b1 : b0;
      bf16x8 (&bn)[J] = (c & 1) ? b0 : b1;
      if (c + 1 < NCH) load_b(c + 1, bn);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < J; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[c], bc[j], acc[j], 0, 0, 0);
      a[c] = load_frag(hnext, gnext, c);
    }
    const int row0 = rt * 64 + wave * 16 + 4 * q;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int col = n0 + j * 16 + r16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float z = acc[j][r] + bv[j];
        if (relu) z = z > 0.f ? z : 0.f;
        if (row0 + r < M && col < N) {
          const int64_t o = static_cast<int64_t>(row0 + r) * N + col;
          if (out_f32) static_cast<float*>(out)[o] = z;
          else static_cast<uint16_t*>(out)[o] = f32_to_bf16(z);
        }
      }
    }
  }
}

template <int NCH>
void launch_bf16_slab(const int32_t* sizes, const uint16_t* hs, const uint16_t* ag, const uint16_t* ws,
                      const uint16_t* wn, const float* bias, int K, int N, int relu, int out_f32,
                      void* out, int64_t cap_rows, hipStream_t s) {
  constexpr int J = 4, BN = 64;
  constexpr int lds = NCH * 4 * BN * 8 * 2;
  constexpr int by_lds = (160 * 1024) / lds;
  const int per_cu = by_lds < 1 ? 1 : (by_lds > kSlabBlocksBf16 ? kSlabBlocksBf16 : by_lds);
  const int col_tiles = (N + BN - 1) / BN;
  int64_t rows = (cap_rows + 63) / 64;
  const int64_t want = (256 * per_cu + col_tiles - 1) / col_tiles;
  if (rows > want) rows = want;
  if (rows < 1) rows = 1;
  const uintptr_t walign = reinterpret_cast<uintptr_t>(ws) | reinterpret_cast<uintptr_t>(wn);
  const int wvec = (N % 8 == 0 && walign % 16 == 0) ? 1 : 0;
  hipLaunchKernelGGL((k_linear_bf16_slab<NCH, J>), dim3(static_cast<unsigned>(rows), col_tiles), dim3(256), 0,
                     s, sizes, hs, ag, ws, wn, bias, K, N, relu, out_f32, wvec, out);
}

}  // namespace

hipError_t launch_mean_aggregate(const int32_t* sizes, const int32_t* indptr, const int32_t* local,
                                 const void* h, int d, int bf16, void* agg, int64_t cap_dst,
                                 int fanout, int64_t max_id, hipStream_t s) {
  const uintptr_t align = reinterpret_cast<uintptr_t>(h) | reinterpret_cast<uintptr_t>(agg);
  if (bf16) {
    if (d % 8 == 0 && align % 16 == 0)
      return mean_dispatch<uint16_t, 8>(sizes, indptr, local, h, d, agg, cap_dst, fanout, max_id, s);
    return mean_dispatch<uint16_t, 1>(sizes, indptr, local, h, d, agg, cap_dst, fanout, max_id, s);
  }
  if (d % 4 == 0 && align % 16 == 0)
    return mean_dispatch<float, 4>(sizes, indptr, local, h, d, agg, cap_dst, fanout, max_id, s);
  return mean_dispatch<float, 1>(sizes, indptr, local, h, d, agg, cap_dst, fanout, max_id, s);
}

hipError_t launch_sage_linear(const int32_t* sizes, const void* h_self, const void* agg,
                              const void* w_self, const void* w_neigh, const float* bias, int d_in,
                              int d_out, int bf16, int relu, int out_f32, void* out,
                              int64_t cap_rows, hipStream_t s) {
  int64_t gm = (cap_rows + kBM - 1) / kBM;
  if (gm < 1) gm = 1;
  const dim3 grid(static_cast<unsigned>(gm), static_cast<unsigned>((d_out + kBN - 1) / kBN)), block(256);
  if (bf16) {
    const uint16_t* hs = static_cast<const uint16_t*>(h_self);
    const uint16_t* ag = static_cast<const uint16_t*>(agg);
    const uint16_t* ws = static_cast<const uint16_t*>(w_self);
    const uint16_t* wn = static_cast<const uint16_t*>(w_neigh);
    const uintptr_t align = reinterpret_cast<uintptr_t>(hs) | reinterpret_cast<uintptr_t>(ag);
    const int nch = (2 * d_in + 31) / 32;
    if (d_in % 8 == 0 && align % 16 == 0 && nch <= 40) {
#define GMB_SLAB16(C) \
  launch_bf16_slab<C>(sizes, hs, ag, ws, wn, bias, d_in, d_out, relu, out_f32, out, cap_rows, s)
      if (nch <= 2) GMB_SLAB16(2);
      else if (nch <= 4) GMB_SLAB16(4);
      else if (nch <= 8) GMB_SLAB16(8);
      else if (nch <= 16) GMB_SLAB16(16);
      else if (nch <= 24) GMB_SLAB16(24);
      else if (nch <= 32) GMB_SLAB16(32);
      else GMB_SLAB16(40);
#undef GMB_SLAB16
      return hipGetLastError();
    }
    hipLaunchKernelGGL(k_linear_bf16, grid, block, 0, s, sizes, hs, ag, ws, wn, bias, d_in, d_out, relu,
                       out_f32, out);
  } else {
    if (!out_f32) return hipErrorInvalidValue;
    const float* hs = static_cast<const float*>(h_self);
    const float* ag = static_cast<const float*>(agg);
    const float* ws = static_cast<const float*>(w_self);
    const float* wn = static_cast<const float*>(w_neigh);
    const uintptr_t align = reinterpret_cast<uintptr_t>(hs) | reinterpret_cast<uintptr_t>(ag);
    const int nch = (2 * d_in + 15) / 16;
    const int nch32 = (2 * d_in + 31) / 32;
    if (d_in % 4 == 0 && align % 16 == 0 && nch32 <= 16) {
      float* o = static_cast<float*>(out);
      bool done;
#define GMB_PARTS(C) done = launch_parts_for<C>(sizes, hs, ag, ws, wn, bias, d_in, d_out, relu, o, cap_rows, s)
      if (nch32 <= 1) GMB_PARTS(1);
      else if (nch32 <= 2) GMB_PARTS(2);
      else if (nch32 <= 4) GMB_PARTS(4);
      else if (nch32 <= 7) GMB_PARTS(7);
      else if (nch32 <= 8) GMB_PARTS(8);
      else if (nch32 <= 12) GMB_PARTS(12);
      else GMB_PARTS(16);
#undef GMB_PARTS
      if (done) return hipGetLastError();
    }
    if (d_in % 4 == 0 && align % 16 == 0 && nch <= 40) {
      float* o = static_cast<float*>(out);
#define GMB_SLAB(C) launch_slab_for<C>(sizes, hs, ag, ws, wn, bias, d_in, d_out, relu, o, cap_rows, s)
      if (nch <= 2) GMB_SLAB(2);
      else if (nch <= 4) GMB_SLAB(4);
      else if (nch <= 8) GMB_SLAB(8);
      else if (nch <= 13) GMB_SLAB(13);
      else if (nch <= 16) GMB_SLAB(16);
      else if (nch <= 24) GMB_SLAB(24);
      else if (nch <= 32) GMB_SLAB(32);
      else GMB_SLAB(40);
#undef GMB_SLAB
      return hipGetLastError();
    }
    hipLaunchKernelGGL(k_linear_f32, grid, block, 0, s, sizes, static_cast<const float*>(h_self),
                       static_cast<const float*>(agg), static_cast<const float*>(w_self),
                       static_cast<const float*>(w_neigh), bias, d_in, d_out, relu,
                       static_cast<float*>(out));
  }
  return hipGetLastError();
}

}  // namespace gmb
