// Runs the C ABI's host code (argument checks, workspace planning, the
// enqueue loops with their pointer arithmetic) in a build with
// AddressSanitizer and UndefinedBehaviorSanitizer whose kernel launchers
// are stand-ins (abi_stubs.cpp): sampling, gather, forward (plain and
// fused), backward (with and without learnable embeddings) and the update,
// on the workloads' shapes and on edge cases, plus argument errors.  Device
// pointers are fake addresses that the host code never dereferences.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "gmb.h"

#define CHECK(c)                                                      \
  do {                                                                \
    if (!(c)) {                                                       \
      std::fprintf(stderr, "check failed at line %d: %s (%s)\n", __LINE__, #c, gmb_last_error()); \
      std::exit(1);                                                   \
    }                                                                 \
  } while (0)

static void* fake(uint64_t k) { return reinterpret_cast<void*>((k + 1) << 36); }

static void run_shape(int32_t B, std::vector<int32_t> fanouts, int64_t N, std::vector<int32_t> dims, bool wide) {
  const int L = static_cast<int>(fanouts.size());
  const size_t ws = gmb_sample_workspace_bytes(B, fanouts.data(), L, N);
  CHECK(ws > 0);
  gmb_csr csr{N, wide ? (int64_t(3) << 31) : 1000, fake(1), wide ? 64 : 32, 0, static_cast<const int32_t*>(fake(2))};
  const size_t sb = gmb_sampler_state_bytes(N);
  CHECK(sb > 0);
  CHECK(gmb_sampler_state_init(fake(3), sb, N, nullptr) == 0);
  gmb_blocks out{};
  CHECK(gmb_sample_blocks(&csr, static_cast<const int32_t*>(fake(4)), B, fanouts.data(), L, 0x1234, fake(3), sb,
                          fake(5), ws, &out, nullptr) == 0);
  CHECK(out.num_layers == L && out.num_seeds == B);
  CHECK(gmb_validate_blocks(&csr, &out, fake(3), nullptr) == 0);
  CHECK(gmb_gather_features(out.blk[0].src_ids, out.blk[0].sizes + 1, out.blk[0].cap_src, fake(6), N, dims[0], 0,
                            fake(7), gmb_state_status_word(fake(3)), nullptr) == 0);
  gmb_sage_weights w{};
  w.num_layers = L;
  w.dtype = GMB_F32;
  for (int l = 0; l <= L; ++l) w.dims[l] = dims[l];
  for (int l = 0; l < L; ++l) {
    w.w_self[l] = fake(10 + l);
    w.w_neigh[l] = fake(20 + l);
    w.bias[l] = static_cast<const float*>(fake(30 + l));
  }
  const size_t fw = gmb_forward_workspace_bytes(&out, &w);
  CHECK(fw > 0);
  CHECK(gmb_forward_hidden_offset(&out, &w, 0) >= (L > 1 ? 0 : -1));
  CHECK(gmb_sage_forward(&out, fake(8), &w, static_cast<float*>(fake(9)), fake(40), fw, nullptr) == 0);
  CHECK(gmb_sage_forward_fused(&out, fake(6), N, fake(41), &w, static_cast<float*>(fake(9)), fake(40), fw,
                               nullptr, nullptr) == 0);
  gmb_sage_grads g{};
  g.num_layers = L;
  for (int l = 0; l < L; ++l) {
    g.d_self[l] = static_cast<float*>(fake(50 + l));
    g.d_neigh[l] = static_cast<float*>(fake(60 + l));
    g.d_bias[l] = static_cast<float*>(fake(70 + l));
  }
  // the same model in bf16: forward, backward on widened copies, the update
  // of fp32 masters
  {
    gmb_sage_weights wb = w;
    wb.dtype = GMB_BF16;
    const size_t fwb = gmb_forward_workspace_bytes(&out, &wb);
    CHECK(fwb > 0);
    CHECK(gmb_sage_forward(&out, fake(8), &wb, static_cast<float*>(fake(9)), fake(40), fwb, nullptr) == 0);
    const size_t bwb = gmb_backward_workspace_bytes(&out, &wb);
    if (bwb > 0) {
      gmb_sage_grads gb{};
      gb.num_layers = L;
      for (int l = 0; l < L; ++l) {
        gb.d_self[l] = static_cast<float*>(fake(80 + l));
        gb.d_neigh[l] = static_cast<float*>(fake(90 + l));
        gb.d_bias[l] = static_cast<float*>(fake(100 + l));
      }
      CHECK(gmb_sage_backward(&out, fake(8), &wb, static_cast<const float*>(fake(9)),
                              static_cast<const int32_t*>(fake(42)), fake(40), fwb, &gb, static_cast<float*>(fake(43)),
                              fake(44), bwb, nullptr) == 0);
      CHECK(gmb_backward_embedding_workspace_bytes(&out, &wb) == 0);
      CHECK(gmb_sgd_update_bf16(&wb, &w, &gb, 0.01f, nullptr) == 0);
      CHECK(gmb_sgd_update_bf16(&w, &w, &gb, 0.01f, nullptr) == GMB_EINVAL);
    }
  }
  const size_t bw = gmb_backward_workspace_bytes(&out, &w);
  if (bw > 0) {
    CHECK(gmb_sage_backward(&out, fake(8), &w, static_cast<const float*>(fake(9)), static_cast<const int32_t*>(fake(42)),
                            fake(40), fw, &g, static_cast<float*>(fake(43)), fake(44), bw, nullptr) == 0);
    const size_t ew = gmb_backward_embedding_workspace_bytes(&out, &w);
    if (ew > 0)
      CHECK(gmb_sage_backward_embedding(&out, fake(8), &w, static_cast<const float*>(fake(9)),
                                        static_cast<const int32_t*>(fake(42)), fake(40), fw, &g,
                                        static_cast<float*>(fake(43)), fake(44), ew, static_cast<float*>(fake(6)), N,
                                        0.1f, nullptr) == 0);
    CHECK(gmb_sgd_update(&w, &g, 0.01f, nullptr) == 0);
  }
  // the no-allocation entry point: its checks pass, then it needs a device
  const int rc = gmb_sample_blocks_noalloc(&csr, static_cast<const int32_t*>(fake(4)), B, fanouts.data(), L, 1,
                                           fake(3), sb, fake(5), ws, &out, nullptr);
  CHECK(rc == 0 || rc == GMB_EDEVICE || rc == GMB_ENOSPC);
}

int main() {
  setenv("GMB_VALIDATE", "1", 1);   // the sampling calls also enqueue the block check
  run_shape(1000, {15, 10, 5}, 2449029, {100, 256, 256, 47}, false);
  run_shape(4000, {25, 10}, 2449029, {128, 256, 47}, false);
  run_shape(1000, {15, 10, 5}, 111059956, {128, 256, 256, 172}, true);
  run_shape(64, {5, 5}, 10000, {16, 16, 8}, false);
  run_shape(0, {5, 5}, 10000, {16, 16, 8}, false);
  run_shape(300, {70}, 3000, {16, 8}, false);
  run_shape(50, {6, 30}, 3000, {16, 12, 8}, false);
  run_shape(7, {1, 1, 1, 1, 1, 1, 1, 1}, 100, {4, 4, 4, 4, 4, 4, 4, 4, 4}, false);
  run_shape(3, {4096}, 1 << 20, {8, 4}, false);
  // argument errors
  std::vector<int32_t> f = {5, 0};
  CHECK(gmb_sample_workspace_bytes(10, f.data(), 2, 100) == 0);
  f = {4097};
  CHECK(gmb_sample_workspace_bytes(10, f.data(), 1, 100000) == 0);
  f = {5};
  CHECK(gmb_sample_workspace_bytes(101, f.data(), 1, 100) == 0);
  CHECK(gmb_sample_workspace_bytes(10, f.data(), 9, 100) == 0);
  gmb_csr csr{100, 500, fake(1), 16, 0, static_cast<const int32_t*>(fake(2))};
  gmb_blocks out{};
  CHECK(gmb_sample_blocks(&csr, static_cast<const int32_t*>(fake(4)), 10, f.data(), 1, 1, fake(3), 1 << 20, fake(5),
                          1 << 30, &out, nullptr) == GMB_EINVAL);
  CHECK(gmb_sample_blocks(nullptr, nullptr, 0, f.data(), 1, 1, nullptr, 0, nullptr, 0, &out, nullptr) == GMB_EINVAL);
  CHECK(gmb_gather_features(nullptr, nullptr, 10, fake(1), 100, 0, 0, fake(2), nullptr, nullptr) == GMB_EINVAL);
  gmb_sage_weights w{};
  CHECK(gmb_forward_workspace_bytes(&out, &w) == 0);
  CHECK(gmb_sgd_update(nullptr, nullptr, 0.1f, nullptr) == GMB_EINVAL);
  std::printf("sanitized C ABI host code: ok\n");
  return 0;
}
