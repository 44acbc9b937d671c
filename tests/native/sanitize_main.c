/* Drives the oracle (oracle/oracle.c) and the input generator
 * (datagen/datagen.c) through their C entry points on small inputs, for a
 * build with AddressSanitizer and UndefinedBehaviorSanitizer: graphs (ER,
 * R-MAT, injected hubs), features, multi-layer sampling with relabel
 * (including a seed out of range and a repeated seed), gather, mean, the
 * linear layers, the loss and the whole backward.  Exits 0 when every call
 * succeeds; any sanitizer report aborts the run. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct orc_blocks orc_blocks;
int orc_sample_blocks(int64_t num_nodes, const int64_t* indptr, const int32_t* indices, const int64_t* seeds,
                      int64_t num_seeds, const int64_t* fanouts, int num_layers, uint64_t seed, orc_blocks** out);
void orc_free_blocks(orc_blocks* b);
int orc_blocks_num_layers(const orc_blocks* b);
void orc_block_sizes(const orc_blocks* b, int l, int64_t sizes[3]);
void orc_block_copy(const orc_blocks* b, int l, int64_t* indptr, int64_t* nbr, int64_t* local, int64_t* src);
int orc_gather(const void* feats, int64_t num_rows, int64_t row_bytes, const int64_t* ids, int64_t n, void* out);
void orc_mean_aggregate(int64_t n_dst, const int64_t* indptr, const int64_t* local, const double* H, int64_t d,
                        double* m);
void orc_sage_linear(int64_t n_dst, int64_t d_in, int64_t d_out, const double* H, const double* m,
                     const double* w_self, const double* w_neigh, const double* bias, int relu, double* out);
double orc_softmax_xent(int64_t n, int64_t C, const double* z, const int64_t* y, double* dz);
void orc_sage_linear_backward(int64_t n, int64_t d_in, int64_t d_out, const double* H, const double* m,
                              const double* w_self, const double* w_neigh, const double* dZ, double* dW_self,
                              double* dW_neigh, double* db, double* dH, double* dM);
void orc_mean_backward(int64_t n_dst, const int64_t* indptr, const int64_t* local, const double* dM, int64_t d,
                       double* dH);
void orc_relu_backward(int64_t n, const double* out, const double* dOut, double* dZ);

int64_t dg_er_count(int64_t n, double p, uint64_t seed, int64_t* indptr);
void dg_er_fill(int64_t n, double p, uint64_t seed, const int64_t* indptr, int32_t* indices);
int64_t dg_rmat(int scale, int64_t n, int64_t draws, double a, double b, double c, uint64_t seed, int64_t* indptr,
                int32_t** indices_out);
int64_t dg_inject_hubs(int64_t n, const int64_t* indptr_in, const int32_t* indices_in, int64_t num_hubs,
                       int64_t hub_deg, uint64_t seed, int64_t* hubs_out, int64_t* indptr_out,
                       int32_t** indices_out);
void dg_features_f32(int64_t rows, int64_t dim, uint64_t seed, float* out);
void dg_features_bf16(int64_t rows, int64_t dim, uint64_t seed, uint16_t* out);
void dg_free(void* p);

#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      exit(1);                                                    \
    }                                                             \
  } while (0)

static double* zeros(int64_t n) {
  double* p = (double*)calloc((size_t)(n > 0 ? n : 1), sizeof(double));
  CHECK(p);
  return p;
}

/* One forward and backward pass of an L-layer model over the blocks. */
static void run_model(const orc_blocks* b, const double* X, const int64_t* dims) {
  const int L = orc_blocks_num_layers(b);
  int64_t* ip[8];
  int64_t* loc[8];
  int64_t sz[8][3];
  double* H[9];
  double* M[8];
  double *ws[8], *wn[8], *bs[8];
  H[0] = (double*)X;
  for (int l = 0; l < L; ++l) {
    orc_block_sizes(b, l, sz[l]);
    ip[l] = (int64_t*)malloc(sizeof(int64_t) * (size_t)(sz[l][0] + 1));
    loc[l] = (int64_t*)malloc(sizeof(int64_t) * (size_t)(sz[l][2] > 0 ? sz[l][2] : 1));
    int64_t* nbr = (int64_t*)malloc(sizeof(int64_t) * (size_t)(sz[l][2] > 0 ? sz[l][2] : 1));
    int64_t* src = (int64_t*)malloc(sizeof(int64_t) * (size_t)(sz[l][1] > 0 ? sz[l][1] : 1));
    CHECK(ip[l] && loc[l] && nbr && src);
    orc_block_copy(b, l, ip[l], nbr, loc[l], src);
    for (int64_t e = 0; e < sz[l][2]; ++e) CHECK(loc[l][e] >= 0 && loc[l][e] < sz[l][1]);
    free(nbr);
    free(src);
    const int64_t di = dims[l], dout = dims[l + 1];
    ws[l] = zeros(di * dout);
    wn[l] = zeros(di * dout);
    bs[l] = zeros(dout);
    for (int64_t i = 0; i < di * dout; ++i) {
      ws[l][i] = 0.01 * (double)((i * 7) % 13 - 6);
      wn[l][i] = 0.01 * (double)((i * 5) % 11 - 5);
    }
    M[l] = zeros(sz[l][0] * di);
    H[l + 1] = zeros(sz[l][0] * dout);
    orc_mean_aggregate(sz[l][0], ip[l], loc[l], H[l], di, M[l]);
    orc_sage_linear(sz[l][0], di, dout, H[l], M[l], ws[l], wn[l], bs[l], l + 1 < L, H[l + 1]);
  }
  const int64_t B = sz[L - 1][0], C = dims[L];
  int64_t* y = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B > 0 ? B : 1));
  CHECK(y);
  for (int64_t i = 0; i < B; ++i) y[i] = i % C;
  double* dZ = zeros(B * C);
  const double loss = orc_softmax_xent(B, C, H[L], y, dZ);
  CHECK(loss == loss);
  for (int l = L - 1; l >= 0; --l) {
    const int64_t di = dims[l], dout = dims[l + 1];
    double* dWs = zeros(di * dout);
    double* dWn = zeros(di * dout);
    double* db = zeros(dout);
    double* dHs = zeros(sz[l][0] * di);
    double* dM = zeros(sz[l][0] * di);
    orc_sage_linear_backward(sz[l][0], di, dout, H[l], M[l], ws[l], wn[l], dZ, dWs, dWn, db, dHs, dM);
    double* dH = zeros(sz[l][1] * di);
    memcpy(dH, dHs, sizeof(double) * (size_t)(sz[l][0] * di));
    orc_mean_backward(sz[l][0], ip[l], loc[l], dM, di, dH);
    double* dZ_below = zeros(sz[l][1] * di);
    if (l > 0) orc_relu_backward(sz[l][1] * di, H[l], dH, dZ_below);
    free(dZ);
    dZ = dZ_below;
    free(dWs);
    free(dWn);
    free(db);
    free(dHs);
    free(dM);
    free(dH);
  }
  free(dZ);
  free(y);
  for (int l = 0; l < L; ++l) {
    free(ip[l]);
    free(loc[l]);
    free(ws[l]);
    free(wn[l]);
    free(bs[l]);
    free(M[l]);
    free(H[l + 1]);
  }
}

static void sample_and_run(int64_t n, const int64_t* indptr, const int32_t* indices, int64_t num_seeds,
                           const int64_t* fanouts, int L, uint64_t key) {
  int64_t* seeds = (int64_t*)malloc(sizeof(int64_t) * (size_t)(num_seeds > 0 ? num_seeds : 1));
  CHECK(seeds);
  for (int64_t i = 0; i < num_seeds; ++i) seeds[i] = (i * 7919) % n;   /* distinct: 7919 is prime, n < 7919 * ... */
  orc_blocks* b = NULL;
  CHECK(orc_sample_blocks(n, indptr, indices, seeds, num_seeds, fanouts, L, key, &b) == 0);
  int64_t sz0[3];
  orc_block_sizes(b, 0, sz0);
  const int64_t D = 8;
  double* X = zeros(sz0[1] * D);
  for (int64_t i = 0; i < sz0[1] * D; ++i) X[i] = (double)(i % 17) / 17.0;
  int64_t dims[9] = {D, 6, 5, 4, 3, 3, 3, 3, 3};
  dims[L] = 3;
  run_model(b, X, dims);
  /* the gather of the input rows */
  int64_t* src = (int64_t*)malloc(sizeof(int64_t) * (size_t)(sz0[1] > 0 ? sz0[1] : 1));
  int64_t* ip = (int64_t*)malloc(sizeof(int64_t) * (size_t)(sz0[0] + 1));
  int64_t* nb = (int64_t*)malloc(sizeof(int64_t) * (size_t)(sz0[2] > 0 ? sz0[2] : 1));
  int64_t* lc = (int64_t*)malloc(sizeof(int64_t) * (size_t)(sz0[2] > 0 ? sz0[2] : 1));
  CHECK(src && ip && nb && lc);
  orc_block_copy(b, 0, ip, nb, lc, src);
  float* feats = (float*)malloc(sizeof(float) * (size_t)(n * 4));
  float* out = (float*)malloc(sizeof(float) * (size_t)((sz0[1] > 0 ? sz0[1] : 1) * 4));
  CHECK(feats && out);
  dg_features_f32(n, 4, 11, feats);
  CHECK(orc_gather(feats, n, 16, src, sz0[1], out) == 0);
  free(feats);
  free(out);
  free(src);
  free(ip);
  free(nb);
  free(lc);
  free(X);
  orc_free_blocks(b);
  /* a seed out of range and a repeated seed are refused */
  if (num_seeds >= 2) {
    seeds[1] = n;
    CHECK(orc_sample_blocks(n, indptr, indices, seeds, num_seeds, fanouts, L, key, &b) == -4);
    seeds[1] = seeds[0];
    CHECK(orc_sample_blocks(n, indptr, indices, seeds, num_seeds, fanouts, L, key, &b) == -5);
  }
  free(seeds);
}

int main(void) {
  /* directed ER */
  const int64_t n = 3000;
  int64_t* indptr = (int64_t*)calloc((size_t)(n + 1), sizeof(int64_t));
  CHECK(indptr);
  const int64_t nnz = dg_er_count(n, 8.0 / (n - 1), 101, indptr);
  CHECK(nnz > 0 && indptr[n] == nnz);
  int32_t* indices = (int32_t*)malloc(sizeof(int32_t) * (size_t)nnz);
  CHECK(indices);
  dg_er_fill(n, 8.0 / (n - 1), 101, indptr, indices);
  const int64_t f2[2] = {4, 3}, f3[3] = {6, 4, 2}, f1[1] = {70};
  sample_and_run(n, indptr, indices, 64, f2, 2, 7);
  sample_and_run(n, indptr, indices, 200, f3, 3, 8);
  sample_and_run(n, indptr, indices, 10, f1, 1, 9);
  sample_and_run(n, indptr, indices, 0, f2, 2, 10);
  /* R-MAT and injected hubs */
  int64_t* rp = (int64_t*)calloc((size_t)(4000 + 1), sizeof(int64_t));
  int32_t* ri = NULL;
  CHECK(rp);
  const int64_t rn = dg_rmat(12, 4000, 20000, 0.57, 0.19, 0.19, 202, rp, &ri);
  CHECK(rn > 0 && ri);
  int64_t hubs[4];
  int64_t* hp = (int64_t*)calloc((size_t)(4000 + 1), sizeof(int64_t));
  int32_t* hi = NULL;
  CHECK(hp);
  const int64_t hn = dg_inject_hubs(4000, rp, ri, 4, 500, 303, hubs, hp, &hi);
  CHECK(hn > rn && hi);
  const int64_t fh[2] = {25, 10};
  sample_and_run(4000, hp, hi, 300, fh, 2, 11);
  sample_and_run(4000, rp, ri, 300, f3, 3, 12);
  uint16_t* bf = (uint16_t*)malloc(sizeof(uint16_t) * 4000 * 8);
  CHECK(bf);
  dg_features_bf16(4000, 8, 5, bf);
  free(bf);
  dg_free(ri);
  dg_free(hi);
  free(rp);
  free(hp);
  free(indices);
  free(indptr);
  printf("sanitized oracle and generator: ok\n");
  return 0;
}
