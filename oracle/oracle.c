/*
 * CPU oracle of the mini-batch GNN hot path.  TEST INFRASTRUCTURE ONLY:
 * only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  It shares no code with the GPU library; the only
 * thing both sides share is the seeded input generator.
 *
 * Plain, slow, single-threaded, fp64 where arithmetic is floating point.
 *
 * What it computes (DistDGL, arXiv 2010.05337):
 *   Section II-B, mini-batch training: take N target vertices, pick at most
 *   K (the fan-out) neighbours of each target at random, repeat recursively
 *   once per GNN layer; the sampled graph plus the extracted features form
 *   the mini-batch, and the targets' representations are computed by
 *   gathering messages from the sampled neighbours (Fig. 1(b): messages flow
 *   from the leaves to the root).
 *   Section II-A, Eq. (1): h_v^(l+1) = g(h_v^(l), (+)_{u in N(v)} f(h_u^(l), ...)),
 *   instantiated as GraphSAGE-mean (Section IV: 3 layers, hidden 256,
 *   fan-outs 15, 10, 5).
 *
 * The paper does not fix the random-number generator, the subset algorithm,
 * edge direction, neighbour order within a row or dedup across targets.  The
 * readings taken here:
 *   - draws come from Philox4x32-10 (Salmon, Moraes, Dror & Shaw, "Parallel
 *     random numbers: as easy as 1, 2, 3", SC'11), key = (lo32(seed),
 *     hi32(seed)), counter = (node v, layer l, draw index i, retry r);
 *   - a draw in [0, m) is Lemire's multiply-and-reject method ("Fast random
 *     integer generation in an interval", ACM TOMACS 2019) on the words
 *     x0, x1, x2, x3 of one Philox block, then on the block with r + 1, ...;
 *   - "at most K" is sampling without replacement, k = min(deg, K), by
 *     Floyd's algorithm (Bentley & Floyd, "Programming pearls: a sample of
 *     brilliance", CACM 30(9), 1987); deg <= K takes the whole row with no
 *     draws;
 *   - neighbours are in-neighbours (the CSR row of v lists the sources of the
 *     edges into v), and a node's sampled slots are reported in ascending
 *     slot order;
 *   - each layer's frontier is de-duplicated: the block's source list is the
 *     destination list followed by the new vertices in order of first
 *     appearance over (destination position, slot).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

/* ------------------------------------------------------------------ */
/* O1: Philox4x32-10 (Salmon et al., SC'11, Section 4 and Table 2).     */

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static void philox_round(uint32_t c[4], const uint32_t k[2]) {
  uint64_t p0 = (uint64_t)PHILOX_M0 * c[0];
  uint64_t p1 = (uint64_t)PHILOX_M1 * c[2];
  uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
  uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
  uint32_t n0 = hi1 ^ c[1] ^ k[0];
  uint32_t n1 = lo1;
  uint32_t n2 = hi0 ^ c[3] ^ k[1];
  uint32_t n3 = lo0;
  c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
}

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  uint32_t k[2] = {key[0], key[1]};
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {           /* the key schedule: add the Weyl constants */
      k[0] += PHILOX_W0;
      k[1] += PHILOX_W1;
    }
    philox_round(c, k);
  }
  memcpy(out, c, sizeof c);
}

/* ------------------------------------------------------------------ */
/* O2: bounded draw in [0, m) from one 32-bit word (Lemire 2019).        */
/* Returns 1 and sets *t when the word is accepted, 0 when rejected.     */

int orc_bounded_from_word(uint32_t x, uint32_t m, uint32_t* t) {
  uint64_t p = (uint64_t)x * (uint64_t)m;
  uint32_t low = (uint32_t)p;
  uint32_t threshold = (uint32_t)((4294967296ULL - (uint64_t)m) % (uint64_t)m);
  if (low < threshold) return 0;
  *t = (uint32_t)(p >> 32);
  return 1;
}

/* Draw i of node v at layer l, uniform in [0, m), m >= 1. */
uint32_t orc_uniform_below(uint64_t seed, uint32_t v, uint32_t l, uint32_t i, uint32_t m) {
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  for (uint32_t r = 0;; ++r) {
    uint32_t ctr[4] = {v, l, i, r};
    uint32_t x[4];
    orc_philox4x32_10(ctr, key, x);
    for (int w = 0; w < 4; ++w) {
      uint32_t t;
      if (orc_bounded_from_word(x[w], m, &t)) return t;
    }
  }
}

/* ------------------------------------------------------------------ */
/* O3: Floyd's algorithm.  Picks k distinct values of {0..d-1}: for       */
/* i = 0..k-1 with j = d-k+i and a draw t_i uniform in [0, j], insert t_i  */
/* unless it is already chosen, in which case insert j.  `draws` holds    */
/* t_0..t_{k-1}; `chosen` receives the values in insertion order.         */

void orc_floyd(uint32_t d, uint32_t k, const uint32_t* draws, uint32_t* chosen) {
  for (uint32_t i = 0; i < k; ++i) {
    uint32_t j = d - k + i;
    uint32_t t = draws[i];
    int present = 0;
    for (uint32_t q = 0; q < i; ++q)
      if (chosen[q] == t) present = 1;
    chosen[i] = present ? j : t;
  }
}

static int cmp_u32(const void* a, const void* b) {
  uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
  return (x > y) - (x < y);
}

/* Sampled slots (row offsets) of node v with in-degree d at layer l with
 * fan-out f, ascending.  Returns k = min(d, f).  `slots` holds >= k. */
int64_t orc_sample_node(uint64_t seed, uint32_t v, uint32_t l, int64_t d, int64_t f,
                        uint32_t* slots) {
  if (d <= f) {
    for (int64_t s = 0; s < d; ++s) slots[s] = (uint32_t)s;
    return d;
  }
  uint32_t k = (uint32_t)f;
  uint32_t* draws = (uint32_t*)malloc(sizeof(uint32_t) * k);
  for (uint32_t i = 0; i < k; ++i) {
    uint32_t j = (uint32_t)d - k + i;
    draws[i] = orc_uniform_below(seed, v, l, i, j + 1);
  }
  orc_floyd((uint32_t)d, k, draws, slots);
  free(draws);
  qsort(slots, k, sizeof(uint32_t), cmp_u32);
  return k;
}

/* ------------------------------------------------------------------ */
/* O4: multi-layer sampling with per-layer relabelling.                   */

typedef struct {
  int64_t n_dst, n_src, nnz;
  int64_t* indptr;    /* [n_dst+1] */
  int64_t* nbr;       /* [nnz] global ids of the sampled in-neighbours */
  int64_t* local;     /* [nnz] position of nbr[e] in src */
  int64_t* src;       /* [n_src] global ids; src[0:n_dst] = the destinations */
} orc_block;

typedef struct {
  int num_layers;
  orc_block* blk;     /* blk[l] for model layer l (l = 0 is the input layer) */
} orc_blocks;

enum { ORC_OK = 0, ORC_EINVAL = -1, ORC_ERANGE = -4, ORC_EDUP = -5, ORC_ENOMEM = -6 };

void orc_free_blocks(orc_blocks* b) {
  if (!b) return;
  for (int l = 0; l < b->num_layers; ++l) {
    free(b->blk[l].indptr); free(b->blk[l].nbr); free(b->blk[l].local); free(b->blk[l].src);
  }
  free(b->blk);
  free(b);
}

/* The seeds and fan-outs define the mini-batch; fanouts[l] belongs to model
 * layer l, so the first hop (from the seeds) uses fanouts[L-1].  Returns a
 * status; on success *out holds the blocks (free with orc_free_blocks). */
int orc_sample_blocks(int64_t num_nodes, const int64_t* indptr, const int32_t* indices,
                      const int64_t* seeds, int64_t num_seeds, const int64_t* fanouts,
                      int num_layers, uint64_t seed, orc_blocks** out) {
  *out = NULL;
  if (num_layers < 1 || num_seeds < 0) return ORC_EINVAL;
  for (int l = 0; l < num_layers; ++l)
    if (fanouts[l] < 1) return ORC_EINVAL;

  /* map[u] = 1 + position of u in the current source list, 0 = absent */
  int64_t* map = (int64_t*)calloc((size_t)num_nodes + 1, sizeof(int64_t));
  orc_blocks* res = (orc_blocks*)calloc(1, sizeof(orc_blocks));
  if (!map || !res) { free(map); free(res); return ORC_ENOMEM; }
  res->num_layers = num_layers;
  res->blk = (orc_block*)calloc((size_t)num_layers, sizeof(orc_block));

  /* frontier = seeds */
  int64_t n_front = num_seeds;
  int64_t* front = (int64_t*)malloc(sizeof(int64_t) * (size_t)(num_seeds > 0 ? num_seeds : 1));
  for (int64_t p = 0; p < num_seeds; ++p) {
    int64_t s = seeds[p];
    if (s < 0 || s >= num_nodes) { free(front); free(map); orc_free_blocks(res); return ORC_ERANGE; }
    if (map[s] != 0) { free(front); free(map); orc_free_blocks(res); return ORC_EDUP; }
    map[s] = p + 1;
    front[p] = s;
  }

  int status = ORC_OK;
  for (int hop = 0; hop < num_layers; ++hop) {
    int l = num_layers - 1 - hop;
    int64_t f = fanouts[l];
    orc_block* B = &res->blk[l];
    B->n_dst = n_front;

    /* sampling: edges in (destination position, slot) order */
    B->indptr = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_front + 1));
    B->indptr[0] = 0;
    for (int64_t p = 0; p < n_front; ++p) {
      int64_t v = front[p];
      int64_t d = indptr[v + 1] - indptr[v];
      B->indptr[p + 1] = B->indptr[p] + (d < f ? d : f);
    }
    B->nnz = B->indptr[n_front];
    B->nbr = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B->nnz > 0 ? B->nnz : 1));
    B->local = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B->nnz > 0 ? B->nnz : 1));
    uint32_t* slots = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)f);
    for (int64_t p = 0; p < n_front; ++p) {
      int64_t v = front[p];
      int64_t d = indptr[v + 1] - indptr[v];
      int64_t k = orc_sample_node(seed, (uint32_t)v, (uint32_t)l, d, f, slots);
      for (int64_t q = 0; q < k; ++q) {
        int64_t u = indices[indptr[v] + slots[q]];
        if (u < 0 || u >= num_nodes) status = ORC_ERANGE;
        B->nbr[B->indptr[p] + q] = u;
      }
    }
    free(slots);
    if (status != ORC_OK) break;

    /* relabel: sources = destinations, then new vertices in first-seen order */
    int64_t n_src = n_front;
    B->src = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_front + B->nnz + 1));
    memcpy(B->src, front, sizeof(int64_t) * (size_t)n_front);
    for (int64_t e = 0; e < B->nnz; ++e) {
      int64_t u = B->nbr[e];
      if (map[u] == 0) {
        B->src[n_src] = u;
        map[u] = n_src + 1;
        ++n_src;
      }
      B->local[e] = map[u] - 1;
    }
    B->n_src = n_src;

    /* the next frontier is this block's source list */
    free(front);
    front = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_src > 0 ? n_src : 1));
    memcpy(front, B->src, sizeof(int64_t) * (size_t)n_src);
    n_front = n_src;
  }
  free(front);
  free(map);
  if (status != ORC_OK) { orc_free_blocks(res); return status; }
  *out = res;
  return ORC_OK;
}

int orc_blocks_num_layers(const orc_blocks* b) { return b->num_layers; }

void orc_block_sizes(const orc_blocks* b, int l, int64_t sizes[3]) {
  sizes[0] = b->blk[l].n_dst;
  sizes[1] = b->blk[l].n_src;
  sizes[2] = b->blk[l].nnz;
}

/* Copies block l out: indptr [n_dst+1], nbr [nnz], local [nnz], src [n_src]. */
void orc_block_copy(const orc_blocks* b, int l, int64_t* indptr, int64_t* nbr, int64_t* local,
                    int64_t* src) {
  const orc_block* B = &b->blk[l];
  memcpy(indptr, B->indptr, sizeof(int64_t) * (size_t)(B->n_dst + 1));
  if (B->nnz) {
    memcpy(nbr, B->nbr, sizeof(int64_t) * (size_t)B->nnz);
    memcpy(local, B->local, sizeof(int64_t) * (size_t)B->nnz);
  }
  if (B->n_src) memcpy(src, B->src, sizeof(int64_t) * (size_t)B->n_src);
}

/* ------------------------------------------------------------------ */
/* O5: feature gather: out row i is a bitwise copy of feats row ids[i].   */

int orc_gather(const void* feats, int64_t num_rows, int64_t row_bytes, const int64_t* ids,
               int64_t n, void* out) {
  for (int64_t i = 0; i < n; ++i) {
    if (ids[i] < 0 || ids[i] >= num_rows) return ORC_ERANGE;
    memcpy((char*)out + i * row_bytes, (const char*)feats + ids[i] * row_bytes, (size_t)row_bytes);
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* O6: GraphSAGE-mean layer, Eq. (1) with f(h_u, .) = h_u, (+) = mean,    */
/* g(h_v, m_v) = act(h_v W_self + m_v W_neigh + b).                        */

/* m[v] = (sum over the block row of H[local[e]]) / k_v, or 0 when k_v = 0.
 * H is [n_src, d] row-major, m is [n_dst, d]. */
void orc_mean_aggregate(int64_t n_dst, const int64_t* indptr, const int64_t* local,
                        const double* H, int64_t d, double* m) {
  for (int64_t v = 0; v < n_dst; ++v) {
    double* row = m + v * d;
    for (int64_t c = 0; c < d; ++c) row[c] = 0.0;
    int64_t k = indptr[v + 1] - indptr[v];
    for (int64_t e = indptr[v]; e < indptr[v + 1]; ++e) {
      const double* h = H + local[e] * d;
      for (int64_t c = 0; c < d; ++c) row[c] += h[c];
    }
    if (k > 0)
      for (int64_t c = 0; c < d; ++c) row[c] = row[c] / (double)k;
  }
}

/* out[v] = act(H[v] W_self + m[v] W_neigh + b) for v < n_dst; H rows are the
 * first n_dst rows of the layer input (the destinations).  W_* are
 * [d_in, d_out] row-major; relu != 0 applies max(z, 0). */
void orc_sage_linear(int64_t n_dst, int64_t d_in, int64_t d_out, const double* H,
                     const double* m, const double* w_self, const double* w_neigh,
                     const double* bias, int relu, double* out) {
  for (int64_t v = 0; v < n_dst; ++v) {
    for (int64_t o = 0; o < d_out; ++o) {
      double z = bias[o];
      for (int64_t c = 0; c < d_in; ++c) z += H[v * d_in + c] * w_self[c * d_out + o];
      for (int64_t c = 0; c < d_in; ++c) z += m[v * d_in + c] * w_neigh[c * d_out + o];
      out[v * d_out + o] = (relu && z < 0.0) ? 0.0 : z;
    }
  }
}

/* ------------------------------------------------------------------ */
/* O7: one training step on the mini-batch (the trainer's iteration of    */
/* Section III-E: forward, backward, gradient update).  The loss is the   */
/* mean softmax cross-entropy of the targets' logits against their labels */
/* (node classification, the task of Section IV; the paper prints no loss */
/* formula, so this is the standard reading).  Gradients follow Eq. (1)   */
/* by the chain rule, layer by layer from the last.                       */

/* loss = (1/n) sum_v -log softmax(z_v)[y_v];  dz_v = (softmax(z_v) - e_{y_v}) / n.
 * z, dz are [n, C] row-major.  Returns the loss. */
double orc_softmax_xent(int64_t n, int64_t C, const double* z, const int64_t* y, double* dz) {
  double loss = 0.0;
  for (int64_t v = 0; v < n; ++v) {
    const double* row = z + v * C;
    double mx = row[0];
    for (int64_t c = 1; c < C; ++c) mx = row[c] > mx ? row[c] : mx;
    double sum = 0.0;
    for (int64_t c = 0; c < C; ++c) sum += exp(row[c] - mx);
    loss += -(row[y[v]] - mx - log(sum));
    for (int64_t c = 0; c < C; ++c) {
      const double p = exp(row[c] - mx) / sum;
      dz[v * C + c] = (p - (c == y[v] ? 1.0 : 0.0)) / (double)n;
    }
  }
  return n > 0 ? loss / (double)n : 0.0;
}

/* Backward of out = H W_self + m W_neigh + b over n rows, given dZ = dL/d(out)
 * [n, d_out] (the activation already applied):
 *   dW_self = H^T dZ, dW_neigh = m^T dZ  [d_in, d_out];  db = column sums of dZ;
 *   dH = dZ W_self^T, dM = dZ W_neigh^T  [n, d_in]  (skipped when NULL). */
void orc_sage_linear_backward(int64_t n, int64_t d_in, int64_t d_out, const double* H,
                              const double* m, const double* w_self, const double* w_neigh,
                              const double* dZ, double* dW_self, double* dW_neigh, double* db,
                              double* dH, double* dM) {
  /* dW[c][o] = sum over v = 0, 1, ..., n-1 in that order; v is the outer
   * loop so that every pass reads two rows of the inputs */
  for (int64_t i = 0; i < d_in * d_out; ++i) dW_self[i] = dW_neigh[i] = 0.0;
  for (int64_t v = 0; v < n; ++v)
    for (int64_t c = 0; c < d_in; ++c) {
      const double hc = H[v * d_in + c], mc = m[v * d_in + c];
      for (int64_t o = 0; o < d_out; ++o) {
        dW_self[c * d_out + o] += hc * dZ[v * d_out + o];
        dW_neigh[c * d_out + o] += mc * dZ[v * d_out + o];
      }
    }
  for (int64_t o = 0; o < d_out; ++o) {
    double s = 0.0;
    for (int64_t v = 0; v < n; ++v) s += dZ[v * d_out + o];
    db[o] = s;
  }
  if (!dH || !dM) return;
  for (int64_t v = 0; v < n; ++v)
    for (int64_t c = 0; c < d_in; ++c) {
      double s = 0.0, t = 0.0;
      for (int64_t o = 0; o < d_out; ++o) {
        s += dZ[v * d_out + o] * w_self[c * d_out + o];
        t += dZ[v * d_out + o] * w_neigh[c * d_out + o];
      }
      dH[v * d_in + c] = s;
      dM[v * d_in + c] = t;
    }
}

/* Backward of the mean: every edge (v <- u) of the block passes dM[v] / k_v
 * to its source, dH[local[e]] += dM[v] / k_v (dH accumulates). */
void orc_mean_backward(int64_t n_dst, const int64_t* indptr, const int64_t* local,
                       const double* dM, int64_t d, double* dH) {
  for (int64_t v = 0; v < n_dst; ++v) {
    const int64_t k = indptr[v + 1] - indptr[v];
    for (int64_t e = indptr[v]; e < indptr[v + 1]; ++e) {
      double* h = dH + local[e] * d;
      for (int64_t c = 0; c < d; ++c) h[c] += dM[v * d + c] / (double)k;
    }
  }
}

/* Backward of out = max(z, 0) through the output: dZ = dOut where out > 0,
 * else 0 (the derivative at 0 is taken as 0). */
void orc_relu_backward(int64_t n, const double* out, const double* dOut, double* dZ) {
  for (int64_t i = 0; i < n; ++i) dZ[i] = out[i] > 0.0 ? dOut[i] : 0.0;
}
