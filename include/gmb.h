/*
 * gmb.h — C ABI of the mini-batch GNN hot path on MI355X (gfx950).
 *
 * The library implements the data-parallel part of one trainer's iteration
 * in DistDGL (arXiv 2010.05337): build a mini-batch by recursive fan-out
 * neighbour sampling (Section II-B), pull the feature rows of the sampled
 * vertices (the KVStore "pull" of Section III-C, here a local gather), and
 * run the GraphSAGE-mean forward pass (Section II-A, Eq. (1); model of
 * Section IV).
 *
 * Conventions shared by every entry point
 *   - Pointers documented "device" are HIP device pointers; "host" are host
 *     pointers.  Device buffers are owned by the caller; the library never
 *     allocates or frees device memory, and keeps none but the fixed scratch
 *     array of gmb_sample_blocks_noalloc (a static device array).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     All device work of a call is enqueued on that stream; a call returns
 *     as soon as the work is enqueued, unless it says it synchronises.
 *   - Return value: GMB_OK (0) or a negative gmb_status.  Argument errors are
 *     detected on the host before anything is enqueued, so nothing runs and
 *     no buffer is touched.  Errors in the data (a vertex id out of range, a
 *     duplicated seed) are found on the device; they set bits of a sticky
 *     status word that gmb_read_status() returns.  Outputs produced under a
 *     data error are unspecified, but every access stays in bounds.
 *   - gmb_last_error() returns a thread-local message for the last failing
 *     call on this thread.
 *   - Layer numbering: model layer l = 0 is the input layer; fanouts[l]
 *     belongs to layer l, so the first hop (from the seeds) uses
 *     fanouts[L-1], and blocks are returned in layer order.
 *   - Vertex ids are int32 (graphs up to 2^31 - 1 vertices); CSR row offsets
 *     may be int32 or int64.
 */
#ifndef GMB_H
#define GMB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GMB_MAX_LAYERS 8
#define GMB_ABI_VERSION 1

typedef enum {
  GMB_OK = 0,
  GMB_EINVAL = -1,   /* bad argument (null pointer, bad size, unsupported shape) */
  GMB_ENOSPC = -2,   /* workspace or state buffer too small */
  GMB_EDEVICE = -3,  /* a HIP runtime call failed */
  GMB_ERANGE = -4,   /* (device) a vertex id outside [0, num_nodes) */
  GMB_EDUP = -5      /* (device) the seed list holds a vertex twice */
} gmb_status;

typedef enum { GMB_F32 = 0, GMB_BF16 = 1 } gmb_dtype;

/* Bits of the device status word. */
#define GMB_STATUS_ERANGE 1u
#define GMB_STATUS_EDUP 2u
#define GMB_STATUS_INTERNAL 4u   /* a bounded wait inside the relabel scan ran out */
#define GMB_STATUS_INVALID 8u    /* gmb_validate_blocks found an inconsistent block */

/* In-neighbour CSR of the input graph G(V, E) (Section II-A): row v lists
 * the sources u of the edges u -> v, so sampling row v samples the vertices
 * whose messages flow into v.  Rows must be sorted ascending and unique;
 * without that, sampled neighbour sets may hold duplicates.
 * All pointers are device pointers, read-only, owned by the caller. */
typedef struct {
  int64_t num_nodes;      /* |V|, 1 .. 2^31 - 1 */
  int64_t num_edges;      /* |E| = indptr[num_nodes] */
  const void* indptr;     /* [num_nodes + 1] int32 or int64 row offsets */
  int32_t indptr_bits;    /* 32 or 64 */
  int32_t reserved;
  const int32_t* indices; /* [num_edges] source vertex of each edge */
} gmb_csr;

/* One bipartite block of the sampled computation graph (Fig. 1(b)): the
 * messages of model layer l flow from the block's sources to its
 * destinations.  Filled in by gmb_sample_blocks with pointers into the
 * caller's workspace; sizes live on the device.
 *   indptr  [cap_dst + 1]  row offsets: edges of destination p are
 *                          [indptr[p], indptr[p+1]), k_p = min(deg, fanout)
 *   indices [cap_nnz]      local source id of each edge: a position in src_ids
 *   nbr     [cap_nnz]      the same edges as global vertex ids, each row in
 *                          ascending CSR-slot order
 *   src_ids [cap_src]      global ids of the sources; the first n_dst entries
 *                          are the destinations, in order, followed by the
 *                          new vertices in order of first appearance over
 *                          (destination position, slot).  All blocks of one
 *                          call share this array: block l uses its first
 *                          n_src(l) entries, and block 0's sources are the
 *                          input vertices whose features are gathered.
 *   sizes   [4]            device int32: n_dst, n_src, nnz, 0
 * cap_* are host-known upper bounds of the device-side sizes. */
typedef struct {
  int32_t* indptr;
  int32_t* indices;
  int32_t* nbr;
  int32_t* src_ids;
  int32_t* sizes;
  int64_t cap_dst, cap_src, cap_nnz;
  int32_t fanout;
  int32_t layer;
} gmb_block;

typedef struct {
  int32_t num_layers;
  int32_t num_seeds;
  gmb_block blk[GMB_MAX_LAYERS];   /* blk[l] = model layer l */
} gmb_blocks;

/* GraphSAGE-mean weights of an L-layer model (Section IV: 3 layers, hidden
 * 256).  Layer l maps dims[l] -> dims[l+1]:
 *   h_v' = act(h_v W_self[l] + mean_{u in sampled N(v)} h_u W_neigh[l] + bias[l])
 * with act = ReLU for l < L-1 and the identity for the last layer.
 * w_self[l], w_neigh[l]: device, [dims[l]][dims[l+1]] row-major, in `dtype`
 * (fp32, or bf16 bit patterns).  bias[l]: device, [dims[l+1]] fp32.  The
 * input features must have the same dtype as the matrices. */
typedef struct {
  int32_t num_layers;
  int32_t dtype;                       /* gmb_dtype */
  int32_t dims[GMB_MAX_LAYERS + 1];
  const void* w_self[GMB_MAX_LAYERS];
  const void* w_neigh[GMB_MAX_LAYERS];
  const float* bias[GMB_MAX_LAYERS];
} gmb_sage_weights;

/* ---- library ---------------------------------------------------------- */

/* GMB_ABI_VERSION of the loaded library. */
int32_t gmb_abi_version(void);

/* Message of the last failing call on this thread ("" if none). */
const char* gmb_last_error(void);

/* ---- sampler state ---------------------------------------------------- */

/* The sampler keeps one 32-bit slot per vertex (the dedup table of the
 * relabel step) plus a status word, in a caller-owned device buffer that
 * outlives calls: gmb_sampler_state_bytes() bytes for `num_nodes` vertices.
 * gmb_sampler_state_init() clears it (enqueued on `stream`); every
 * gmb_sample_blocks call leaves the table clear again.  One state serves
 * one call at a time: calls that share a state must be ordered on one
 * stream.  Returns 0 for num_nodes outside 1 .. 2^31 - 1. */
size_t gmb_sampler_state_bytes(int64_t num_nodes);
int gmb_sampler_state_init(void* state, size_t state_bytes, int64_t num_nodes, void* stream);

/* Device address of the state's status word (uint32, GMB_STATUS_* bits),
 * for passing to gmb_gather_features; NULL for a NULL state. */
uint32_t* gmb_state_status_word(void* state);

/* Synchronises `stream`, reads and clears the status word and returns the
 * matching status (GMB_ERANGE before GMB_EDUP before GMB_EDEVICE for
 * GMB_STATUS_INTERNAL or GMB_STATUS_INVALID), or GMB_OK.  After GMB_STATUS_INTERNAL it also
 * clears the state's table again (and synchronises once more), since the
 * failed call may have left slots behind. */
int gmb_read_status(void* state, void* stream);

/* ---- sampling (Section II-B, steps (i)-(ii), recursive per layer) ------- */

/* Bytes of workspace gmb_sample_blocks needs for these shapes (0 for bad
 * arguments). */
size_t gmb_sample_workspace_bytes(int32_t num_seeds, const int32_t* fanouts, int32_t num_layers,
                                  int64_t num_nodes);

/* Samples an L-layer mini-batch.
 *   seeds     device int32[num_seeds]: the target vertices, distinct, in
 *             [0, num_nodes) (a duplicate sets GMB_STATUS_EDUP, an id out of
 *             range GMB_STATUS_ERANGE).  num_seeds may be 0.
 *   fanouts   host int32[num_layers], each >= 1: at most fanouts[l]
 *             in-neighbours of each destination of layer l are picked,
 *             uniformly without replacement; a vertex with in-degree
 *             <= fanouts[l] keeps all of them.
 *   seed      64-bit key.  The sample of vertex v at layer l depends only on
 *             (seed, v, l) and the CSR row of v: Philox4x32-10 keyed by
 *             (lo32(seed), hi32(seed)) with counter (v, l, i, r) draws the
 *             i-th number of Floyd's algorithm by Lemire's
 *             multiply-and-reject on words x0..x3 of block r = 0, 1, ...
 *   state     the sampler state of this graph (see above).
 *   ws        device workspace of >= gmb_sample_workspace_bytes(...) bytes,
 *             256-byte aligned; the blocks point into it and stay valid
 *             until the workspace is reused.
 *   out       host struct filled with the blocks' pointers and capacities.
 * No host synchronisation: the sizes stay on the device (gmb_read_sizes). */
int gmb_sample_blocks(const gmb_csr* csr, const int32_t* seeds, int32_t num_seeds,
                      const int32_t* fanouts, int32_t num_layers, uint64_t seed,
                      void* state, size_t state_bytes, void* ws, size_t ws_bytes,
                      gmb_blocks* out, void* stream);

/* ---- sampling without allocation ---------------------------------------- */

/* Bytes of the fixed device scratch of gmb_sample_blocks_noalloc. */
#define GMB_NOALLOC_SCRATCH_BYTES (32u << 20)

/* For callers that cannot allocate device memory or cannot pass a
 * workspace: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  The same sampling as gmb_sample_blocks (same
 * kernels, the same blocks bit for bit), with the scratch that the call
 * needs besides its outputs (the relabel scans' look-back words and tickets,
 * the running edge counts, the dedup's routed pairs and answers) in a fixed
 * array of GMB_NOALLOC_SCRATCH_BYTES
 * that the library holds in device memory, one copy per GPU, from the first
 * call on that GPU until the process ends.  The call allocates nothing.
 *   out_buf    device buffer for the blocks, 256-byte aligned, caller-owned;
 *              gmb_sample_workspace_bytes(...) bytes for the same shapes
 *              always suffice (the blocks take its first part).  The blocks
 *              point into it and stay valid until it is reused.
 *   others     as for gmb_sample_blocks.
 * Errors: those of gmb_sample_blocks, and GMB_ENOSPC when the shapes need
 * more scratch than the fixed array holds (about 12 bytes per edge and per
 * destination of the last hop's capacity: 13 MB for 1000 seeds and fan-outs
 * 15, 10, 5); nothing is enqueued then.  The scratch is cleared by
 * the call's own first kernel.  Every call on one GPU shares that GPU's
 * array: calls that overlap in time on one GPU (other streams, other host
 * threads) race and give wrong blocks, so order them on one stream. */
int gmb_sample_blocks_noalloc(const gmb_csr* csr, const int32_t* seeds, int32_t num_seeds,
                              const int32_t* fanouts, int32_t num_layers, uint64_t seed,
                              void* state, size_t state_bytes, void* out_buf, size_t out_bytes,
                              gmb_blocks* out, void* stream);

/* Debug check of sampled blocks (run after every gmb_sample_blocks and
 * gmb_sample_blocks_noalloc call when the environment variable GMB_VALIDATE
 * is set to 1): enqueues on `stream` a device check of each block's
 * invariants (sizes within the capacities; row offsets rising from 0 to nnz
 * with at most `fanout` edges per row; every edge's local id below n_src and
 * naming the edge's sampled vertex in src_ids; every sampled vertex inside
 * the graph).  A violation sets GMB_STATUS_INVALID in the state's status
 * word, which gmb_read_status reports as GMB_EDEVICE.  The check reads only
 * within the blocks' capacities, whatever their size words hold.  It does
 * not check that src_ids is duplicate-free (the oracle tests do). */
int gmb_validate_blocks(const gmb_csr* csr, const gmb_blocks* blocks, void* state, void* stream);

/* Synchronises `stream` and copies the device sizes to host
 * sizes[num_layers][3] = {n_dst, n_src, nnz} (layer order). */
int gmb_read_sizes(const gmb_blocks* blocks, int64_t* sizes, void* stream);

/* ---- feature gather (KVStore pull, Section III-C) ---------------------- */

/* out[i, :] = feats[ids[i], :] bit for bit, for i < n, where n = *n_dev
 * (device int32, e.g. block 0's n_src) clamped to n_cap, or n = n_cap when
 * n_dev is NULL.  Rows at i >= n are not written.
 *   ids    device int32[n_cap]
 *   feats  device [num_nodes, dim] row-major, element size from dtype
 *   out    device [n_cap, dim]
 *   status device uint32 status word or NULL: an id outside [0, num_nodes)
 *          sets GMB_STATUS_ERANGE there and its output row is zero-filled. */
int gmb_gather_features(const int32_t* ids, const int32_t* n_dev, int64_t n_cap, const void* feats,
                        int64_t num_nodes, int32_t dim, int32_t dtype, void* out, uint32_t* status,
                        void* stream);

/* ---- GraphSAGE-mean forward (Eq. (1), Section IV model) ----------------- */

/* Bytes of workspace gmb_sage_forward needs (0 for bad arguments). */
size_t gmb_forward_workspace_bytes(const gmb_blocks* blocks, const gmb_sage_weights* weights);

/* Byte offset in the forward workspace of the output of layer l < L-1
 * (the hidden activations, [n_dst(l), dims[l+1]] in the weights' dtype);
 * -1 for a bad layer. */
int64_t gmb_forward_hidden_offset(const gmb_blocks* blocks, const gmb_sage_weights* weights,
                                  int32_t layer);

/* Runs the L layers over the blocks (the workspace keeps every layer's
 * mean and hidden output, which gmb_sage_backward reads).
 *   x       device [blocks->blk[0].cap_src, dims[0]] in weights->dtype: the
 *           gathered input features of block 0's sources (rows beyond
 *           n_src are not read).
 *   logits  device fp32 [num_seeds, dims[L]].
 *   ws      device workspace of >= gmb_forward_workspace_bytes() bytes,
 *           256-byte aligned.
 * Per layer: the mean of the sampled in-neighbours' rows (0 for a vertex
 * with none) accumulated in fp32, then the two products and the bias in
 * one matrix-core GEMM with fp32 accumulation.  In bf16 mode the mean and
 * the hidden activations are rounded to bf16 before the next product.
 * An empty batch (num_seeds == 0) has no rows in any layer: nothing is
 * enqueued, and x and logits may be NULL. */
int gmb_sage_forward(const gmb_blocks* blocks, const void* x, const gmb_sage_weights* weights,
                     float* logits, void* ws, size_t ws_bytes, void* stream);

/* The forward of gmb_sage_forward with the feature pull of Section III-C
 * folded into layer 0: instead of a gathered copy of every input row, the
 * layer-0 mean reads the sampled neighbours' rows straight from the feature
 * table by their global ids (block 0's nbr array), and only block 0's
 * destination rows, which its linear term h_v W_self needs, are gathered
 * into x_dst.  The results are bit for bit those of gmb_sage_forward on
 * the same blocks and weights (the same rows are summed in the same order).
 *   feats      device [num_nodes, dims[0]] in weights->dtype, read-only.
 *   num_nodes  rows of feats (1 .. 2^31 - 1).
 *   x_dst      device [blocks->blk[0].cap_dst, dims[0]] in weights->dtype,
 *              caller-owned, written with the destination rows; it stands
 *              for `x` in a later gmb_sage_backward (which reads layer 0's
 *              destination rows only).
 *   status     NULL or the sampler state's status word
 *              (gmb_state_status_word): an id outside [0, num_nodes) in
 *              the gather sets GMB_STATUS_ERANGE there and gives a zero row;
 *              in the mean it is read as row 0.
 *   others     as for gmb_sage_forward (same workspace size; with
 *              num_seeds == 0 nothing is enqueued and x_dst and logits
 *              may be NULL). */
int gmb_sage_forward_fused(const gmb_blocks* blocks, const void* feats, int64_t num_nodes, void* x_dst,
                           const gmb_sage_weights* weights, float* logits, void* ws, size_t ws_bytes,
                           uint32_t* status, void* stream);

/* ---- training step (the trainer's iteration of Section III-E) ---------- */

/* Gradient arrays of an L-layer model, one per weight array, fp32 and laid
 * out like the weights (d_self[l], d_neigh[l]: [dims[l]][dims[l+1]],
 * d_bias[l]: [dims[l+1]]).  Device pointers, caller-owned. */
typedef struct {
  int32_t num_layers;
  int32_t reserved;
  float* d_self[GMB_MAX_LAYERS];
  float* d_neigh[GMB_MAX_LAYERS];
  float* d_bias[GMB_MAX_LAYERS];
} gmb_sage_grads;

/* Bytes of workspace gmb_sage_backward needs (0 for bad arguments,
 * including a model the training step does not support: hidden dims not a
 * multiple of 4, a dims[l] above 640 for l >= 2).  For bf16 weights it
 * includes fp32 copies of what the backward reads. */
size_t gmb_backward_workspace_bytes(const gmb_blocks* blocks, const gmb_sage_weights* weights);

/* Gradients of the loss L = (1/B) sum over the B seeds of the softmax
 * cross-entropy of the seed's logits against its label, in every weight
 * and bias (the input features are not trained).  Node classification is
 * the task the paper trains (Section IV); its loss is not printed, this is
 * the standard one.  The backward follows Eq. (1) layer by layer from the
 * last: with dZ the gradient at a layer's pre-activation (ReLU passes it
 * where the layer's output is > 0), dW_self = H_dst^T dZ, dW_neigh = M^T dZ,
 * db = the column sums of dZ, and the layer input receives dZ W_self^T on
 * its destination rows plus, over every block edge (v <- u), its share
 * (dZ W_neigh^T)[v] / k_v of the mean.
 *   blocks, x, weights  as given to the gmb_sage_forward call that produced
 *                       `logits`, fp32 or bf16.  A bf16 model's backward
 *                       first widens block 0's destination rows of x, every
 *                       layer's kept mean and hidden output and the matrices
 *                       to fp32 (inside `ws`), then runs the fp32 backward
 *                       on them: fp32 products, fp32 gradients (update
 *                       with gmb_sgd_update_bf16).
 *   logits   device fp32 [num_seeds, dims[L]] from that call.
 *   labels   device int32 [num_seeds], the class of each seed in
 *            [0, dims[L]) (a label outside it is a data error: that row's
 *            loss term is 0 and its gradient unspecified, in bounds).
 *   fwd_ws   that call's workspace (it keeps every layer's mean and hidden
 *            output), unchanged since; fwd_ws_bytes its size.
 *   grads    where the gradients go (overwritten).
 *   loss     device fp32 scalar receiving L, or NULL.
 *   ws       device workspace of >= gmb_backward_workspace_bytes() bytes,
 *            256-byte aligned.
 * An empty batch (num_seeds == 0): the loss, a mean over no seeds, is
 * taken as 0, every gradient array is set to 0, and x, logits and labels
 * may be NULL.
 * Each weight gradient is summed over the rows in a fixed order (no
 * atomics), so the last layer's gradients are the same on every run.  The
 * gradient that flows into the input of layers >= 1 is pulled per source
 * vertex from a transpose of the block whose entries take their slots by
 * atomic counters, so each source's terms are summed in an order that can
 * change between runs, and the gradients of the layers below the last can
 * differ in their last bits.  The transpose's offsets come from a
 * single-pass scan whose tiles wait for their predecessors in a bounded
 * loop (about 4M short sleeps); only a GPU that stalls a running tile for
 * that long makes a wait give up, and then the input gradients of that
 * call are wrong (the call reports no status for it). */
int gmb_sage_backward(const gmb_blocks* blocks, const void* x, const gmb_sage_weights* weights,
                      const float* logits, const int32_t* labels, const void* fwd_ws, size_t fwd_ws_bytes,
                      const gmb_sage_grads* grads, float* loss, void* ws, size_t ws_bytes, void* stream);

/* ---- learnable vertex embeddings (Section III-C, Section III-E) -------- */

/* Bytes of workspace gmb_sage_backward_embedding needs (0 for bad arguments,
 * including a model it does not support: those of gmb_sage_backward, and
 * dims[0] or dims[1] breaking the same limits as the hidden widths). */
size_t gmb_backward_embedding_workspace_bytes(const gmb_blocks* blocks, const gmb_sage_weights* weights);

/* gmb_sage_backward for a model whose layer-0 inputs are learnable vertex
 * embeddings (the transductive case of Section III-C): besides the weight
 * gradients it takes the gradient in layer 0's input rows,
 * dX = dZ_0 W_self^T on the destination rows plus, over every block-0 edge
 * (v <- u), (dZ_0 W_neigh^T)[v] / k_v on row u (no activation acts on the
 * input), and applies it at once as the sparse SGD step of the paper's
 * embeddings (Section III-E): table[src_ids[u]] -= emb_lr * dX[u] for every
 * input vertex u of block 0.  dX is never stored.
 *   x          as for gmb_sage_backward: the gathered input rows (those
 *              of table), or x_dst of gmb_sage_forward_fused run on table.
 *   table      device fp32 [num_nodes, dims[0]], 16-byte aligned, updated
 *              in place (rows of vertices outside the mini-batch are not
 *              touched).
 *   emb_lr     the embeddings' step size.
 *   ws         >= gmb_backward_embedding_workspace_bytes() bytes.
 * The rows of one mini-batch are distinct, so the update needs no atomics;
 * calls in flight together on several streams update the shared table
 * without locks (asynchronous SGD as in Hogwild, as the paper updates its
 * embeddings), and a gather running meanwhile may see old or new rows.
 * An empty batch changes no row (the gradients and the loss as for
 * gmb_sage_backward). */
int gmb_sage_backward_embedding(const gmb_blocks* blocks, const void* x, const gmb_sage_weights* weights,
                                const float* logits, const int32_t* labels, const void* fwd_ws, size_t fwd_ws_bytes,
                                const gmb_sage_grads* grads, float* loss, void* ws, size_t ws_bytes, float* table,
                                int64_t num_nodes, float emb_lr, void* stream);

/* One SGD step: every weight array W -= lr * dW, every bias b -= lr * db,
 * in place on the device arrays that `weights` points to (fp32). */
int gmb_sgd_update(const gmb_sage_weights* weights, const gmb_sage_grads* grads, float lr, void* stream);

/* One SGD step of a bf16 model (the trainer's update of Section III-E with
 * the dense parameters kept in fp32): the fp32 master weights `master`
 * (same dims, dtype GMB_F32) take W -= lr * dW and b -= lr * db, then
 * every bf16 matrix of `weights` becomes its master rounded to the nearest
 * bf16 (ties to even), and each bias of `weights`, when it is not the
 * master's own array, a copy of the master's.  All device arrays,
 * caller-owned, updated in place on `stream`. */
int gmb_sgd_update_bf16(const gmb_sage_weights* weights, const gmb_sage_weights* master, const gmb_sage_grads* grads,
                        float lr, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GMB_H */
