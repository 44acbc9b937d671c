"""GPU parity of the training step (softmax cross-entropy, the backward
through the GraphSAGE-mean layers, SGD) against the oracle's fp64 step.

The ReLU mask is a decision taken on floating-point values, and an fp32
pre-activation within rounding of zero can fall on the other side of it than
the fp64 one.  These cases remove the ambiguity by making the forward exact
in fp32: integer features, weights and biases that are multiples of 1/16,
fan-outs that are powers of two with every in-degree 0 or >= the largest
fan-out (so every neighbour count is a power of two and every mean is
exact), and sizes for which every partial sum of a hidden layer stays below
2^24 times its granularity (asserted from the oracle's values).  The hidden
activations then agree bit for bit and so do the masks; the gradients differ
only by the rounding of the fp32 backward.

Tolerances: the loss within 1e-5 relative; every gradient array within 1e-4
of its largest magnitude (fp32 sums of at most a few thousand terms, split
into partial sums; the layer-input gradients sum each source's terms in
an order that atomic slot claims set anew each run); the SGD result within
lr * that error plus one fp32 rounding.
"""
import types

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU on this machine", allow_module_level=True)

import paper_2010_05337_amd as gmb  # noqa: E402
from gpu_util import (assert_blocks_equal, compare_train_step, csr_on_device, gpu_blocks, max_rel,  # noqa: E402
                      run_train_step, to_torch_weights)

from gpu_util import TOL_GRAD, bf16_bits, compare_train_step_bf16  # noqa: E402


def exact_graph(n, seed, min_deg=8, spread=9, broadcaster=None):
    """In-degree 0 for every 7th vertex, else min_deg .. min_deg+spread-1
    distinct sources (no self-loops).  With a broadcaster vertex b, b is
    one of the sources of every other non-empty row, so it is sampled by
    many destinations and its transpose list is long on every layer."""
    rng = np.random.default_rng(seed)
    deg = np.where(np.arange(n) % 7 == 0, 0, min_deg + rng.integers(0, spread, n))
    indptr = np.zeros(n + 1, dtype=np.int64)
    indptr[1:] = np.cumsum(deg)
    rows = []
    for v, d in enumerate(deg):
        u = rng.choice(n - 1, int(d), replace=False)
        u[u >= v] += 1
        if broadcaster is not None and d and v != broadcaster and broadcaster not in u:
            u[0] = broadcaster
        rows.append(np.sort(u))
    indices = np.concatenate(rows).astype(np.int32) if rows else np.zeros(0, np.int32)
    return types.SimpleNamespace(num_nodes=n, indptr=indptr, indices=indices)


def exact_model(dg, n, dims, seed):
    rng = np.random.default_rng(seed)
    feats = rng.integers(-2, 3, (n, dims[0])).astype(np.float32)
    ws, wn, bs = [], [], []
    for l in range(len(dims) - 1):
        ws.append((rng.integers(-2, 3, (dims[l], dims[l + 1])) / 16).astype(np.float32))
        wn.append((rng.integers(-2, 3, (dims[l], dims[l + 1])) / 16).astype(np.float32))
        bs.append((rng.integers(-2, 3, dims[l + 1]) / 16).astype(np.float32))
    return feats, dg.Weights(list(dims), ws, wn, bs, "f32")


def assert_hidden_exact(orc, ref_blocks, X, w):
    """Every partial sum of every hidden layer is a multiple of the layer's
    granularity below 2^24 times it, so fp32 computes it exactly in any
    order."""
    ws, wn, bs = w.as_f64()
    H, gran = X, 1.0
    for l, blk in enumerate(ref_blocks[:-1]):
        # the sums of up to 8 neighbour rows behind the mean
        assert np.abs(H).max(initial=0.0) * 8 < 2.0 ** 24 * gran, (l, np.abs(H).max())
        m = orc.mean_aggregate(blk, H)
        gran = gran / 8 / 16
        bound = np.abs(H[:blk.n_dst]) @ np.abs(ws[l]) + np.abs(m) @ np.abs(wn[l]) + np.abs(bs[l])
        assert bound.max(initial=0.0) < 2.0 ** 24 * gran, (l, bound.max(), gran)
        H = np.maximum(H[:blk.n_dst] @ ws[l] + m @ wn[l] + bs[l], 0.0)


CASES = [
    # dims, fan-outs, seeds
    ([16, 32, 8], [4, 2], 64),
    ([10, 12, 7], [8, 4], 37),             # ragged input width, 7 classes (padded dZ rows)
    ([24, 64, 640, 10], [2, 4, 8], 50),    # 640-wide hidden layer, three layers
    ([100, 256, 256, 47], [8, 4, 2], 200), # the benchmark model's widths
    ([12, 5], [4], 33),                    # one layer: no ReLU, no input gradient
    ([8, 16, 4], [2, 2], 1),               # one seed
]


@pytest.mark.parametrize("dims,fanouts,n_seeds", CASES)
def test_train_step_matches_the_oracle(orc, dg, dims, fanouts, n_seeds):
    n = 3000
    g = exact_graph(n, 11 + len(dims))
    feats, w = exact_model(dg, n, dims, 12 + dims[1])
    seeds = dg.permutation(n, 13)[:n_seeds]
    labels = dg.labels(n, dims[-1], 14)[seeds]
    key, lr = 15, 0.25
    print(f"dims {dims} fan-outs {fanouts} seeds {n_seeds}", flush=True)
    csr = csr_on_device(g)
    wt = to_torch_weights(w)
    ft = torch.from_numpy(feats).cuda()
    out = run_train_step(csr, seeds, fanouts, key, ft, wt, labels, lr)
    ref_blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, key)
    assert_blocks_equal(out["host"], ref_blocks)
    X = orc.gather(feats, ref_blocks[0].src).astype(np.float64)
    assert_hidden_exact(orc, ref_blocks, X, w)
    compare_train_step(orc, out, ref_blocks, X, w, labels, lr, wt, exact_hidden=True)
    csr.check_status()


@pytest.mark.parametrize("dims,fanouts,n_seeds", [([16, 32, 32, 6], [4, 4, 8], 120),
                                                  ([100, 47], [8], 600)])
def test_repeated_backward(orc, dg, dims, fanouts, n_seeds):
    """The last layer's gradients are summed in a fixed order: identical bits
    on every run; the layers below take the fp32 atomic adds of the mean's
    backward and agree within the tolerance.  The one-layer case puts the
    last layer's products in a launch of their own (the part-product weight
    gradient: two column tiles, several row ranges)."""
    n = 3000
    g = exact_graph(n, 21)
    feats, w = exact_model(dg, n, dims, 22)
    seeds = dg.permutation(n, 23)[:n_seeds]
    labels = torch.from_numpy(dg.labels(n, dims[-1], 24)[seeds]).cuda()
    csr = csr_on_device(g)
    wt = to_torch_weights(w)
    ft = torch.from_numpy(feats).cuda()
    blocks, _ = gpu_blocks(csr, seeds, fanouts, 25)
    x = gmb.gather_features(blocks, ft)
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), ft.device)[1]
    logits = gmb.sage_forward(blocks, x, wt, workspace=ws_fwd)
    g1, l1 = gmb.sage_backward(blocks, x, wt, logits, labels, ws_fwd)
    first = [[t.clone() for t in a] for a in (g1.d_self, g1.d_neigh, g1.d_bias)]
    g2, l2 = gmb.sage_backward(blocks, x, wt, logits, labels, ws_fwd)
    assert torch.equal(l1, l2)
    L = len(dims) - 1
    for a, b in zip(first, (g2.d_self, g2.d_neigh, g2.d_bias)):
        assert torch.equal(a[L - 1], b[L - 1])
        for l in range(L - 1):
            assert max_rel(b[l].cpu().numpy(), a[l].cpu().numpy().astype(np.float64)) <= TOL_GRAD


def test_sgd_steps_lower_the_loss(dg):
    """Five GPU training steps on one batch of Gaussian data: the loss goes
    down at every step."""
    n, dims, fanouts = 10000, [32, 64, 64, 10], [5, 10, 15]
    g = dg.er_directed(n, 12.0, 31)
    feats = dg.features(n, dims[0], 32, "f32")
    w = dg.sage_weights(dims, 33)
    seeds = dg.permutation(n, 34)[:256]
    labels = torch.from_numpy(dg.labels(n, dims[-1], 35)[seeds]).cuda()
    csr = csr_on_device(g)
    wt = to_torch_weights(w)
    ft = torch.from_numpy(feats).cuda()
    blocks, _ = gpu_blocks(csr, seeds, fanouts, 36)
    x = gmb.gather_features(blocks, ft)
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), ft.device)[1]
    losses = []
    for _ in range(6):
        logits = gmb.sage_forward(blocks, x, wt, workspace=ws_fwd)
        grads, loss = gmb.sage_backward(blocks, x, wt, logits, labels, ws_fwd)
        gmb.sgd_update(wt, grads, 0.5)
        losses.append(float(loss.item()))
    print("losses", losses, flush=True)
    assert all(b < a for a, b in zip(losses, losses[1:])), losses


def test_backward_rejects_unsupported_models(dg):
    """Hidden widths that are not a multiple of 4 are refused before any
    launch, and so are learnable embeddings with bf16 weights; the bf16
    backward itself is accepted."""
    n = 2000
    g = dg.er_directed(n, 8.0, 41)
    csr = csr_on_device(g)
    seeds = dg.permutation(n, 42)[:16]
    blocks, _ = gpu_blocks(csr, seeds, [3, 3], 43)
    labels = torch.zeros(16, dtype=torch.int32, device="cuda")
    for dims, dtype in (([8, 6, 4], "f32"), ([8, 8, 4], "bf16")):
        w = dg.sage_weights(dims, 44, dtype)
        wt = to_torch_weights(w)
        ft = torch.from_numpy(dg.features(n, dims[0], 45, dtype).view(np.int16) if dtype == "bf16"
                              else dg.features(n, dims[0], 45, dtype)).cuda()
        if dtype == "bf16":
            ft = ft.view(torch.bfloat16)
        x = gmb.gather_features(blocks, ft)
        ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), ft.device)[1]
        logits = gmb.sage_forward(blocks, x, wt, workspace=ws_fwd)
        if dtype == "bf16":
            assert gmb.backward_workspace_bytes(blocks, wt) > 0
            assert gmb.backward_embedding_workspace_bytes(blocks, wt) == 0
            continue
        assert gmb.backward_workspace_bytes(blocks, wt) == 0
        with pytest.raises(gmb.GmbError):
            gmb.sage_backward(blocks, x, wt, logits, labels, ws_fwd)


def test_train_step_on_fused_forward(orc, dg):
    """The training step fed by the fused forward: x_dst (block 0's
    destination rows) stands for the gathered input in the backward."""
    n, dims, fanouts, n_seeds = 3000, [24, 32, 32, 6], [4, 2, 8], 90
    g = exact_graph(n, 71)
    feats, w = exact_model(dg, n, dims, 72)
    seeds = dg.permutation(n, 73)[:n_seeds]
    labels = dg.labels(n, dims[-1], 74)[seeds]
    csr = csr_on_device(g)
    wt = to_torch_weights(w)
    ft = torch.from_numpy(feats).cuda()
    blocks, host = gpu_blocks(csr, seeds, fanouts, 75)
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), ft.device)[1]
    logits, x_dst, hidden = gmb.sage_forward_fused(blocks, ft, wt, workspace=ws_fwd, return_hidden=True)
    y = torch.from_numpy(labels).cuda()
    grads, loss = gmb.sage_backward(blocks, x_dst, wt, logits, y, ws_fwd)
    before = [[t.clone() for t in arrs] for arrs in (wt.w_self, wt.w_neigh, wt.bias)]
    gmb.sgd_update(wt, grads, 0.25)
    torch.cuda.synchronize()
    ref_blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, 75)
    assert_blocks_equal(host, ref_blocks)
    X = orc.gather(feats, ref_blocks[0].src).astype(np.float64)
    assert_hidden_exact(orc, ref_blocks, X, w)
    out = dict(hidden=hidden, grads=grads, loss=float(loss.item()), before=before)
    compare_train_step(orc, out, ref_blocks, X, w, labels, 0.25, wt, exact_hidden=True)
    csr.check_status()


# ---- learnable vertex embeddings ---------------------------------------------

def check_embedding_update(orc, table_before, table_after, ref_blocks, ref_table, dX, emb_lr):
    """Rows of the batch's input vertices against the oracle's update; every
    other row untouched, bit for bit."""
    got = table_after.cpu().numpy()
    before = table_before.cpu().numpy()
    src = np.asarray(ref_blocks[0].src, dtype=np.int64)
    rest = np.ones(len(before), dtype=bool)
    rest[src] = False
    assert np.array_equal(got[rest], before[rest]), "rows outside the mini-batch changed"
    want = ref_table[src]
    bound = emb_lr * TOL_GRAD * max(np.abs(dX).max(), 1e-30) + 2.0 ** -23 * np.abs(want).max()
    err = np.abs(got[src].astype(np.float64) - want).max()
    print(f"embedding rows: {len(src)} updated, max error {err:.2e} (bound {bound:.2e})", flush=True)
    assert err <= bound, (err, bound)
    assert np.abs(dX).max() == 0.0 or not np.array_equal(got[src], before[src])


@pytest.mark.parametrize("dims,fanouts,n_seeds,fused", [([16, 32, 8], [4, 2], 64, False),
                                                         ([24, 64, 640, 10], [2, 4, 8], 50, True),
                                                         ([100, 256, 256, 47], [8, 4, 2], 200, False),
                                                         ([100, 256, 256, 47], [8, 4, 2], 200, True),
                                                         ([12, 5], [4], 33, True)])
def test_embedding_train_step_matches_the_oracle(orc, dg, dims, fanouts, n_seeds, fused):
    """Inputs are learnable vertex embeddings: the weight gradients, the loss
    and the sparse update of the table rows against the oracle, through the
    gathered or the fused forward."""
    n = 3000
    g = exact_graph(n, 81 + len(dims))
    table_np, w = exact_model(dg, n, dims, 82 + dims[1])
    seeds = dg.permutation(n, 83)[:n_seeds]
    labels = dg.labels(n, dims[-1], 84)[seeds]
    key, lr, emb_lr = 85, 0.25, 0.5
    print(f"dims {dims} fan-outs {fanouts} seeds {n_seeds} fused {fused}", flush=True)
    csr = csr_on_device(g)
    wt = to_torch_weights(w)
    table = torch.from_numpy(table_np.copy()).cuda()
    blocks, host = gpu_blocks(csr, seeds, fanouts, key)
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), table.device)[1]
    if fused:
        logits, x, hidden = gmb.sage_forward_fused(blocks, table, wt, workspace=ws_fwd, return_hidden=True)
    else:
        x = gmb.gather_features(blocks, table)
        logits, hidden = gmb.sage_forward(blocks, x, wt, workspace=ws_fwd, return_hidden=True)
    table_before = table.clone()
    y = torch.from_numpy(labels).cuda()
    grads, loss = gmb.sage_backward(blocks, x, wt, logits, y, ws_fwd, embedding=table, emb_lr=emb_lr)
    before = [[t.clone() for t in arrs] for arrs in (wt.w_self, wt.w_neigh, wt.bias)]
    gmb.sgd_update(wt, grads, lr)
    torch.cuda.synchronize()
    ref_blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, key)
    assert_blocks_equal(host, ref_blocks)
    X = table_np[np.asarray(ref_blocks[0].src, dtype=np.int64)].astype(np.float64)
    assert_hidden_exact(orc, ref_blocks, X, w)
    out = dict(hidden=hidden, grads=grads, loss=float(loss.item()), before=before)
    compare_train_step(orc, out, ref_blocks, X, w, labels, lr, wt, exact_hidden=True)
    ws, wn, bs = w.as_f64()
    _, _, dX, _, ref_table = orc.sage_train_step_embed(ref_blocks, table_np.astype(np.float64), ws, wn, bs, labels,
                                                        lr, emb_lr)
    check_embedding_update(orc, table_before, table, ref_blocks, ref_table, dX, emb_lr)
    csr.check_status()


def test_embedding_backward_rejects_unsupported(dg):
    """An input width that is not a multiple of 4 is refused before any
    launch."""
    n = 2000
    g = dg.er_directed(n, 8.0, 91)
    csr = csr_on_device(g)
    seeds = dg.permutation(n, 92)[:16]
    blocks, _ = gpu_blocks(csr, seeds, [3, 3], 93)
    w = dg.sage_weights([10, 8, 4], 94)
    wt = to_torch_weights(w)
    table = torch.from_numpy(dg.features(n, 10, 95, "f32")).cuda()
    x = gmb.gather_features(blocks, table)
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), table.device)[1]
    logits = gmb.sage_forward(blocks, x, wt, workspace=ws_fwd)
    labels = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(gmb.GmbError):
        gmb.sage_backward(blocks, x, wt, logits, labels, ws_fwd, embedding=table, emb_lr=0.1)


@pytest.mark.parametrize("embed", [False, True])
def test_long_transpose_lists(orc, dg, embed):
    """A broadcaster vertex sampled by hundreds of destinations on every
    layer: its transpose lists take the workgroup-per-row kernel (the masked
    pull on the hidden layers, the table update on layer 0)."""
    n, dims, fanouts, n_seeds = 3000, [16, 32, 32, 6], [4, 8, 4], 400
    g = exact_graph(n, 101, broadcaster=5)
    table_np, w = exact_model(dg, n, dims, 102)
    seeds = dg.permutation(n, 103)[:n_seeds]
    seeds = seeds[seeds != 5]
    labels = dg.labels(n, dims[-1], 104)[seeds]
    lr, emb_lr = 0.25, 0.5
    csr = csr_on_device(g)
    wt = to_torch_weights(w)
    table = torch.from_numpy(table_np.copy()).cuda()
    blocks, host = gpu_blocks(csr, seeds, fanouts, 105)
    for l, h in enumerate(host):
        k = int((h["nbr"] == 5).sum())
        print(f"layer {l}: the broadcaster is sampled {k} times", flush=True)
        assert k > 16
    x = gmb.gather_features(blocks, table)
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), table.device)[1]
    logits, hidden = gmb.sage_forward(blocks, x, wt, workspace=ws_fwd, return_hidden=True)
    table_before = table.clone()
    y = torch.from_numpy(labels).cuda()
    kw = dict(embedding=table, emb_lr=emb_lr) if embed else {}
    grads, loss = gmb.sage_backward(blocks, x, wt, logits, y, ws_fwd, **kw)
    before = [[t.clone() for t in arrs] for arrs in (wt.w_self, wt.w_neigh, wt.bias)]
    gmb.sgd_update(wt, grads, lr)
    torch.cuda.synchronize()
    ref_blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, 105)
    assert_blocks_equal(host, ref_blocks)
    X = table_np[np.asarray(ref_blocks[0].src, dtype=np.int64)].astype(np.float64)
    assert_hidden_exact(orc, ref_blocks, X, w)
    out = dict(hidden=hidden, grads=grads, loss=float(loss.item()), before=before)
    compare_train_step(orc, out, ref_blocks, X, w, labels, lr, wt, exact_hidden=True)
    if embed:
        ws, wn, bs = w.as_f64()
        _, _, dX, _, ref_table = orc.sage_train_step_embed(ref_blocks, table_np.astype(np.float64), ws, wn, bs,
                                                            labels, lr, emb_lr)
        check_embedding_update(orc, table_before, table, ref_blocks, ref_table, dX, emb_lr)
    csr.check_status()


def test_empty_batch(dg):
    """No seeds: the forwards leave no rows, the backward writes a zero loss
    and zero gradients (the mean over no seeds taken as 0) over arrays that
    held other values, and the embedding step changes no table row."""
    g = dg.er_directed(2000, 6.0, 5)
    csr = csr_on_device(g)
    X = dg.features(2000, 12, 6, "f32")
    ft = torch.from_numpy(X).cuda()
    wt = to_torch_weights(dg.sage_weights([12, 8, 5], 7))
    blocks, host = gpu_blocks(csr, np.zeros(0, dtype=np.int64), [3, 4], 8)
    assert all(h["n_dst"] == 0 and h["n_src"] == 0 and h["nnz"] == 0 for h in host)
    x = gmb.gather_features(blocks, ft)
    ws = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), ft.device)[1]
    logits = gmb.sage_forward(blocks, x, wt, workspace=ws)
    assert tuple(logits.shape) == (0, 5)
    labels = torch.zeros(0, dtype=torch.int32, device="cuda")
    for embedding in (None, ft.clone()):
        grads = gmb.SageGrads(wt)
        for a in grads.d_self + grads.d_neigh + grads.d_bias:
            a.fill_(7.0)
        loss = torch.full((1,), 7.0, dtype=torch.float32, device="cuda")
        before = None if embedding is None else embedding.clone()
        grads, loss = gmb.sage_backward(blocks, x, wt, logits, labels, ws, grads=grads, loss=loss,
                                        embedding=embedding, emb_lr=0.5)
        torch.cuda.synchronize()
        assert float(loss.item()) == 0.0
        for a in grads.d_self + grads.d_neigh + grads.d_bias:
            assert bool((a == 0).all())
        if embedding is not None:
            assert torch.equal(embedding, before)
    logits_f, x_dst = gmb.sage_forward_fused(blocks, ft, wt, workspace=ws)
    assert tuple(logits_f.shape) == (0, 5) and x_dst.shape[0] == 0
    csr.check_status()



@pytest.mark.parametrize("dims,fanouts,n_seeds", [([16, 32, 8], [4, 2], 64), ([128, 256, 47], [8, 4], 150),
                                                  ([24, 64, 32, 12], [2, 4, 8], 50)])
def test_bf16_train_step_matches_the_oracle(orc, dg, dims, fanouts, n_seeds):
    """A bf16 model (bf16 features and matrices, exact in bf16: integers and
    multiples of 1/16) trains through fp32 copies and fp32 master weights:
    loss and gradients against the oracle's fp64 step within 2e-2, the
    update exact on the masters, the bf16 matrices their rounding.  The
    hidden biases keep every pre-activation far from zero, so that the bf16
    rounding of the hidden layers cannot flip a ReLU."""
    import types
    from gpu_util import margin_biases
    n = 3000
    g = exact_graph(n, 51 + len(dims))
    feats32, w32 = exact_model(dg, n, dims, 52 + dims[1])
    seeds = dg.permutation(n, 53)[:n_seeds]
    labels = dg.labels(n, dims[-1], 54)[seeds]
    key, lr = 55, 0.25
    ref_blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, key)
    X = orc.gather(feats32, ref_blocks[0].src).astype(np.float64)
    w = types.SimpleNamespace(dims=list(dims), w_self=[bf16_bits(a) for a in w32.w_self],
                              w_neigh=[bf16_bits(a) for a in w32.w_neigh], bias=w32.bias, dtype="bf16")
    w.bias = margin_biases(orc, ref_blocks, X, types.SimpleNamespace(
        bias=w32.bias, as_f64=lambda: w32.as_f64()))
    w.as_f64 = lambda: ([a.astype(np.float64) for a in w32.w_self], [a.astype(np.float64) for a in w32.w_neigh],
                        [b.astype(np.float64) for b in w.bias])
    print(f"bf16 training: dims {dims} fan-outs {fanouts} seeds {n_seeds}", flush=True)
    csr = csr_on_device(g)
    wt = to_torch_weights(w)
    master = wt.master()
    ft = torch.from_numpy(bf16_bits(feats32).view(np.int16)).cuda().view(torch.bfloat16)
    blocks, host = gpu_blocks(csr, seeds, fanouts, key)
    assert_blocks_equal(host, ref_blocks)
    x = gmb.gather_features(blocks, ft)
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), ft.device)[1]
    logits = gmb.sage_forward(blocks, x, wt, workspace=ws_fwd)
    y = torch.from_numpy(labels).cuda()
    grads, loss = gmb.sage_backward(blocks, x, wt, logits, y, ws_fwd)
    before = [[t.clone() for t in arrs] for arrs in (master.w_self, master.w_neigh, master.bias)]
    gmb.sgd_update_bf16(wt, master, grads, lr)
    torch.cuda.synchronize()
    compare_train_step_bf16(orc, float(loss.item()), grads, ref_blocks, X, w, labels, lr, before, master, wt)
    csr.check_status()


def test_bf16_sgd_steps_lower_the_loss(dg):
    """Five bf16 training steps on one batch of Gaussian data: the loss goes
    down at every step."""
    n, dims, fanouts = 10000, [32, 64, 64, 10], [5, 10, 15]
    g = dg.er_directed(n, 12.0, 61)
    feats = dg.features(n, dims[0], 62, "bf16")
    w = dg.sage_weights(dims, 63, "bf16")
    seeds = dg.permutation(n, 64)[:256]
    labels = torch.from_numpy(dg.labels(n, dims[-1], 65)[seeds]).cuda()
    csr = csr_on_device(g)
    wt = to_torch_weights(w)
    master = wt.master()
    ft = torch.from_numpy(feats.view(np.int16)).cuda().view(torch.bfloat16)
    blocks, _ = gpu_blocks(csr, seeds, fanouts, 66)
    x = gmb.gather_features(blocks, ft)
    ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(blocks, wt), ft.device)[1]
    losses = []
    for _ in range(6):
        logits = gmb.sage_forward(blocks, x, wt, workspace=ws_fwd)
        grads, loss = gmb.sage_backward(blocks, x, wt, logits, labels, ws_fwd)
        gmb.sgd_update_bf16(wt, master, grads, 0.5)
        losses.append(float(loss.item()))
    print("bf16 losses", losses, flush=True)
    assert all(b < a for a, b in zip(losses, losses[1:])), losses
