"""Pins of the oracle's training step (O7): softmax cross-entropy, the
backward through the GraphSAGE-mean layers, and SGD.

Two references that share nothing with the oracle's backward formulas:
  - central finite differences of the loss (computed by the oracle's
    forward only) in every parameter, in fp64;
  - with every fan-out >= the maximum degree the mini-batch loss equals the
    loss of the dense full-graph model at the targets, as a function of the
    weights; torch autograd (fp64, CPU) differentiates the dense model.
"""
import numpy as np
import pytest
import torch


def _setup(orc, dg, dims, fanouts, n_seeds=12, n_nodes=2000, seed=3):
    g = dg.er_directed(n_nodes, 6.0, 50 + seed)
    w = dg.sage_weights(dims, 60 + seed)
    ws, wn, bs = w.as_f64()
    X = np.random.default_rng(seed).standard_normal((n_nodes, dims[0]))
    seeds = dg.permutation(n_nodes, 70 + seed)[:n_seeds]
    blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, 80 + seed)
    y = dg.labels(n_nodes, dims[-1], 90 + seed)[seeds]
    return g, blocks, X[blocks[0].src], ws, wn, bs, y, seeds, X


def _loss(orc, blocks, X0, ws, wn, bs, y):
    logits, _ = orc.sage_forward(blocks, X0, ws, wn, bs)
    return orc.softmax_xent(logits, y)[0]


def test_softmax_xent_value_and_gradient(orc):
    rng = np.random.default_rng(4)
    z = rng.standard_normal((7, 5)) * 3
    y = rng.integers(0, 5, 7)
    loss, dz = orc.softmax_xent(z, y)
    # the definition written out with numpy's logsumexp-free form
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    assert abs(loss - np.mean(-np.log(p[np.arange(7), y]))) < 1e-12
    h = 1e-6
    for i in range(7):
        for c in range(5):
            zp, zm = z.copy(), z.copy()
            zp[i, c] += h
            zm[i, c] -= h
            fd = (orc.softmax_xent(zp, y)[0] - orc.softmax_xent(zm, y)[0]) / (2 * h)
            assert abs(fd - dz[i, c]) < 1e-8
    # each row's gradient sums to zero
    assert np.allclose(dz.sum(axis=1), 0.0, atol=1e-15)


def test_backward_matches_finite_differences(orc, dg):
    """Every weight and bias entry of a three-layer model."""
    dims, fanouts = [5, 4, 4, 3], [2, 3, 2]
    g, blocks, X0, ws, wn, bs, y, _, _ = _setup(orc, dg, dims, fanouts)
    assert blocks[0].nnz > 0 and blocks[1].nnz > 0
    logits, hidden, means = orc.sage_forward_train(blocks, X0, ws, wn, bs)
    _, dz = orc.softmax_xent(logits, y)
    dWs, dWn, dbs = orc.sage_backward(blocks, X0, ws, wn, hidden, means, dz)
    h = 1e-6
    for l in range(len(dims) - 1):
        for name, P, G in (("W_self", ws, dWs), ("W_neigh", wn, dWn), ("b", bs, dbs)):
            it = np.nditer(P[l], flags=["multi_index"])
            for _ in it:
                idx = it.multi_index
                keep = P[l][idx]
                P[l][idx] = keep + h
                up = _loss(orc, blocks, X0, ws, wn, bs, y)
                P[l][idx] = keep - h
                dn = _loss(orc, blocks, X0, ws, wn, bs, y)
                P[l][idx] = keep
                fd = (up - dn) / (2 * h)
                scale = max(1.0, np.abs(G[l]).max())
                assert abs(fd - G[l][idx]) < 1e-6 * scale, (l, name, idx, fd, G[l][idx])


def _dense_loss_grads(g, X, ws, wn, bs, seeds, y):
    """Dense full-graph GraphSAGE-mean in torch, fp64; gradient of the mean
    cross-entropy at the seeds by autograd."""
    n = g.num_nodes
    A = torch.zeros((n, n), dtype=torch.float64)
    for v in range(n):
        row = g.indices[g.indptr[v]:g.indptr[v + 1]]
        if len(row):
            A[v, torch.from_numpy(row.astype(np.int64))] = 1.0 / len(row)
    params = []
    for l in range(len(ws)):
        params += [torch.tensor(ws[l], requires_grad=True), torch.tensor(wn[l], requires_grad=True),
                   torch.tensor(bs[l], requires_grad=True)]
    H = torch.from_numpy(X)
    L = len(ws)
    for l in range(L):
        Ws, Wn, b = params[3 * l:3 * l + 3]
        Z = H @ Ws + (A @ H) @ Wn + b
        H = torch.relu(Z) if l < L - 1 else Z
    loss = torch.nn.functional.cross_entropy(H[torch.from_numpy(seeds.astype(np.int64))],
                                             torch.from_numpy(y.astype(np.int64)))
    grads = torch.autograd.grad(loss, params)
    return loss.item(), [t.detach().numpy() for t in grads]


@pytest.mark.parametrize("L", [1, 2, 3])
def test_full_neighbourhood_gradients_equal_dense_autograd(orc, dg, L):
    g = dg.er_directed(300, 4.0, 11)
    fo = [int(g.degrees().max()) + 1] * L
    dims = [6] + [7] * (L - 1) + [4]
    w = dg.sage_weights(dims, 5)
    ws, wn, bs = w.as_f64()
    X = np.random.default_rng(1).standard_normal((300, 6))
    seeds = dg.permutation(300, 2)[:40]
    y = dg.labels(300, dims[-1], 9)[seeds]
    blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fo, 77)
    loss, logits, (dWs, dWn, dbs), _ = orc.sage_train_step(blocks, X[blocks[0].src], ws, wn, bs, y, 0.1)
    ref_loss, ref = _dense_loss_grads(g, X, ws, wn, bs, seeds, y)
    assert abs(loss - ref_loss) < 1e-12
    for l in range(L):
        for got, want in ((dWs[l], ref[3 * l]), (dWn[l], ref[3 * l + 1]), (dbs[l], ref[3 * l + 2])):
            assert np.allclose(got, want, rtol=1e-10, atol=1e-12), (l, np.abs(got - want).max())


def test_sgd_step(orc, dg):
    dims, fanouts = [5, 4, 3], [2, 3]
    g, blocks, X0, ws, wn, bs, y, _, _ = _setup(orc, dg, dims, fanouts)
    loss, _, (dWs, dWn, dbs), (nws, nwn, nbs) = orc.sage_train_step(blocks, X0, ws, wn, bs, y, 0.5)
    for l in range(2):
        assert np.array_equal(nws[l], ws[l] - 0.5 * dWs[l])
        assert np.array_equal(nwn[l], wn[l] - 0.5 * dWn[l])
        assert np.array_equal(nbs[l], bs[l] - 0.5 * dbs[l])
    # a small step along the negative gradient lowers the loss
    _, _, _, (sws, swn, sbs) = orc.sage_train_step(blocks, X0, ws, wn, bs, y, 1e-3)
    assert _loss(orc, blocks, X0, sws, swn, sbs, y) < loss


# ---- learnable vertex embeddings: the input-row gradient and its update ----

def test_input_gradient_matches_finite_differences(orc, dg):
    """Every entry of the layer-0 input rows of a three-layer model."""
    dims, fanouts = [5, 4, 4, 3], [2, 3, 2]
    g, blocks, X0, ws, wn, bs, y, _, _ = _setup(orc, dg, dims, fanouts)
    logits, hidden, means = orc.sage_forward_train(blocks, X0, ws, wn, bs)
    _, dz = orc.softmax_xent(logits, y)
    _, _, _, dX = orc.sage_backward(blocks, X0, ws, wn, hidden, means, dz, input_grad=True)
    assert dX.shape == X0.shape
    h = 1e-6
    scale = max(1.0, np.abs(dX).max())
    for idx in np.ndindex(*X0.shape):
        keep = X0[idx]
        X0[idx] = keep + h
        up = _loss(orc, blocks, X0, ws, wn, bs, y)
        X0[idx] = keep - h
        dn = _loss(orc, blocks, X0, ws, wn, bs, y)
        X0[idx] = keep
        fd = (up - dn) / (2 * h)
        assert abs(fd - dX[idx]) < 1e-6 * scale, (idx, fd, dX[idx])


@pytest.mark.parametrize("L", [1, 2, 3])
def test_input_gradient_equals_dense_autograd(orc, dg, L):
    """Full neighbourhoods: the gradient in the input rows equals torch
    autograd of the dense full-graph model in the feature matrix, at the
    rows of the sampled input vertices (every other row's gradient is 0)."""
    g = dg.er_directed(300, 4.0, 11)
    fo = [int(g.degrees().max()) + 1] * L
    dims = [6] + [7] * (L - 1) + [4]
    w = dg.sage_weights(dims, 5)
    ws, wn, bs = w.as_f64()
    X = np.random.default_rng(1).standard_normal((300, 6))
    seeds = dg.permutation(300, 2)[:40]
    y = dg.labels(300, dims[-1], 9)[seeds]
    blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fo, 77)
    _, _, dX, _, _ = orc.sage_train_step_embed(blocks, X, ws, wn, bs, y, 0.1, 0.1)
    n = g.num_nodes
    A = torch.zeros((n, n), dtype=torch.float64)
    for v in range(n):
        row = g.indices[g.indptr[v]:g.indptr[v + 1]]
        if len(row):
            A[v, torch.from_numpy(row.astype(np.int64))] = 1.0 / len(row)
    Xt = torch.tensor(X, requires_grad=True)
    H = Xt
    for l in range(L):
        Z = H @ torch.from_numpy(ws[l]) + (A @ H) @ torch.from_numpy(wn[l]) + torch.from_numpy(bs[l])
        H = torch.relu(Z) if l < L - 1 else Z
    loss = torch.nn.functional.cross_entropy(H[torch.from_numpy(seeds.astype(np.int64))],
                                             torch.from_numpy(y.astype(np.int64)))
    (gX,) = torch.autograd.grad(loss, [Xt])
    gX = gX.numpy()
    src = np.asarray(blocks[0].src, dtype=np.int64)
    assert np.allclose(dX, gX[src], rtol=1e-10, atol=1e-12), np.abs(dX - gX[src]).max()
    rest = np.setdiff1d(np.arange(n), src)
    assert np.abs(gX[rest]).max(initial=0.0) == 0.0


def test_embedding_sgd(orc, dg):
    rng = np.random.default_rng(5)
    table = rng.standard_normal((50, 6))
    rows = np.array([7, 3, 41, 0])
    dX = rng.standard_normal((4, 6))
    new = orc.embedding_sgd(table, rows, dX, 0.5)
    untouched = np.setdiff1d(np.arange(50), rows)
    assert np.array_equal(new[untouched], table[untouched])
    for i, r in enumerate(rows):
        assert np.array_equal(new[r], table[r] - 0.5 * dX[i])
    with pytest.raises(ValueError):
        orc.embedding_sgd(table, np.array([1, 1]), dX[:2], 0.5)
    # a small step on the embeddings (weights held) lowers the loss
    dims, fanouts = [5, 4, 3], [2, 3]
    g, blocks, X0, ws, wn, bs, y, seeds, Xall = _setup(orc, dg, dims, fanouts)
    loss0, _, _, _, tab = orc.sage_train_step_embed(blocks, Xall, ws, wn, bs, y, 0.0, 1e-2)
    X1 = tab[np.asarray(blocks[0].src, dtype=np.int64)]
    assert _loss(orc, blocks, X1, ws, wn, bs, y) < loss0
