"""Pins of the oracle's block construction, gather and GraphSAGE forward
(CPU only)."""
import numpy as np
import pytest


def check_blocks(g, seeds, fanouts, blocks, orc=None, seed=None):
    """Invariants that hold for any correct sample + relabel; together the
    relabel ones determine src and local uniquely from nbr."""
    L = len(fanouts)
    dst = np.asarray(seeds, dtype=np.int64)
    for hop in range(L):
        l = L - 1 - hop
        b = blocks[l]
        f = fanouts[l]
        assert b.n_dst == len(dst)
        assert np.array_equal(b.src[:b.n_dst], dst)
        deg = g.indptr[dst + 1] - g.indptr[dst]
        assert np.array_equal(np.diff(b.indptr), np.minimum(deg, f))
        for p in range(b.n_dst):
            row = b.nbr[b.indptr[p]:b.indptr[p + 1]]
            true = g.indices[g.indptr[dst[p]]:g.indptr[dst[p] + 1]]
            assert np.all(np.isin(row, true))          # subset of true in-neighbours
            assert np.all(np.diff(row) > 0)           # distinct, ascending slot order
            if orc is not None:
                slots = orc.sample_node(seed, int(dst[p]), l, len(true), f)
                assert np.array_equal(row, true[slots])
        # relabel
        assert b.nnz == 0 or (b.local.min() >= 0 and b.local.max() < b.n_src)
        assert np.array_equal(b.src[b.local], b.nbr)          # round trip local -> global
        assert len(np.unique(b.src)) == b.n_src               # distinct
        new = b.src[b.n_dst:]
        first = {}
        for e, u in enumerate(b.nbr):
            first.setdefault(int(u), e)
        assert all(int(u) in first for u in new)               # every new node is sampled
        pos = [first[int(u)] for u in new]
        assert np.all(np.diff(pos) > 0)                        # first-appearance order
        assert not np.any(np.isin(new, dst))
        missing = set(int(u) for u in b.nbr) - set(int(u) for u in b.src)
        assert not missing
        dst = b.src
    return True


@pytest.fixture(scope="module")
def tiny(dg):
    return dg.er_directed(10000, 10.0, 101)


def test_tiny_blocks_invariants(orc, dg, tiny):
    seeds = dg.permutation(10000, 104)[:64]
    blocks = orc.sample_blocks(tiny.indptr, tiny.indices, seeds, [5, 5], 105)
    check_blocks(tiny, seeds, [5, 5], blocks, orc, 105)


def test_rmat_blocks_invariants_with_hubs(orc, dg):
    g = dg.rmat(14, 12000, 150000, (0.57, 0.19, 0.19), 7)
    assert g.degrees().max() > 200
    hubs = np.argsort(-g.degrees())[:20]
    seeds = np.concatenate([hubs, dg.permutation(12000, 8)[:300]])
    seeds = seeds[np.sort(np.unique(seeds, return_index=True)[1])]
    fo = [15, 10, 5]
    blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fo, 99)
    check_blocks(g, seeds, fo, blocks, orc, 99)


def test_block_degree_cases(orc):
    # star-ish graph: node 0 has in-degree 0, node 1 degree 3, node 2 degree 5,
    # node 3 degree 9 (fan-out 5 => < f, = f, > f and 0).
    rows = {0: [], 1: [4, 5, 6], 2: [4, 5, 6, 7, 8], 3: [4, 5, 6, 7, 8, 9, 10, 11, 12]}
    n = 13
    indptr = [0]
    indices = []
    for v in range(n):
        indices += rows.get(v, [])
        indptr.append(len(indices))
    indptr, indices = np.array(indptr), np.array(indices, dtype=np.int32)

    class G:
        pass
    g = G()
    g.indptr, g.indices = indptr, indices
    blocks = orc.sample_blocks(indptr, indices, [0, 1, 2, 3], [5], 3)
    b = blocks[0]
    assert list(np.diff(b.indptr)) == [0, 3, 5, 5]
    check_blocks(g, [0, 1, 2, 3], [5], blocks, orc, 3)
    # the empty mini-batch
    e = orc.sample_blocks(indptr, indices, [], [5, 5], 3)
    assert all(x.n_dst == 0 and x.nnz == 0 and x.n_src == 0 for x in e)


def test_samples_independent_of_batch_composition(orc, dg, tiny):
    """A node's sample depends only on (key, node, layer), not on the other
    targets in the mini-batch, so dedup changes no output value."""
    a_seeds = dg.permutation(10000, 1)[:50]
    b_seeds = np.concatenate([a_seeds[25:], dg.permutation(10000, 2)[:40]])
    b_seeds = b_seeds[np.sort(np.unique(b_seeds, return_index=True)[1])]
    A = orc.sample_blocks(tiny.indptr, tiny.indices, a_seeds, [5, 5], 42)
    B = orc.sample_blocks(tiny.indptr, tiny.indices, b_seeds, [5, 5], 42)
    for l in range(2):
        rows_a = {int(A[l].src[p]): tuple(A[l].nbr[A[l].indptr[p]:A[l].indptr[p + 1]])
                  for p in range(A[l].n_dst)}
        rows_b = {int(B[l].src[p]): tuple(B[l].nbr[B[l].indptr[p]:B[l].indptr[p + 1]])
                  for p in range(B[l].n_dst)}
        common = set(rows_a) & set(rows_b)
        assert len(common) > 10
        for v in common:
            assert rows_a[v] == rows_b[v]
    C = orc.sample_blocks(tiny.indptr, tiny.indices, a_seeds, [5, 5], 43)
    assert not np.array_equal(A[1].nbr, C[1].nbr)


def test_error_statuses(orc, tiny):
    with pytest.raises(orc.OracleError) as e:
        orc.sample_blocks(tiny.indptr, tiny.indices, [1, 2, 10000], [5], 1)
    assert e.value.code == -4
    with pytest.raises(orc.OracleError) as e:
        orc.sample_blocks(tiny.indptr, tiny.indices, [1, 2, 1], [5], 1)
    assert e.value.code == -5
    with pytest.raises(orc.OracleError) as e:
        orc.sample_blocks(tiny.indptr, tiny.indices, [1, 2], [5, 0], 1)
    assert e.value.code == -1


def test_gather_is_a_bit_copy(orc, dg):
    f32 = dg.features(500, 16, 9, "f32")
    b16 = dg.features(500, 128, 9, "bf16")
    ids = np.array([3, 499, 0, 3, 250], dtype=np.int64)
    assert np.array_equal(orc.gather(f32, ids).view(np.uint32), f32[ids].view(np.uint32))
    assert np.array_equal(orc.gather(b16, ids), b16[ids])
    with pytest.raises(orc.OracleError):
        orc.gather(f32, [500])
    # rows that carry their own index: entry (r, c) = r * 16 + c, exact in
    # fp32, so every gathered row decodes to the id it was asked for
    own = np.arange(500 * 16, dtype=np.float32).reshape(500, 16)
    got = orc.gather(own, ids)
    assert np.array_equal(got[:, 0].astype(np.int64) // 16, ids)
    assert np.array_equal(got - got[:, :1], np.tile(np.arange(16, dtype=np.float32), (len(ids), 1)))


def test_mean_aggregate_matches_dense(orc, dg, tiny):
    seeds = dg.permutation(10000, 3)[:64]
    blocks = orc.sample_blocks(tiny.indptr, tiny.indices, seeds, [5, 5], 7)
    rng = np.random.default_rng(0)
    for b in blocks:
        H = rng.standard_normal((b.n_src, 12))
        A = np.zeros((b.n_dst, b.n_src))
        for p in range(b.n_dst):
            k = b.indptr[p + 1] - b.indptr[p]
            for e in range(b.indptr[p], b.indptr[p + 1]):
                A[p, b.local[e]] += 1.0 / k
        want = A @ H
        got = orc.mean_aggregate(b, H)
        assert np.allclose(got, want, rtol=1e-12, atol=1e-12)
        zero_rows = np.diff(b.indptr) == 0
        assert np.all(got[zero_rows] == 0.0)


def _dense_sage(indptr, indices, X, ws, wn, bs):
    n = len(indptr) - 1
    A = np.zeros((n, n))
    for v in range(n):
        nb = indices[indptr[v]:indptr[v + 1]]
        if len(nb):
            A[v, nb] = 1.0 / len(nb)
    H = X
    outs = []
    for l in range(len(ws)):
        Z = H @ ws[l] + (A @ H) @ wn[l] + bs[l]
        H = np.maximum(Z, 0.0) if l < len(ws) - 1 else Z
        outs.append(H)
    return outs


@pytest.mark.parametrize("L", [1, 2, 3])
def test_full_neighbourhood_equals_dense_sage(orc, dg, L):
    """With every fan-out >= the maximum degree, the mini-batch forward at
    the targets equals the full-graph dense GraphSAGE-mean forward
    H' = act(H W_self + D^-1 A H W_neigh + b), restricted to the targets."""
    g = dg.er_directed(300, 4.0, 11)
    fo = [int(g.degrees().max()) + 1] * L
    dims = [6] + [7] * (L - 1) + [3]
    w = dg.sage_weights(dims, 5)
    ws, wn, bs = w.as_f64()
    X = np.random.default_rng(1).standard_normal((300, 6))
    seeds = dg.permutation(300, 2)[:40]
    blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fo, 77)
    check_blocks(g, seeds, fo, blocks)
    logits, hidden = orc.sage_forward(blocks, X[blocks[0].src], ws, wn, bs)
    full = _dense_sage(g.indptr, g.indices, X, ws, wn, bs)
    for l in range(L):
        nodes = blocks[l].src[:blocks[l].n_dst]
        assert np.allclose(hidden[l], full[l][nodes], rtol=1e-12, atol=1e-12)
    assert np.allclose(logits, full[-1][seeds], rtol=1e-12, atol=1e-12)


def test_sage_linear_relu_and_bias(orc):
    H = np.array([[1.0, -2.0]])
    m = np.array([[0.5, 0.25]])
    ws = np.array([[1.0, 0.0], [0.0, 1.0]])
    wn = np.array([[2.0, 0.0], [0.0, 4.0]])
    b = np.array([0.5, -0.5])
    # z = [1 + 1 + 0.5, -2 + 1 - 0.5] = [2.5, -1.5]
    assert np.array_equal(orc.sage_linear(H, m, ws, wn, b, relu=False), [[2.5, -1.5]])
    assert np.array_equal(orc.sage_linear(H, m, ws, wn, b, relu=True), [[2.5, 0.0]])
