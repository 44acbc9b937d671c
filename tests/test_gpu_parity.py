"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Sampling, relabelling and gather must match bit for bit; the GraphSAGE
forward within a row-wise max relative error of 1e-4 (fp32 features) or
2e-2 (bf16 features), on the logits and on every hidden layer.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU on this machine", allow_module_level=True)

import paper_2010_05337_amd as gmb  # noqa: E402
from gpu_util import (assert_blocks_equal, csr_on_device, gpu_blocks, rowwise_rel_err,  # noqa: E402
                      tensor_bits, tensor_f64, to_torch_feats, to_torch_weights)

TOL_F32, TOL_BF16 = 1e-4, 2e-2


@pytest.fixture(scope="module")
def tiny(dg):
    return dg.er_directed(10000, 10.0, 101)


def _star_graph():
    class G:
        pass
    rows = {0: [], 1: [4, 5, 6], 2: [4, 5, 6, 7, 8], 3: list(range(4, 13))}
    g = G()
    g.num_nodes = 13
    idx, ptr = [], [0]
    for v in range(13):
        idx += rows.get(v, [])
        ptr.append(len(idx))
    g.indptr = np.array(ptr, dtype=np.int64)
    g.indices = np.array(idx, dtype=np.int32)
    return g


def test_library_is_the_hip_build():
    L = gmb.lib()
    assert L.gmb_abi_version() == 1
    assert torch.cuda.get_device_properties(0).gcnArchName.startswith("gfx950")


@pytest.mark.parametrize("fanouts", [[5, 5], [1], [3, 7, 2], [16, 16], [33, 9], [70]])
def test_sampling_tiny_bitexact(orc, dg, tiny, fanouts):
    print(f"tiny ER, fanouts={fanouts}", flush=True)
    csr = csr_on_device(tiny)
    seeds = dg.permutation(10000, 104)[:64]
    _, host = gpu_blocks(csr, seeds, fanouts, 105)
    ref = orc.sample_blocks(tiny.indptr, tiny.indices, seeds, fanouts, 105)
    assert_blocks_equal(host, ref, f"fanouts {fanouts}")
    csr.check_status()


def test_sampling_degree_cases_and_empty(orc):
    g = _star_graph()
    csr = csr_on_device(g)
    for seeds, fo in [([0, 1, 2, 3], [5]), ([3, 2, 1, 0], [5, 2]), ([], [5, 5]), ([0], [3])]:
        _, host = gpu_blocks(csr, seeds, fo, 3)
        ref = orc.sample_blocks(g.indptr, g.indices, seeds, fo, 3)
        assert_blocks_equal(host, ref, f"seeds {seeds} fanouts {fo}")
    csr.check_status()


@pytest.mark.parametrize("wide", [False, True])
def test_sampling_rmat_hubs_bitexact(orc, dg, wide):
    """Hubs well above every fan-out, many tiles of the look-back scans, and
    int32 / int64 row offsets."""
    g = dg.rmat(16, 60000, 900000, (0.57, 0.19, 0.19), 7)
    g = dg.inject_hubs(g, 5, 20000, 3)
    print(f"rmat N={g.num_nodes} nnz={g.num_edges} max deg={g.degrees().max()} wide={wide}", flush=True)
    csr = csr_on_device(g, wide=wide)
    seeds = np.concatenate([g.hubs, dg.permutation(60000, 8)[:3000]]).astype(np.int64)
    seeds = seeds[np.sort(np.unique(seeds, return_index=True)[1])]
    for fo, key in [([15, 10, 5], 99), ([25, 10], 7)]:
        _, host = gpu_blocks(csr, seeds, fo, key)
        ref = orc.sample_blocks(g.indptr, g.indices, seeds, fo, key)
        assert_blocks_equal(host, ref, f"fanouts {fo}")
        assert ref[0].nnz > 2 * 2048   # several scan tiles
    csr.check_status()


def test_sampling_wide_fanouts_on_hubs(orc, dg):
    """Fan-outs above 64 on rows far longer than the fan-out: 65 to 128 (a
    wave per destination, two draws per lane), 129 to 256 (four per lane),
    above 256 (one thread per destination, slots sorted in place), and a
    fan-out of exactly 64 (the widest lane group)."""
    g = dg.rmat(14, 16000, 240000, (0.57, 0.19, 0.19), 17)
    g = dg.inject_hubs(g, 4, 5000, 18)
    csr = csr_on_device(g)
    seeds = np.concatenate([g.hubs, dg.permutation(16000, 19)[:400]]).astype(np.int64)
    seeds = seeds[np.sort(np.unique(seeds, return_index=True)[1])]
    deg = g.degrees()
    for fo, key in [([100], 21), ([70, 3], 22), ([64], 23), ([128], 24), ([129], 25), ([200], 26),
                    ([256], 27), ([300], 28), ([65, 2], 29)]:
        _, host = gpu_blocks(csr, seeds, fo, key)
        ref = orc.sample_blocks(g.indptr, g.indices, seeds, fo, key)
        assert_blocks_equal(host, ref, f"fanouts {fo}")
        assert (deg[seeds] > max(fo)).sum() >= 4   # Floyd runs on every hub
    csr.check_status()


def test_sampling_is_deterministic_and_keyed(dg, tiny):
    csr = csr_on_device(tiny)
    seeds = dg.permutation(10000, 5)[:500]
    _, a = gpu_blocks(csr, seeds, [10, 10], 11)
    _, b = gpu_blocks(csr, seeds, [10, 10], 11)
    _, c = gpu_blocks(csr, seeds, [10, 10], 12)
    for x, y in zip(a, b):
        for k in x:
            assert np.array_equal(x[k], y[k])
    assert not np.array_equal(a[1]["nbr"], c[1]["nbr"])


def _table_is_clear(csr):
    torch.cuda.synchronize()
    table = csr.state[256:256 + 4 * csr.num_nodes].view(torch.int32)
    return bool((table == -1).all())


@pytest.mark.parametrize("n, num_seeds, fanouts, whole", [
    (10000, 64, [5, 5], True), (10000, 8, [2], False), (10003, 64, [5, 5], True), (10003, 8, [2], False),
    (200_000, 8, [3, 3], False)])
def test_state_is_clean_after_each_call(orc, dg, n, num_seeds, fanouts, whole):
    """The cleanup clears the dedup table in one of two ways: all of it
    with 16-byte stores when it holds at most eight slots per possible
    source of the batch, else the slots of the batch's vertices one by one;
    10,003 vertices leave three slots past the last 16-byte group."""
    print(f"ER N={n}, {num_seeds} seeds, fanouts={fanouts}", flush=True)
    g = dg.er_directed(n, 10.0, 101)
    csr = csr_on_device(g)
    seeds = dg.permutation(n, 6)[:num_seeds]
    for key in (1, 2):
        blocks, host = gpu_blocks(csr, seeds, fanouts, key)
        assert (n <= 8 * blocks.input_capacity) == whole
        assert_blocks_equal(host, orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, key), f"key {key}")
        assert _table_is_clear(csr)
    csr.check_status()


def test_device_errors_are_reported(orc, dg, tiny):
    csr = csr_on_device(tiny)
    gpu_blocks(csr, [1, 2, 10000], [5], 1)
    with pytest.raises(gmb.GmbError) as e:
        csr.check_status()
    assert e.value.code == -4
    gpu_blocks(csr, [1, 2, 1], [5, 5], 1)
    with pytest.raises(gmb.GmbError) as e:
        csr.check_status()
    assert e.value.code == -5
    assert _table_is_clear(csr)
    # a repeated seed under fan-outs above 64 (the one-thread sampler)
    gpu_blocks(csr, [7, 3, 9, 3], [70], 1)
    with pytest.raises(gmb.GmbError) as e:
        csr.check_status()
    assert e.value.code == -5
    assert _table_is_clear(csr)
    # the state is usable again afterwards
    seeds = dg.permutation(10000, 9)[:64]
    _, host = gpu_blocks(csr, seeds, [5, 5], 2)
    assert_blocks_equal(host, orc.sample_blocks(tiny.indptr, tiny.indices, seeds, [5, 5], 2))
    csr.check_status()


def test_host_argument_errors(tiny):
    csr = csr_on_device(tiny)
    s = torch.arange(10, dtype=torch.int32, device="cuda")
    with pytest.raises(gmb.GmbError) as e:
        gmb.sample_blocks(csr, s, [5, 0], 1)
    assert e.value.code == -1
    small = torch.empty(256, dtype=torch.uint8, device="cuda")
    need = gmb.sample_workspace_bytes(10, [5, 5], csr.num_nodes)
    assert need > 256
    # a too-small workspace is replaced by the binding; through the ABI it is ENOSPC
    blocks = gmb.sample_blocks(csr, s, [5, 5], 1, workspace=small)
    assert blocks.workspace.numel() >= need


@pytest.mark.parametrize("dim,dtype", [(16, "f32"), (100, "f32"), (7, "f32"), (128, "bf16"),
                                       (3, "bf16"), (256, "f32")])
def test_gather_bitexact(orc, dg, tiny, dim, dtype):
    feats = dg.features(10000, dim, 77, dtype)
    ft = to_torch_feats(feats)
    csr = csr_on_device(tiny)
    seeds = dg.permutation(10000, 104)[:64]
    blocks, host = gpu_blocks(csr, seeds, [5, 5], 105)
    x = gmb.gather_features(blocks, ft)
    n_in = host[0]["n_src"]
    got = tensor_bits(x)[:n_in]
    ref = orc.gather(feats, host[0]["src"])
    assert got.view(np.uint8).tobytes() == ref.view(np.uint8).tobytes()
    # explicit id list with a ragged count
    ids = torch.from_numpy(dg.permutation(10000, 3)[:1001]).cuda()
    y = gmb.gather_features(ids, ft, n=999)
    assert np.array_equal(tensor_bits(y).view(np.uint8),
                          orc.gather(feats, ids.cpu().numpy()[:999]).view(np.uint8))
    csr.check_status()


def _forward_case(orc, dg, g, feats, w, seeds, fanouts, key, tol):
    csr = csr_on_device(g)
    ft = to_torch_feats(feats)
    wt = to_torch_weights(w)
    blocks, host = gpu_blocks(csr, seeds, fanouts, key)
    x = gmb.gather_features(blocks, ft)
    logits, hidden = gmb.sage_forward(blocks, x, wt, return_hidden=True)
    ref_blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, key)
    assert_blocks_equal(host, ref_blocks)
    X = orc.widen(orc.gather(feats, ref_blocks[0].src), w.dtype)
    ws, wn, bs = w.as_f64()
    ref_logits, ref_hidden = orc.sage_forward(ref_blocks, X, ws, wn, bs)
    errs = [rowwise_rel_err(tensor_f64(h), r) for h, r in zip(hidden, ref_hidden[:-1])]
    errs.append(rowwise_rel_err(tensor_f64(logits), ref_logits))
    print(f"forward rel. errors per layer: {errs}", flush=True)
    assert all(e <= tol for e in errs), errs
    csr.check_status()
    return errs


@pytest.mark.parametrize("fanouts", [[5, 5], [2, 9]])
def test_forward_tiny_f32(orc, dg, tiny, fanouts):
    feats = dg.features(10000, 16, 102, "f32")
    w = dg.sage_weights([16, 16, 8], 103)
    seeds = dg.permutation(10000, 104)[:64]
    _forward_case(orc, dg, tiny, feats, w, seeds, fanouts, 105, TOL_F32)


def test_forward_ragged_dims_f32(orc, dg, tiny):
    """Dims that are not multiples of the vector width or of the 64-wide
    output tile, three layers."""
    feats = dg.features(10000, 37, 1, "f32")
    w = dg.sage_weights([37, 70, 65, 5], 2)
    seeds = dg.permutation(10000, 3)[:200]
    _forward_case(orc, dg, tiny, feats, w, seeds, [4, 3, 6], 4, TOL_F32)


def test_forward_bf16(orc, dg, tiny):
    feats = dg.features(10000, 128, 5, "bf16")
    w = dg.sage_weights([128, 256, 47], 6, "bf16")
    seeds = dg.permutation(10000, 7)[:300]
    _forward_case(orc, dg, tiny, feats, w, seeds, [25, 10], 8, TOL_BF16)


@pytest.mark.parametrize("dims,fanouts", [([12, 40, 5], [3, 6]), ([64, 256, 47], [10, 4]),
                                          ([256, 64, 130], [2, 3])])
def test_forward_bf16_shapes(orc, dg, tiny, dims, fanouts):
    """bf16 layers on the LDS-slab kernel (d_in a multiple of 8: 40, 64, 256,
    K up to 512, output widths 5, 47, 130) and on the general kernel
    (d_in = 12)."""
    feats = dg.features(10000, dims[0], 41, "bf16")
    w = dg.sage_weights(dims, 42, "bf16")
    seeds = dg.permutation(10000, 43)[:300]
    _forward_case(orc, dg, tiny, feats, w, seeds, fanouts, 44, TOL_BF16)


def test_forward_wide_model_f32(orc, dg):
    """The paper's model shape (3 layers, hidden 256, fan-outs 15/10/5) on a
    small power-law graph: many rows of the 64-row tiles, K = 200 and 512."""
    g = dg.rmat(15, 30000, 300000, (0.57, 0.19, 0.19), 21)
    feats = dg.features(30000, 100, 22, "f32")
    w = dg.sage_weights([100, 256, 256, 47], 23)
    seeds = dg.permutation(30000, 24)[:256]
    errs = _forward_case(orc, dg, g, feats, w, seeds, [15, 10, 5], 25, TOL_F32)
    # the layers take the split-K tilings of the part-product linear (32
    # columns on layer 0, 16 on the smaller two): fp32-level accuracy, well
    # inside the tolerance (about 1e-6 measured; a dropped part product would
    # show as 1e-5 or more)
    assert max(errs) <= 5e-6, errs


@pytest.mark.parametrize("d_in,d_hid", [(64, 300), (128, 256), (100, 256)])
def test_forward_large_layer_eight_waves_f32(orc, dg, d_in, d_hid):
    """A first layer with 17.5k destination rows: the part-product linear
    on eight waves per workgroup (K = 2 d_in of 128, 256 and 200, the last
    not a multiple of the 32-wide chunk), ragged rows, and 300 outputs (a
    ragged fifth column tile); fp32-level accuracy."""
    g = dg.rmat(16, 60000, 1500000, (0.57, 0.19, 0.19), 91)
    feats = dg.features(60000, d_in, 92, "f32")
    w = dg.sage_weights([d_in, d_hid, 8], 93)
    seeds = dg.permutation(60000, 94)[:8000]
    # 17,502 destination rows in layer 0: 137 tiles of 128 rows per column tile
    errs = _forward_case(orc, dg, g, feats, w, seeds, [3, 12], 95, TOL_F32)
    assert max(errs) <= 5e-6, errs


@pytest.mark.parametrize("dims,fanouts", [([8, 300, 20], [6, 3]), ([64, 130, 12], [4, 7]),
                                          ([128, 64, 40, 3], [3, 2, 5])])
def test_forward_more_shapes_f32(orc, dg, tiny, dims, fanouts):
    """Output widths above 256 (several column tiles), a narrow input, and
    deep small layers."""
    feats = dg.features(10000, dims[0], 31, "f32")
    w = dg.sage_weights(dims, 32)
    seeds = dg.permutation(10000, 33)[:150]
    _forward_case(orc, dg, tiny, feats, w, seeds, fanouts, 34, TOL_F32)


@pytest.mark.parametrize("d_in", [192, 256, 320])
def test_forward_wide_inputs_many_rows_f32(orc, dg, tiny, d_in):
    """K = 2 d_in of 384, 512 and 640 on a layer with over 8192 rows and 256
    outputs: the fp32 slab kernel with one wave per 16 rows and 64 columns
    at its widest slabs (96, 128 and 160 KB of LDS), which the smaller
    shapes of the other cases never reach."""
    feats = dg.features(10000, d_in, 61, "f32")
    w = dg.sage_weights([d_in, 256, 8], 62)
    seeds = dg.permutation(10000, 63)[:600]
    _forward_case(orc, dg, tiny, feats, w, seeds, [3, 15], 64, TOL_F32)


# ---- the forward with the feature pull folded into layer 0 -----------------

def _fused_case(orc, dg, g, feats, w, seeds, fanouts, key, tol):
    """The fused forward against the three-call path on the same blocks: the
    logits and every hidden layer bit for bit, x_dst = the gathered rows of
    block 0's destinations bit for bit; and the logits against the oracle."""
    csr = csr_on_device(g)
    ft = to_torch_feats(feats)
    wt = to_torch_weights(w)
    blocks, host = gpu_blocks(csr, seeds, fanouts, key)
    x = gmb.gather_features(blocks, ft)
    logits, hidden = gmb.sage_forward(blocks, x, wt, return_hidden=True)
    logits2, x_dst, hidden2 = gmb.sage_forward_fused(blocks, ft, wt, return_hidden=True)
    csr.check_status()
    n_dst0 = host[0]["n_dst"]
    assert torch.equal(tensor_bits_t(x_dst[:n_dst0]), tensor_bits_t(x[:n_dst0])), "x_dst"
    assert torch.equal(logits, logits2), "logits"
    for l, (h1, h2) in enumerate(zip(hidden, hidden2)):
        assert torch.equal(tensor_bits_t(h1), tensor_bits_t(h2)), f"hidden layer {l}"
    ref_blocks = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, key)
    X = orc.widen(orc.gather(feats, ref_blocks[0].src), w.dtype)
    ws, wn, bs = w.as_f64()
    ref_logits, _ = orc.sage_forward(ref_blocks, X, ws, wn, bs)
    err = rowwise_rel_err(tensor_f64(logits2), ref_logits)
    print(f"fused forward: equal to the three-call path; logits rel. error {err:.2e}", flush=True)
    assert err <= tol


def tensor_bits_t(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


@pytest.mark.parametrize("dims,fanouts,dtype", [([16, 16, 8], [5, 5], "f32"), ([10, 12, 7], [8, 4], "f32"),
                                                ([64, 256, 47], [10, 4], "bf16"), ([12, 40, 5], [3, 6], "bf16"),
                                                ([128, 64, 40, 3], [3, 2, 5], "f32")])
def test_forward_fused_equals_three_calls(orc, dg, tiny, dims, fanouts, dtype):
    feats = dg.features(10000, dims[0], 51, dtype)
    w = dg.sage_weights(dims, 52, dtype)
    seeds = dg.permutation(10000, 53)[:200]
    _fused_case(orc, dg, tiny, feats, w, seeds, fanouts, 54, TOL_F32 if dtype == "f32" else TOL_BF16)


def test_forward_fused_hubs(orc, dg):
    """The 100k-degree hub graph shape on the fused path (bf16 x128, fan-outs
    25/10): hubs as seeds among ordinary vertices."""
    g = dg.inject_hubs(dg.er_directed(20000, 8.0, 61), 5, 3000, 62)
    feats = dg.features(20000, 128, 63, "bf16")
    w = dg.sage_weights([128, 256, 47], 64, "bf16")
    seeds = np.concatenate([np.asarray(g.hubs, np.int32),
                            dg.permutation(20000, 65)[:300][~np.isin(dg.permutation(20000, 65)[:300], g.hubs)]])
    _fused_case(orc, dg, g, feats, w, seeds.astype(np.int32), [25, 10], 66, TOL_BF16)


@pytest.mark.parametrize("fanouts, num_seeds", [([12, 8, 5], 3000), ([70], 300), ([6, 30], 800)])
def test_owner_overflow_path(orc, dg, fanouts, num_seeds, monkeypatch):
    """An owner whose vertices do not fit its LDS table redoes its pairs
    through the state's per-vertex table: forced here with a 64-slot limit
    (the test hook GMB_OWNER_TABLE_SLOTS), every block must still equal the
    oracle's, repeated seeds must still be reported, and the table must be
    clear afterwards."""
    monkeypatch.setenv("GMB_OWNER_TABLE_SLOTS", "64")
    g = dg.rmat(15, 30_000, 250_000, (0.57, 0.19, 0.19), 9)
    csr = csr_on_device(g)
    seeds = dg.permutation(g.num_nodes, 4)[:num_seeds]
    for key in (3, 4):
        print(f"overflow path: fanouts {fanouts}, {num_seeds} seeds, key {key}", flush=True)
        _, host = gpu_blocks(csr, seeds, fanouts, key)
        assert_blocks_equal(host, orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, key), f"key {key}")
        assert _table_is_clear(csr)
    csr.check_status()
    gpu_blocks(csr, np.concatenate([seeds[:50], seeds[:1]]), fanouts, 5)
    with pytest.raises(gmb.GmbError) as e:
        csr.check_status()
    assert e.value.code == -5
    assert _table_is_clear(csr)


def test_validation_mode_passes_on_real_blocks(orc, dg, tiny, monkeypatch):
    """GMB_VALIDATE=1: every sampling call also runs the device check of its
    blocks; on the library's own output it finds nothing (ER, R-MAT with
    hubs, fan-outs above 64, the owners' overflow path)."""
    monkeypatch.setenv("GMB_VALIDATE", "1")
    csr = csr_on_device(tiny)
    gpu_blocks(csr, dg.permutation(10000, 5)[:500], [10, 10], 3)
    csr.check_status()
    g = dg.rmat(15, 30_000, 250_000, (0.57, 0.19, 0.19), 9)
    csr = csr_on_device(g)
    seeds = dg.permutation(g.num_nodes, 4)[:800]
    for fo in ([15, 10, 5], [70], [6, 30]):
        gpu_blocks(csr, seeds, fo, 7)
        csr.check_status()
    monkeypatch.setenv("GMB_OWNER_TABLE_SLOTS", "64")
    gpu_blocks(csr, seeds, [12, 8], 8)
    csr.check_status()


def test_validation_finds_a_corrupted_block(dg, tiny):
    """The check reports a block whose local id names the wrong vertex, one
    whose local id is out of range and one whose row offsets fall; the
    state works again afterwards."""
    csr = csr_on_device(tiny)
    seeds = dg.permutation(10000, 5)[:300]
    for what in ("wrong vertex", "out of range", "falling offsets"):
        print(f"corruption: {what}", flush=True)
        blocks = gmb.sample_blocks(csr, torch.from_numpy(seeds).cuda(), [5, 5], 3)
        blocks.validate()
        csr.check_status()
        b = blocks.blocks()[0]
        if what == "wrong vertex":
            b.indices[0] = (b.indices[0] + 1) % b.n_src
        elif what == "out of range":
            b.indices[1] = b.n_src
        else:
            b.indptr[2] = b.indptr[1] - 1
        blocks.validate()
        with pytest.raises(gmb.GmbError) as e:
            csr.check_status()
        assert e.value.code == -3
    blocks = gmb.sample_blocks(csr, torch.from_numpy(seeds).cuda(), [5, 5], 4)
    blocks.validate()
    csr.check_status()
