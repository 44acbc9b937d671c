"""GPU parity at the full sizes of the benchmark workloads.

The 1M-node R-MAT graph (fp32 x100, fan-outs 15/10/5, batch 1000), the
2.4M-node power-law graph (the benchmark's workload) and the same graph with
100 hubs of in-degree 100k (bf16 x128, fan-outs 25/10, batch 4000), each run
through the C ABI exactly as bench.py runs them (caller-owned workspaces,
reused across batches).  Whole batches are compared with the oracle:
sampling, relabel and gather bit for bit, the forward within 1e-4 (fp32) or
2e-2 (bf16) row-wise relative error on every layer, and on the fp32
workloads one whole training step (loss, every gradient, the SGD update).
"""
import types

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU on this machine", allow_module_level=True)

import paper_2010_05337_amd as gmb  # noqa: E402
from datagen.configs import make_workload  # noqa: E402
from gpu_util import (margin_biases, assert_blocks_equal, compare_train_step, rowwise_rel_err, tensor_bits,  # noqa: E402
                      tensor_f64, to_torch_feats, to_torch_weights)

TOL = {"f32": 1e-4, "bf16": 2e-2}


class Lane:
    """One set of device buffers, sized for a full batch, as bench.py keeps
    per stream."""

    def __init__(self, csr, wl, feats, weights, stream=None):
        cfg = wl.cfg
        self.csr, self.stream = csr, stream
        dev = torch.device("cuda")
        self.ws_sample = gmb._aligned_bytes(gmb.sample_workspace_bytes(cfg.batch, list(cfg.fanouts),
                                                                       cfg.num_nodes), dev)[1]
        probe = gmb.sample_blocks(csr, torch.from_numpy(wl.batches[0]).cuda(), list(cfg.fanouts),
                                  wl.batch_key(0), workspace=self.ws_sample)
        self.x = torch.empty((probe.input_capacity, cfg.feat_dim), dtype=feats.dtype, device=dev)
        self.ws_fwd = gmb._aligned_bytes(gmb.forward_workspace_bytes(probe, weights), dev)[1]
        self.logits = torch.empty((cfg.batch, cfg.dims[-1]), dtype=torch.float32, device=dev)

    def run(self, wl, feats, weights, b, seeds=None):
        cfg = wl.cfg
        s = torch.from_numpy(wl.batches[b] if seeds is None else seeds).cuda()
        blocks = gmb.sample_blocks(self.csr, s, list(cfg.fanouts), wl.batch_key(b), workspace=self.ws_sample)
        x = gmb.gather_features(blocks, feats, out=self.x)
        logits, hidden = gmb.sage_forward(blocks, x, weights, workspace=self.ws_fwd,
                                          logits=self.logits[:s.numel()], return_hidden=True)
        return blocks, x, logits, hidden


def host_blocks(blocks):
    out = []
    for b in blocks.blocks():
        out.append(dict(n_dst=b.n_dst, n_src=b.n_src, nnz=b.nnz,
                        indptr=b.indptr.cpu().numpy().astype(np.int64),
                        local=b.indices.cpu().numpy().astype(np.int64),
                        nbr=b.nbr.cpu().numpy().astype(np.int64),
                        src=b.src_ids.cpu().numpy().astype(np.int64)))
    return out


def check_batch(orc, wl, lane, feats, weights, b, seeds=None):
    cfg, g = wl.cfg, wl.graph
    seeds_np = wl.batches[b] if seeds is None else seeds
    print(f"{cfg.name}: batch {b}, {len(seeds_np)} seeds", flush=True)
    blocks, x, logits, hidden = lane.run(wl, feats, weights, b, seeds)
    host = host_blocks(blocks)
    ref = orc.sample_blocks(g.indptr, g.indices, seeds_np, list(cfg.fanouts), wl.batch_key(b))
    assert_blocks_equal(host, ref, f"{cfg.name} batch {b}")
    X = orc.gather(wl.feats, ref[0].src)
    got = tensor_bits(x)[:ref[0].n_src]
    assert got.view(np.uint8).tobytes() == X.view(np.uint8).tobytes(), "gathered rows differ"
    ws, wn, bs = wl.weights.as_f64()
    ref_logits, ref_hidden = orc.sage_forward(ref, orc.widen(X, cfg.feat_dtype), ws, wn, bs)
    errs = [rowwise_rel_err(tensor_f64(h), r) for h, r in zip(hidden, ref_hidden[:-1])]
    errs.append(rowwise_rel_err(tensor_f64(logits), ref_logits))
    print(f"  sizes {[(r.n_dst, r.n_src, r.nnz) for r in ref]}, forward errors {errs}", flush=True)
    assert all(e <= TOL[cfg.feat_dtype] for e in errs), errs
    return blocks, logits


@pytest.fixture(scope="module", params=["rmat1m", "products2m", "hubs2m"])
def setup(request):
    wl = make_workload(request.param)
    g = wl.graph
    print(f"{request.param}: N={g.num_nodes} E={g.num_edges} max deg={g.degrees().max()}", flush=True)
    ip = torch.from_numpy(g.indptr.astype(np.int32)).cuda()
    ix = torch.from_numpy(g.indices).cuda()
    csr = gmb.CSRGraph(ip, ix)
    feats = to_torch_feats(wl.feats)
    weights = to_torch_weights(wl.weights)
    yield wl, csr, feats, weights, ip, ix
    del csr, feats, weights
    torch.cuda.empty_cache()


def test_full_size_batches_match_the_oracle(orc, setup):
    """First, middle and last (partial) batch of the epoch, one set of
    reused buffers."""
    wl, csr, feats, weights, _, _ = setup
    lane = Lane(csr, wl, feats, weights)
    nb = len(wl.batches)
    for b in sorted({0, nb // 2, nb - 1}):
        check_batch(orc, wl, lane, feats, weights, b)
    csr.check_status()


def test_hub_seeds(orc, setup):
    """Every hub as a seed next to ordinary vertices (the hubs2m graph; on
    the others, the 100 highest-degree vertices)."""
    wl, csr, feats, weights, _, _ = setup
    g = wl.graph
    deg = g.degrees()
    hubs = np.asarray(g.hubs) if getattr(g, "hubs", None) is not None and len(g.hubs) else \
        np.argsort(-deg, kind="stable")[:100]
    rest = wl.batches[0][~np.isin(wl.batches[0], hubs)][:wl.cfg.batch - len(hubs)]
    seeds = np.concatenate([hubs.astype(np.int32), rest.astype(np.int32)])
    assert len(np.unique(seeds)) == len(seeds)
    lane = Lane(csr, wl, feats, weights)
    check_batch(orc, wl, lane, feats, weights, 0, seeds=seeds)
    csr.check_status()


def test_streams_reproduce_one_stream(setup):
    """Batches run four at a time on four streams (each stream with its own
    sampler state and buffers, as in the benchmark) give the same blocks and
    the same logits, bit for bit, as the same batches on one stream."""
    wl, csr, feats, weights, ip, ix = setup
    streams = [torch.cuda.Stream() for _ in range(4)]
    lanes = [Lane(gmb.CSRGraph(ip, ix), wl, feats, weights, st) for st in streams]
    single = Lane(csr, wl, feats, weights)
    nb = min(8, len(wl.batches))
    torch.cuda.synchronize()
    for g0 in range(0, nb, 4):
        group = []
        for b in range(g0, min(g0 + 4, nb)):
            ln = lanes[b % 4]
            with torch.cuda.stream(ln.stream):
                blocks, _, logits, _ = ln.run(wl, feats, weights, b)
            group.append((b, blocks, logits))
        torch.cuda.synchronize()
        for b, blocks, logits in group:
            got, lg = host_blocks(blocks), logits.clone()
            blocks1, _, logits1, _ = single.run(wl, feats, weights, b)
            ref = host_blocks(blocks1)
            for l, (h, r) in enumerate(zip(got, ref)):
                for k in ("n_dst", "n_src", "nnz", "indptr", "local", "nbr", "src"):
                    assert np.array_equal(h[k], r[k]), f"batch {b} layer {l} {k}"
            assert torch.equal(lg, logits1), f"batch {b} logits"
    for ln in lanes:
        ln.csr.check_status()


def test_full_size_training_step(orc, dg, setup):
    """Batch 0 of the epoch: sample, gather, forward, loss, backward and one
    SGD step on the device, in the buffers bench.py's training mode uses,
    against the oracle's fp64 step."""
    wl, csr, feats, _, _, _ = setup
    cfg, g = wl.cfg, wl.graph
    seeds = wl.batches[0]
    ref = orc.sample_blocks(g.indptr, g.indices, seeds, list(cfg.fanouts), wl.batch_key(0))
    X = orc.widen(orc.gather(wl.feats, ref[0].src), cfg.feat_dtype)
    if cfg.feat_dtype == "bf16":
        return _bf16_training_step(orc, dg, wl, csr, feats, ref, X)
    w = types.SimpleNamespace(**vars(wl.weights))
    w.bias = margin_biases(orc, ref, X, wl.weights)
    w.as_f64 = lambda: ([a.astype(np.float64) for a in w.w_self], [a.astype(np.float64) for a in w.w_neigh],
                        [b.astype(np.float64) for b in w.bias])
    wt = to_torch_weights(w)
    lane = Lane(csr, wl, feats, wt)
    print(f"{cfg.name}: training step on batch 0, {len(seeds)} seeds", flush=True)
    blocks, x, logits, hidden = lane.run(wl, feats, wt, 0)
    assert_blocks_equal(host_blocks(blocks), ref, f"{cfg.name} batch 0")
    labels = dg.labels(g.num_nodes, cfg.dims[-1], 7)[seeds]
    y = torch.from_numpy(labels).cuda()
    grads, loss = gmb.sage_backward(blocks, x, wt, logits, y, lane.ws_fwd)
    before = [[t.clone() for t in arrs] for arrs in (wt.w_self, wt.w_neigh, wt.bias)]
    lr = 0.1
    gmb.sgd_update(wt, grads, lr)
    torch.cuda.synchronize()
    out = dict(hidden=hidden, grads=grads, loss=float(loss.item()), before=before)
    compare_train_step(orc, out, ref, X, w, labels, lr, wt, exact_hidden=False)
    csr.check_status()


def _bf16_training_step(orc, dg, wl, csr, feats, ref, X):
    """test_full_size_training_step for a bf16 workload: fp32 master weights,
    the oracle's fp64 step within 2e-2 (see test_bf16_train_step_matches_the_oracle)."""
    from gpu_util import compare_train_step_bf16
    cfg, g = wl.cfg, wl.graph
    w = types.SimpleNamespace(**vars(wl.weights))
    w.bias = margin_biases(orc, ref, X, wl.weights)
    base = wl.weights.as_f64()
    w.as_f64 = lambda: (base[0], base[1], [b.astype(np.float64) for b in w.bias])
    wt = to_torch_weights(w)
    master = wt.master()
    lane = Lane(csr, wl, feats, wt)
    print(f"{cfg.name}: bf16 training step on batch 0, {len(wl.batches[0])} seeds", flush=True)
    blocks, x, logits, _ = lane.run(wl, feats, wt, 0)
    assert_blocks_equal(host_blocks(blocks), ref, f"{cfg.name} batch 0")
    labels = dg.labels(g.num_nodes, cfg.dims[-1], 7)[wl.batches[0]]
    grads, loss = gmb.sage_backward(blocks, x, wt, logits, torch.from_numpy(labels).cuda(), lane.ws_fwd)
    before = [[t.clone() for t in arrs] for arrs in (master.w_self, master.w_neigh, master.bias)]
    gmb.sgd_update_bf16(wt, master, grads, 0.1)
    torch.cuda.synchronize()
    compare_train_step_bf16(orc, float(loss.item()), grads, ref, X, w, labels, 0.1, before, master, wt)
    csr.check_status()


def test_full_size_fused_forward(setup):
    """The fused forward (layer-0 mean straight from the feature table, only
    the destination rows gathered) against the three-call path, bit for
    bit, on the first and last batch, in bench.py's buffers."""
    wl, csr, feats, weights, _, _ = setup
    lane = Lane(csr, wl, feats, weights)
    nb = len(wl.batches)
    for b in sorted({0, nb - 1}):
        blocks, x, logits, hidden = lane.run(wl, feats, weights, b)
        lg = logits.clone()
        hid = [h.clone() for h in hidden]
        n_dst0 = blocks.sizes()[0][0]
        x_dst = torch.empty((gmb.dst_capacity(blocks), wl.cfg.feat_dim), dtype=feats.dtype, device="cuda")
        logits2, x_dst, hidden2 = gmb.sage_forward_fused(blocks, feats, weights, x_dst=x_dst,
                                                         workspace=lane.ws_fwd, return_hidden=True)
        bits = (lambda t: t.view(torch.int16)) if feats.dtype == torch.bfloat16 else (lambda t: t.view(torch.int32))
        assert torch.equal(bits(x_dst[:n_dst0]), bits(x[:n_dst0])), f"batch {b} x_dst"
        assert torch.equal(logits2, lg), f"batch {b} logits"
        for l, (h1, h2) in enumerate(zip(hid, hidden2)):
            assert torch.equal(bits(h1), bits(h2)), f"batch {b} hidden {l}"
        print(f"{wl.cfg.name}: batch {b}: fused forward equal to the three-call path", flush=True)
    csr.check_status()


def test_every_batch_of_the_epoch(orc, setup):
    """Sampling, relabel and gather of every batch of the epoch bit for bit,
    and the forward of the first 16 batches within the tolerance, against
    the oracle run on host threads (its C calls release the interpreter
    lock; at most 32 batches in flight)."""
    import os
    from concurrent.futures import ThreadPoolExecutor

    wl, csr, feats, weights, _, _ = setup
    cfg, g = wl.cfg, wl.graph
    lane = Lane(csr, wl, feats, weights)
    nb = len(wl.batches)
    n_fwd = min(16, nb)
    ws, wn, bs = wl.weights.as_f64()
    orc.lib()

    def oracle_batch(b):
        ref = orc.sample_blocks(g.indptr, g.indices, wl.batches[b], list(cfg.fanouts), wl.batch_key(b))
        X = orc.gather(wl.feats, ref[0].src)
        logits = orc.sage_forward(ref, orc.widen(X, cfg.feat_dtype), ws, wn, bs)[0] if b < n_fwd else None
        return ref, X, logits

    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    worst = 0.0
    with ThreadPoolExecutor(max_workers=threads) as ex:
        futs = {}
        for b in range(min(32, nb)):
            futs[b] = ex.submit(oracle_batch, b)
        for b in range(nb):
            blocks, x, logits, _ = lane.run(wl, feats, weights, b)
            host = host_blocks(blocks)
            ref, X, ref_logits = futs.pop(b).result()
            if b + 32 < nb:
                futs[b + 32] = ex.submit(oracle_batch, b + 32)
            assert_blocks_equal(host, ref, f"{cfg.name} batch {b}")
            got = tensor_bits(x)[:ref[0].n_src]
            assert got.view(np.uint8).tobytes() == X.view(np.uint8).tobytes(), f"batch {b}: gathered rows differ"
            if ref_logits is not None:
                e = rowwise_rel_err(tensor_f64(logits), ref_logits)
                worst = max(worst, e)
                assert e <= TOL[cfg.feat_dtype], (b, e)
            del ref, X
    csr.check_status()
    print(f"{cfg.name}: {nb} batches bit-exact (sampling, relabel, gather); forward of the first {n_fwd}: "
          f"max rel. error {worst:.2e}", flush=True)


def test_full_size_embedding_step(orc, dg, setup):
    """Batch 0 with the features as learnable vertex embeddings (fp32
    workloads): the sparse update of the table against the oracle, every
    row outside the batch untouched (margin biases as in the training-step
    test)."""
    wl, csr, feats, _, _, _ = setup
    cfg, g = wl.cfg, wl.graph
    seeds = wl.batches[0]
    ref = orc.sample_blocks(g.indptr, g.indices, seeds, list(cfg.fanouts), wl.batch_key(0))
    X = orc.widen(orc.gather(wl.feats, ref[0].src), cfg.feat_dtype)
    if cfg.feat_dtype == "bf16":
        return _bf16_training_step(orc, dg, wl, csr, feats, ref, X)
    w = types.SimpleNamespace(**vars(wl.weights))
    w.bias = margin_biases(orc, ref, X, wl.weights)
    w.as_f64 = lambda: ([a.astype(np.float64) for a in w.w_self], [a.astype(np.float64) for a in w.w_neigh],
                        [b.astype(np.float64) for b in w.bias])
    wt = to_torch_weights(w)
    table = feats.clone()
    lane = Lane(csr, wl, table, wt)
    blocks, x, logits, _ = lane.run(wl, table, wt, 0)
    labels = dg.labels(g.num_nodes, cfg.dims[-1], 7)[seeds]
    emb_lr = 0.5
    _, loss = gmb.sage_backward(blocks, x, wt, logits, torch.from_numpy(labels).cuda(), lane.ws_fwd,
                                embedding=table, emb_lr=emb_lr)
    torch.cuda.synchronize()
    ws, wn, bs = w.as_f64()
    ref_loss, _, dX, _, _ = orc.sage_train_step_embed(ref, wl.feats, ws, wn, bs, labels, 0.0, 0.0)
    assert abs(loss.item() - ref_loss) <= 1e-5 * max(1.0, abs(ref_loss))
    src = np.asarray(ref[0].src, dtype=np.int64)
    got = table.cpu().numpy()
    rest = np.ones(g.num_nodes, dtype=bool)
    rest[src] = False
    assert np.array_equal(got[rest], wl.feats[rest]), "rows outside the mini-batch changed"
    want = wl.feats[src].astype(np.float64) - emb_lr * dX
    bound = emb_lr * 1e-4 * np.abs(dX).max() + 2.0 ** -23 * np.abs(want).max()
    err = np.abs(got[src].astype(np.float64) - want).max()
    print(f"{cfg.name}: {len(src)} embedding rows updated, max error {err:.2e} (bound {bound:.2e})", flush=True)
    assert err <= bound
    csr.check_status()
