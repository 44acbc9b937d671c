"""Helpers of the GPU parity tests: run the HIP path through the binding and
compare it with the oracle."""
import numpy as np
import torch

import paper_2010_05337_amd as gmb


def csr_on_device(g, wide: bool = False):
    ip = torch.from_numpy(g.indptr.astype(np.int64 if wide else np.int32)).cuda()
    ix = torch.from_numpy(np.ascontiguousarray(g.indices, dtype=np.int32)).cuda()
    return gmb.CSRGraph(ip, ix)


def gpu_blocks(csr, seeds, fanouts, key):
    s = torch.from_numpy(np.ascontiguousarray(seeds, dtype=np.int32)).cuda()
    blocks = gmb.sample_blocks(csr, s, fanouts, key)
    host = []
    for b in blocks.blocks():
        host.append(dict(n_dst=b.n_dst, n_src=b.n_src, nnz=b.nnz,
                         indptr=b.indptr.cpu().numpy().astype(np.int64),
                         local=b.indices.cpu().numpy().astype(np.int64),
                         nbr=b.nbr.cpu().numpy().astype(np.int64),
                         src=b.src_ids.cpu().numpy().astype(np.int64)))
    return blocks, host


def assert_blocks_equal(host, ref, what=""):
    """Bit-exact comparison of every array of every block."""
    assert len(host) == len(ref)
    for l, (h, r) in enumerate(zip(host, ref)):
        tag = f"{what} layer {l}"
        assert (h["n_dst"], h["n_src"], h["nnz"]) == (r.n_dst, r.n_src, r.nnz), tag
        assert np.array_equal(h["indptr"], r.indptr), tag + " indptr"
        assert np.array_equal(h["nbr"], r.nbr), tag + " sampled ids"
        assert np.array_equal(h["local"], r.local), tag + " local ids"
        assert np.array_equal(h["src"], r.src), tag + " src ids"


def rowwise_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max over rows v of ||g_v - r_v||_inf / max(||r_v||_inf, 1e-30)."""
    if ref.size == 0:
        return 0.0
    num = np.abs(got.astype(np.float64) - ref).max(axis=1)
    den = np.maximum(np.abs(ref).max(axis=1), 1e-30)
    return float((num / den).max())


def to_torch_feats(feats: np.ndarray) -> torch.Tensor:
    if feats.dtype == np.uint16:
        return torch.from_numpy(feats.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(feats).cuda()


def to_torch_weights(w) -> "gmb.SageWeights":
    def mat(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
        return torch.from_numpy(a).cuda()
    return gmb.SageWeights([mat(a) for a in w.w_self], [mat(a) for a in w.w_neigh],
                           [torch.from_numpy(b).cuda() for b in w.bias])


def tensor_bits(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def tensor_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)
