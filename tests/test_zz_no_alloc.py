"""The no-allocation sampling entry point (gmb_sample_blocks_noalloc),
called through the C ABI: its blocks equal those of gmb_sample_blocks bit
for bit (and the oracle's), on two calls in a row, the second smaller, so
that the second call runs on the scratch the first one left behind."""
import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU on this machine", allow_module_level=True)

import paper_2010_05337_amd as gmb  # noqa: E402
from datagen import rmat  # noqa: E402
from gpu_util import assert_blocks_equal, csr_on_device  # noqa: E402


def _host(blocks):
    out = []
    for b in blocks.blocks():
        out.append(dict(n_dst=b.n_dst, n_src=b.n_src, nnz=b.nnz,
                        indptr=b.indptr.cpu().numpy().astype(np.int64),
                        local=b.indices.cpu().numpy().astype(np.int64),
                        nbr=b.nbr.cpu().numpy().astype(np.int64),
                        src=b.src_ids.cpu().numpy().astype(np.int64)))
    return out


def _noalloc(csr, seeds, fanouts, key):
    L = gmb.lib()
    s = torch.from_numpy(np.ascontiguousarray(seeds, dtype=np.int32)).cuda()
    fo = (ctypes.c_int32 * len(fanouts))(*fanouts)
    need = L.gmb_sample_workspace_bytes(len(seeds), fo, len(fanouts), csr.num_nodes)
    assert need > 0
    _, buf = gmb._aligned_bytes(need, s.device)
    out = gmb.BlocksStruct()
    print(f"no-alloc call: {len(seeds)} seeds, fan-outs {fanouts}, key {key}", flush=True)
    rc = L.gmb_sample_blocks_noalloc(ctypes.byref(csr.struct), ctypes.c_void_p(s.data_ptr()), len(seeds), fo,
                                     len(fanouts), key, ctypes.c_void_p(csr.state.data_ptr()), csr.state_bytes,
                                     ctypes.c_void_p(buf.data_ptr()), buf.numel(), ctypes.byref(out),
                                     gmb._stream_handle())
    assert rc == 0, L.gmb_last_error()
    blocks = gmb.Blocks(out, buf, csr)
    host = _host(blocks)
    csr.check_status()
    return host


def _regular(csr, seeds, fanouts, key):
    s = torch.from_numpy(np.ascontiguousarray(seeds, dtype=np.int32)).cuda()
    host = _host(gmb.sample_blocks(csr, s, fanouts, key))
    csr.check_status()
    return host


def test_noalloc_matches_sample_blocks_twice(orc):
    g = rmat(16, 60_000, 500_000, (0.57, 0.19, 0.19), 7)
    csr = csr_on_device(g)
    rng = np.random.default_rng(3)
    cases = [(rng.permutation(g.num_nodes)[:3000].astype(np.int32), [12, 8, 5], 0x1234),
             (rng.permutation(g.num_nodes)[:200].astype(np.int32), [6, 3], 0x99)]
    for seeds, fanouts, key in cases:
        want = _regular(csr, seeds, fanouts, key)
        got = _noalloc(csr, seeds, fanouts, key)
        ref = orc.sample_blocks(g.indptr, g.indices, seeds, fanouts, key)
        assert_blocks_equal(got, ref, f"no-alloc {len(seeds)} seeds")
        for l, (a, b) in enumerate(zip(got, want)):
            for k in a:
                assert np.array_equal(np.asarray(a[k]), np.asarray(b[k])), (len(seeds), l, k)
