"""The C-ABI library loads on the CPU, exports every symbol the header
declares, and rejects bad arguments on the host before touching any device
memory (no compute call is made here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gmb.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(gmb_[a-z_0-9]+)\s*\(", text)
    return sorted(set(names))


@pytest.fixture(scope="module")
def L():
    import paper_2010_05337_amd as gmb
    if not os.path.exists(gmb.LIB_PATH):
        from paper_2010_05337_amd import build
        build.build()
    return gmb.lib()


def test_every_declared_symbol_is_exported(L):
    import paper_2010_05337_amd as gmb
    names = _declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(L, n), n
    assert sorted(gmb.EXPORTS) == names


def test_no_oracle_symbols_in_library(L):
    for n in ("orc_philox4x32_10", "orc_sample_blocks", "orc_sage_linear"):
        with pytest.raises(AttributeError):
            getattr(L, n)


def test_product_and_oracle_share_no_code():
    """The HIP path and the oracle are written apart: no source of the
    package names the oracle, no source of the oracle names the package or
    its kernels' sources, and neither includes a header of the other."""
    def sources(d, exts):
        for base, _, files in os.walk(os.path.join(ROOT, d)):
            if "__pycache__" in base or "_build" in base:
                continue
            for f in files:
                if f.endswith(exts):
                    yield os.path.join(base, f)
    prod = list(sources("paper_2010_05337_amd", (".py", ".hip", ".hpp", ".h", ".cpp")))
    orc = list(sources("oracle", (".py", ".c", ".h")))
    assert prod and orc
    for f in prod:
        text = open(f).read()
        assert not re.search(r"^\s*(import|from)\s+oracle\b|\borc_[a-z]|\boracle\.", text, re.M), f
    for f in orc:
        text = open(f).read()
        assert not re.search(r"^\s*(import|from)\s+paper_2010_05337_amd\b|#\s*include\s*[<\"].*"
                             r"(gmb\.h|kernels\.hpp|common\.hpp|scan\.hpp|philox\.hpp)", text, re.M), f


def test_abi_version(L):
    assert L.gmb_abi_version() == 1


def test_state_bytes(L):
    assert L.gmb_sampler_state_bytes(0) == 0
    assert L.gmb_sampler_state_bytes(1 << 31) == 0
    assert L.gmb_sampler_state_bytes(10) == 256 + 256
    assert L.gmb_sampler_state_bytes(2449029) >= 256 + 4 * 2449029


def _fo(*f):
    return (ctypes.c_int32 * len(f))(*f)


def test_workspace_bytes_and_caps(L):
    assert L.gmb_sample_workspace_bytes(1000, _fo(15, 10, 5), 3, 2449029) > 0
    assert L.gmb_sample_workspace_bytes(0, _fo(5), 1, 10) > 0
    assert L.gmb_sample_workspace_bytes(10, _fo(5, 0), 2, 100) == 0
    assert b"fanouts[1]" in L.gmb_last_error()
    assert L.gmb_sample_workspace_bytes(10, _fo(5), 0, 100) == 0
    assert L.gmb_sample_workspace_bytes(10, _fo(*([2] * 9)), 9, 100) == 0
    assert L.gmb_sample_workspace_bytes(101, _fo(5), 1, 100) == 0
    # a hop whose capacity would not fit 31-bit positions
    assert L.gmb_sample_workspace_bytes(1 << 20, _fo(1 << 12), 1, (1 << 31) - 1) == 0
    assert b"exceeds" in L.gmb_last_error()
    # larger fan-outs never need less space
    a = L.gmb_sample_workspace_bytes(1000, _fo(15, 10, 5), 3, 2449029)
    b = L.gmb_sample_workspace_bytes(1000, _fo(16, 10, 5), 3, 2449029)
    assert b >= a


def test_sample_blocks_rejects_bad_arguments_on_host(L):
    import paper_2010_05337_amd as gmb
    fake = ctypes.c_void_p(1 << 20)   # never dereferenced: every case fails validation first
    csr = gmb.CsrStruct(100, 500, 1 << 20, 32, 0, 1 << 21)
    out = gmb.BlocksStruct()

    def call(csr_, nseeds, fo, L_, state_bytes=1 << 20, ws_bytes=1 << 30):
        return L.gmb_sample_blocks(ctypes.byref(csr_), fake, nseeds, fo, L_, 1, fake, state_bytes,
                                   fake, ws_bytes, ctypes.byref(out), None)

    assert call(csr, 10, _fo(5, 0), 2) == -1
    assert call(csr, 10, _fo(5), 9) == -1
    bad = gmb.CsrStruct(100, 500, 1 << 20, 16, 0, 1 << 21)
    assert call(bad, 10, _fo(5), 1) == -1
    assert b"indptr_bits" in L.gmb_last_error()
    assert call(csr, 10, _fo(5), 1, state_bytes=16) == -2
    assert call(csr, 10, _fo(5), 1, ws_bytes=64) == -2
    assert b"workspace" in L.gmb_last_error()
    assert L.gmb_sample_blocks(None, fake, 10, _fo(5), 1, 1, fake, 1 << 20, fake, 1 << 30,
                               ctypes.byref(out), None) == -1


def test_gather_rejects_bad_arguments_on_host(L):
    fake = ctypes.c_void_p(1 << 20)
    assert L.gmb_gather_features(fake, None, 10, fake, 100, 0, 0, fake, None, None) == -1
    assert L.gmb_gather_features(fake, None, 10, fake, 100, 16, 7, fake, None, None) == -1
    assert L.gmb_gather_features(fake, None, -1, fake, 100, 16, 0, fake, None, None) == -1
    assert L.gmb_gather_features(None, None, 10, fake, 100, 16, 0, fake, None, None) == -1
    # nothing to copy is not an error
    assert L.gmb_gather_features(None, None, 0, None, 100, 16, 0, None, None, None) == 0


def test_forward_rejects_bad_arguments_on_host(L):
    import paper_2010_05337_amd as gmb
    b = gmb.BlocksStruct()
    w = gmb.WeightsStruct()
    assert L.gmb_forward_workspace_bytes(ctypes.byref(b), ctypes.byref(w)) == 0
    b.num_layers = 2
    for l in range(2):
        for f in ("indptr", "indices", "src_ids", "sizes", "nbr"):
            setattr(b.blk[l], f, 1 << 20)
    b.blk[1].cap_dst, b.blk[1].cap_src, b.blk[1].cap_nnz = 64, 384, 320
    b.blk[0].cap_dst, b.blk[0].cap_src, b.blk[0].cap_nnz = 384, 2304, 1920
    w.num_layers, w.dtype = 2, 0
    for i, d in enumerate([16, 16, 8]):
        w.dims[i] = d
    for l in range(2):
        w.w_self[l] = w.w_neigh[l] = w.bias[l] = 1 << 20
    assert L.gmb_forward_workspace_bytes(ctypes.byref(b), ctypes.byref(w)) > 0
    assert L.gmb_forward_hidden_offset(ctypes.byref(b), ctypes.byref(w), 0) >= 0
    assert L.gmb_forward_hidden_offset(ctypes.byref(b), ctypes.byref(w), 1) == -1
    w.dtype = 5
    assert L.gmb_forward_workspace_bytes(ctypes.byref(b), ctypes.byref(w)) == 0
    w.dtype = 0
    b.blk[1].cap_src = 385    # block 1's sources must be block 0's destinations
    assert L.gmb_forward_workspace_bytes(ctypes.byref(b), ctypes.byref(w)) == 0
    assert b"destinations" in L.gmb_last_error()


def test_sample_noalloc_rejects_bad_arguments_on_host(L):
    """The no-allocation entry point checks its output buffer and the
    sampling arguments before it touches the device (or its scratch)."""
    import paper_2010_05337_amd as gmb
    fake = ctypes.c_void_p(1 << 20)
    csr = gmb.CsrStruct(100, 500, 1 << 20, 32, 0, 1 << 21)
    out = gmb.BlocksStruct()
    need = L.gmb_sample_workspace_bytes(10, _fo(5, 3), 2, 100)
    assert need > 0

    def call(buf, nbytes, fo=_fo(5, 3), L_=2):
        return L.gmb_sample_blocks_noalloc(ctypes.byref(csr), fake, 10, fo, L_, 1, fake, 1 << 20, buf, nbytes,
                                           ctypes.byref(out), None)

    assert call(None, need) == -1
    assert b"output buffer" in L.gmb_last_error()
    assert call(ctypes.c_void_p((1 << 20) + 64), need) == -1
    assert b"aligned" in L.gmb_last_error()
    assert call(fake, 256) == -2
    assert b"output buffer holds" in L.gmb_last_error()
    assert call(fake, need, fo=_fo(5, 0)) == -1
    assert call(fake, need, L_=9) == -1
