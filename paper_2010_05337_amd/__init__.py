"""Mini-batch GNN hot path on MI355X: Python binding of libgmb.so.

Argument marshalling only: every step runs in the HIP kernels behind the C
ABI declared in include/gmb.h.  PyTorch provides device memory and the
current stream.  There is no CPU fallback: without the built library (or
without a GPU) every call raises.

    csr = CSRGraph(indptr, indices)                 # device tensors
    blocks = sample_blocks(csr, seeds, [15, 10, 5], seed=0)
    x = gather_features(blocks, feats)              # [cap_src0, D]
    logits = sage_forward(blocks, x, weights)       # [B, C] fp32

The three calls follow DistDGL (arXiv 2010.05337) Section II-B (sampling a
mini-batch), Section III-C (pulling its vertex features) and Section II-A
Eq. (1) with the GraphSAGE-mean model of Section IV.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgmb.so")

GMB_MAX_LAYERS = 8
GMB_F32, GMB_BF16 = 0, 1
STATUS = {0: "OK", -1: "EINVAL", -2: "ENOSPC", -3: "EDEVICE", -4: "ERANGE", -5: "EDUP"}
EXPORTS = (
    "gmb_abi_version", "gmb_last_error", "gmb_sampler_state_bytes", "gmb_sampler_state_init",
    "gmb_state_status_word", "gmb_read_status", "gmb_sample_workspace_bytes", "gmb_sample_blocks",
    "gmb_read_sizes", "gmb_gather_features", "gmb_forward_workspace_bytes",
    "gmb_forward_hidden_offset", "gmb_sage_forward", "gmb_sage_forward_fused", "gmb_backward_workspace_bytes",
    "gmb_sage_backward", "gmb_sgd_update", "gmb_backward_embedding_workspace_bytes",
    "gmb_sage_backward_embedding", "gmb_sample_blocks_noalloc",
    "gmb_validate_blocks", "gmb_sgd_update_bf16",
)


class GmbError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class CsrStruct(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("num_edges", ctypes.c_int64),
                ("indptr", ctypes.c_void_p), ("indptr_bits", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("indices", ctypes.c_void_p)]


class BlockStruct(ctypes.Structure):
    _fields_ = [("indptr", ctypes.c_void_p), ("indices", ctypes.c_void_p), ("nbr", ctypes.c_void_p),
                ("src_ids", ctypes.c_void_p), ("sizes", ctypes.c_void_p),
                ("cap_dst", ctypes.c_int64), ("cap_src", ctypes.c_int64), ("cap_nnz", ctypes.c_int64),
                ("fanout", ctypes.c_int32), ("layer", ctypes.c_int32)]


class BlocksStruct(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_seeds", ctypes.c_int32),
                ("blk", BlockStruct * GMB_MAX_LAYERS)]


class WeightsStruct(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("dims", ctypes.c_int32 * (GMB_MAX_LAYERS + 1)),
                ("w_self", ctypes.c_void_p * GMB_MAX_LAYERS),
                ("w_neigh", ctypes.c_void_p * GMB_MAX_LAYERS),
                ("bias", ctypes.c_void_p * GMB_MAX_LAYERS)]


class GradsStruct(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("d_self", ctypes.c_void_p * GMB_MAX_LAYERS),
                ("d_neigh", ctypes.c_void_p * GMB_MAX_LAYERS),
                ("d_bias", ctypes.c_void_p * GMB_MAX_LAYERS)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded C ABI; raises if libgmb.so has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2010_05337_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, u64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                                 ctypes.c_size_t)
        L.gmb_abi_version.restype = i32
        L.gmb_last_error.restype = ctypes.c_char_p
        L.gmb_sampler_state_bytes.restype = sz
        L.gmb_sampler_state_bytes.argtypes = [i64]
        L.gmb_sampler_state_init.restype = ctypes.c_int
        L.gmb_sampler_state_init.argtypes = [vp, sz, i64, vp]
        L.gmb_state_status_word.restype = vp
        L.gmb_state_status_word.argtypes = [vp]
        L.gmb_read_status.restype = ctypes.c_int
        L.gmb_read_status.argtypes = [vp, vp]
        L.gmb_sample_workspace_bytes.restype = sz
        L.gmb_sample_workspace_bytes.argtypes = [i32, vp, i32, i64]
        L.gmb_sample_blocks.restype = ctypes.c_int
        L.gmb_sample_blocks.argtypes = [ctypes.POINTER(CsrStruct), vp, i32, vp, i32, u64, vp, sz, vp,
                                        sz, ctypes.POINTER(BlocksStruct), vp]
        L.gmb_sample_blocks_noalloc.restype = ctypes.c_int
        L.gmb_sample_blocks_noalloc.argtypes = [ctypes.POINTER(CsrStruct), vp, i32, vp, i32, u64, vp, sz, vp,
                                                sz, ctypes.POINTER(BlocksStruct), vp]
        L.gmb_validate_blocks.restype = ctypes.c_int
        L.gmb_validate_blocks.argtypes = [ctypes.POINTER(CsrStruct), ctypes.POINTER(BlocksStruct), vp, vp]
        L.gmb_read_sizes.restype = ctypes.c_int
        L.gmb_read_sizes.argtypes = [ctypes.POINTER(BlocksStruct), vp, vp]
        L.gmb_gather_features.restype = ctypes.c_int
        L.gmb_gather_features.argtypes = [vp, vp, i64, vp, i64, i32, i32, vp, vp, vp]
        L.gmb_forward_workspace_bytes.restype = sz
        L.gmb_forward_workspace_bytes.argtypes = [ctypes.POINTER(BlocksStruct),
                                                  ctypes.POINTER(WeightsStruct)]
        L.gmb_forward_hidden_offset.restype = i64
        L.gmb_forward_hidden_offset.argtypes = [ctypes.POINTER(BlocksStruct),
                                                ctypes.POINTER(WeightsStruct), i32]
        L.gmb_sage_forward.restype = ctypes.c_int
        L.gmb_sage_forward.argtypes = [ctypes.POINTER(BlocksStruct), vp, ctypes.POINTER(WeightsStruct),
                                       vp, vp, sz, vp]
        L.gmb_sage_forward_fused.restype = ctypes.c_int
        L.gmb_sage_forward_fused.argtypes = [ctypes.POINTER(BlocksStruct), vp, ctypes.c_int64, vp,
                                             ctypes.POINTER(WeightsStruct), vp, vp, sz, vp, vp]
        L.gmb_backward_workspace_bytes.restype = sz
        L.gmb_backward_workspace_bytes.argtypes = [ctypes.POINTER(BlocksStruct),
                                                   ctypes.POINTER(WeightsStruct)]
        L.gmb_sage_backward.restype = ctypes.c_int
        L.gmb_sage_backward.argtypes = [ctypes.POINTER(BlocksStruct), vp, ctypes.POINTER(WeightsStruct), vp, vp,
                                        vp, sz, ctypes.POINTER(GradsStruct), vp, vp, sz, vp]
        L.gmb_backward_embedding_workspace_bytes.restype = sz
        L.gmb_backward_embedding_workspace_bytes.argtypes = [ctypes.POINTER(BlocksStruct),
                                                             ctypes.POINTER(WeightsStruct)]
        L.gmb_sage_backward_embedding.restype = ctypes.c_int
        L.gmb_sage_backward_embedding.argtypes = [ctypes.POINTER(BlocksStruct), vp, ctypes.POINTER(WeightsStruct),
                                                  vp, vp, vp, sz, ctypes.POINTER(GradsStruct), vp, vp, sz, vp,
                                                  ctypes.c_int64, ctypes.c_float, vp]
        L.gmb_sgd_update_bf16.restype = ctypes.c_int
        L.gmb_sgd_update_bf16.argtypes = [ctypes.POINTER(WeightsStruct), ctypes.POINTER(WeightsStruct),
                                          ctypes.POINTER(GradsStruct), ctypes.c_float, vp]
        L.gmb_sgd_update.restype = ctypes.c_int
        L.gmb_sgd_update.argtypes = [ctypes.POINTER(WeightsStruct), ctypes.POINTER(GradsStruct),
                                     ctypes.c_float, vp]
        _lib = L
    return _lib


def _check(code: int):
    if code != 0:
        raise GmbError(code, lib().gmb_last_error().decode(errors="replace"))


def _stream_handle():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _require_cuda(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _aligned_bytes(nbytes: int, device) -> tuple:
    """A uint8 device buffer with a 256-byte aligned view of nbytes."""
    buf = torch.empty(max(nbytes, 1) + 256, dtype=torch.uint8, device=device)
    off = (-buf.data_ptr()) % 256
    return buf, buf[off:off + max(nbytes, 1)]


class CSRGraph:
    """In-neighbour CSR on the device (row v lists the sources of the edges
    into v), plus the sampler state (a per-vertex dedup table) that
    sample_blocks needs."""

    def __init__(self, indptr: torch.Tensor, indices: torch.Tensor):
        _require_cuda(indptr, "indptr")
        _require_cuda(indices, "indices")
        if indptr.dtype not in (torch.int32, torch.int64):
            raise TypeError("indptr must be int32 or int64")
        if indices.dtype != torch.int32:
            raise TypeError("indices must be int32")
        self.indptr, self.indices = indptr, indices
        self.num_nodes = indptr.numel() - 1
        self.num_edges = indices.numel()
        self.struct = CsrStruct(self.num_nodes, self.num_edges, indptr.data_ptr(),
                                32 if indptr.dtype == torch.int32 else 64, 0,
                                indices.data_ptr() if self.num_edges else None)
        nbytes = lib().gmb_sampler_state_bytes(self.num_nodes)
        if nbytes == 0:
            raise GmbError(-1, f"num_nodes={self.num_nodes} unsupported")
        self._state_buf, self.state = _aligned_bytes(nbytes, indptr.device)
        self.state_bytes = nbytes
        _check(lib().gmb_sampler_state_init(ctypes.c_void_p(self.state.data_ptr()), nbytes,
                                            self.num_nodes, _stream_handle()))

    @property
    def status_word(self) -> int:
        return lib().gmb_state_status_word(ctypes.c_void_p(self.state.data_ptr()))

    def check_status(self):
        """Synchronises, then raises GmbError for a data error found on the device."""
        _check(lib().gmb_read_status(ctypes.c_void_p(self.state.data_ptr()), _stream_handle()))


class Block:
    """Host view of one block after the sizes were read (tensors are views
    into the workspace, cut to the device-side sizes)."""

    def __init__(self, n_dst, n_src, nnz, indptr, indices, nbr, src_ids, fanout, layer):
        self.n_dst, self.n_src, self.nnz = n_dst, n_src, nnz
        self.indptr, self.indices, self.nbr, self.src_ids = indptr, indices, nbr, src_ids
        self.fanout, self.layer = fanout, layer


class Blocks:
    """The L blocks of one mini-batch (index 0 = input layer).  Sizes stay on
    the device until sizes() is called."""

    def __init__(self, struct: BlocksStruct, workspace: torch.Tensor, csr: CSRGraph):
        self.struct = struct
        self.workspace = workspace
        self.csr = csr
        self.num_layers = struct.num_layers
        self.num_seeds = struct.num_seeds

    def _view(self, ptr: int, n: int) -> torch.Tensor:
        off = ptr - self.workspace.data_ptr()
        return self.workspace[off:off + 4 * n].view(torch.int32)

    @property
    def input_ids(self) -> torch.Tensor:
        """Block 0's source ids at full capacity (valid prefix: n_src of block 0)."""
        b = self.struct.blk[0]
        return self._view(b.src_ids, b.cap_src)

    @property
    def input_count_ptr(self) -> int:
        """Device address of block 0's n_src word."""
        return self.struct.blk[0].sizes + 4 * 1

    @property
    def input_capacity(self) -> int:
        return int(self.struct.blk[0].cap_src)

    def sizes(self):
        """[(n_dst, n_src, nnz)] per layer (synchronises the stream)."""
        out = (ctypes.c_int64 * (3 * self.num_layers))()
        _check(lib().gmb_read_sizes(ctypes.byref(self.struct), out, _stream_handle()))
        return [tuple(int(out[3 * l + i]) for i in range(3)) for l in range(self.num_layers)]

    def validate(self):
        """Enqueues the device consistency check of the blocks; a violation
        shows in the next csr.check_status() (GmbError EDEVICE)."""
        _check(lib().gmb_validate_blocks(ctypes.byref(self.csr.struct), ctypes.byref(self.struct),
                                         ctypes.c_void_p(self.csr.state.data_ptr()), _stream_handle()))

    def blocks(self):
        """Per-layer Block views cut to the device sizes (synchronises)."""
        res = []
        for l, (n_dst, n_src, nnz) in enumerate(self.sizes()):
            b = self.struct.blk[l]
            res.append(Block(n_dst, n_src, nnz, self._view(b.indptr, n_dst + 1),
                             self._view(b.indices, nnz), self._view(b.nbr, nnz),
                             self._view(b.src_ids, n_src), int(b.fanout), int(b.layer)))
        return res


def sample_workspace_bytes(num_seeds: int, fanouts, num_nodes: int) -> int:
    fo = (ctypes.c_int32 * len(fanouts))(*fanouts)
    return lib().gmb_sample_workspace_bytes(num_seeds, fo, len(fanouts), num_nodes)


def sample_blocks(csr: CSRGraph, seeds: torch.Tensor, fanouts, seed: int,
                  workspace: torch.Tensor | None = None) -> Blocks:
    """Samples an L-layer mini-batch from `seeds` (device int32, distinct);
    fanouts[l] belongs to model layer l (l = 0 is the input layer)."""
    _require_cuda(seeds, "seeds")
    if seeds.dtype != torch.int32:
        raise TypeError("seeds must be int32")
    fanouts = [int(f) for f in fanouts]
    fo = (ctypes.c_int32 * len(fanouts))(*fanouts)
    need = lib().gmb_sample_workspace_bytes(seeds.numel(), fo, len(fanouts), csr.num_nodes)
    if need == 0:
        _check(-1)
    if workspace is None or workspace.numel() < need or workspace.data_ptr() % 256:
        _, workspace = _aligned_bytes(need, seeds.device)
    out = BlocksStruct()
    _check(lib().gmb_sample_blocks(ctypes.byref(csr.struct),
                                   ctypes.c_void_p(seeds.data_ptr()) if seeds.numel() else None,
                                   seeds.numel(), fo, len(fanouts), seed & 0xFFFFFFFFFFFFFFFF,
                                   ctypes.c_void_p(csr.state.data_ptr()), csr.state_bytes,
                                   ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                   ctypes.byref(out), _stream_handle()))
    return Blocks(out, workspace, csr)


def gather_features(ids, feats: torch.Tensor, n: int | None = None,
                    out: torch.Tensor | None = None, status_word: int | None = None) -> torch.Tensor:
    """out[i] = feats[ids[i]] bit for bit.  `ids` is a Blocks (its input
    vertices; the count stays on the device and the result has the blocks'
    input capacity in rows) or a device int32 tensor (all of it, or the
    first n)."""
    _require_cuda(feats, "feats")
    if feats.dim() != 2:
        raise ValueError("feats must be [num_nodes, dim]")
    if feats.dtype == torch.float32:
        dtype = GMB_F32
    elif feats.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        dtype = GMB_BF16
    else:
        raise TypeError("feats must be float32 or bfloat16")
    n_dev = None
    if isinstance(ids, Blocks):
        cap = ids.input_capacity
        n_dev = ctypes.c_void_p(ids.input_count_ptr)
        if status_word is None:
            status_word = ids.csr.status_word
        ids_t = ids.input_ids
    else:
        _require_cuda(ids, "ids")
        if ids.dtype != torch.int32:
            raise TypeError("ids must be int32")
        ids_t = ids
        cap = ids.numel() if n is None else int(n)
        if cap > ids.numel():
            raise ValueError("n exceeds ids")
    if out is None:
        out = torch.empty((cap, feats.shape[1]), dtype=feats.dtype, device=feats.device)
    elif out.shape[0] < cap or out.shape[1] != feats.shape[1] or out.dtype != feats.dtype:
        raise ValueError("out has the wrong shape or dtype")
    _check(lib().gmb_gather_features(ctypes.c_void_p(ids_t.data_ptr()) if cap else None, n_dev, cap,
                                     ctypes.c_void_p(feats.data_ptr()), feats.shape[0], feats.shape[1],
                                     dtype, ctypes.c_void_p(out.data_ptr()) if cap else None,
                                     ctypes.c_void_p(status_word) if status_word else None,
                                     _stream_handle()))
    return out


class SageWeights:
    """GraphSAGE-mean weights on the device: W_self[l], W_neigh[l]
    [dims[l], dims[l+1]] (float32 or bfloat16) and bias[l] float32."""

    def __init__(self, w_self, w_neigh, bias):
        if not (len(w_self) == len(w_neigh) == len(bias)) or not w_self:
            raise ValueError("one W_self, W_neigh and bias per layer")
        if len(w_self) > GMB_MAX_LAYERS:
            raise ValueError("too many layers")
        self.w_self = [w.contiguous() for w in w_self]
        self.w_neigh = [w.contiguous() for w in w_neigh]
        self.bias = [b.contiguous().float() for b in bias]
        dt = self.w_self[0].dtype
        self.dtype = GMB_BF16 if dt == torch.bfloat16 else GMB_F32
        if dt not in (torch.float32, torch.bfloat16):
            raise TypeError("weights must be float32 or bfloat16")
        dims = [self.w_self[0].shape[0]] + [w.shape[1] for w in self.w_self]
        for l, (a, b) in enumerate(zip(self.w_self, self.w_neigh)):
            if a.shape != b.shape or a.shape != (dims[l], dims[l + 1]) or a.dtype != dt or b.dtype != dt:
                raise ValueError(f"layer {l}: W_self/W_neigh shapes or dtypes disagree")
            _require_cuda(a, "w_self")
            _require_cuda(b, "w_neigh")
            _require_cuda(self.bias[l], "bias")
        self.dims = dims
        s = WeightsStruct()
        s.num_layers = len(self.w_self)
        s.dtype = self.dtype
        for i, d in enumerate(dims):
            s.dims[i] = d
        for l in range(len(self.w_self)):
            s.w_self[l] = self.w_self[l].data_ptr()
            s.w_neigh[l] = self.w_neigh[l].data_ptr()
            s.bias[l] = self.bias[l].data_ptr()
        self.struct = s

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == GMB_BF16 else torch.float32

    def master(self) -> "SageWeights":
        """fp32 copies of the matrices (the biases are shared): the master
        weights that sgd_update_bf16 updates for a bf16 model."""
        return SageWeights([w.float() for w in self.w_self], [w.float() for w in self.w_neigh], self.bias)


def forward_workspace_bytes(blocks: Blocks, weights: SageWeights) -> int:
    return lib().gmb_forward_workspace_bytes(ctypes.byref(blocks.struct), ctypes.byref(weights.struct))


def sage_forward(blocks: Blocks, feats: torch.Tensor, weights: SageWeights,
                 workspace: torch.Tensor | None = None, logits: torch.Tensor | None = None,
                 return_hidden: bool = False):
    """GraphSAGE-mean forward over the blocks; feats holds the gathered input
    rows of block 0's sources.  Returns logits [num_seeds, C] float32 (and,
    with return_hidden, the hidden activations cut to their row counts)."""
    _require_cuda(feats, "feats")
    if feats.dtype != weights.torch_dtype:
        raise TypeError("feats and weights must have the same dtype")
    if feats.dim() != 2 or feats.shape[1] != weights.dims[0] or feats.shape[0] < blocks.input_capacity:
        raise ValueError("feats must be [input capacity, dims[0]]")
    need = lib().gmb_forward_workspace_bytes(ctypes.byref(blocks.struct), ctypes.byref(weights.struct))
    if need == 0:
        _check(-1)
    if workspace is None or workspace.numel() < need or workspace.data_ptr() % 256:
        _, workspace = _aligned_bytes(need, feats.device)
    B, C = blocks.num_seeds, weights.dims[-1]
    if logits is None:
        logits = torch.empty((max(B, 0), C), dtype=torch.float32, device=feats.device)
    _check(lib().gmb_sage_forward(ctypes.byref(blocks.struct), ctypes.c_void_p(feats.data_ptr()),
                                  ctypes.byref(weights.struct), ctypes.c_void_p(logits.data_ptr()),
                                  ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                  _stream_handle()))
    if not return_hidden:
        return logits
    return logits, _hidden_views(blocks, weights, workspace)


def _hidden_views(blocks: Blocks, weights: SageWeights, workspace: torch.Tensor):
    hidden = []
    sizes = blocks.sizes()
    es = 2 if weights.dtype == GMB_BF16 else 4
    for l in range(blocks.num_layers - 1):
        off = lib().gmb_forward_hidden_offset(ctypes.byref(blocks.struct), ctypes.byref(weights.struct), l)
        n = sizes[l][0]
        d = weights.dims[l + 1]
        h = workspace[off:off + n * d * es].view(weights.torch_dtype).view(n, d)
        hidden.append(h)
    return hidden


def dst_capacity(blocks: Blocks) -> int:
    """Rows of block 0's destinations (the x_dst buffer of the fused forward)."""
    return int(blocks.struct.blk[0].cap_dst)


def sage_forward_fused(blocks: Blocks, feats: torch.Tensor, weights: SageWeights,
                       x_dst: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                       logits: torch.Tensor | None = None, return_hidden: bool = False):
    """The forward with the feature pull folded into layer 0: `feats` is the
    whole feature table [num_nodes, dims[0]]; block 0's destination rows are
    gathered into x_dst ([dst capacity, dims[0]]), the layer-0 mean reads
    the table directly.  Returns (logits, x_dst) (and the hidden
    activations with return_hidden); x_dst serves as `x` of sage_backward."""
    _require_cuda(feats, "feats")
    if feats.dtype != weights.torch_dtype:
        raise TypeError("feats and weights must have the same dtype")
    if feats.dim() != 2 or feats.shape[1] != weights.dims[0]:
        raise ValueError("feats must be [num_nodes, dims[0]]")
    need = lib().gmb_forward_workspace_bytes(ctypes.byref(blocks.struct), ctypes.byref(weights.struct))
    if need == 0:
        _check(-1)
    if workspace is None or workspace.numel() < need or workspace.data_ptr() % 256:
        _, workspace = _aligned_bytes(need, feats.device)
    if x_dst is None:
        x_dst = torch.empty((dst_capacity(blocks), weights.dims[0]), dtype=feats.dtype, device=feats.device)
    if x_dst.dtype != feats.dtype or x_dst.dim() != 2 or x_dst.shape[1] != weights.dims[0] or \
            x_dst.shape[0] < dst_capacity(blocks) or not x_dst.is_contiguous():
        raise ValueError("x_dst must be a contiguous [dst capacity, dims[0]] tensor of the features' dtype")
    B, C = blocks.num_seeds, weights.dims[-1]
    if logits is None:
        logits = torch.empty((max(B, 0), C), dtype=torch.float32, device=feats.device)
    _check(lib().gmb_sage_forward_fused(ctypes.byref(blocks.struct), ctypes.c_void_p(feats.data_ptr()),
                                        feats.shape[0], ctypes.c_void_p(x_dst.data_ptr()),
                                        ctypes.byref(weights.struct), ctypes.c_void_p(logits.data_ptr()),
                                        ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                        ctypes.c_void_p(blocks.csr.status_word), _stream_handle()))
    if not return_hidden:
        return logits, x_dst
    return logits, x_dst, _hidden_views(blocks, weights, workspace)


# ---------------------------------------------------------------- training

class SageGrads:
    """fp32 gradient arrays laid out like the weights (device tensors)."""

    def __init__(self, weights: SageWeights):
        dev = weights.w_self[0].device
        self.d_self = [torch.zeros(w.shape, dtype=torch.float32, device=dev) for w in weights.w_self]
        self.d_neigh = [torch.zeros(w.shape, dtype=torch.float32, device=dev) for w in weights.w_neigh]
        self.d_bias = [torch.zeros(b.shape, dtype=torch.float32, device=dev) for b in weights.bias]
        g = GradsStruct()
        g.num_layers = len(self.d_self)
        for l in range(g.num_layers):
            g.d_self[l] = self.d_self[l].data_ptr()
            g.d_neigh[l] = self.d_neigh[l].data_ptr()
            g.d_bias[l] = self.d_bias[l].data_ptr()
        self.struct = g


def backward_workspace_bytes(blocks: Blocks, weights: SageWeights) -> int:
    return lib().gmb_backward_workspace_bytes(ctypes.byref(blocks.struct), ctypes.byref(weights.struct))


def backward_embedding_workspace_bytes(blocks: Blocks, weights: SageWeights) -> int:
    return lib().gmb_backward_embedding_workspace_bytes(ctypes.byref(blocks.struct), ctypes.byref(weights.struct))


def sage_backward(blocks: Blocks, feats: torch.Tensor, weights: SageWeights, logits: torch.Tensor,
                  labels: torch.Tensor, fwd_workspace: torch.Tensor, grads: SageGrads | None = None,
                  loss: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                  embedding: torch.Tensor | None = None, emb_lr: float = 0.0):
    """Gradients of the mean softmax cross-entropy of `logits` (from the
    sage_forward call that used `fwd_workspace`) against `labels` (device
    int32, one per seed).  Returns (grads, loss) with loss a 1-element
    float32 device tensor.  With `embedding` (the fp32 [num_nodes, dims[0]]
    table the layer-0 inputs were taken from) the gradient in the input
    rows is applied to the table as an SGD step of size emb_lr."""
    _require_cuda(labels, "labels")
    if labels.dtype != torch.int32 or labels.numel() < blocks.num_seeds:
        raise TypeError("labels must be int32 with one entry per seed")
    if embedding is not None:
        _require_cuda(embedding, "embedding")
        if embedding.dtype != torch.float32 or embedding.dim() != 2 or embedding.shape[1] != weights.dims[0] \
                or not embedding.is_contiguous():
            raise ValueError("embedding must be a contiguous float32 [num_nodes, dims[0]] tensor")
        need = backward_embedding_workspace_bytes(blocks, weights)
    else:
        need = backward_workspace_bytes(blocks, weights)
    if need == 0:
        _check(-1)
    if workspace is None or workspace.numel() < need or workspace.data_ptr() % 256:
        _, workspace = _aligned_bytes(need, feats.device)
    if grads is None:
        grads = SageGrads(weights)
    if loss is None:
        loss = torch.empty(1, dtype=torch.float32, device=feats.device)
    common = (ctypes.byref(blocks.struct), ctypes.c_void_p(feats.data_ptr()), ctypes.byref(weights.struct),
              ctypes.c_void_p(logits.data_ptr()), ctypes.c_void_p(labels.data_ptr()),
              ctypes.c_void_p(fwd_workspace.data_ptr()), fwd_workspace.numel(), ctypes.byref(grads.struct),
              ctypes.c_void_p(loss.data_ptr()), ctypes.c_void_p(workspace.data_ptr()), workspace.numel())
    if embedding is None:
        _check(lib().gmb_sage_backward(*common, _stream_handle()))
    else:
        _check(lib().gmb_sage_backward_embedding(*common, ctypes.c_void_p(embedding.data_ptr()),
                                                 embedding.shape[0], float(emb_lr), _stream_handle()))
    return grads, loss


def sgd_update(weights: SageWeights, grads: SageGrads, lr: float):
    """W -= lr * dW and b -= lr * db in place (fp32 weights)."""
    _check(lib().gmb_sgd_update(ctypes.byref(weights.struct), ctypes.byref(grads.struct), float(lr),
                                _stream_handle()))


def sgd_update_bf16(weights: SageWeights, master: SageWeights, grads: SageGrads, lr: float):
    """One SGD step of a bf16 model: the fp32 master weights W -= lr * dW,
    then the bf16 matrices become the new masters rounded to nearest even
    (the biases, fp32 in both, are updated in the master and copied)."""
    _check(lib().gmb_sgd_update_bf16(ctypes.byref(weights.struct), ctypes.byref(master.struct),
                                     ctypes.byref(grads.struct), float(lr), _stream_handle()))
