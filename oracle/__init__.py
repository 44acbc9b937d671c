"""CPU oracle of the mini-batch GNN hot path (TEST INFRASTRUCTURE).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg
may import this package.  The product path (``paper_2010_05337_amd``) never
imports it and shares no code with it.

The arithmetic lives in ``oracle.c`` (plain C, fp64, single-threaded); this
module compiles it with gcc, loads it with ctypes and composes the layers.
Every step follows DistDGL (arXiv 2010.05337) Section II-B (mini-batch
construction) and Section II-A Eq. (1) (message passing) as read in the
header of ``oracle.c``.

Parity status per function:
  philox4x32_10     pinned: published known-answer vectors (tests/golden)
  bounded_from_word pinned: exhaustive enumeration of all 2^32 words
  floyd             pinned: brute force over all draw sequences, d <= 8
  sample_node       pinned: chi-square uniformity, invariants
  sample_blocks     pinned: relabel invariants that determine it uniquely,
                    batch-composition independence
  gather            pinned: numpy fancy indexing
  mean_aggregate    pinned: dense D^-1 A H with numpy
  sage_forward      pinned: full-neighbourhood special case == full-graph
                    dense GraphSAGE (numpy)
  softmax_xent,     pinned: central finite differences of the loss in every
  sage_backward     parameter (fp64), and the full-neighbourhood special
                    case == torch autograd (fp64, CPU) of the dense
                    full-graph model; its input-row gradient likewise
                    (finite differences in every input entry, autograd of
                    the dense model in the feature matrix)
  embedding_sgd     pinned: rows outside the batch unchanged bit for bit,
                    the touched rows against the formula, repeated rows
                    refused; a small step lowers the loss
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

STATUS = {0: "OK", -1: "EINVAL", -4: "ERANGE", -5: "EDUP", -6: "ENOMEM"}


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle status {code} ({STATUS.get(code, '?')})")
        self.code = code


def build(force: bool = False) -> str:
    """Compile liboracle.so: gcc -O2, no fast-math, no SIMD intrinsics."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-Wall", _SRC,
                               "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        vp, i64, u32, u64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64
        L.orc_philox4x32_10.restype = None
        L.orc_philox4x32_10.argtypes = [vp, vp, vp]
        L.orc_bounded_from_word.restype = ctypes.c_int
        L.orc_bounded_from_word.argtypes = [u32, u32, ctypes.POINTER(u32)]
        L.orc_uniform_below.restype = u32
        L.orc_uniform_below.argtypes = [u64, u32, u32, u32, u32]
        L.orc_floyd.restype = None
        L.orc_floyd.argtypes = [u32, u32, vp, vp]
        L.orc_sample_node.restype = i64
        L.orc_sample_node.argtypes = [u64, u32, u32, i64, i64, vp]
        L.orc_sample_blocks.restype = ctypes.c_int
        L.orc_sample_blocks.argtypes = [i64, vp, vp, vp, i64, vp, ctypes.c_int, u64,
                                        ctypes.POINTER(vp)]
        L.orc_free_blocks.restype = None
        L.orc_free_blocks.argtypes = [vp]
        L.orc_block_sizes.restype = None
        L.orc_block_sizes.argtypes = [vp, ctypes.c_int, vp]
        L.orc_block_copy.restype = None
        L.orc_block_copy.argtypes = [vp, ctypes.c_int, vp, vp, vp, vp]
        L.orc_gather.restype = ctypes.c_int
        L.orc_gather.argtypes = [vp, i64, i64, vp, i64, vp]
        L.orc_mean_aggregate.restype = None
        L.orc_mean_aggregate.argtypes = [i64, vp, vp, vp, i64, vp]
        L.orc_sage_linear.restype = None
        L.orc_sage_linear.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, ctypes.c_int, vp]
        L.orc_softmax_xent.restype = ctypes.c_double
        L.orc_softmax_xent.argtypes = [i64, i64, vp, vp, vp]
        L.orc_sage_linear_backward.restype = None
        L.orc_sage_linear_backward.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.orc_mean_backward.restype = None
        L.orc_mean_backward.argtypes = [i64, vp, vp, vp, i64, vp]
        L.orc_relu_backward.restype = None
        L.orc_relu_backward.argtypes = [i64, vp, vp, vp]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a.size else None


# ---------------------------------------------------------------- O1 / O2 / O3

def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def bounded_from_word(x: int, m: int):
    """Lemire's draw from one word: the value in [0, m), or None if rejected."""
    t = ctypes.c_uint32(0)
    ok = lib().orc_bounded_from_word(x, m, ctypes.byref(t))
    return t.value if ok else None


def uniform_below(seed: int, v: int, l: int, i: int, m: int) -> int:
    return lib().orc_uniform_below(seed, v, l, i, m)


def floyd(d: int, k: int, draws) -> np.ndarray:
    t = np.ascontiguousarray(draws, dtype=np.uint32)
    out = np.zeros(max(k, 1), dtype=np.uint32)
    lib().orc_floyd(d, k, _p(t), _p(out))
    return out[:k]


def sample_node(seed: int, v: int, l: int, deg: int, fanout: int) -> np.ndarray:
    """Ascending row slots sampled for node v at layer l."""
    out = np.zeros(max(min(deg, fanout), 1), dtype=np.uint32)
    k = lib().orc_sample_node(seed, v, l, deg, fanout, _p(out))
    return out[:k]


# ---------------------------------------------------------------- O4

@dataclass
class Block:
    """Bipartite block of model layer l: destinations = src[:n_dst]."""
    n_dst: int
    n_src: int
    nnz: int
    indptr: np.ndarray   # int64 [n_dst+1]
    nbr: np.ndarray      # int64 [nnz] global ids of sampled in-neighbours
    local: np.ndarray    # int64 [nnz] positions in src
    src: np.ndarray      # int64 [n_src] global ids


def sample_blocks(indptr, indices, seeds, fanouts, seed: int):
    """Blocks for model layers 0..L-1 (index 0 = input layer)."""
    ip = np.ascontiguousarray(indptr, dtype=np.int64)
    ix = np.ascontiguousarray(indices, dtype=np.int32)
    sd = np.ascontiguousarray(seeds, dtype=np.int64)
    fo = np.ascontiguousarray(fanouts, dtype=np.int64)
    h = ctypes.c_void_p()
    st = lib().orc_sample_blocks(len(ip) - 1, _p(ip), _p(ix), _p(sd), len(sd), _p(fo), len(fo),
                                 seed & 0xFFFFFFFFFFFFFFFF, ctypes.byref(h))
    if st != 0:
        raise OracleError(st)
    try:
        blocks = []
        for l in range(len(fo)):
            sz = np.zeros(3, dtype=np.int64)
            lib().orc_block_sizes(h, l, _p(sz))
            n_dst, n_src, nnz = (int(x) for x in sz)
            b = Block(n_dst, n_src, nnz, np.zeros(n_dst + 1, np.int64), np.zeros(nnz, np.int64),
                      np.zeros(nnz, np.int64), np.zeros(n_src, np.int64))
            lib().orc_block_copy(h, l, _p(b.indptr), _p(b.nbr), _p(b.local), _p(b.src))
            blocks.append(b)
    finally:
        lib().orc_free_blocks(h)
    return blocks


# ---------------------------------------------------------------- O5

def gather(feats: np.ndarray, ids) -> np.ndarray:
    """Rows of `feats` at `ids`, copied bit for bit (any dtype)."""
    f = np.ascontiguousarray(feats)
    ii = np.ascontiguousarray(ids, dtype=np.int64)
    out = np.empty((len(ii),) + f.shape[1:], dtype=f.dtype)
    row_bytes = f.strides[0] if f.ndim > 1 else f.itemsize
    st = lib().orc_gather(_p(f), f.shape[0], row_bytes, _p(ii), len(ii), _p(out))
    if st != 0:
        raise OracleError(st)
    return out


def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact stored values as float64 (bf16 arrives as uint16 bit patterns)."""
    if dtype == "bf16":
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


# ---------------------------------------------------------------- O6

def mean_aggregate(block: Block, H: np.ndarray) -> np.ndarray:
    H = np.ascontiguousarray(H, dtype=np.float64)
    d = H.shape[1]
    m = np.zeros((block.n_dst, d), dtype=np.float64)
    lib().orc_mean_aggregate(block.n_dst, _p(block.indptr), _p(block.local), _p(H), d, _p(m))
    return m


def sage_linear(H_dst: np.ndarray, m: np.ndarray, w_self, w_neigh, bias, relu: bool) -> np.ndarray:
    H_dst = np.ascontiguousarray(H_dst, dtype=np.float64)
    m = np.ascontiguousarray(m, dtype=np.float64)
    ws = np.ascontiguousarray(w_self, dtype=np.float64)
    wn = np.ascontiguousarray(w_neigh, dtype=np.float64)
    b = np.ascontiguousarray(bias, dtype=np.float64)
    n, d_in = m.shape
    d_out = ws.shape[1]
    out = np.zeros((n, d_out), dtype=np.float64)
    lib().orc_sage_linear(n, d_in, d_out, _p(H_dst), _p(m), _p(ws), _p(wn), _p(b), int(relu),
                          _p(out))
    return out


def sage_forward(blocks, X: np.ndarray, w_self, w_neigh, bias):
    """GraphSAGE-mean over the blocks (layer 0 first).  X is the fp64 input
    of blocks[0]'s sources.  Returns (logits [B, C], [H_1, ..., H_L])."""
    H = np.ascontiguousarray(X, dtype=np.float64)
    outs = []
    L = len(blocks)
    for l, blk in enumerate(blocks):
        m = mean_aggregate(blk, H)
        H = sage_linear(H[:blk.n_dst], m, w_self[l], w_neigh[l], bias[l], relu=(l < L - 1))
        outs.append(H)
    return H, outs


# ---------------------------------------------------------------- O7

def softmax_xent(logits: np.ndarray, labels) -> tuple:
    """Mean softmax cross-entropy of the rows against labels and its
    gradient dL/dlogits.  Returns (loss, dlogits)."""
    z = np.ascontiguousarray(logits, dtype=np.float64)
    y = np.ascontiguousarray(labels, dtype=np.int64)
    n, C = z.shape
    if y.shape != (n,) or (n and (y.min() < 0 or y.max() >= C)):
        raise ValueError("labels must be [n] in [0, C)")
    dz = np.zeros_like(z)
    loss = lib().orc_softmax_xent(n, C, _p(z), _p(y), _p(dz))
    return float(loss), dz


def sage_forward_train(blocks, X: np.ndarray, w_self, w_neigh, bias):
    """The forward of sage_forward that also keeps each layer's mean.
    Returns (logits, [H_1, ..., H_L], [m_0, ..., m_{L-1}])."""
    H = np.ascontiguousarray(X, dtype=np.float64)
    outs, means = [], []
    L = len(blocks)
    for l, blk in enumerate(blocks):
        m = mean_aggregate(blk, H)
        H = sage_linear(H[:blk.n_dst], m, w_self[l], w_neigh[l], bias[l], relu=(l < L - 1))
        outs.append(H)
        means.append(m)
    return H, outs, means


def sage_backward(blocks, X: np.ndarray, w_self, w_neigh, hidden, means, dlogits, input_grad: bool = False):
    """Gradients of the loss in every parameter, from dL/dlogits back to
    layer 0.  hidden and means come from sage_forward_train.  Returns
    (dW_self, dW_neigh, db), lists by layer; with input_grad also dX, the
    gradient in the layer-0 input rows X [n_src(0), D] (the input has no
    activation, so nothing masks it)."""
    L = len(blocks)
    dWs, dWn, dbs = [None] * L, [None] * L, [None] * L
    dOut = np.ascontiguousarray(dlogits, dtype=np.float64)
    for l in range(L - 1, -1, -1):
        blk = blocks[l]
        Hin = np.ascontiguousarray(X if l == 0 else hidden[l - 1], dtype=np.float64)
        ws = np.ascontiguousarray(w_self[l], dtype=np.float64)
        wn = np.ascontiguousarray(w_neigh[l], dtype=np.float64)
        d_in, d_out = ws.shape
        n = blk.n_dst
        if l == L - 1:
            dZ = dOut
        else:
            out = np.ascontiguousarray(hidden[l], dtype=np.float64)
            dZ = np.zeros_like(out)
            lib().orc_relu_backward(out.size, _p(out), _p(dOut), _p(dZ))
        dZ = np.ascontiguousarray(dZ)
        dWs[l] = np.zeros((d_in, d_out))
        dWn[l] = np.zeros((d_in, d_out))
        dbs[l] = np.zeros(d_out)
        Hd = np.ascontiguousarray(Hin[:n])
        m = np.ascontiguousarray(means[l], dtype=np.float64)
        if l > 0 or input_grad:
            dH = np.zeros((blk.n_src, d_in))
            dM = np.zeros((n, d_in))
            dHd = np.zeros((n, d_in))
            lib().orc_sage_linear_backward(n, d_in, d_out, _p(Hd), _p(m), _p(ws), _p(wn), _p(dZ),
                                           _p(dWs[l]), _p(dWn[l]), _p(dbs[l]), _p(dHd), _p(dM))
            dH[:n] = dHd
            lib().orc_mean_backward(n, _p(blk.indptr), _p(blk.local), _p(dM), d_in, _p(dH))
            dOut = dH
        else:
            lib().orc_sage_linear_backward(n, d_in, d_out, _p(Hd), _p(m), _p(ws), _p(wn), _p(dZ),
                                           _p(dWs[l]), _p(dWn[l]), _p(dbs[l]), None, None)
    if input_grad:
        return dWs, dWn, dbs, dOut
    return dWs, dWn, dbs


def sgd(params, grads, lr: float):
    """p - lr * g for every array."""
    return [np.asarray(p, dtype=np.float64) - lr * np.asarray(g, dtype=np.float64)
            for p, g in zip(params, grads)]


def embedding_sgd(table: np.ndarray, rows, dX: np.ndarray, lr: float) -> np.ndarray:
    """The sparse update of learnable vertex embeddings (Section III-E: SGD
    on the rows a mini-batch touched): table[rows[u]] -= lr * dX[u].  The
    rows of one mini-batch are distinct (its input vertices).  Returns the
    updated copy."""
    out = np.array(table, dtype=np.float64, copy=True)
    rows = np.asarray(rows, dtype=np.int64)
    if len(np.unique(rows)) != len(rows):
        raise ValueError("the rows of one mini-batch must be distinct")
    out[rows] -= lr * np.asarray(dX, dtype=np.float64)
    return out


def sage_train_step_embed(blocks, table: np.ndarray, w_self, w_neigh, bias, labels, lr: float, emb_lr: float):
    """A training step whose layer-0 inputs are learnable vertex embeddings:
    X = table[src(0)], forward, loss, backward down to X, SGD on the dense
    weights and on the embedding rows.  Returns (loss, (dW_self, dW_neigh,
    db), dX, (new W_self, new W_neigh, new b), new table)."""
    X = np.asarray(table, dtype=np.float64)[np.asarray(blocks[0].src, dtype=np.int64)]
    logits, hidden, means = sage_forward_train(blocks, X, w_self, w_neigh, bias)
    loss, dz = softmax_xent(logits, labels)
    dWs, dWn, dbs, dX = sage_backward(blocks, X, w_self, w_neigh, hidden, means, dz, input_grad=True)
    return (loss, (dWs, dWn, dbs), dX, (sgd(w_self, dWs, lr), sgd(w_neigh, dWn, lr), sgd(bias, dbs, lr)),
            embedding_sgd(table, blocks[0].src, dX, emb_lr))


def sage_train_step(blocks, X: np.ndarray, w_self, w_neigh, bias, labels, lr: float):
    """Forward, loss, backward and one SGD step.  Returns (loss, logits,
    (dW_self, dW_neigh, db), (new W_self, new W_neigh, new b))."""
    logits, hidden, means = sage_forward_train(blocks, X, w_self, w_neigh, bias)
    loss, dz = softmax_xent(logits, labels)
    dWs, dWn, dbs = sage_backward(blocks, X, w_self, w_neigh, hidden, means, dz)
    return loss, logits, (dWs, dWn, dbs), (sgd(w_self, dWs, lr), sgd(w_neigh, dWn, lr), sgd(bias, dbs, lr))
