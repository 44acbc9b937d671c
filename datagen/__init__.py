"""Seeded synthetic inputs shared by the oracle and the GPU path.

This package produces *inputs only*: CSR graphs, feature tables, SAGE
weights, training sets and seed batches.  It holds none of the method's
arithmetic.  The heavy generators live in ``datagen.c`` (host C, threaded,
deterministic for any thread count); small arrays (weights, permutations)
come from numpy's PCG64 generator.

The workloads stand in for the two Open Graph Benchmark datasets the paper
evaluates on (Table I: a 2.4M-node product co-purchase graph with 100-d
features and a 111M-node citation graph with 128-d features); only their
shapes are reproduced.  No dataset record is used or reproduced.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "datagen.c")
_LIB = os.path.join(_HERE, "libdatagen.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile libdatagen.so with gcc (host only)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-pthread",
                               "-Wall", "-Wno-unused-function", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        i64, u64, i32p, i64p = ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p
        lib.dg_er_count.restype = i64
        lib.dg_er_count.argtypes = [i64, ctypes.c_double, u64, i64p]
        lib.dg_er_fill.restype = None
        lib.dg_er_fill.argtypes = [i64, ctypes.c_double, u64, i64p, i32p]
        lib.dg_rmat.restype = i64
        lib.dg_rmat.argtypes = [ctypes.c_int, i64, i64, ctypes.c_double, ctypes.c_double,
                                ctypes.c_double, u64, i64p, ctypes.POINTER(ctypes.c_void_p)]
        lib.dg_inject_hubs.restype = i64
        lib.dg_inject_hubs.argtypes = [i64, i64p, i32p, i64, i64, u64, i64p, i64p,
                                       ctypes.POINTER(ctypes.c_void_p)]
        lib.dg_features_f32.restype = None
        lib.dg_features_f32.argtypes = [i64, i64, u64, ctypes.c_void_p]
        lib.dg_features_bf16.restype = None
        lib.dg_features_bf16.argtypes = [i64, i64, u64, ctypes.c_void_p]
        lib.dg_free.restype = None
        lib.dg_free.argtypes = [ctypes.c_void_p]
        lib.dg_set_threads.restype = None
        lib.dg_set_threads.argtypes = [ctypes.c_int]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _take_indices(lib, handle: ctypes.c_void_p, nnz: int) -> np.ndarray:
    if nnz == 0:
        lib.dg_free(handle)
        return np.zeros(0, dtype=np.int32)
    buf = (ctypes.c_int32 * nnz).from_address(handle.value)
    out = np.frombuffer(buf, dtype=np.int32).copy()
    lib.dg_free(handle)
    return out


@dataclass
class Graph:
    """In-neighbour CSR: row v lists the sources u of the edges u -> v,
    ascending and unique, no self-loops."""
    num_nodes: int
    indptr: np.ndarray   # int64 [N+1]
    indices: np.ndarray  # int32 [nnz]
    hubs: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))

    @property
    def num_edges(self) -> int:
        return int(self.indptr[-1])

    def degrees(self) -> np.ndarray:
        return np.diff(self.indptr)


def er_directed(n: int, avg_deg: float, seed: int) -> Graph:
    """Directed G(n, p) with p = avg_deg / (n - 1) (Batagelj-Brandes skipping)."""
    lib = _load()
    p = avg_deg / (n - 1)
    indptr = np.zeros(n + 1, dtype=np.int64)
    nnz = lib.dg_er_count(n, p, seed, _ptr(indptr))
    indices = np.zeros(max(nnz, 1), dtype=np.int32)[:nnz]
    lib.dg_er_fill(n, p, seed, _ptr(indptr), _ptr(indices) if nnz else None)
    return Graph(n, indptr, indices)


def rmat(scale: int, n: int, draws: int, abc=(0.57, 0.19, 0.19), seed: int = 0) -> Graph:
    """Symmetrised R-MAT graph on n <= 2^scale vertices (permuted, rejected >= n)."""
    lib = _load()
    indptr = np.zeros(n + 1, dtype=np.int64)
    h = ctypes.c_void_p()
    nnz = lib.dg_rmat(scale, n, draws, abc[0], abc[1], abc[2], seed, _ptr(indptr), ctypes.byref(h))
    if nnz < 0:
        raise MemoryError("dg_rmat failed")
    return Graph(n, indptr, _take_indices(lib, h, nnz))


def inject_hubs(g: Graph, num_hubs: int, hub_deg: int, seed: int) -> Graph:
    lib = _load()
    indptr = np.zeros(g.num_nodes + 1, dtype=np.int64)
    hubs = np.zeros(num_hubs, dtype=np.int64)
    h = ctypes.c_void_p()
    nnz = lib.dg_inject_hubs(g.num_nodes, _ptr(g.indptr), _ptr(g.indices), num_hubs, hub_deg, seed,
                             _ptr(hubs), _ptr(indptr), ctypes.byref(h))
    if nnz < 0:
        raise MemoryError("dg_inject_hubs failed")
    return Graph(g.num_nodes, indptr, _take_indices(lib, h, nnz), hubs)


def features(rows: int, dim: int, seed: int, dtype: str = "f32") -> np.ndarray:
    """N(0,1) feature table [rows, dim]: float32, or bf16 bit patterns (uint16)."""
    lib = _load()
    if dtype == "f32":
        out = np.empty((rows, dim), dtype=np.float32)
        lib.dg_features_f32(rows, dim, seed, _ptr(out))
    elif dtype == "bf16":
        out = np.empty((rows, dim), dtype=np.uint16)
        lib.dg_features_bf16(rows, dim, seed, _ptr(out))
    else:
        raise ValueError(dtype)
    return out


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 -> bf16 (nearest-even), returned as uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclass
class Weights:
    """GraphSAGE-mean weights: per layer W_self, W_neigh [d_l, d_{l+1}] and bias
    [d_{l+1}].  ``dtype`` is "f32" (float32 arrays) or "bf16" (matrices as
    uint16 bf16 bit patterns; bias stays float32)."""
    dims: list
    w_self: list
    w_neigh: list
    bias: list
    dtype: str = "f32"

    def as_f64(self):
        conv = (lambda a: bf16_bits_to_f32(a).astype(np.float64)) if self.dtype == "bf16" \
            else (lambda a: a.astype(np.float64))
        return ([conv(w) for w in self.w_self], [conv(w) for w in self.w_neigh],
                [b.astype(np.float64) for b in self.bias])


def sage_weights(dims, seed: int, dtype: str = "f32") -> Weights:
    """Xavier-uniform (Glorot & Bengio 2010) matrices, U(-0.1, 0.1) biases."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ws, wn, bs = [], [], []
    for l in range(len(dims) - 1):
        a = np.sqrt(6.0 / (dims[l] + dims[l + 1]))
        s = rng.uniform(-a, a, size=(dims[l], dims[l + 1])).astype(np.float32)
        n = rng.uniform(-a, a, size=(dims[l], dims[l + 1])).astype(np.float32)
        b = rng.uniform(-0.1, 0.1, size=(dims[l + 1],)).astype(np.float32)
        if dtype == "bf16":
            s, n = bf16_bits_from_f32(s), bf16_bits_from_f32(n)
        ws.append(s)
        wn.append(n)
        bs.append(b)
    return Weights(list(dims), ws, wn, bs, dtype)


def labels(n: int, num_classes: int, seed: int) -> np.ndarray:
    """A class label per vertex, uniform in [0, num_classes), int32."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(0, num_classes, size=n).astype(np.int32)


def permutation(n: int, seed: int) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.permutation(n).astype(np.int32)


def train_set(n: int, fraction: float, seed: int) -> np.ndarray:
    """A seeded random subset of round(fraction * n) distinct vertices."""
    k = int(round(fraction * n))
    return permutation(n, seed)[:k].copy()


def epoch_batches(train: np.ndarray, batch: int, epoch_seed: int):
    """Seeded Fisher-Yates shuffle of the training set, then consecutive
    chunks of `batch` seeds; the last partial batch is kept."""
    rng = np.random.Generator(np.random.PCG64(epoch_seed))
    perm = train[rng.permutation(len(train))]
    return [perm[i:i + batch].copy() for i in range(0, len(perm), batch)]


def batch_seed(base: int, b: int) -> int:
    """Per-batch sampling key: the base key XOR the batch index."""
    return (base ^ b) & 0xFFFFFFFFFFFFFFFF
