"""The arithmetic of the fp32 linear layers and input gradients on the bf16
matrix cores, checked on the CPU: every fp32 value is cut by truncation into
three bf16 parts, x = x0 + x1 + x2 exactly, and a product a b is taken as
the six part products a0 b0 + a0 b1 + a1 b0 + a0 b2 + a1 b1 + a2 b0 (each
exact in fp32), summed in fp32.

These tests restate that rule in numpy (not the kernels' code) and check the
claims the kernels rely on: the cut is exact and its parts are bf16 values
of at most 8 significant bits; values with few significant bits give exact
products; the dropped terms stay below 2^-21 of the product; and on long
random dot products the error against the fp64 dot product is of the order
of fp32's own rounding, while leaving out any one of the six kept terms is
visibly worse.  The GPU parity tests then check that the kernels compute
this (rows within 5e-6 of the fp64 oracle).
"""
import numpy as np

EDGE_MASK = np.uint32(0xFFFF0000)


def cut3(x):
    """x (fp32) -> three fp32 arrays holding bf16 values, x = x0 + x1 + x2."""
    x = np.asarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    x0 = (u & EDGE_MASK).view(np.float32)
    r1 = (x - x0).astype(np.float32)
    x1 = (r1.view(np.uint32) & EDGE_MASK).view(np.float32)
    x2 = (r1 - x1).astype(np.float32)
    return x0, x1, x2


def parts_dot(a, b, terms=((0, 0), (0, 1), (1, 0), (0, 2), (1, 1), (2, 0))):
    """Row-wise sum_k a[:, k] b[:, k] from the part products `terms`, each
    product exact in fp32 (checked), summed in fp32 in the order k, then
    term."""
    pa, pb = cut3(a), cut3(b)
    acc = np.zeros(a.shape[0], dtype=np.float32)
    for k in range(a.shape[1]):
        for i, j in terms:
            p = pa[i][:, k] * pb[j][:, k]
            assert np.array_equal(p.astype(np.float64), pa[i][:, k].astype(np.float64) * pb[j][:, k])
            acc = (acc + p).astype(np.float32)
    return acc


def test_cut_is_exact_into_bf16_parts():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(20000), rng.uniform(-1e6, 1e6, 2000),
                        rng.uniform(-1e-6, 1e-6, 2000), [0.0, -0.0, 1.0, -3.5]]).astype(np.float32)
    x0, x1, x2 = cut3(x)
    assert np.array_equal((x0.astype(np.float64) + x1 + x2), x.astype(np.float64))
    for p in (x0, x1, x2):
        assert np.all((p.view(np.uint32) & np.uint32(0xFFFF)) == 0)   # a bf16 value
    nz = x != 0
    assert np.all(np.abs(x1[nz]) < 2.0 ** -7 * np.abs(x[nz]))
    assert np.all(np.abs(x2[nz]) < 2.0 ** -15 * np.abs(x[nz]))


def test_few_significant_bits_give_exact_products():
    """Integers and multiples of 1/16 (the exact training cases): at most 8
    significant bits, so x1 = x2 = 0 and the part sum is the product."""
    rng = np.random.default_rng(2)
    a = rng.integers(-200, 201, 4096).astype(np.float32)
    b = (rng.integers(-40, 41, 4096) / 16).astype(np.float32)
    for x in (a, b):
        _, x1, x2 = cut3(x)
        assert not x1.any() and not x2.any()
    # 16-bit values: x2 = 0, every dropped term vanishes
    c = (rng.integers(-30000, 30001, 4096) / 64).astype(np.float32)
    assert not cut3(c)[2].any()
    a0, a1, a2 = cut3(c)
    b0, b1, b2 = cut3(b)
    kept = (a0 * b0 + a0 * b1 + a1 * b0 + a0 * b2 + a1 * b1 + a2 * b0).astype(np.float64)
    assert np.array_equal(kept, c.astype(np.float64) * b.astype(np.float64))


def test_dropped_terms_are_below_2_to_minus_21():
    rng = np.random.default_rng(3)
    a = rng.standard_normal(50000).astype(np.float32)
    b = rng.standard_normal(50000).astype(np.float32)
    a0, a1, a2 = (p.astype(np.float64) for p in cut3(a))
    b0, b1, b2 = (p.astype(np.float64) for p in cut3(b))
    dropped = a1 * b2 + a2 * b1 + a2 * b2
    prod = a.astype(np.float64) * b.astype(np.float64)
    assert np.all(np.abs(dropped) <= 2.0 ** -21 * np.abs(prod))


def test_dot_products_at_fp32_level():
    """K = 512 (the widest part-product layer) on N(0,1) data: relative to
    the sum of |a_k b_k|, the six-term fp32 sum is within a few fp32
    roundings of the fp64 dot product, like a plain fp32 sum; dropping any
    one kept term costs far more."""
    rng = np.random.default_rng(4)
    K, trials = 512, 64
    a = rng.standard_normal((trials, K)).astype(np.float32)
    b = rng.standard_normal((trials, K)).astype(np.float32)
    exact = (a.astype(np.float64) * b).sum(axis=1)
    scale = np.abs(a.astype(np.float64) * b).sum(axis=1)
    terms = ((0, 0), (0, 1), (1, 0), (0, 2), (1, 1), (2, 0))
    e6 = np.abs(parts_dot(a, b, terms) - exact) / scale
    acc = np.zeros(trials, dtype=np.float32)
    for k in range(K):
        acc = (acc + (a[:, k] * b[:, k]).astype(np.float32)).astype(np.float32)
    e32 = np.abs(acc - exact) / scale
    assert np.median(e6) < 4 * max(np.median(e32), 2.0 ** -24), (np.median(e6), np.median(e32))
    assert e6.max() < 2.0 ** -18
    for drop in terms[1:]:
        e5 = np.abs(parts_dot(a, b, tuple(t for t in terms if t != drop)) - exact) / scale
        assert np.median(e5) > 8 * np.median(e6), (drop, np.median(e5), np.median(e6))
