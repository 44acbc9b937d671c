"""The pins must catch plausible mistakes in the oracle.

Each case copies the oracle source, plants one mistake, builds it on the CPU
in a temporary directory and runs the pin meant to catch it against the
mutant, which must fail.  Nothing here touches the GPU.
"""
import ctypes
import importlib.util
import os
import subprocess
import sys

import numpy as np
import pytest

import test_oracle_blocks as tb
import test_oracle_rng as tr
import test_oracle_sampling as ts
import test_oracle_train as tt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    # Philox: multipliers swapped between the two lanes
    "philox_multipliers_swapped": ("(uint64_t)PHILOX_M0 * c[0]", "(uint64_t)PHILOX_M1 * c[0]"),
    # Philox: key bumped before the first round as well
    "philox_key_schedule": ("if (round > 0) {", "if (round >= 0) {"),
    # Philox: output lanes mixed up
    "philox_output_order": ("uint32_t n1 = lo1;", "uint32_t n1 = lo0;"),
    # bounded draw: no rejection (biased modulo-like draw)
    "bounded_no_rejection": ("if (low < threshold) return 0;", "(void)threshold;"),
    # Floyd: inserts the draw even when it is already chosen
    "floyd_insert_wrong": ("chosen[i] = present ? j : t;", "chosen[i] = present ? t : j;"),
    # Floyd: draw range off by one ([0, j) instead of [0, j])
    "floyd_draw_range": ("orc_uniform_below(seed, v, l, i, j + 1)", "orc_uniform_below(seed, v, l, i, j)"),
    # relabel: local ids off by one
    "relabel_off_by_one": ("B->local[e] = map[u] - 1;", "B->local[e] = map[u];"),
    # relabel: new nodes not recorded in the map (duplicates in src)
    "relabel_no_dedup": ("map[u] = n_src + 1;\n", "\n"),
    # mean: divides by the fan-out instead of the sampled count
    "mean_divides_by_wrong_count": ("row[c] = row[c] / (double)k;", "row[c] = row[c] / (double)(k + 1);"),
    # SAGE: neighbour weights applied transposed
    "sage_transposed_weight": ("m[v * d_in + c] * w_neigh[c * d_out + o]", "m[v * d_in + c] * w_neigh[o * d_in + c]"),
    # SAGE: bias dropped
    "sage_no_bias": ("double z = bias[o];", "double z = 0.0;"),
    # sampling: slots mapped to the row in reverse
    "sample_slots_reversed": ("int64_t u = indices[indptr[v] + slots[q]];",
                              "int64_t u = indices[indptr[v] + (d - 1 - slots[q])];"),
    # sampling: fan-out of the wrong layer (hop index instead of layer index)
    "sample_wrong_layer_fanout": ("int64_t f = fanouts[l];", "int64_t f = fanouts[hop];"),
    # backward: ReLU mask dropped
    "bwd_no_relu_mask": ("dZ[i] = out[i] > 0.0 ? dOut[i] : 0.0;", "dZ[i] = dOut[i];"),
    # backward: mean's 1/k missing on the way back
    "bwd_mean_unscaled": ("h[c] += dM[v * d + c] / (double)k;", "h[c] += dM[v * d + c];"),
    # backward: input gradient through W_self transposed
    "bwd_self_transposed": ("s += dZ[v * d_out + o] * w_self[c * d_out + o];",
                            "s += dZ[v * d_out + o] * w_self[o * d_in + c];"),
    # backward: loss gradient not divided by the batch size
    "bwd_xent_not_mean": ("dz[v * C + c] = (p - (c == y[v] ? 1.0 : 0.0)) / (double)n;",
                          "dz[v * C + c] = (p - (c == y[v] ? 1.0 : 0.0));"),
    # gather: the row before the named one
    "gather_wrong_row": ("(const char*)feats + ids[i] * row_bytes",
                         "(const char*)feats + (ids[i] > 0 ? ids[i] - 1 : 0) * row_bytes"),
    # seeds: a repeated seed accepted instead of refused
    "seed_duplicate_accepted": ("if (map[s] != 0) { free(front);", "if (0) { free(front);"),
    # sampling: the drawn slots left in Floyd's order instead of ascending
    "sample_slots_unsorted": ("qsort(slots, k, sizeof(uint32_t), cmp_u32);", "(void)cmp_u32;"),
    # sampling: a row of degree <= fan-out taken back to front
    "sample_small_row_reversed": ("for (int64_t s = 0; s < d; ++s) slots[s] = (uint32_t)s;",
                                  "for (int64_t s = 0; s < d; ++s) slots[s] = (uint32_t)(d - 1 - s);"),
    # SAGE: the ReLU applied on every layer, the last one too
    "sage_relu_everywhere": ("out[v * d_out + o] = (relu && z < 0.0) ? 0.0 : z;",
                             "out[v * d_out + o] = (z < 0.0) ? 0.0 : z;"),
    # mean: a row without edges divided by its count as well (0 / 0)
    "mean_empty_row_divided": ("    if (k > 0)\n      for (int64_t c = 0; c < d; ++c) row[c] = row[c] / (double)k;",
                               "    for (int64_t c = 0; c < d; ++c) row[c] = row[c] / (double)k;"),
    # loss: the label's class shifted by one
    "xent_label_shifted": ("loss += -(row[y[v]] - mx - log(sum));", "loss += -(row[(y[v] + 1) % C] - mx - log(sum));"),
    # backward: the bias gradient summed over one row only
    "bwd_bias_one_row": ("for (int64_t v = 0; v < n; ++v) s += dZ[v * d_out + o];", "s += dZ[o];"),
    # backward: the ReLU mask letting the clamped units through
    "bwd_relu_mask_at_zero": ("dZ[i] = out[i] > 0.0 ? dOut[i] : 0.0;", "dZ[i] = out[i] >= 0.0 ? dOut[i] : 0.0;"),
    # backward: the mean's gradient sent to the destination instead of the source
    "bwd_mean_to_destination": ("double* h = dH + local[e] * d;", "double* h = dH + v * d;"),
    # backward: neighbour weight gradient taken from the self input
    "bwd_neigh_from_self": ("const double hc = H[v * d_in + c], mc = m[v * d_in + c];",
                            "const double hc = H[v * d_in + c], mc = H[v * d_in + c];"),
}


def _build_mutant(tmpdir, name):
    old, new = MUTANTS[name]
    src = open(os.path.join(ROOT, "oracle", "oracle.c")).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    d = os.path.join(tmpdir, name)
    os.makedirs(d, exist_ok=True)
    path = os.path.join(d, "oracle.c")
    with open(path, "w") as fh:
        fh.write(src.replace(old, new))
    # a file name of its own: a shared object is matched by name when another
    # library asks for it, so the mutant must not be called liboracle.so
    so = os.path.join(d, f"liboracle_{name}.so")
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-w", path, "-o", so, "-lm"])
    spec = importlib.util.spec_from_file_location(f"oracle_mutant_{name}",
                                                  os.path.join(ROOT, "oracle", "__init__.py"))
    mod = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = mod
    spec.loader.exec_module(mod)
    mod._LIB = so
    mod._lib = None
    pins_so = os.path.join(d, "libpins.so")
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-pthread",
                           os.path.join(ROOT, "tests", "native", "pins.c"), "-o", pins_so,
                           "-L" + d, f"-l:liboracle_{name}.so", "-Wl,-rpath," + d])
    pins = ctypes.CDLL(pins_so)
    vp, u32, u64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64
    pins.pin_bounded_exhaustive.restype = ctypes.c_int
    pins.pin_bounded_exhaustive.argtypes = [u32, vp, ctypes.POINTER(u64), ctypes.c_int]
    for fn in ("pin_subset_hist", "pin_subset_hist_nodes", "pin_marginals"):
        getattr(pins, fn).restype = ctypes.c_int
        getattr(pins, fn).argtypes = [u32, u32, u32, u32, u64, u64, vp]
    return mod, pins


def _fails(fn):
    """True when the pin rejects the mutant: an assertion fails, or a
    pytest.raises in it sees no error where one is due.  Any other
    exception does not count as a catch."""
    try:
        fn()
    except (AssertionError, pytest.fail.Exception):
        return True
    except Exception:
        return False
    return False


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path, dg):
    mut, pins = _build_mutant(str(tmp_path), name)
    tiny = dg.er_directed(10000, 10.0, 101)
    checks = {
        "philox": lambda: tr.test_philox_known_answers(mut),
        "bounded": lambda: tr.test_bounded_draw_exhaustive(pins, 7),
        "floyd": lambda: ts.test_floyd_brute_force_exact_uniformity(mut, 5),
        "chi2": lambda: ts.test_keyed_subsets_uniform_over_keys(pins, 8, 3, 200000),
        "blocks": lambda: tb.test_tiny_blocks_invariants(mut, dg, tiny),
        "errors": lambda: tb.test_error_statuses(mut, tiny),
        "gather": lambda: tb.test_gather_is_a_bit_copy(mut, dg),
        "rmat": lambda: tb.test_rmat_blocks_invariants_with_hubs(mut, dg),
        "mean": lambda: tb.test_mean_aggregate_matches_dense(mut, dg, tiny),
        "dense": lambda: tb.test_full_neighbourhood_equals_dense_sage(mut, dg, 2),
        "xent": lambda: tt.test_softmax_xent_value_and_gradient(mut),
        "train_fd": lambda: tt.test_backward_matches_finite_differences(mut, dg),
        "train_dense": lambda: tt.test_full_neighbourhood_gradients_equal_dense_autograd(mut, dg, 2),
        "input_fd": lambda: tt.test_input_gradient_matches_finite_differences(mut, dg),
        "input_dense": lambda: tt.test_input_gradient_equals_dense_autograd(mut, dg, 2),
    }
    caught = next((k for k, fn in checks.items() if _fails(fn)), None)
    assert caught is not None, f"mutant {name} passed every pin"
