"""Plant plausible mistakes in a copy of the oracle and check a pin catches each.

The copy is compiled on the CPU into a temporary directory; the real oracle
is untouched.  Each mutant must fail at least one pin of
test_oracle_pins / test_plan_oracle.
"""
import os

import numpy as np
import pytest

import oracle
from oracle.build import HERE, build
import test_fm_oracle as FP
import test_oracle_pins as LP
import test_plan_oracle as PP
import test_sched_oracle as SP

MUTANTS = {
    "mean_divisor": ("o[c] /= (double)len;", "o[c] /= (double)(len + 1);"),
    "always_mean": ("if (pooling && pooling[t] == 1 && len > 0)", "if (len > 0)"),
    "ids_local_index": ("ids[id_base[t] + j]", "ids[id_base[t] + j - start]"),
    "previous_col_base": ("out + b * total_d + col_base[t];", "out + b * total_d + col_base[t > 0 ? t - 1 : 0];"),
    "half_bias": ("e - 25);", "e - 24);"),
    "half_subnormal": ("ldexp((double)m, -24)", "ldexp((double)m, -23)"),
    "half_sign": ("return sign ? -v : v;", "return v;"),
    "onehot_index": ("start = b;\n      end = b + 1;", "start = (b + 1) % B;\n      end = start + 1;"),
    "drop_last_id": ("for (int64_t j = start; j < end; ++j)", "for (int64_t j = start; j < end - 1; ++j)"),
    "items_floor": ("int64_t n = (L + C - 1) / C;", "int64_t n = L / C;"),
    "out_bytes_every_chunk": ("return rows * row_bytes + (j == 0 ? out_bytes : 0) + K;",
                              "return rows * row_bytes + out_bytes + K;"),
    "no_item_constant": ("return rows * row_bytes + (j == 0 ? out_bytes : 0) + K;",
                         "return rows * row_bytes + (j == 0 ? out_bytes : 0) + (j == 0 ? K : 1);"),
    "chunk_rows_shifted": ("int64_t lo = j * C, hi = (j + 1) * C;", "int64_t lo = j * C, hi = (j + 1) * C + 1;"),
    "target_floor": ("(int64_t)((num + (uint64_t)W - 1) / (uint64_t)W)", "(int64_t)(num / (uint64_t)W)"),
    "slack_wide": ("S / (2 * W)", "S / W"),
    "snap_backward": ("begin = bag_item_base[bag + 1];", "begin = bag_item_base[bag];"),
    "split_double_count": ("if (b0 > bag_item_base[bag] && bag != last_split)", "if (b0 > bag_item_base[bag])"),
    "no_wave_clamp": ("waves_requested < N ? waves_requested : N", "waves_requested"),
    "id_base_onehot": ("int64_t nnz = offsets ? offsets[t * (B + 1) + B] : B;",
                       "int64_t nnz = offsets ? offsets[t * (B + 1) + B] : B - (t > 0);"),
    "fm_no_half": ("out[b] = 0.5 * y;", "out[b] = y;"),
    "fm_no_square_sum": ("y += s * s - q;", "y += s * s;"),
    "fm_field_stride": ("b * row_stride + (int64_t)t * dim + c", "b * row_stride + (int64_t)t + c"),
    "fm_sample_stride": ("b * row_stride + (int64_t)t * dim + c", "b * num_fields * dim + (int64_t)t * dim + c"),
    "fm_abs_sum": ("s += e;", "s += fabs(e);"),
    "fm_mag_signed": ("sa += fabs(e);", "sa += e;"),
    "fm_mag_no_half": ("if (mag) mag[b] = 0.5 * m;", "if (mag) mag[b] = m;"),
    "fm_mag_minus_squares": ("m += sa * sa + q;", "m += sa * sa - q;"),
    "fm_mag_no_squares": ("m += sa * sa + q;", "m += sa * sa;"),
    "waves_head_first_previous": ("head_first[w] = (int32_t)v;", "head_first[w] = (int32_t)(w - 1);"),
    "waves_pieces_count_empty": ("if (wave_item_begin[u] < wave_item_begin[u + 1]) ++pieces;", "++pieces;"),
    "waves_inside_at_bag_start": ("if (i >= N || i <= wave_bag_base[w]) continue;",
                                  "if (i >= N || i < wave_bag_base[w]) continue;"),
    "waves_base_of_next_bag": ("wave_bag_base[w] = bag_item_base[wave_bag[w]];",
                               "wave_bag_base[w] = bag_item_base[wave_bag[w] + (wave_bag[w] < TB)];"),
    "waves_split_last_first": ("split_last[v] = (int32_t)w;", "if (split_last[v] < 0) split_last[v] = (int32_t)w;"),
}

# Mistakes planted in the oracle's Python interaction head (dcn_forward's magnitudes).
PY_MUTANTS = {
    "dcn_mag_signed_weights": ("ax = ax0 * (ax @ np.abs(W).T + np.abs(b)) + ax",
                               "ax = ax0 * (ax @ W.T + np.abs(b)) + ax"),
    "dcn_mag_no_bias": ("ax = ax0 * (ax @ np.abs(W).T + np.abs(b)) + ax", "ax = ax0 * (ax @ np.abs(W).T) + ax"),
    "dcn_mag_signed_x0": ("ax = ax0 * (ax @ np.abs(W).T + np.abs(b)) + ax",
                          "ax = x0 * (ax @ np.abs(W).T + np.abs(b)) + ax"),
    "mlp_mag_signed_bias": ("ah = ah @ np.abs(V).T + np.abs(c)", "ah = ah @ np.abs(V).T + c"),
    "mlp_mag_from_cross": ("h, ah = x0.copy(), ax0.copy()", "h, ah = x0.copy(), ax.copy()"),
    "mag_scaled": ("return x, h, ax, ah", "return x, h, 0.5 * ax, ah"),
}


def _pins():
    yield lambda: LP.test_golden_lookup("lookup_fig5_onehot.txt")
    yield lambda: LP.test_golden_lookup("lookup_multihot_mixed.txt")
    yield lambda: LP.test_onehot_equals_algorithm1(1, None)
    yield lambda: LP.test_pooled_equals_embedding_bag(5, 128, None)
    yield LP.test_empty_bags_are_zero
    yield LP.test_one_hot_bag_is_the_row
    yield LP.test_mean_is_sum_over_length
    yield LP.test_binary16_decode_all_patterns
    for name in ("plan_small_w3.txt", "plan_small_w3_exact.txt", "plan_small_w8.txt"):
        yield (lambda n: (lambda: PP.test_golden_plan(n)))(name)
    for seed in range(8):
        yield (lambda s: (lambda: PP.test_random_small_plans(s)))(seed)
    yield FP.test_golden_fm
    yield FP.test_golden_fm_magnitude
    yield lambda: FP.test_magnitude_equals_pairwise_form(3, 5, np.float32)
    yield FP.test_magnitude_closed_forms
    yield PP.test_wave_arrays_brute_force
    yield lambda: FP.test_equals_pairwise_dot_products(3, 5, np.float32)
    yield lambda: FP.test_equals_pairwise_dot_products(7, 16, np.float16)
    yield FP.test_closed_forms


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path, monkeypatch):
    old, new = MUTANTS[name]
    src = open(os.path.join(HERE, "oracle.c")).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    mutated = src.replace(old, new, 1)
    path = tmp_path / "oracle_mutant.c"
    path.write_text(mutated)
    lib = build(source=str(path), out=str(tmp_path / f"liboracle_{name}.so"))
    monkeypatch.setattr(oracle, "LIB", lib)
    caught = []
    for pin in _pins():
        try:
            pin()
        except (AssertionError, oracle.OracleError, IndexError, ValueError):
            caught.append(pin)
            break
    assert caught, f"no pin catches mutant {name}"


def test_unmutated_copy_passes(tmp_path, monkeypatch):
    src = open(os.path.join(HERE, "oracle.c")).read()
    path = tmp_path / "oracle_copy.c"
    path.write_text(src)
    lib = build(source=str(path), out=str(tmp_path / "liboracle_copy.so"))
    monkeypatch.setattr(oracle, "LIB", lib)
    for pin in _pins():
        pin()


def _py_pins():
    yield SP.test_dcn_magnitude_hand_typed
    yield SP.test_dcn_magnitude_identity_on_nonnegative_inputs
    yield SP.test_dcn_magnitude_sign_invariance_and_bound


@pytest.mark.parametrize("name", sorted(PY_MUTANTS))
def test_python_mutant_is_caught(name, monkeypatch):
    """The oracle's dcn_forward with one planted mistake (its source edited and
    compiled into a function that replaces it for this test only)."""
    import inspect
    import textwrap
    old, new = PY_MUTANTS[name]
    src = textwrap.dedent(inspect.getsource(oracle.dcn_forward))
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    ns = dict(vars(oracle))
    exec(compile(src.replace(old, new, 1), f"<mutant {name}>", "exec"), ns)
    monkeypatch.setattr(oracle, "dcn_forward", ns["dcn_forward"])
    caught = False
    for pin in _py_pins():
        try:
            pin()
        except AssertionError:
            caught = True
            break
    assert caught, f"no pin catches mutant {name}"


def test_python_pins_pass_unmutated():
    for pin in _py_pins():
        pin()
