"""Plant plausible mistakes in copies of the oracle; the pins must catch each.

Every mutant is a one-line source edit of oracle/bpc_oracle.py loaded as a
separate module, so the real oracle is never touched.
"""

import importlib.util
import os

import pytest

from oracle_pins import ALL_PINS

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "bpc_oracle.py")

MUTANTS = {
    "alg1_sign_of_zero": ("        u = np.where(a >= 0.0, 1.0, -1.0)\n        fragile += _fragile_count(a)\n        s = ",
                          "        u = np.where(a > 0.0, 1.0, -1.0)\n        fragile += _fragile_count(a)\n        s = "),
    "alg1_divisor": ("v = s / np.float64(N) if", "v = s / np.float64(N + 1) if"),
    "alg1_residual_sign": ("R = R - u[:, None] * P[i]", "R = R + u[:, None] * P[i]"),
    "alg1_unrounded_update": ("R = R - u[:, None] * P[i].astype(np.float64)[None, :]", "R = R - u[:, None] * v[None, :]"),
    "alg1_reversed_u": ("s = pairwise_tree_sum(R * u[:, None])", "s = pairwise_tree_sum(R * u[::-1, None])"),
    "alg1_fixed_direction": ("g = G[i].astype(np.float64)", "g = G[0].astype(np.float64)"),
    "alg1_transposed_direction": ("a = canonical_dot(R, g)", "a = canonical_dot(R, g[::-1])"),
    "alg2_residual_sign": ("r = r - u[:, None] * Pd[i][None, :]", "r = r + u[:, None] * Pd[i][None, :]"),
    "alg2_one_shot": ("a = canonical_dot(r, Pd[i])", "a = canonical_dot(bf16_bits_to_f64(K_bits), Pd[i])"),
    "alg2_row_index": ("a = canonical_dot(r, Pd[i])", "a = canonical_dot(r, Pd[L - 1 - i])"),
    "quant_scale": ("y = (x * 127.0) / m", "y = (x * 128.0) / m"),
    "quant_first_head_only": ("        x = x + xs[g]\n", "        x = x + 0.0 * xs[g]\n"),
    "quant_sign_plane": ("planes[0] = np.where(p >= 0, 1, -1)", "planes[0] = np.where(p > 0, -1, 1)"),
    "quant_plane_order": ("planes[1 + j] = np.where(((mag >> j) & 1) == 1, 1, -1)",
                          "planes[7 - j] = np.where(((mag >> j) & 1) == 1, 1, -1)"),
    "score_abs": ("    return H @ p\n", "    return H @ np.abs(p)\n"),
    "score_bit_order": ("bits = (c[:, :, None] >> shifts[None, None, :]) & np.uint32(1)",
                        "bits = (c[:, :, None] >> (31 - shifts)[None, None, :]) & np.uint32(1)"),
    "select_tie_high": ("order = np.lexsort((np.arange(N), -c))", "order = np.lexsort((-np.arange(N), -c))"),
    "select_smallest": ("order = np.lexsort((np.arange(N), -c))", "order = np.lexsort((np.arange(N), c))"),
    "attend_no_scale": ("logits = (q @ Ks.T) * np.float64(sm_scale)", "logits = (q @ Ks.T)"),
    "attend_values_are_keys": ("Vs = bf16_bits_to_f64(np.asarray(V_bits)[idx])", "Vs = bf16_bits_to_f64(np.asarray(K_bits)[idx])"),
    "dot_block_order": ("    return (parts[0] + parts[1]) + (parts[2] + parts[3])\n\n\ndef canonical_sumsq",
                        "    return ((parts[0] + parts[1]) + parts[2]) + parts[3]\n\n\ndef canonical_sumsq"),
    "tree_sequential": ("        s = T[0:even:2] + T[1:even:2]\n", "        return np.cumsum(T, axis=0)[-1]\n"),
    "budget_floor": ("return -((-N * num) // den)", "return (N * num) // den"),
    "bf16_wrong_shift": ("<< np.uint32(16)", "<< np.uint32(15)"),
    "hard_tie_high": ("order = np.lexsort((np.arange(N), -key))", "order = np.lexsort((-np.arange(N), -key))"),
    "hard_smallest": ("order = np.lexsort((np.arange(N), -key))", "order = np.lexsort((np.arange(N), key))"),
    "hard_plain_bits": ("key = np.where(u >= (1 << 31), (~u) & 0xFFFFFFFF, u | (1 << 31))", "key = u"),
    "eas_intersection": ("union = np.union1d(idx, serr)", "union = np.intersect1d(idx, serr)"),
    "eas_added_inverted": ("added = (~np.isin(serr, idx)).astype(np.int32)", "added = np.isin(serr, idx).astype(np.int32)"),
    "eas_budget_floor": ("m = min(-(-budget * num // den), budget - 1)", "m = min(budget * num // den, budget - 1)"),
    "perq_group_selection": ("heads = [decode_head(q_bits[g:g + 1], K_bits, V_bits, codes, P, k, sm_scale)",
                             "heads = [decode_head(q_bits, K_bits, V_bits, codes, P, k, sm_scale)"),
    "perq_first_head_only": ("heads = [decode_head(q_bits[g:g + 1], K_bits,", "heads = [decode_head(q_bits[0:1], K_bits,"),
    "decode_attends_all": ("    out = attend(q_bits, K_bits, V_bits, idx, sm_scale)\n    return {\"p\"",
                           "    out = attend(q_bits, K_bits, V_bits, np.arange(len(c)), sm_scale)\n    return {\"p\""),
    "perq_head_order": ("for g in range(q_bits.shape[0])]", "for g in range(q_bits.shape[0])][::-1]"),
}


def _load_mutant(name, old, new):
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) >= 1, f"mutant {name}: pattern not found"
    text = text.replace(old, new, 1)
    spec = importlib.util.spec_from_loader(f"oracle_mutant_{name}", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(text, f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    mod = _load_mutant(name, *MUTANTS[name])
    caught = None
    for pin in ALL_PINS:
        try:
            pin(mod)
        except Exception:  # an assertion, or the mutant crashing on a pin input
            caught = pin.__name__
            break
    assert caught, f"no pin catches mutant {name}"
