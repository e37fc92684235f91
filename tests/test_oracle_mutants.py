"""Planted mistakes: each test copies the oracle's source, plants one plausible mistake in
the copy (a dropped term, a flipped sign, a transposed operand, a wrong row index, a
wrong tie-break, a missing mask or gate ...), loads the copy as a separate module and
runs the pins of tests/test_oracle.py against it with the copy in place of the oracle.
Every mutant must make at least one named pin fail; the real oracle passes them all.

This shows that the pins constrain the oracle's arithmetic, not only that the oracle
agrees with itself. The copy lives only in memory; the oracle file is never changed.
"""
import inspect
import itertools
import sys
import types

import numpy as np
import pytest

from oracle import pmpe_oracle as O
from tests import test_oracle as TO

SOURCE = inspect.getsource(O)


def mutant(old: str, new: str) -> types.ModuleType:
    """The oracle with `old` replaced by `new` (which must occur exactly once)."""
    assert SOURCE.count(old) == 1, f"mutation site not unique: {old!r}"
    name = f"pmpe_oracle_mutant_{next(_COUNTER)}"
    m = types.ModuleType(name)
    sys.modules[name] = m  # dataclasses resolve annotations through sys.modules
    try:
        exec(compile(SOURCE.replace(old, new), f"<{name}>", "exec"), m.__dict__)
    finally:
        del sys.modules[name]
    return m


_COUNTER = itertools.count()


def pin_fails(monkeypatch, module, pin, *args) -> bool:
    """Run pin(*args) from tests/test_oracle.py with `module` as the oracle."""
    monkeypatch.setattr(TO, "O", module)
    try:
        pin(*args)
    except AssertionError:
        return True
    finally:
        monkeypatch.setattr(TO, "O", O)
    return False


def backward_autograd(mode, soft=False, shared=False):
    return lambda: TO.test_backward_equals_autograd_of_textbook_forward(mode, soft, shared)


# (id, mutation site, replacement, pins of which at least one must fail)
MUTANTS = [
    # --- Sec. 3.2 private-only backward ---
    ("backward_dropped_silu_prime_term",
     "dG = dA * U * S * (1.0 + G * (1.0 - S))", "dG = dA * U * S",
     [backward_autograd("renorm"), TO.test_backward_central_differences]),
    ("backward_flipped_renorm_softmax_jacobian_sign",
     "dz[sel_pos] = g * (dg - (g * dg).sum())", "dz[sel_pos] = g * (dg + (g * dg).sum())",
     [backward_autograd("renorm"), TO.test_backward_central_differences]),
    ("backward_flipped_pool_softmax_jacobian_sign",
     "dz = p * (up - (p[sel_pos] * dg).sum())", "dz = p * (up + (p[sel_pos] * dg).sum())",
     [backward_autograd("pool_softmax")]),
    ("backward_transposed_down_projection",
     "dA = dY @ w2                        # [n, I]", "dA = dY @ w2.T",
     [lambda: TO.test_backward_square_expert_equals_autograd()]),
    ("backward_wrong_row_index",
     "dx[rows] += dX", "dx[np.roll(rows, 1)] += dX",
     [backward_autograd("renorm"), TO.test_backward_central_differences]),
    ("backward_router_gradient_on_wrong_token",
     "dwr[ids[priv] - n_pub] += dz[priv][:, None] * x64[t][None, :]",
     "dwr[ids[priv] - n_pub] += dz[priv][:, None] * x64[(t + 1) % T][None, :]",
     [backward_autograd("renorm")]),
    # --- Sec. 3.1 resolver, mask and top-k ---
    ("resolver_accepts_truthy_values",
     "if type(v) is bool and v is True:", "if v:",
     [TO.test_resolver_rejects_non_python_bool]),
    ("policy_word_fails_open_on_malformed_words",
     "return 1 if int(word) == ALLOW_WORD else 0", "return 1 if int(word) != DENY_WORD else 0",
     [TO.test_word_decode_single_allow_value, TO.test_mask_invariant_and_adversarial_override]),
    ("topk_highest_id_wins_ties",
     "key=lambda i: (-zz[i], int(ids[i])))", "key=lambda i: (-zz[i], -int(ids[i])))",
     [lambda: TO.test_topk_brute_force_heavy_ties(0), TO.test_forced_ties_zero_input_selects_first_ids]),
    ("topk_nan_not_ranked_last",
     "zz = np.where(np.isnan(zz), -np.inf, zz) + 0.0", "zz = zz + 0.0",
     [TO.test_topk_zero_signs_tie_and_nan_last]),
    ("logits_bias_dropped",
     "z = (z + np.asarray(bias, np.float32)[None, :]).astype(np.float32)", "z = z",
     [TO.test_logits_bias_single_fp32_add]),
    ("logits_rounded_to_bf16_like_precision",
     "z = (np.asarray(x_rows, np.float64) @ np.asarray(wr_rows, np.float64).T).astype(np.float32)",
     "z = (np.asarray(x_rows, np.float64) @ np.asarray(wr_rows, np.float64).T).astype(np.float16).astype(np.float32)",
     [TO.test_logits_match_exactly_rounded_sums]),
    # --- gates ---
    ("renorm_gate_normalised_over_pool",
     "    if mode == GATE_RENORM:\n        den = num.sum()",
     "    if mode == GATE_RENORM:\n        den = np.exp(np.asarray(z_pool, np.float64) - m).sum()",
     [TO.test_gates_closed_forms]),
    # --- dispatch ---
    ("dispatch_tokens_descending_within_expert",
     "tokens = np.nonzero(hit.any(axis=1))[0]", "tokens = np.nonzero(hit.any(axis=1))[0][::-1]",
     [lambda: TO.test_dispatch_is_stable_counting_sort(0)]),
    # --- experts and combine ---
    ("swiglu_sigmoid_instead_of_silu",
     "A = G / (1.0 + np.exp(-G)) * U", "A = 1.0 / (1.0 + np.exp(-G)) * U",
     [TO.test_one_expert_pool_is_dense_swiglu_mlp]),
    ("swiglu_gate_and_up_swapped",
     "    G = X @ w13[:I].T\n    U = X @ w13[I:].T\n    A = G / (1.0 + np.exp(-G)) * U",
     "    G = X @ w13[I:].T\n    U = X @ w13[:I].T\n    A = G / (1.0 + np.exp(-G)) * U",
     [TO.test_one_expert_pool_is_dense_swiglu_mlp]),
    ("combine_gate_dropped",
     "acc += np.float64(rt.gate[t, j]) * y[(int(t), int(rt.idx[t, j]))]",
     "acc += y[(int(t), int(rt.idx[t, j]))]",
     [TO.test_all_deny_equals_public_only_moe]),
    # --- audit (App. F.1 hooks) ---
    ("audit_hook_counts_routed_not_executed_rows_twice",
     "        hook.rows[int(t)] += 1", "        hook.rows[int(t)] += 2",
     [TO.test_audit_closed_form_and_hooks_equal_route_log]),
    ("audit_call_counted_per_row",
     "    if len(tokens) > 0:\n        hook.calls[p] += 1", "    hook.calls[p] += len(tokens)",
     [TO.test_audit_closed_form_and_hooks_equal_route_log]),
    # --- request-gated LoRA control (Sec. 4.2; App. F.2) ---
    ("lora_tile_gate_uses_first_row_only",
     "run = any(taus[u] == 1 for u in tile)", "run = taus[tile[0]] == 1",
     [TO.test_lora_tile_gate_known_by_construction]),
    ("lora_tile_of_32_rows",
     "LORA_TILE_ROWS = 64", "LORA_TILE_ROWS = 32",
     [TO.test_lora_tile_gate_known_by_construction]),
]


@pytest.mark.parametrize("name,old,new,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(monkeypatch, name, old, new, pins):
    m = mutant(old, new)
    failed = [getattr(p, "__name__", "pin") for p in pins if pin_fails(monkeypatch, m, p)]
    assert failed, f"{name}: no pin failed"


@pytest.mark.parametrize("name,old,new,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_unmutated_oracle_passes_the_same_pins(name, old, new, pins):
    for p in pins:
        p()


def test_mutant_loader_reproduces_the_oracle():
    """The copy mechanism itself changes nothing: an identity 'mutation' gives the
    oracle's results."""
    m = mutant("NEAR_TIE = 1e-5", "NEAR_TIE = 1e-5")
    z = np.array([0.3, 0.9, 0.1, 0.7], np.float32)
    assert [list(a) for a in (m.topk(z, np.arange(4), 2)[0],)] == [list(O.topk(z, np.arange(4), 2)[0])]
