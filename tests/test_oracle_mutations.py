"""Plant plausible mistakes in the CPU oracle and check that a pin catches each.

A pin that passes for a wrong oracle proves nothing; every mutation below is a
slip one could make writing Alg. 1 from the paper (a dropped normalisation, a
sign error in the head, the wrong tie rule, pruning by the wrong key, the wrong
parent's row, a depth-blind global order, a transposed or shifted head matrix).  The
mistakes are planted in the oracle module only, on the CPU, and undone by
``monkeypatch`` after each case.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import pctree_oracle as O
import test_oracle_pins as P

PINS = [P.pin_brute_force, P.pin_best_first, P.pin_chain, P.pin_shared_markov,
        P.pin_independent, P.pin_w_zero, P.pin_row_normalised, P.pin_hand_worked, P.pin_invariants]


def _some_pin_fails():
    for pin in PINS:
        try:
            pin()
        except Exception:  # noqa: BLE001 - any failure counts as caught
            return True
    return False


def test_unmutated_oracle_passes_every_pin():
    assert not _some_pin_fails()


def _mut_no_lse(monkeypatch):
    orig = O.child_logprobs

    def f(L_d, E, W, h_d, p, dtype):
        z, lse, lp = orig(L_d, E, W, h_d, p, dtype)
        return z, lse, z  # forgot to subtract the log-normaliser
    monkeypatch.setattr(O, "child_logprobs", f)


def _mut_silu_sign(monkeypatch):
    def f(E_row, h_row, dtype):
        x = E_row.astype(np.float64) + h_row.astype(np.float64)
        with np.errstate(over="ignore"):
            u = (x / (1.0 + np.exp(x))).astype(np.float32)  # sign slip in the exponent
        return u.astype(np.float64)
    monkeypatch.setattr(O, "activation", f)


def _mut_tie_rule(monkeypatch):
    def f(logpi, k):
        V = logpi.shape[0]
        return np.lexsort((-np.arange(V), -logpi))[:k]  # ties to the highest id
    monkeypatch.setattr(O, "local_topk", f)


def _mut_prune_by_token(monkeypatch):
    monkeypatch.setattr(O, "_layer_key", lambda n: (n.token, n.slot))


def _mut_wrong_parent(monkeypatch):
    orig = O.child_logprobs
    monkeypatch.setattr(O, "child_logprobs",
                        lambda L_d, E, W, h_d, p, dt: orig(L_d, E, W, h_d, 0, dt))


def _mut_depth_desc(monkeypatch):
    monkeypatch.setattr(O, "_glob_key", lambda n: (-n.score, -n.depth, n.token, n.slot))


def _mut_transposed_head(monkeypatch):
    orig = O.child_logprobs

    def f(L_d, E, W, h_d, p, dtype):
        r, V = W.shape
        if r == V:
            return orig(L_d, E, W.T, h_d, p, dtype)
        Wp = np.roll(W, 1, axis=0)  # rank index off by one
        return orig(L_d, E, Wp, h_d, p, dtype)
    monkeypatch.setattr(O, "child_logprobs", f)


def _mut_independent_unnormalised(monkeypatch):
    monkeypatch.setattr(O, "position_rows", lambda L_d: L_d.astype(np.float64))  # no lse


@pytest.mark.parametrize("mutate", [_mut_independent_unnormalised, _mut_no_lse, _mut_silu_sign, _mut_tie_rule,
                                    _mut_prune_by_token, _mut_wrong_parent,
                                    _mut_depth_desc, _mut_transposed_head])
def test_mutation_is_caught(monkeypatch, mutate):
    mutate(monkeypatch)
    assert _some_pin_fails(), f"no pin caught {mutate.__name__}"
