"""The acceptance parity rule's own arithmetic, on the CPU: the admissible count of final-draw
near-ties stays finite and covers every sequence when all the draws are near-ties (a nearly
flat distribution at a high temperature)."""
import types

import numpy as np

import gpu_util as G
import oracle


def test_tie_bound_with_probabilities_rounded_above_one():
    ref = types.SimpleNamespace(sample_tie_p=np.array([1.0 + 4e-16, 1.0, 1.0 - 1e-16, 0.25]))
    b = G.sample_tie_bound(ref, np.ones(4, bool))
    assert np.isfinite(b) and b >= 4.0


def test_flat_distribution_every_draw_a_near_tie():
    """Equal logits over a vocabulary whose every token's interval is narrower than twice the
    band: the oracle's tie probability is one (up to rounding) and the bound admits all S."""
    S, V = 3, 120_000
    target = np.zeros((S, V), np.float32)  # one anchor row per sequence: bonus draws only
    u = np.array([0.1, 0.5, 0.9], np.float32)
    r = oracle.accept(target, np.zeros((0, V), np.float32), np.zeros(0, np.int32), u, np.ones(S, np.int32),
                      np.arange(S + 1, dtype=np.int32), 20.0, band=G.BAND)
    assert np.allclose(r.sample_tie_p, 1.0, atol=1e-12)
    assert G.sample_tie_bound(r, np.ones(S, bool)) >= S
    # the drawn token is the one at u*V, up to the band
    assert np.all(np.abs(r.next_token - u.astype(np.float64) * V) <= 2 + G.BAND * V)
