"""Pins of the block-size policy oracle: an independent torch fp64 implementation of the same
network, closed forms with selector weights and zeroed layers, softmax shift invariance, the
lowest-candidate tie rule, and planted mistakes that must fail."""
import numpy as np
import pytest
import scipy.special
import torch

import oracle.policy as OP
from paper_2606_31315_amd import workloads as W


def _small(seed=5, P=3, V=512, H=64, radius=2):
    return W.make_policy(seed, P=P, V=V, H=H, radius=radius, dtype="f32")


def _run(pp, fn=None):
    fn = fn or OP.block_size_policy
    return fn(pp.logits, pp.w1, pp.b1, pp.w2, pp.b2, pp.w3, pp.b3, pp.base_block, pp.radius)


def test_matches_torch_sequential_fp64():
    pp = _small()
    net = torch.nn.Sequential(torch.nn.Linear(pp.V, pp.H), torch.nn.ReLU(), torch.nn.Linear(pp.H, pp.H),
                              torch.nn.ReLU(), torch.nn.Linear(pp.H, 2 * pp.radius + 1)).double()
    with torch.no_grad():
        for lin, w, b in zip([net[0], net[2], net[4]], [pp.w1, pp.w2, pp.w3], [pp.b1, pp.b2, pp.b3]):
            lin.weight.copy_(w.double())
            lin.bias.copy_(torch.from_numpy(b).double())
        o = net(torch.softmax(pp.logits.double(), dim=1)).numpy()
    r = _run(pp)
    assert np.abs(r.scores - o).max() < 1e-12
    assert np.array_equal(r.block_size, pp.base_block - pp.radius + np.argmax(o, axis=1))


def test_selector_weights_give_probabilities():
    """W1 rows pick single vocabulary entries, W2 = I, W3 = I (H = 2k+1): scores = p[sel] + b."""
    pp = _small(H=5)
    V = pp.V
    sel = np.array([3, 100, 7, 511, 0])
    w1 = torch.zeros(5, V, dtype=torch.bfloat16)
    w1[np.arange(5), sel] = 1.0
    pp.w1 = w1
    pp.w2 = torch.eye(5, dtype=torch.bfloat16)
    pp.w3 = torch.eye(5, dtype=torch.bfloat16)
    pp.b1[:] = 0.0
    pp.b2[:] = 0.0
    r = _run(pp)
    p = scipy.special.softmax(pp.logits.double().numpy(), axis=1)
    assert np.abs(r.scores - (p[:, sel] + pp.b3)).max() < 1e-14


def test_zero_network_takes_the_bias_argmax_and_lowest_tie():
    pp = _small(radius=3)
    pp.w3 = torch.zeros_like(pp.w3)
    pp.b3 = np.array([0.1, 0.5, -1.0, 0.5, 0.2, 0.0, 0.5], np.float32)
    r = _run(pp)
    assert (r.block_size == pp.base_block - 3 + 1).all()  # three candidates tie at 0.5: the smallest wins


def test_relu_zeroes_negative_preactivations():
    pp = _small()
    pp.w1 = torch.zeros_like(pp.w1)
    pp.b1[:] = -1.0
    r = _run(pp)
    expect = np.maximum(pp.b2.astype(np.float64), 0) @ pp.w3.double().numpy().T + pp.b3
    assert np.abs(r.scores - expect[None, :]).max() < 1e-14


def test_softmax_shift_invariance():
    pp = _small()
    r0 = _run(pp)
    pp.logits = pp.logits.double() + 7.0  # shifted exactly in fp64
    r1 = _run(pp)
    assert np.abs(r0.scores - r1.scores).max() < 1e-12


def _mutant(kind):
    """The oracle's network with one plausible mistake."""
    def f(logits, w1, b1, w2, b2, w3, b3, base_block, radius):
        z = OP._f64(logits)
        p = OP.softmax_rows(z)
        if kind == "double_softmax":
            p = OP.softmax_rows(p)
        if kind == "logits_as_input":
            p = z
        act = (lambda x: x) if kind == "no_relu" else (lambda x: np.maximum(x, 0.0))
        h1 = act(p @ OP._f64(w1).T + OP._f64(b1))
        h2 = act(h1 @ OP._f64(w2).T + OP._f64(b2))
        o = h2 @ OP._f64(w3).T + OP._f64(b3)
        best = np.argmax(o, axis=1)
        if kind == "highest_tie":
            best = o.shape[1] - 1 - np.argmax(o[:, ::-1], axis=1)
        return OP.PolicyResult(o, (base_block - radius + best).astype(np.int32), np.zeros(o.shape[0]))
    return f


@pytest.mark.parametrize("mutant", ["no_relu", "double_softmax", "highest_tie", "logits_as_input"])
def test_planted_mistakes_fail_a_pin(mutant, monkeypatch):
    monkeypatch.setattr(OP, "block_size_policy", _mutant(mutant))
    pins = [test_matches_torch_sequential_fp64, test_selector_weights_give_probabilities,
            test_zero_network_takes_the_bias_argmax_and_lowest_tie, test_relu_zeroes_negative_preactivations]
    failed = 0
    for pin in pins:
        try:
            pin()
        except AssertionError:
            failed += 1
    assert failed > 0, f"mutant {mutant} passed every pin"


def test_unmutated_network_passes_every_pin(monkeypatch):
    """The mutant harness itself: the network without a mistake passes."""
    monkeypatch.setattr(OP, "block_size_policy", _mutant("none"))
    for pin in [test_matches_torch_sequential_fp64, test_selector_weights_give_probabilities,
                test_zero_network_takes_the_bias_argmax_and_lowest_tie, test_relu_zeroes_negative_preactivations,
                test_softmax_shift_invariance]:
        pin()
