"""Pins of the prefix-survival oracle (App. A): numpy's own Philox4x64-10 bit generator,
the expectation of L_b by enumerating every accept pattern, the distribution of L_b, the
geometric closed form (Eq. tau_geometric), closed cases of the block-size argmax, the
regret bound of App. A.3, Monte-Carlo agreement within four standard errors, and planted
mistakes that must fail."""
import itertools
import sys
import types

import numpy as np
import pytest

import oracle.survival as OS
from paper_2606_31315_amd import workloads as W


# ---------------------------------------------------------------------------------------- #
# pin checks, parameterised by the oracle module so planted mistakes can be run through them
# ---------------------------------------------------------------------------------------- #
def check_philox(S):
    """numpy's Philox bit generator increments its 256-bit counter, then emits the four words
    of Philox4x64-10 of the new counter."""
    for key, ctr in [((0, 0), (0, 0, 0, 0)), ((0x1234, 0x5678), (7, 0, 0, 0)),
                     ((2**64 - 1, 7), (2**64 - 1, 5, 9, 11)), ((123456789, 987654321), (2**64 - 1, 2**64 - 1, 3, 0))]:
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(ctr, dtype=np.uint64))
        ref = bg.random_raw(8)
        c = list(ctr)
        blocks = []
        for _ in range(2):
            for w in range(4):        # add one with carry
                c[w] = (c[w] + 1) % 2**64
                if c[w] != 0:
                    break
            blocks.append(list(c))
        mine = S.philox4x64(np.array(blocks, dtype=np.uint64), key).reshape(-1)
        assert np.array_equal(ref, mine), (key, ctr)
        # numpy's doubles take the top 53 bits of each word
        gen = np.random.Generator(np.random.Philox(key=np.array(key, dtype=np.uint64),
                                                   counter=np.array(ctr, dtype=np.uint64)))
        assert np.array_equal(gen.random(8), S.uniform53(mine)), (key, ctr)


def _enumerated_mean(q):
    """E[L] as the sum over all 2^b accept/reject patterns of P(pattern) * (leading accepts)."""
    b = len(q)
    total = 0.0
    for pat in itertools.product([0, 1], repeat=b):
        pr = 1.0
        for a, qi in zip(pat, q):
            pr *= qi if a else 1.0 - qi
        lead = b if all(pat) else pat.index(0)
        total += pr * lead
    return total


def check_enumeration(S):
    rng = np.random.default_rng(3)
    for b, B, alpha in [(1, 1, 0.0), (4, 3, 0.05), (7, 8, 0.02), (9, 9, 0.3), (10, 6, 0.01)]:
        g = rng.uniform(0.05, 1.0, size=12).astype(np.float32)
        q = g[:b].astype(np.float64) * np.exp(-alpha * (b - B) ** 2)
        assert abs(S.tau(g, b, B, alpha) - _enumerated_mean(q)) < 1e-12, (b, B, alpha)


def check_distribution_mean(S):
    """E[L] = sum_l l P(L = l) with P(L = l) = q_1..q_l (1 - q_{l+1}), P(L = b) = q_1..q_b."""
    rng = np.random.default_rng(4)
    for b in (8, 16, 24, 32):
        g = rng.uniform(0.5, 1.0, size=40).astype(np.float32)
        q = g[:b].astype(np.float64) * np.exp(-0.01 * (b - 16) ** 2)
        mean, run = 0.0, 1.0
        for l in range(b + 1):
            p_l = run * (1.0 - q[l]) if l < b else run
            mean += l * p_l
            if l < b:
                run *= q[l]
        assert abs(S.tau(g, b, 16, 0.01) - mean) < 1e-12 * max(1.0, mean), b


def check_geometric(S):
    """Constant predictability: tau = rho (1 - rho^b) / (1 - rho), rho = gamma r(b; B)."""
    for gam, b, B, alpha in [(0.9, 16, 16, 0.01), (0.75, 14, 16, 0.02), (0.97, 20, 16, 0.005), (0.5, 3, 10, 0.0)]:
        g = np.full(32, gam, dtype=np.float32)
        rho = float(np.float32(gam)) * np.exp(-alpha * (b - B) ** 2)
        closed = rho * (1.0 - rho ** b) / (1.0 - rho)
        assert abs(S.tau(g, b, B, alpha) - closed) < 1e-12 * closed


def check_certain_positions(S):
    """gamma = 1 at the training block size: every drafted position is accepted, tau = b."""
    g = np.ones(32, dtype=np.float32)
    for B in (1, 8, 16, 32):
        assert S.tau(g, B, B, 0.3) == float(B)


def check_argmax_cases(S):
    cands = [12, 14, 16, 18, 20]
    N = 3
    zero = np.zeros((N, 32), dtype=np.float32)
    r = S.survival_tau(zero, cands, 16, 0.01)
    assert (r.tau == 0).all() and (r.b_star == 12).all()           # all tied: smallest size
    one = np.ones((N, 32), dtype=np.float32)
    r = S.survival_tau(one, cands, 16, 0.0)
    assert (r.b_star == 20).all()                                    # no retention loss: longest
    assert np.allclose(r.tau, np.array(cands, dtype=np.float64)[None, :])
    r = S.survival_tau(one, cands, 16, 5.0)
    assert (r.b_star == 16).all()                                    # sharp retention: the training size
    g = np.full((1, 32), 0.9, dtype=np.float32)
    r = S.survival_tau(g, [16], 16, 0.01)
    assert r.b_star[0] == 16 and r.margin[0] == 0.0 and r.lipschitz[0] == 0.0


def check_regret(S):
    p = W.make_survival(21, N=64, P=32, train_block=16, radius=3, alpha=0.02)
    r = S.survival_tau(p.gamma, p.cands, p.train_block, p.alpha, p.b_hat)
    assert (r.regret >= 0).all()
    assert (r.regret[p.b_hat == r.b_star] == 0).all()
    # App. A.3: R(x) <= L_tau |B*(x) - B_hat(x)|
    assert (r.regret <= r.lipschitz * np.abs(r.b_star - p.b_hat) + 1e-12).all()
    # and L_tau is attained: some adjacent-or-not pair has exactly that slope
    for n in range(8):
        slopes = [abs(r.tau[n, i] - r.tau[n, j]) / (p.cands[j] - p.cands[i])
                  for i in range(len(p.cands)) for j in range(i + 1, len(p.cands))]
        assert r.lipschitz[n] == max(slopes)
    bad = p.b_hat.copy()
    bad[0] = 99
    assert np.isnan(S.survival_tau(p.gamma[:2], p.cands, 16, p.alpha, bad[:2]).regret[0])


def check_monte_carlo(S):
    p = W.make_survival(22, N=6, P=32, train_block=16, radius=2, alpha=0.01)
    trials = 4000
    hist, mean = S.survival_sample(p.gamma, p.cands, p.train_block, p.alpha, seed=77, trials=trials)
    assert (hist.sum(axis=2) == trials).all()
    for c, b in enumerate(p.cands):
        assert (hist[:, c, b + 1:] == 0).all()                       # L_b <= b
    r = S.survival_tau(p.gamma, p.cands, p.train_block, p.alpha)
    L = np.arange(p.P + 1)
    var = (hist * L[None, None, :] ** 2).sum(axis=2) / trials - mean ** 2
    se = np.sqrt(var / trials)
    assert (np.abs(mean - r.tau) <= 4 * se + 1e-12).all(), np.abs(mean - r.tau) / se
    # empirical survival P(L >= i) against the prefix product prod_{j<=i} q_j (App. A.1)
    n, c = 2, 2
    b = int(p.cands[c])
    surv = hist[n, c, ::-1].cumsum()[::-1][1:b + 1] / trials          # P(L >= i), i = 1..b
    q = p.gamma[n, :b].astype(np.float64) * np.exp(-p.alpha * (b - p.train_block) ** 2)
    pref = np.cumprod(q)
    assert (np.abs(surv - pref) <= 4 * np.sqrt(pref * (1 - pref) / trials) + 1e-9).all()


def check_never_below_training_size(S):
    """Shorter blocks than B lose both terms and retention (r <= 1 = r(B; B)), so with B among
    the candidates B* >= B for every sample."""
    for seed, alpha in ((24, 0.001), (25, 0.02), (26, 0.3)):
        p = W.make_survival(seed, N=40, P=32, train_block=16, radius=4, alpha=alpha, gamma_lo=0.3, gamma_hi=1.0,
                            jitter=0.2)
        r = S.survival_tau(p.gamma, p.cands, p.train_block, p.alpha)
        assert (r.b_star >= 16).all()
        assert (r.tau[:, :4] <= r.tau[:, 4:5]).all()


PINS = [check_never_below_training_size, check_philox, check_enumeration, check_distribution_mean, check_geometric, check_certain_positions,
        check_argmax_cases, check_regret, check_monte_carlo]


@pytest.mark.parametrize("pin", PINS, ids=[f.__name__ for f in PINS])
def test_pin(pin):
    pin(OS)


def test_counter_layout_is_the_documented_one():
    """Trial t, candidate c, sample n, position i draws word (i-1) % 4 of the Philox block at
    counter ((i-1) // 4, t, c, n): rebuild one trial's uniforms by hand and replay it."""
    p = W.make_survival(23, N=3, P=32)
    n, c, t, seed = 2, 3, 5, 99
    b = int(p.cands[c])
    words = [OS.philox4x64(np.array([[blk, t, c, n]], dtype=np.uint64), (seed, 0))[0] for blk in range((b + 3) // 4)]
    u = OS.uniform53(np.concatenate(words))[:b]
    q = p.gamma[n, :b].astype(np.float64) * np.exp(-p.alpha * (b - p.train_block) ** 2)
    lead = 0
    while lead < b and u[lead] < q[lead]:
        lead += 1
    assert OS.sample_lengths(p.gamma[n], b, p.train_block, p.alpha, seed, n, c, t + 1)[t] == lead


# ---------------------------------------------------------------------------------------- #
# planted mistakes: each must fail at least one pin
# ---------------------------------------------------------------------------------------- #
MUTANTS = {
    "horizon_b_minus_1": ("return float(np.cumprod(q).sum())", "return float(np.cumprod(q)[:-1].sum())"),
    "retention_linear": ("np.exp(-float(alpha) * d * d)", "np.exp(-float(alpha) * np.abs(d))"),
    "retention_once": ("np.asarray(gamma_row[:b], dtype=np.float64) * retention(b, train_block, alpha)",
                       "np.asarray(gamma_row[:b], dtype=np.float64) * np.r_[retention(b, train_block, alpha), np.ones(b - 1)]"),
    "shifted_position": ("np.asarray(gamma_row[:b], dtype=np.float64)", "np.asarray(gamma_row[1:b + 1], dtype=np.float64)"),
    "ties_to_largest": ("if t[n, c] > t[n, best[n]]:", "if t[n, c] >= t[n, best[n]]:"),
    "regret_sign": ("regret[n] = t[n, best[n]] - t[n, cands.index(int(bh[n]))]",
                    "regret[n] = t[n, cands.index(int(bh[n]))] - t[n, best[n]]"),
    "lipschitz_undivided": ("abs(t[n, c1] - t[n, c2]) / (cands[c2] - cands[c1])", "abs(t[n, c1] - t[n, c2])"),
    "mc_off_by_one": ("np.argmin(accepted, axis=1))", "np.argmin(accepted, axis=1) + 1)"),
    "mc_accept_inverted": ("accepted = u < q[None, :]", "accepted = u > q[None, :]"),
    "philox_multiplier": ("PHILOX_M1 = 0xCA5A826395121157", "PHILOX_M1 = 0xCA5A826395121156"),
    "philox_nine_rounds": ("for r in range(10):", "for r in range(9):"),
    "philox_key_not_bumped": ("k1 = (k1 + PHILOX_W1) & (2**64 - 1)", "k1 = k1"),
    "uniform_low_bits": ("(words >> np.uint64(11))", "(words & np.uint64(2**53 - 1))"),
}


def _mutant(name):
    old, new = MUTANTS[name]
    src = open(OS.__file__).read()
    assert src.count(old) == 1, name
    mod = types.ModuleType(f"survival_mutant_{name}")
    sys.modules[mod.__name__] = mod  # dataclasses look their module up by name
    try:
        exec(compile(src.replace(old, new), f"<{name}>", "exec"), mod.__dict__)
    finally:
        del sys.modules[mod.__name__]
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(name):
    mod = _mutant(name)
    failed = []
    for pin in PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
