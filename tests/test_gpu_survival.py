"""GPU parity of the prefix-survival model (sd_survival_tau, sd_survival_sample) against the fp64
oracle.

Tolerances.  tau, the regret and L_tau are fp64 on both sides; the sums run in a different
order (the oracle sums the prefix products pairwise, the kernel left to right) and the two
exp() implementations may differ in the last bit, so they agree to a few ulps: the test
allows 1e-12 relative.  B* must equal the oracle's unless the oracle's best two candidates
lie within that band (counted; then the device's choice must be one of them).  The
Monte-Carlo histograms are integers decided by u < q in fp64 on both sides from the same
Philox4x64-10 words: they must be identical.  A decision could only differ if u fell within
an ulp of q, where the two exp() results may differ; the test reports how close the nearest
draw came and allows no difference."""
import numpy as np
import pytest
import torch

import gpu_util as G
import oracle.survival as OS
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu
REL = 1e-12


def _tau_check(p, rows=None):
    dev = G.dev()
    G.log(f"sd_survival_tau N={p.N} P={p.P} C={len(p.cands)} alpha={p.alpha}")
    tau, b_star, regret, lip = sd.survival_tau(torch.from_numpy(p.gamma).to(dev), p.cands, p.train_block, p.alpha,
                                               torch.from_numpy(p.b_hat).to(dev))
    torch.cuda.synchronize()
    tau, b_star, regret, lip = (x.cpu().numpy() for x in (tau, b_star, regret, lip))
    idx = np.arange(p.N) if rows is None else rows
    ref = OS.survival_tau(p.gamma[idx], p.cands, p.train_block, p.alpha, p.b_hat[idx])
    tau, b_star, regret, lip = tau[idx], b_star[idx], regret[idx], lip[idx]
    scale = np.maximum(np.abs(ref.tau), 1e-300)
    assert (np.abs(tau - ref.tau) <= REL * scale + 1e-300).all(), np.max(np.abs(tau - ref.tau) / scale)
    near = ref.margin <= 4 * REL * np.abs(ref.tau).max(axis=1)
    assert np.array_equal(b_star[~near], ref.b_star[~near])
    for n in np.nonzero(near)[0]:
        top2 = np.asarray(p.cands)[np.argsort(ref.tau[n], kind="stable")[-2:]]
        assert b_star[n] in top2 or ref.tau[n].max() == ref.tau[n].min()
    nan = np.isnan(ref.regret)
    assert np.array_equal(np.isnan(regret), nan)
    rscale = np.abs(ref.tau).max(axis=1)[~nan]
    assert (np.abs(regret[~nan] - ref.regret[~nan]) <= 4 * REL * rscale).all()
    assert (np.abs(lip - ref.lipschitz) <= 4 * REL * np.maximum(ref.lipschitz, 1e-300)).all()
    G.log(f"  max rel tau error {np.max(np.abs(tau - ref.tau) / scale):.2e}; near-ties {int(near.sum())}")
    return tau, b_star


def test_tau_several_workgroups_and_a_ragged_tail():
    _tau_check(W.make_survival(31, N=1000, P=32, radius=2, alpha=0.01))


def test_tau_wide_interval_rows_not_a_vector_multiple():
    p = W.make_survival(32, N=300, P=30, train_block=16, radius=7, alpha=0.02)
    p.b_hat[::7] = 99                     # not a candidate: regret NaN
    _tau_check(p)


def test_tau_64_candidates_128_positions():
    p = W.make_survival(33, N=200, P=128, train_block=64, radius=2, alpha=0.001, gamma_lo=0.9, gamma_hi=0.995)
    p.cands = np.arange(1, 128, 2, dtype=np.int32)[:64]          # 64 odd sizes up to 127
    p.b_hat = p.cands[np.arange(p.N) % 64].astype(np.int32)
    _tau_check(p)


def test_tau_degenerate_cases():
    p = W.make_survival(34, N=70, P=16, train_block=8, radius=3, alpha=0.05)
    p.gamma[:10] = 0.0                    # every tau 0: B* is the smallest candidate
    p.gamma[10:20] = 1.0                  # certain positions
    tau, b_star = _tau_check(p)
    assert (b_star[:10] == p.cands[0]).all() and (tau[:10] == 0).all()
    one = W.make_survival(35, N=1, P=8, train_block=4, radius=0, alpha=0.1)
    _tau_check(one)


def test_tau_full_size_sampled_rows():
    """The benchmark's population (2^20 samples) in the benchmark's launch; 512 sampled rows,
    including the first and last workgroup, checked against the oracle."""
    p = W.make_survival(36, N=1 << 20, P=32, radius=2, alpha=0.01)
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([np.arange(256), np.arange(p.N - 256, p.N), rng.choice(p.N, 512)]))
    _tau_check(p, rows)


def _sample_check(p, seed, trials, pairs=None):
    dev = G.dev()
    G.log(f"sd_survival_sample N={p.N} P={p.P} C={len(p.cands)} trials={trials} seed={seed}")
    mean, hist = sd.survival_sample(torch.from_numpy(p.gamma).to(dev), p.cands, p.train_block, p.alpha, seed, trials)
    torch.cuda.synchronize()
    mean, hist = mean.cpu().numpy(), hist.cpu().numpy()
    if pairs is None:
        ref_hist, ref_mean = OS.survival_sample(p.gamma, p.cands, p.train_block, p.alpha, seed, trials)
        assert np.array_equal(hist, ref_hist)
        assert np.array_equal(mean, ref_mean)
    else:
        for n, c in pairs:
            L = OS.sample_lengths(p.gamma[n].astype(np.float64), int(p.cands[c]), p.train_block, p.alpha, seed, n, c,
                                  trials)
            assert np.array_equal(hist[n, c], np.bincount(L, minlength=p.P + 1)), (n, c)
            assert mean[n, c] == L.sum() / trials
    assert (hist.sum(axis=2) == trials).all()
    return mean, hist


def test_sample_bit_exact_small():
    _sample_check(W.make_survival(41, N=9, P=32, radius=2, alpha=0.01), seed=12345, trials=3000)


def test_sample_trials_not_a_wave_multiple_odd_positions():
    _sample_check(W.make_survival(42, N=5, P=30, train_block=12, radius=3, alpha=0.03), seed=2**64 - 5, trials=999)


def test_sample_certain_and_impossible_positions():
    p = W.make_survival(43, N=4, P=20, train_block=10, radius=1, alpha=0.0)
    p.gamma[0] = 1.0
    p.gamma[1] = 0.0
    mean, hist = _sample_check(p, seed=7, trials=130)
    assert (mean[0] == p.cands).all() and (mean[1] == 0).all()


def test_sample_full_size_sampled_pairs():
    """The benchmark's Monte-Carlo launch (2^16 samples x 5 candidates x 1024 trials); 24 sampled
    (sample, candidate) pairs replayed by the oracle trial by trial."""
    p = W.make_survival(44, N=1 << 16, P=32, radius=2, alpha=0.01)
    rng = np.random.default_rng(1)
    pairs = [(0, 0), (p.N - 1, 4)] + [(int(n), int(c)) for n, c in zip(rng.choice(p.N, 22), rng.integers(0, 5, 22))]
    _sample_check(p, seed=2024, trials=1024, pairs=pairs)
