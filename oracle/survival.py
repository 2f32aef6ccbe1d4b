"""fp64 CPU oracle of the prefix-survival model of acceptance length.

TEST INFRASTRUCTURE ONLY: the test suite and the benchmark's CPU-baseline leg are the only
callers.  Plain numpy, fp64, written from App. A of the paper:

  App. A.1 (prefix-survival identity, Eq. tau_prefix_survival): with q_j(x, b) the probability
    that drafted position j is accepted given that positions 1..j-1 were,
        tau(b; x) = E[L_b(x)] = sum_{i=1..b} prod_{j=1..i} q_j(x, b).
  App. A.2 (predictability-retention decomposition): q_j(x, b) = gamma_j(x) r(b; B) with the
    retention r(b; B) = exp(-alpha (b - B)^2), B the drafter's training block size.
  App. A.2 (local candidate interval): B*(x) = argmax over the candidate set of tau(b; x).
  App. A.3 (regret): R(x) = tau(B*(x); x) - tau(B_hat(x); x), bounded by
    L_tau |B*(x) - B_hat(x)| when tau is L_tau-Lipschitz over the candidates.

Readings (the paper is silent on them):
  * argmax ties go to the smallest block size;
  * L_tau(x) is the smallest constant that satisfies the discrete Lipschitz condition for
    sample x: the largest |tau(b1) - tau(b2)| / |b1 - b2| over candidate pairs;
  * the Monte-Carlo sampler draws the uniform of drafted position i (1-based) of trial t,
    candidate c, sample n from Philox4x64-10 (Salmon et al., SC'11) with key (seed, 0) and
    counter ((i-1) div 4, t, c, n): word (i-1) mod 4 of the block, as the top 53 bits over
    2^53.  Position i is accepted iff u < q_i(x, b); L is the number of leading acceptances.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

# ---------------------------------------------------------------------------------------- #
# Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
# SC'11): ten rounds of two 64x64 -> 128-bit multiplies on a 4-word counter, with the
# 2-word key advanced by the Weyl constants between rounds.
# ---------------------------------------------------------------------------------------- #
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15  # golden ratio
PHILOX_W1 = 0xBB67AE8584CAA73B  # sqrt(3) - 1
_M32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo(a: int, b: np.ndarray):
    """(high, low) 64-bit halves of the 128-bit product of the constant a and the words b."""
    a_lo, a_hi = np.uint64(a & 0xFFFFFFFF), np.uint64(a >> 32)
    b_lo, b_hi = b & _M32, b >> _S32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> _S32) + (lh & _M32) + (hl & _M32)
    hi = hh + (lh >> _S32) + (hl >> _S32) + (mid >> _S32)
    lo = (mid << _S32) | (ll & _M32)
    return hi, lo


def philox4x64(counter, key) -> np.ndarray:
    """Philox4x64-10 of counters [..., 4] under key (k0, k1); returns [..., 4] uint64."""
    c = np.array(counter, dtype=np.uint64)
    c0, c1, c2, c3 = (c[..., i].copy() for i in range(4))
    k0, k1 = int(key[0]) & (2**64 - 1), int(key[1]) & (2**64 - 1)
    with np.errstate(over="ignore"):
        for r in range(10):
            hi0, lo0 = _mulhilo(PHILOX_M0, c0)
            hi1, lo1 = _mulhilo(PHILOX_M1, c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0
            k0 = (k0 + PHILOX_W0) & (2**64 - 1)
            k1 = (k1 + PHILOX_W1) & (2**64 - 1)
    return np.stack([c0, c1, c2, c3], axis=-1)


def uniform53(words: np.ndarray) -> np.ndarray:
    """[0, 1) doubles from the top 53 bits of 64-bit words."""
    return (words >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)


# ---------------------------------------------------------------------------------------- #
# the model
# ---------------------------------------------------------------------------------------- #
def retention(b, train_block: int, alpha: float):
    """r(b; B) = exp(-alpha (b - B)^2)  (App. A.2)."""
    d = np.asarray(b, dtype=np.float64) - float(train_block)
    return np.exp(-float(alpha) * d * d)


def acceptance_probs(gamma_row: np.ndarray, b: int, train_block: int, alpha: float) -> np.ndarray:
    """q_j(x, b) = gamma_j(x) r(b; B) for j = 1..b  (App. A.2)."""
    return np.asarray(gamma_row[:b], dtype=np.float64) * retention(b, train_block, alpha)


def tau(gamma_row: np.ndarray, b: int, train_block: int, alpha: float) -> float:
    """tau(b; x) = sum_{i=1..b} prod_{j<=i} q_j(x, b)  (Eq. tau_prefix_survival)."""
    q = acceptance_probs(gamma_row, b, train_block, alpha)
    return float(np.cumprod(q).sum())


@dataclass
class SurvivalResult:
    tau: np.ndarray        # [N, C] fp64
    b_star: np.ndarray     # [N] int32
    regret: Optional[np.ndarray]     # [N] fp64 (None without b_hat)
    lipschitz: np.ndarray  # [N] fp64
    margin: np.ndarray     # [N] fp64: tau(B*) minus the best other candidate's tau (0 if C == 1)


def survival_tau(gamma, cands, train_block: int, alpha: float, b_hat=None) -> SurvivalResult:
    """tau(b; x) for every sample x (rows of gamma [N, P]) and candidate b; B*(x); the regret of
    b_hat [N] (App. A.3; NaN where b_hat is not a candidate); L_tau(x)."""
    g = np.asarray(gamma, dtype=np.float64)
    cands = [int(b) for b in cands]
    N, C = g.shape[0], len(cands)
    t = np.zeros((N, C))
    for n in range(N):
        for c, b in enumerate(cands):
            t[n, c] = tau(g[n], b, train_block, alpha)
    best = np.zeros(N, dtype=np.int64)
    for n in range(N):
        for c in range(1, C):          # strict: ties keep the smaller block size
            if t[n, c] > t[n, best[n]]:
                best[n] = c
    b_star = np.array([cands[c] for c in best], dtype=np.int32)
    margin = np.zeros(N)
    if C > 1:
        for n in range(N):
            others = [t[n, c] for c in range(C) if c != best[n]]
            margin[n] = t[n, best[n]] - max(others)
    lip = np.zeros(N)
    for n in range(N):
        for c1 in range(C):
            for c2 in range(c1 + 1, C):
                lip[n] = max(lip[n], abs(t[n, c1] - t[n, c2]) / (cands[c2] - cands[c1]))
    regret = None
    if b_hat is not None:
        bh = np.asarray(b_hat, dtype=np.int64)
        regret = np.full(N, np.nan)
        for n in range(N):
            if int(bh[n]) in cands:
                regret[n] = t[n, best[n]] - t[n, cands.index(int(bh[n]))]
    return SurvivalResult(t, b_star, regret, lip, margin)


def sample_lengths(gamma_row: np.ndarray, b: int, train_block: int, alpha: float, seed: int, n: int, c: int,
                   trials: int) -> np.ndarray:
    """L_b(x) of each trial t < trials for sample n, candidate index c: the length of the
    longest prefix of drafted positions all accepted, position i accepted iff u < q_i(x, b)."""
    q = acceptance_probs(gamma_row, b, train_block, alpha)
    t = np.arange(trials, dtype=np.uint64)
    nblk = (b + 3) // 4
    ctr = np.zeros((trials, nblk, 4), dtype=np.uint64)
    ctr[:, :, 0] = np.arange(nblk, dtype=np.uint64)[None, :]
    ctr[:, :, 1] = t[:, None]
    ctr[:, :, 2] = np.uint64(c)
    ctr[:, :, 3] = np.uint64(n)
    u = uniform53(philox4x64(ctr, (seed, 0)).reshape(trials, nblk * 4))[:, :b]
    accepted = u < q[None, :]
    # leading run of acceptances: the first rejected position, or b if none
    first_reject = np.where(accepted.all(axis=1), b, np.argmin(accepted, axis=1))
    return first_reject.astype(np.int64)


def survival_sample(gamma, cands, train_block: int, alpha: float, seed: int, trials: int):
    """Monte-Carlo L_b(x) over `trials` trials for every sample and candidate: returns
    (histogram [N, C, P + 1] int64 of L = 0..P, mean [N, C] fp64)."""
    g = np.asarray(gamma, dtype=np.float64)
    N, P = g.shape
    C = len(cands)
    hist = np.zeros((N, C, P + 1), dtype=np.int64)
    for n in range(N):
        for c, b in enumerate(cands):
            L = sample_lengths(g[n], int(b), train_block, alpha, seed, n, c, trials)
            hist[n, c] = np.bincount(L, minlength=P + 1)
    mean = (hist * np.arange(P + 1)[None, None, :]).sum(axis=2) / float(trials)
    return hist, mean
