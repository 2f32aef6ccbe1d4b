"""Pins for the fp64 oracle: checks against what the paper and the mathematics fix,
independent of the oracle's own code.

Each ``pin_*`` takes an ``oracle.Oracle`` handle and raises AssertionError when the
oracle disagrees.  The same functions run against the real oracle
(test_oracle_pins.py) and against mutated builds of it (test_oracle_mutants.py),
which shows that a plausible mistake in the oracle fails at least one pin.

What pins what:
  attention   torch's scaled_dot_product_attention (fp64, explicit boolean mask,
              enable_gqa) as a library routine; closed forms (zero query -> mean of
              the visible values; constant values -> that constant; a single
              dominant key -> its value); invariants (B=1 is decode attention, row
              independence, bidirectional rows = unmasked attention over ctx+B keys,
              GQA = MHA after repeat_kv, permutation of context rows).
  acceptance  numpy argmax (first occurrence) for greedy T=0; constructed cases;
              lossless property by chi-square (the committed token distributions
              equal the target's, Sec. 1 and Sec. 3.1 "Metrics"); expected accepted
              length = prefix-survival sum (App. A.1) with per-position acceptance
              probability 1 - TV(p, q); geometric closed form for equal positions
              (App. A.2); u = 0 edge; temperature scaling.
"""
from __future__ import annotations

import numpy as np
import scipy.special
import scipy.stats
import torch
import torch.nn.functional as F

CAUSAL, BIDIR = 0, 1


# --------------------------------------------------------------------------- #
# small problem builders (inputs only)
# --------------------------------------------------------------------------- #

def _offsets(bl):
    off = np.zeros(len(bl) + 1, dtype=np.int32)
    off[1:] = np.cumsum(bl)
    return off


def _attn_case(rng, ctx, bl, Hq=4, Hkv=2, D=16, Lmax=None):
    ctx = np.asarray(ctx, dtype=np.int32)
    bl = np.asarray(bl, dtype=np.int32)
    S = len(ctx)
    if Lmax is None:
        Lmax = int((ctx + bl).max()) + 3
    off = _offsets(bl)
    q = rng.standard_normal((int(off[-1]), Hq, D)).astype(np.float32)
    k = rng.standard_normal((S, Hkv, Lmax, D)).astype(np.float32)
    v = rng.standard_normal((S, Hkv, Lmax, D)).astype(np.float32)
    return q, k, v, ctx, bl, off


def _sdpa_reference(q, k, v, ctx, bl, off, mask_mode, Hq, Hkv):
    """torch SDPA in fp64 with an explicit boolean mask and grouped kv heads."""
    out = np.zeros(q.shape, dtype=np.float64)
    for s in range(len(ctx)):
        c, b = int(ctx[s]), int(bl[s])
        if b == 0:
            continue
        n = c + b
        qs = torch.from_numpy(q[off[s]:off[s] + b].astype(np.float64)).permute(1, 0, 2)  # [Hq,B,D]
        ks = torch.from_numpy(k[s, :, :n].astype(np.float64))                             # [Hkv,n,D]
        vs = torch.from_numpy(v[s, :, :n].astype(np.float64))
        j = torch.arange(n)[None, :]
        i = torch.arange(b)[:, None]
        allowed = (j <= c + i) if mask_mode == CAUSAL else torch.ones(b, n, dtype=torch.bool)
        o = F.scaled_dot_product_attention(qs[None], ks[None], vs[None], attn_mask=allowed,
                                           enable_gqa=(Hq != Hkv))[0]
        out[off[s]:off[s] + b] = o.permute(1, 0, 2).numpy()
    return out


# --------------------------------------------------------------------------- #
# attention pins
# --------------------------------------------------------------------------- #

def pin_attn_sdpa(orc):
    """Library routine: fp64 SDPA with an explicit (bottom-right aligned) mask."""
    rng = np.random.default_rng(11)
    for (Hq, Hkv, D) in [(4, 2, 16), (6, 3, 8), (4, 4, 12), (8, 1, 16)]:
        q, k, v, ctx, bl, off = _attn_case(rng, [0, 5, 9, 3], [3, 1, 4, 6], Hq, Hkv, D)
        for mode in (CAUSAL, BIDIR):
            got = orc.block_attn(q, k, v, ctx, bl, off, mode)
            ref = _sdpa_reference(q, k, v, ctx, bl, off, mode, Hq, Hkv)
            err = np.abs(got - ref).max()
            assert err < 1e-12, f"SDPA mismatch {err} (Hq={Hq},Hkv={Hkv},mode={mode})"


def pin_attn_zero_query(orc):
    """Zero query => equal scores => output is the mean of exactly the visible values."""
    rng = np.random.default_rng(12)
    q, k, v, ctx, bl, off = _attn_case(rng, [4, 0, 7], [5, 3, 2], Hq=4, Hkv=2, D=8)
    q[:] = 0
    for mode in (CAUSAL, BIDIR):
        got = orc.block_attn(q, k, v, ctx, bl, off, mode)
        for s in range(3):
            for i in range(int(bl[s])):
                n = int(ctx[s]) + (i + 1 if mode == CAUSAL else int(bl[s]))
                for h in range(4):
                    ref = v[s, h // 2, :n].astype(np.float64).mean(axis=0)
                    assert np.abs(got[off[s] + i, h] - ref).max() < 1e-12, (mode, s, i, h)


def pin_attn_dominant_key(orc):
    """A key with a much larger score than all others takes all the weight, unless masked.

    Causal row i: the key at ctx+i is visible and dominant, the key at ctx+i+1 is even
    larger but must be masked, so the output is V[ctx+i].  Bidirectional rows see the
    larger key.
    """
    D, Hq, Hkv = 8, 2, 1
    ctx, B = 6, 4
    for i in range(B):
        k = np.zeros((1, Hkv, ctx + B + 2, D), dtype=np.float32)
        v = np.random.default_rng(13 + i).standard_normal((1, Hkv, ctx + B + 2, D)).astype(np.float32)
        q = np.zeros((B, Hq, D), dtype=np.float32)
        q[:, :, 0] = 1.0
        k[0, 0, ctx + i, 0] = 400.0
        if ctx + i + 1 < ctx + B:
            k[0, 0, ctx + i + 1, 0] = 800.0
        off = _offsets([B])
        got_c = orc.block_attn(q, k, v, [ctx], [B], off, CAUSAL)
        assert np.abs(got_c[i, 0] - v[0, 0, ctx + i]).max() < 1e-9, ("causal", i)
        got_b = orc.block_attn(q, k, v, [ctx], [B], off, BIDIR)
        top = ctx + i + 1 if i + 1 < B else ctx + i
        assert np.abs(got_b[0, 0] - v[0, 0, top]).max() < 1e-9, ("bidir", i)


def pin_attn_b1_is_decode(orc):
    """B=1: causal and bidirectional both reduce to decode attention over ctx+1 keys."""
    rng = np.random.default_rng(14)
    q, k, v, ctx, bl, off = _attn_case(rng, [0, 9, 17], [1, 1, 1], Hq=4, Hkv=2, D=16)
    c = orc.block_attn(q, k, v, ctx, bl, off, CAUSAL)
    b = orc.block_attn(q, k, v, ctx, bl, off, BIDIR)
    assert np.abs(c - b).max() < 1e-13
    for s in range(3):
        n = int(ctx[s]) + 1
        qs = torch.from_numpy(q[s].astype(np.float64))[:, None, :]                   # [Hq,1,D]
        ks = torch.from_numpy(k[s, :, :n].astype(np.float64)).repeat_interleave(2, 0)
        vs = torch.from_numpy(v[s, :, :n].astype(np.float64)).repeat_interleave(2, 0)
        ref = F.scaled_dot_product_attention(qs, ks, vs)[:, 0].numpy()
        assert np.abs(c[s] - ref).max() < 1e-12


def pin_attn_row_independence(orc):
    """Causal row i equals a B=1 call at ctx+i; a bidirectional row equals a B=1 call at ctx+B-1."""
    rng = np.random.default_rng(15)
    q, k, v, ctx, bl, off = _attn_case(rng, [5], [6], Hq=4, Hkv=1, D=8)
    c = orc.block_attn(q, k, v, ctx, bl, off, CAUSAL)
    b = orc.block_attn(q, k, v, ctx, bl, off, BIDIR)
    one = _offsets([1])
    for i in range(6):
        ci = orc.block_attn(q[i:i + 1], k, v, [5 + i], [1], one, CAUSAL)
        assert np.abs(c[i] - ci[0]).max() < 1e-13, i
        bi = orc.block_attn(q[i:i + 1], k, v, [5 + 6 - 1], [1], one, CAUSAL)
        assert np.abs(b[i] - bi[0]).max() < 1e-13, i


def pin_attn_gqa_repeat(orc):
    """GQA equals MHA after repeating each kv head over its group of query heads."""
    rng = np.random.default_rng(16)
    q, k, v, ctx, bl, off = _attn_case(rng, [3, 8], [4, 2], Hq=8, Hkv=2, D=8)
    kr = np.repeat(k, 4, axis=1)
    vr = np.repeat(v, 4, axis=1)
    for mode in (CAUSAL, BIDIR):
        g = orc.block_attn(q, k, v, ctx, bl, off, mode)
        m = orc.block_attn(q, kr, vr, ctx, bl, off, mode)
        assert np.abs(g - m).max() < 1e-13


def pin_attn_permutation(orc):
    """Jointly permuting context rows of K and V changes nothing; permuting in-block rows
    changes nothing for the bidirectional mask."""
    rng = np.random.default_rng(17)
    q, k, v, ctx, bl, off = _attn_case(rng, [9], [5], Hq=4, Hkv=2, D=8)
    perm = rng.permutation(9)
    k2, v2 = k.copy(), v.copy()
    k2[:, :, :9] = k[:, :, perm]
    v2[:, :, :9] = v[:, :, perm]
    for mode in (CAUSAL, BIDIR):
        a = orc.block_attn(q, k, v, ctx, bl, off, mode)
        b = orc.block_attn(q, k2, v2, ctx, bl, off, mode)
        assert np.abs(a - b).max() < 1e-12
    pb = 9 + rng.permutation(5)
    k3, v3 = k.copy(), v.copy()
    k3[:, :, 9:14] = k[:, :, pb]
    v3[:, :, 9:14] = v[:, :, pb]
    a = orc.block_attn(q, k, v, ctx, bl, off, BIDIR)
    b = orc.block_attn(q, k3, v3, ctx, bl, off, BIDIR)
    assert np.abs(a - b).max() < 1e-12


def pin_attn_constant_values(orc):
    """Constant value rows => the output is that constant for every row and mask."""
    rng = np.random.default_rng(18)
    q, k, v, ctx, bl, off = _attn_case(rng, [4, 0], [3, 2], Hq=4, Hkv=2, D=8)
    v[:] = 0.375
    for mode in (CAUSAL, BIDIR):
        o = orc.block_attn(q, k, v, ctx, bl, off, mode)
        assert np.abs(o - 0.375).max() < 1e-13


def pin_attn_scale(orc):
    """Default scale is 1/sqrt(D); an explicit scale s equals scaling q by s*sqrt(D)."""
    rng = np.random.default_rng(19)
    q, k, v, ctx, bl, off = _attn_case(rng, [6], [3], Hq=2, Hkv=1, D=16)
    a = orc.block_attn(q, k, v, ctx, bl, off, CAUSAL)
    b = orc.block_attn(q, k, v, ctx, bl, off, CAUSAL, scale=0.25)
    assert np.abs(a - b).max() < 1e-13
    c = orc.block_attn(q, k, v, ctx, bl, off, CAUSAL, scale=0.5)
    d = orc.block_attn(q * 2, k, v, ctx, bl, off, CAUSAL, scale=0.25)
    assert np.abs(c - d).max() < 1e-12


ATTN_PINS = [pin_attn_sdpa, pin_attn_zero_query, pin_attn_dominant_key, pin_attn_b1_is_decode,
             pin_attn_row_independence, pin_attn_gqa_repeat, pin_attn_permutation,
             pin_attn_constant_values, pin_attn_scale]


# --------------------------------------------------------------------------- #
# acceptance pins
# --------------------------------------------------------------------------- #

def pin_greedy_numpy_prefix(orc):
    """T=0: accept_len = longest prefix where the draft equals numpy's first-occurrence argmax;
    next token = argmax of the target row at accept_len."""
    rng = np.random.default_rng(21)
    bl = rng.integers(1, 8, size=40).astype(np.int32)
    off = _offsets(bl)
    V = 37
    t = rng.standard_normal((int(off[-1]), V)).astype(np.float32)
    t[rng.random(len(t)) < 0.2, 5] = 9.0  # plant some exact ties at the max
    t[rng.random(len(t)) < 0.2, 2] = 9.0
    am = np.argmax(t, axis=1)
    tok = np.empty(int(off[-1]) - len(bl), dtype=np.int32)
    for s in range(len(bl)):
        for j in range(int(bl[s]) - 1):
            tok[off[s] - s + j] = am[off[s] + j] if rng.random() < 0.75 else rng.integers(V)
    r = orc.accept(t, None, tok, None, bl, off, 0.0)
    for s in range(len(bl)):
        n = int(bl[s]) - 1
        a = 0
        while a < n and tok[off[s] - s + a] == am[off[s] + a]:
            a += 1
        assert r.accept_len[s] == a, s
        assert r.next_token[s] == am[off[s] + a], s


def pin_greedy_constructed(orc):
    """All drafts equal the argmax => accept everything, bonus = argmax of the last row;
    a mismatch at position 0 => accept nothing, next = argmax of row 0; B=1 => next = argmax."""
    V = 20
    t = np.zeros((5, V), dtype=np.float32)
    for i in range(5):
        t[i, (3 * i + 1) % V] = 1.0
    off = _offsets([5])
    tok = np.array([(3 * i + 1) % V for i in range(4)], dtype=np.int32)
    r = orc.accept(t, None, tok, None, [5], off, 0.0)
    assert r.accept_len[0] == 4 and r.next_token[0] == 13
    tok0 = tok.copy()
    tok0[0] = 0
    r = orc.accept(t, None, tok0, None, [5], off, 0.0)
    assert r.accept_len[0] == 0 and r.next_token[0] == 1
    r = orc.accept(t[:1], None, np.zeros(0, np.int32), None, [1], _offsets([1]), 0.0)
    assert r.accept_len[0] == 0 and r.next_token[0] == 1


def pin_greedy_ties_lowest(orc):
    """Tied maxima resolve to the lowest index: a draft of the higher tied index is rejected."""
    V = 16
    t = np.zeros((2, V), dtype=np.float32)
    t[:, 3] = t[:, 7] = 2.0
    off = _offsets([2])
    r = orc.accept(t, None, np.array([7], np.int32), None, [2], off, 0.0)
    assert r.accept_len[0] == 0 and r.next_token[0] == 3
    r = orc.accept(t, None, np.array([3], np.int32), None, [2], off, 0.0)
    assert r.accept_len[0] == 1 and r.next_token[0] == 3


def _softmax(x, T=1.0):
    return scipy.special.softmax(np.asarray(x, dtype=np.float64) / T)


def pin_sampling_identical_rows(orc):
    """delta == t => p/q = 1 => every draft is accepted for any u < 1; the bonus token is the
    inverse-CDF draw from p_n (numpy searchsorted on scipy's softmax)."""
    rng = np.random.default_rng(23)
    V, B = 30, 6
    t = rng.normal(0, 2, (B, V)).astype(np.float32)
    tok = rng.integers(0, V, B - 1).astype(np.int32)
    for trial in range(20):
        u = rng.random(B, dtype=np.float32)
        u[0] = np.float32(0.99999994)
        r = orc.accept(t, t[:B - 1], tok, u, [B], _offsets([B]), 1.0)
        assert r.accept_len[0] == B - 1
        cdf = np.cumsum(_softmax(t[B - 1]))
        ref = int(np.searchsorted(cdf, float(u[B - 1]) * cdf[-1], side="right"))
        if r.sample_margin[0] > 1e-12:
            assert r.next_token[0] == ref, trial


def pin_sampling_residual(orc):
    """A draft token the target gives almost no mass is rejected; the resample is the
    inverse-CDF draw from max(0, p - q) normalised (numpy on scipy's softmax)."""
    rng = np.random.default_rng(24)
    V = 12
    for trial in range(20):
        t = rng.normal(0, 1.5, (2, V)).astype(np.float32)
        dl = rng.normal(0, 1.5, (1, V)).astype(np.float32)
        t[0, 4] = -60.0
        dl[0, 4] = 6.0
        u = np.array([rng.random() * 0.99 + 0.005, rng.random()], dtype=np.float32)
        r = orc.accept(t, dl, np.array([4], np.int32), u, [2], _offsets([2]), 1.0)
        assert r.accept_len[0] == 0
        res = np.maximum(0.0, _softmax(t[0]) - _softmax(dl[0]))
        cdf = np.cumsum(res)
        ref = int(np.searchsorted(cdf, float(u[1]) * cdf[-1], side="right"))
        if r.sample_margin[0] > 1e-12:
            assert r.next_token[0] == ref, trial
        assert r.next_token[0] != 4


def pin_sampling_u_zero(orc):
    """u = 0 accepts exactly when p(d) > 0; the final draw at u* = 0 is the first token with
    nonzero residual mass."""
    V = 8
    t = np.zeros((3, V), dtype=np.float32)
    dl = np.zeros((2, V), dtype=np.float32)
    t[1, 5] = -1e30  # p_1(5) underflows to exactly 0 in fp64
    tok = np.array([2, 5], np.int32)
    u = np.zeros(3, dtype=np.float32)
    r = orc.accept(t, dl, tok, u, [3], _offsets([3]), 1.0)
    assert r.accept_len[0] == 1
    # residual at row 1: p_1 - q_1 > 0 everywhere except token 5 -> first positive is 0
    assert r.next_token[0] == 0
    dl2 = dl.copy()
    dl2[1, :3] = 5.0  # q_1 large on 0..2 -> residual zero there
    r = orc.accept(t, dl2, tok, u, [3], _offsets([3]), 1.0)
    assert r.accept_len[0] == 1 and r.next_token[0] == 3


def pin_sampling_temperature(orc):
    """Softmax at temperature T on logits x equals softmax at T=1 on x/T (exact halving)."""
    rng = np.random.default_rng(25)
    bl = np.array([4, 3, 5], np.int32)
    off = _offsets(bl)
    V = 25
    t = rng.normal(0, 2, (int(off[-1]), V)).astype(np.float32)
    dl = (t[np.concatenate([np.arange(off[s], off[s] + bl[s] - 1) for s in range(3)])]
          + rng.normal(0, 1, (int(off[-1]) - 3, V))).astype(np.float32)
    tok = rng.integers(0, V, int(off[-1]) - 3).astype(np.int32)
    for trial in range(10):
        u = rng.random(int(off[-1]), dtype=np.float32)
        a = orc.accept(t, dl, tok, u, bl, off, 2.0)
        b = orc.accept(t * np.float32(0.5), dl * np.float32(0.5), tok, u, bl, off, 1.0)
        assert (a.accept_len == b.accept_len).all()
        ok = (a.sample_margin > 1e-12)
        assert (a.next_token[ok] == b.next_token[ok]).all()


# Rows with exactly known distributions: logits of 0 and -inf give probabilities that are
# exact binary fractions (1/4, 1/2, 1/8), so every margin, interval edge and band below is
# a hand-computed number, not a re-evaluation of the oracle's formulas.
NEG = np.float32(-np.inf)


def _quarter_row(V=4):
    """Target row with p = 1/4 on tokens 0..3 and 0 elsewhere."""
    t = np.full(V, NEG, dtype=np.float32)
    t[:4] = 0.0
    return t


def _half_row(V=4):
    """Draft row with q = 1/2 on tokens 0 and 1 and 0 elsewhere."""
    d = np.full(V, NEG, dtype=np.float32)
    d[:2] = 0.0
    return d


def pin_accept_margin(orc):
    """The accept near-tie margin is |u - min(1, rho)| at the tested positions only (the
    parity rule's band, exempting positions whose test the rounding could flip).

    p = (1/4,1/4,1/4,1/4), q = (1/2,1/2,0,0) and a draft of token 0 give rho = 1/2 exactly;
    q = 1/8 everywhere with the same p gives rho = 2, whose accept probability min(1, rho)
    is 1.  Expected margins are the hand-computed distances of the chosen fp32 uniforms."""
    t, d = _quarter_row(), _half_row()
    off = _offsets([2])
    tok = np.array([0], np.int32)
    # rho = 1/2, u just above: rejected, margin 2^-15 (outside the 1e-5 band)
    r = orc.accept(np.stack([t, t]), d[None], tok, np.array([0.5 + 2 ** -15, 0.3], np.float32), [2], off, 1.0)
    assert r.accept_len[0] == 0 and r.accept_margin[0] == 2.0 ** -15, (r.accept_len, r.accept_margin)
    # rho = 1/2, u just below: accepted, margin 2^-18 (a near-tie inside the band)
    r = orc.accept(np.stack([t, t]), d[None], tok, np.array([0.5 - 2 ** -18, 0.3], np.float32), [2], off, 1.0)
    assert r.accept_len[0] == 1 and r.accept_margin[0] == 2.0 ** -18, (r.accept_len, r.accept_margin)
    # rho = 2: accept probability 1, margin 1 - u = 2^-17, not |u - rho|
    t8 = _quarter_row(8)
    d8 = np.zeros(8, np.float32)
    r = orc.accept(np.stack([t8, t8]), d8[None], np.array([1], np.int32),
                   np.array([1 - 2 ** -17, 0.3], np.float32), [2], off, 1.0)
    assert r.accept_len[0] == 1 and r.accept_margin[0] == 2.0 ** -17, (r.accept_len, r.accept_margin)
    # three drafts, rho = 1/2 each: position 0 accepted at margin 2^-13, position 1 rejected at
    # margin 0.4 - 0.5 in fp32, position 2 untested (its margin 2^-20 must not count): the margin
    # is the minimum over the tested positions, 2^-13
    u = np.array([0.5 - 2 ** -13, 0.9, 0.5 + 2 ** -20, 0.3], np.float32)
    r = orc.accept(np.stack([t] * 4), np.stack([d] * 3), np.zeros(3, np.int32), u, [4], _offsets([4]), 1.0)
    assert r.accept_len[0] == 1 and r.accept_margin[0] == 2.0 ** -13, (r.accept_len, r.accept_margin)
    # no tested position (B = 1) and greedy acceptance: no accept margin
    r = orc.accept(t[None], np.zeros((1, 4), np.float32), np.zeros(0, np.int32), np.array([0.5], np.float32),
                   [1], _offsets([1]), 1.0)
    assert r.accept_margin[0] == np.inf
    r = orc.accept(np.stack([t, t]), None, tok, None, [2], off, 0.0)
    assert r.accept_margin[0] == np.inf and r.sample_margin[0] == np.inf and r.sample_tie_p[0] == 0.0
    assert r.sample_lo[0] == r.sample_hi[0] == r.next_token[0]


# (u*, token, margin, band low token, band high token) for a final draw from the bonus row
# p = (1/4,1/4,1/4,1/4): interval edges at 0, 1/4, 1/2, 3/4, 1; band 1e-5
_BONUS_CASES = [
    (0.5 + 2 ** -20, 2, 2.0 ** -20, 1, 2),   # just past the edge at 1/2
    (0.5, 2, 0.0, 1, 2),                     # exactly on an edge: the upper token, margin 0
    (0.375, 1, 0.125, 1, 1),                 # mid-interval
    (0.0, 0, 0.0, 0, 0),                     # the bottom edge; the band clamps at 0
    (0.25 - 2 ** -21, 0, 2.0 ** -21, 0, 1),  # just below the edge at 1/4
    (1 - 2 ** -24, 3, 2.0 ** -24, 3, 3),     # top: the band clamps at S, whose draw is the last token
]
# the same for the residual max(0, p - q) = (0, 0, 1/4, 1/4) of q = (1/2,1/2,0,0), S = 1/2:
# edges at 0 (tokens 0 and 1 have no mass), 1/4 and 1/2 of S = relative 0, 1/2, 1
_RESIDUAL_CASES = [
    (0.5 + 2 ** -16, 3, 2.0 ** -16, 3, 3),   # margin 2^-17 absolute is 2^-16 of S; band = 1e-5 S
    (0.5 - 2 ** -18, 2, 2.0 ** -18, 2, 3),
    (0.25, 2, 0.25, 2, 2),
    (0.0, 2, 0.0, 2, 2),                     # the first token with mass, not token 0
]


def pin_sample_margin_band(orc):
    """The final draw's near-tie margin (distance of u* S to the chosen token's interval
    edges, relative to S) and the band of tokens reachable from (u* -/+ 1e-5) S, on
    distributions whose cumulative masses are exact binary fractions."""
    t, d = _quarter_row(), _half_row()
    for ustar, x, m, lo, hi in _BONUS_CASES:
        r = orc.accept(t[None], np.zeros((1, 4), np.float32), np.zeros(0, np.int32), np.array([ustar], np.float32),
                       [1], _offsets([1]), 1.0, band=1e-5)
        got = (int(r.next_token[0]), float(r.sample_margin[0]), int(r.sample_lo[0]), int(r.sample_hi[0]))
        assert got[0] == x and abs(got[1] - m) <= 1e-15 and got[2:] == (lo, hi), ("bonus", ustar, got)
    for ustar, x, m, lo, hi in _RESIDUAL_CASES:
        # draft token 0, u_0 = 0.75 >= rho = 1/2: rejected at position 0, residual draw
        r = orc.accept(np.stack([t, t]), d[None], np.array([0], np.int32), np.array([0.75, ustar], np.float32),
                       [2], _offsets([2]), 1.0, band=1e-5)
        got = (int(r.next_token[0]), float(r.sample_margin[0]), int(r.sample_lo[0]), int(r.sample_hi[0]))
        assert r.accept_len[0] == 0, "draft must be rejected"
        assert got[0] == x and abs(got[1] - m) <= 1e-15 and got[2:] == (lo, hi), ("residual", ustar, got)


def pin_sample_tie_probability(orc):
    """The reported near-tie probability of the final draw: hand values on exact
    distributions (each token of p = 1/4 contributes twice the band; tokens without mass
    nothing; a token narrower than twice the band all of its mass), then the frequency of
    sample_margin < band over many uniform u* on a row with wide and narrow tokens, which
    ties the probability to the margin it predicts."""
    t, d = _quarter_row(), _half_row()
    one = _offsets([1])
    r = orc.accept(t[None], np.zeros((1, 4), np.float32), np.zeros(0, np.int32), np.array([0.3], np.float32),
                   [1], one, 1.0, band=1e-5)
    assert abs(r.sample_tie_p[0] - 8e-5) < 1e-18, r.sample_tie_p
    r = orc.accept(np.stack([t, t]), d[None], np.array([0], np.int32), np.array([0.75, 0.3], np.float32),
                   [2], _offsets([2]), 1.0, band=1e-5)
    assert abs(r.sample_tie_p[0] - 4e-5) < 1e-18, r.sample_tie_p
    # p = (1/2, 1/4, 1/8, 1/16, 1/16) from logits 0, -ln2, -2ln2, ... is not exact in fp32;
    # use -inf padding instead: masses 1/2 and 1/2 over tokens 0, 1 with band 0.3 -> each
    # interval (width 1/2) is narrower than 2 band = 0.6, so the probability is 1
    two = np.full(6, NEG, np.float32)
    two[:2] = 0.0
    r = orc.accept(two[None], np.zeros((1, 6), np.float32), np.zeros(0, np.int32), np.array([0.3], np.float32),
                   [1], one, 1.0, band=0.3)
    assert abs(r.sample_tie_p[0] - 1.0) < 1e-15, r.sample_tie_p
    # frequency check: one token with almost all mass and 40 narrow ones
    rng = np.random.default_rng(29)
    V, N, band = 41, 40_000, 0.01
    row = np.full(V, -4.0, np.float32)
    row[0] = 0.0
    u = rng.random(N, dtype=np.float32)
    r = orc.accept(np.tile(row, (N, 1)), np.zeros((1, V), np.float32), np.zeros(0, np.int32), u,
                   np.ones(N, np.int32), _offsets(np.ones(N, np.int32)), 1.0, band=band)
    p = float(r.sample_tie_p[0])
    assert np.allclose(r.sample_tie_p, p)
    w = _softmax(row)
    assert w[1] < 2 * band < w[0]  # the row has both kinds of interval
    freq = float((r.sample_margin < band).mean())
    se = np.sqrt(p * (1 - p) / N)
    assert abs(freq - p) < 4 * se, (freq, p, se)


def _lossless_trials(orc, N, seed):
    """N independent steps over one fixed block: B=4 (3 drafts), V=16.  Draft tokens are
    drawn from q_j, uniforms iid U[0,1)."""
    rng = np.random.default_rng(seed)
    V, B = 16, 4
    n = B - 1
    t = rng.normal(0, 1.5, (B, V)).astype(np.float32)
    dl = (t[:n] + rng.normal(0, 1.0, (n, V))).astype(np.float32)
    p = np.stack([_softmax(t[i]) for i in range(B)])
    q = np.stack([_softmax(dl[i]) for i in range(n)])
    bl = np.full(N, B, dtype=np.int32)
    off = _offsets(bl)
    T_all = np.tile(t, (N, 1))
    D_all = np.tile(dl, (N, 1))
    tok = np.stack([rng.choice(V, size=N, p=q[j]) for j in range(n)], axis=1).astype(np.int32)
    u = rng.random((N, B), dtype=np.float32)
    r = orc.accept(T_all, D_all, tok.reshape(-1), u.reshape(-1), bl, off, 1.0)
    return p, q, tok, r


def _chi2_pvalue(samples, probs):
    counts = np.bincount(samples, minlength=len(probs))
    exp = probs * len(samples)
    keep = exp > 0
    return scipy.stats.chisquare(counts[keep], exp[keep]).pvalue


def pin_lossless_chi2(orc, N=200_000):
    """Lossless property (Sec. 1; Sec. 3.1): committed tokens are distributed as the target's.
    First committed token ~ p_0; second (given accept_len >= 1) ~ p_1; bonus (given accept_len
    = n) ~ p_n.  Chi-square p-value must exceed 1e-3 (fixed seed)."""
    p, q, tok, r = _lossless_trials(orc, N, seed=26)
    al, nt = r.accept_len, r.next_token
    first = np.where(al >= 1, tok[:, 0], nt)
    assert _chi2_pvalue(first, p[0]) > 1e-3, "first committed token is not ~ p_0"
    m = al >= 1
    second = np.where(al[m] >= 2, tok[m, 1], nt[m])
    assert _chi2_pvalue(second, p[1]) > 1e-3, "second committed token is not ~ p_1"
    m = al == 3
    assert m.sum() > 1000
    assert _chi2_pvalue(nt[m], p[3]) > 1e-3, "bonus token is not ~ p_n"


def pin_expected_accept_len(orc, N=200_000):
    """Prefix-survival identity (App. A.1): E[accept_len] = sum_i prod_{j<=i} alpha_j, where the
    per-position acceptance probability of speculative sampling is alpha_j = sum_x min(p_j, q_j).
    The sample mean must lie within 4 standard errors."""
    p, q, tok, r = _lossless_trials(orc, N, seed=27)
    alpha = np.minimum(p[:3], q).sum(axis=1)
    expect = sum(np.prod(alpha[:i + 1]) for i in range(3))
    al = r.accept_len.astype(np.float64)
    se = al.std() / np.sqrt(N)
    assert abs(al.mean() - expect) < 4 * se, (al.mean(), expect, se)


def pin_geometric_form(orc, N=100_000):
    """Equal positions (same target/draft rows at every position) make the survival factor
    constant: E[accept_len] = rho (1 - rho^n) / (1 - rho) (App. A.2, geometric form)."""
    rng = np.random.default_rng(28)
    V, B = 10, 6
    n = B - 1
    t1 = rng.normal(0, 1, V).astype(np.float32)
    d1 = (t1 + rng.normal(0, 0.8, V)).astype(np.float32)
    p, q = _softmax(t1), _softmax(d1)
    rho = np.minimum(p, q).sum()
    bl = np.full(N, B, np.int32)
    T_all = np.tile(t1, (N * B, 1))
    D_all = np.tile(d1, (N * n, 1))
    tok = rng.choice(V, size=N * n, p=q).astype(np.int32)
    u = rng.random(N * B, dtype=np.float32)
    r = orc.accept(T_all, D_all, tok, u, bl, _offsets(bl), 1.0)
    expect = rho * (1 - rho ** n) / (1 - rho)
    al = r.accept_len.astype(np.float64)
    assert abs(al.mean() - expect) < 4 * al.std() / np.sqrt(N), (al.mean(), expect)


ACCEPT_PINS = [pin_greedy_numpy_prefix, pin_greedy_constructed, pin_greedy_ties_lowest,
               pin_sampling_identical_rows, pin_sampling_residual, pin_sampling_u_zero,
               pin_sampling_temperature, pin_accept_margin, pin_sample_margin_band, pin_sample_tie_probability,
               pin_lossless_chi2, pin_expected_accept_len, pin_geometric_form]

ALL_PINS = ATTN_PINS + ACCEPT_PINS


def run_all(orc, names=None):
    """Run pins, returning {name: None if passed else error text}."""
    out = {}
    for fn in ALL_PINS:
        if names is not None and fn.__name__ not in names:
            continue
        try:
            fn(orc)
            out[fn.__name__] = None
        except Exception as e:  # noqa: BLE001 -- a pin failure of any kind counts
            out[fn.__name__] = f"{type(e).__name__}: {e}"
    return out
