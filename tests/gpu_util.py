"""Helpers for the GPU parity tests: run a seeded problem through the HIP library (via the
C ABI binding) and through the fp64 oracle, and compare under the stated tolerances.

Tolerances
  attention  max-abs 1e-5 for fp32 inputs; 2e-2 for bf16 inputs (fp32 accumulation).
  greedy acceptance (T = 0): accept_len and next_token bit-exact.
  sampling acceptance (T > 0): a sequence whose tested positions all have
    |u_i - min(1, p_i/q_i)| >= 1e-5 (in the oracle's fp64) must have the same accept_len;
    its next token must equal the oracle's when u* S lies at least 1e-5 S from the
    chosen token's CDF edges, and otherwise lie in the oracle's range of tokens
    reachable from (u* -/+ 1e-5) S.  Sequences with a closer acceptance margin are
    counted, not compared.
  near-tie counts: accept near-ties at most max(1, 5% of S) (each tested position is one
    with probability about 2e-5); final-draw near-ties at most E + 4 sd + 1, where E and
    sd^2 are the sum of the oracle's per-sequence near-tie probabilities p_s and of
    p_s (1 - p_s).  A final draw lands in a token's edge band with probability
    sum_x min(r(x)/S, 2e-5), which is large for flat residuals whose tokens are narrower
    than the band, so a fixed cap would not hold; more near-ties than this bound means
    the band is being used far more often than the distributions allow.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2606_31315_amd as sd
from paper_2606_31315_amd.workloads import AcceptProblem, AttnProblem

ATTN_TOL = {"f32": 1e-5, "bf16": 2e-2}
BAND = 1e-5


def dev():
    return torch.device("cuda:0")


def log(msg: str) -> None:
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def attn_to_device(p: AttnProblem, device=None):
    device = device or dev()
    return dict(q=p.q.to(device), k=p.k_cache.to(device), v=p.v_cache.to(device),
                ctx=torch.from_numpy(p.ctx_lens).to(device), bl=torch.from_numpy(p.block_lens).to(device),
                off=torch.from_numpy(p.q_offsets).to(device))


def run_attn(p: AttnProblem, d=None, workspace=None, out=None) -> torch.Tensor:
    d = d or attn_to_device(p)
    log(f"sd_block_attn {p.name} S={p.S} Hq={p.Hq} Hkv={p.Hkv} D={p.D} dtype={p.dtype} mask={p.mask_mode} "
        f"ctx<={p.max_ctx} B<={p.max_block} total_q={p.total_q}")
    if p.S:  # the per-sequence device values meet the documented ranges
        st = sd.check_attn_inputs(d["ctx"], d["bl"], d["off"], total_q=p.total_q, max_ctx=p.max_ctx,
                                  max_block=p.max_block)
        assert st.cpu().tolist() == [0, -1, 0], st
    o = sd.block_attn(d["q"], d["k"], d["v"], d["ctx"], d["bl"], d["off"], p.mask_mode, max_ctx=p.max_ctx,
                      max_block=p.max_block, scale=p.scale, workspace=workspace, out=out)
    torch.cuda.synchronize()
    return o


def sample_rows(p: AttnProblem, per_seq=6, seed=0):
    """Deterministic sample of (token, head) rows: first/last block row, first/last head, and random ones."""
    rng = np.random.default_rng(seed)
    toks, heads = [], []
    for s in range(p.S):
        B = int(p.block_lens[s])
        if B == 0:
            continue
        base = int(p.q_offsets[s])
        picks = {(0, 0), (B - 1, p.Hq - 1)}
        while len(picks) < min(per_seq, B * p.Hq):
            picks.add((int(rng.integers(B)), int(rng.integers(p.Hq))))
        for i, h in sorted(picks):
            toks.append(base + i)
            heads.append(h)
    return np.array(toks, dtype=np.int64), np.array(heads, dtype=np.int32)


def oracle_attn_rows(p: AttnProblem, toks, heads):
    """Oracle on selected rows, one sequence at a time (slices the cache of that sequence only)."""
    out = np.zeros((len(toks), p.D), dtype=np.float64)
    seq_of = np.searchsorted(p.q_offsets, toks, side="right") - 1
    for s in np.unique(seq_of):
        sel = np.nonzero(seq_of == s)[0]
        b = int(p.block_lens[s])
        base = int(p.q_offsets[s])
        q = p.q[base:base + b]
        res = oracle.block_attn(q, p.k_cache[s:s + 1], p.v_cache[s:s + 1], p.ctx_lens[s:s + 1],
                                p.block_lens[s:s + 1], np.array([0, b], np.int32), p.mask_mode, p.scale,
                                rows=(toks[sel] - base, heads[sel]))
        out[sel] = res
    return out


def check_attn(p: AttnProblem, full=True, per_seq=6, tol=None):
    tol = ATTN_TOL[p.dtype] if tol is None else tol
    got = run_attn(p).float().cpu().numpy().astype(np.float64)
    assert np.isfinite(got).all(), "non-finite attention output"
    if full:
        ref = oracle.block_attn(p.q, p.k_cache, p.v_cache, p.ctx_lens, p.block_lens, p.q_offsets, p.mask_mode,
                                p.scale)
        err = np.abs(got - ref).max() if got.size else 0.0
    else:
        toks, heads = sample_rows(p, per_seq)
        ref = oracle_attn_rows(p, toks, heads)
        err = np.abs(got[toks, heads] - ref).max()
    log(f"  max-abs error {err:.3e} (tol {tol:g})")
    assert err <= tol, f"attention max-abs error {err} > {tol}"
    return err


def accept_to_device(p: AcceptProblem, device=None):
    device = device or dev()
    d = dict(t=p.target.to(device), tok=torch.from_numpy(np.ascontiguousarray(p.draft_tokens)).to(device),
             bl=torch.from_numpy(p.block_lens).to(device), off=torch.from_numpy(p.q_offsets).to(device))
    d["tok"] = d["tok"] if d["tok"].numel() else torch.zeros(1, dtype=torch.int32, device=device)
    if p.temperature > 0:
        d["d"] = p.draft.to(device)
        d["u"] = torch.from_numpy(p.uniforms).to(device)
    else:
        d["d"] = None
        d["u"] = None
    return d


def run_accept(p: AcceptProblem, d=None, workspace=None):
    d = d or accept_to_device(p)
    log(f"sd_accept {p.name} S={p.S} V={p.V} total_q={p.total_q} B<={p.max_block} T={p.temperature} dtype={p.dtype}")
    if p.S:  # the per-sequence device values meet the documented ranges
        st = sd.check_accept_inputs(d["tok"], d["u"], d["bl"], d["off"], p.temperature, vocab=p.V,
                                    total_q=p.total_q, max_block=p.max_block)
        assert st.cpu().tolist() == [0, -1, 0], st
    al, nt = sd.accept(d["t"], d["d"], d["tok"], d["u"], d["bl"], d["off"], p.temperature, max_block=p.max_block,
                       workspace=workspace)
    torch.cuda.synchronize()
    return al.cpu().numpy(), nt.cpu().numpy()


def oracle_accept(p: AcceptProblem):
    return oracle.accept(p.target, p.draft, p.draft_tokens, p.uniforms, p.block_lens, p.q_offsets,
                         p.temperature, band=BAND)


def sample_tie_bound(ref, compared_mask) -> float:
    """Largest admissible count of final-draw near-ties among the compared sequences."""
    # each is a probability: where every interval is narrower than the band the oracle's sum of the
    # masses can round a few ulps above one, which would make the variance term negative
    ps = np.clip(np.asarray(ref.sample_tie_p, dtype=np.float64)[compared_mask], 0.0, 1.0)
    return float(ps.sum() + 4.0 * np.sqrt((ps * (1.0 - ps)).sum()) + 1.0)


def compare_accept(p: AcceptProblem, al, nt, ref, max_tie_frac=0.05):
    """Apply the parity rule; returns (compared, near_tie_accept, near_tie_sample)."""
    if p.temperature == 0:
        bad = np.nonzero((al != ref.accept_len) | (nt != ref.next_token))[0]
        assert len(bad) == 0, (f"greedy mismatch at sequences {bad[:10]}: gpu {al[bad[:5]]},{nt[bad[:5]]} "
                               f"oracle {ref.accept_len[bad[:5]]},{ref.next_token[bad[:5]]}")
        return p.S, 0, 0
    compared = tie_a = tie_s = 0
    for s in range(p.S):
        if ref.accept_margin[s] < BAND:
            tie_a += 1
            continue
        compared += 1
        assert al[s] == ref.accept_len[s], (s, al[s], ref.accept_len[s], ref.accept_margin[s])
        if ref.sample_margin[s] >= BAND:
            assert nt[s] == ref.next_token[s], (s, nt[s], ref.next_token[s], ref.sample_margin[s])
        else:
            tie_s += 1
            assert ref.sample_lo[s] <= nt[s] <= ref.sample_hi[s], (s, nt[s], ref.sample_lo[s], ref.sample_hi[s])
    assert tie_a <= max(1, max_tie_frac * p.S), f"{tie_a} accept near-ties in {p.S} sequences"
    bound = sample_tie_bound(ref, np.asarray(ref.accept_margin) >= BAND)
    assert tie_s <= bound, f"{tie_s} final-draw near-ties, more than the bound {bound:.2f}"
    return compared, tie_a, tie_s


def check_accept(p: AcceptProblem, max_tie_frac=0.05):
    al, nt = run_accept(p)
    ref = oracle_accept(p)
    assert (al >= 0).all() and (nt >= 0).all() and (nt < p.V).all()
    compared, tie_a, tie_s = compare_accept(p, al, nt, ref, max_tie_frac)
    log(f"  compared {compared}/{p.S} sequences, accept near-ties {tie_a}, sample near-ties {tie_s}; "
        f"mean accept_len {al.mean():.3f}")
    assert tie_a <= max(1, max_tie_frac * p.S)
    return al, nt, ref
