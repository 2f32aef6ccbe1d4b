"""GPU parity of sd_block_attn_append: the block's keys and values come from the new-row arrays,
not the cache, and the same launch writes them into the cache.

Each case starts from an oracle problem whose caches already hold the block rows at
[ctx_s, ctx_s + B_s), takes those rows out as k_new / v_new [total_q, Hkv, D], and poisons
them in the device caches with NaN.  Then
  - the caches after the call must equal the problem's caches bit for bit (every block row
    written, nothing else touched, NaN tails intact);
  - the output must match the fp64 oracle within the bf16 attention tolerance (a poisoned row
    read from the cache would make it NaN);
  - the output must equal sd_block_attn's on the caches with the rows already in place, bit for
    bit (same splits, same tiles, same arithmetic).
Cases cover a block split across two workgroups (small contexts, B = 64), empty contexts and
blocks, head_dim 64 and 128, both masks, and the multi-wave plan with dense split numbering."""
import zlib

import numpy as np
import pytest
import torch

import gpu_util as G
import oracle
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu

CAUSAL, BIDIR = W.MASK_CAUSAL_IN_BLOCK, W.MASK_BIDIR_IN_BLOCK


def _take_block_rows(p):
    """k_new, v_new [total_q, Hkv, D] from the problem's caches, and device caches with those
    rows poisoned."""
    k_new = torch.empty((p.total_q, p.Hkv, p.D), dtype=p.k_cache.dtype)
    v_new = torch.empty_like(k_new)
    kc, vc = p.k_cache.clone(), p.v_cache.clone()
    for s in range(p.S):
        c, b, o = int(p.ctx_lens[s]), int(p.block_lens[s]), int(p.q_offsets[s])
        if b == 0:
            continue
        k_new[o:o + b] = p.k_cache[s, :, c:c + b].transpose(0, 1)
        v_new[o:o + b] = p.v_cache[s, :, c:c + b].transpose(0, 1)
        kc[s, :, c:c + b] = float("nan")
        vc[s, :, c:c + b] = float("nan")
    return k_new, v_new, kc, vc


def _check(p, with_oracle=True):
    dev = G.dev()
    k_new, v_new, kc, vc = _take_block_rows(p)
    d = G.attn_to_device(p)
    dk, dv = kc.to(dev), vc.to(dev)
    G.log(f"sd_block_attn_append {p.name} S={p.S} Hq={p.Hq} Hkv={p.Hkv} D={p.D} mask={p.mask_mode} "
          f"ctx<={p.max_ctx} B<={p.max_block} total_q={p.total_q}")
    out = sd.block_attn_append(d["q"], k_new.to(dev), v_new.to(dev), dk, dv, d["ctx"], d["bl"], d["off"],
                               p.mask_mode, max_ctx=p.max_ctx, max_block=p.max_block, scale=p.scale)
    torch.cuda.synchronize()
    for got, want in ((dk, p.k_cache), (dv, p.v_cache)):
        assert np.array_equal(got.float().cpu().numpy(), want.float().numpy(), equal_nan=True)
    o = out.float().cpu().numpy().astype(np.float64)
    assert np.isfinite(o).all(), "a poisoned cache row reached the output"
    if with_oracle:
        ref = oracle.block_attn(p.q, p.k_cache, p.v_cache, p.ctx_lens, p.block_lens, p.q_offsets, p.mask_mode,
                                p.scale)
        err = np.abs(o - ref).max() if o.size else 0.0
        G.log(f"  max-abs error {err:.3e}")
        assert err <= G.ATTN_TOL["bf16"]
    two_call = G.run_attn(p, d)
    assert torch.equal(out.view(torch.int16), two_call.view(torch.int16)), "differs from sd_block_attn"


CASES = [
    # name, S, Hq, Hkv, D, ctx, B, mode
    ("straddle_small_ctx", 3, 8, 2, 128, [10, 100, 0], [64, 64, 64], CAUSAL),
    ("straddle_bidir", 3, 8, 2, 128, [10, 100, 0], [64, 64, 64], BIDIR),
    ("straddle_D64", 3, 16, 4, 64, [10, 100, 50], [64, 40, 64], CAUSAL),
    ("ctx0_and_empty_block", 4, 8, 2, 128, [0, 0, 300, 17], [5, 16, 0, 1], CAUSAL),
    ("maxrows_long", 2, 32, 8, 128, [300, 2000], [64, 33], CAUSAL),
    ("mha_G1", 2, 8, 8, 128, [77, 1030], [7, 12], BIDIR),
    ("D64_ragged", 3, 16, 4, 64, [64, 65, 2000], [3, 16, 30], BIDIR),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_append_cases(case):
    name, S, Hq, Hkv, D, ctx, B, mode = case
    rs = W._streams(zlib.crc32(("append_" + name).encode()) % 10000)
    _check(W.make_attn(rs, S=S, Hq=Hq, Hkv=Hkv, D=D, ctx_lens=ctx, block_lens=B, dtype="bf16", mask_mode=mode,
                       name=name))


def test_append_ragged_qwen3_4b():
    """The ragged Qwen3-4B verify batch (8 sequences, ctx 4096, B 8..24, causal)."""
    _check(W.c3_ragged(temperatures=(), dtype="bf16").attn)


@pytest.mark.parametrize("mode", [CAUSAL, BIDIR])
def test_append_dense_plan(mode):
    """100 sequences x 2 kv heads (more than one wave of workgroups: dense split numbering),
    with an empty context and empty blocks."""
    rs = W._streams(7302)
    S = 100
    ctx = rs["ctx"].integers(2000, 5000, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(0, 24, endpoint=True, size=S).astype(np.int32)
    ctx[3] = 0
    B[[0, 63, 64, 65]] = [0, 0, 7, 0]
    B[3] = max(int(B[3]), 1)
    _check(W.make_attn(rs, S=S, Hq=8, Hkv=2, D=128, ctx_lens=ctx, block_lens=B, dtype="bf16", mask_mode=mode,
                       name="append_dense"))


@pytest.mark.parametrize("S,ctx_hi", [(40, 14000), (80, 12000)], ids=["ranked_S40", "seq_order_S80"])
def test_append_dense_plan_long_splits(S, ctx_hi):
    """The fused append on plans at the 4096-key split cap (full splits, then partial splits
    longest first), including a block whose keys straddle two splits."""
    from test_gpu_attn import _long_split_sequences
    _check(_long_split_sequences(7600 + S, S, ctx_hi, BIDIR, f"append_long_splits_S{S}"))
