"""GPU parity of sd_block_attn against the fp64 oracle on the same seeded inputs."""
import zlib

import numpy as np
import pytest
import torch

import gpu_util as G
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu

CAUSAL, BIDIR = W.MASK_CAUSAL_IN_BLOCK, W.MASK_BIDIR_IN_BLOCK


def test_tiny_fp32():
    """Tiny CPU-checkable step: 4 q heads / 1 kv head, D=64, fp32, ctx 256, B=8, causal."""
    G.check_attn(W.c1_tiny().attn)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_qwen3_4b_verify(dtype):
    """Qwen3-4B verify step (32/8/128, ctx 2048, B=16, causal); fp32 inputs pin the mask at 1e-5."""
    G.check_attn(W.c2_qwen3_4b_verify(temperatures=(), dtype=dtype).attn)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ragged_blocks(dtype):
    """8 sequences, ctx 4096, ragged B in {8..24}, causal; every output row compared."""
    G.check_attn(W.c3_ragged(temperatures=(), dtype=dtype).attn)


def test_drafter_bidirectional():
    """16 sequences, ctx U{1024..8192}, B U{8..32}, bidirectional-in-block; every row compared."""
    G.check_attn(W.c4_drafter().attn)


@pytest.fixture(scope="module")
def long_context_run():
    """The long-context batch (32 sequences, ctx U{8192..32768}, B U{4..32}) through the GPU once."""
    p = W.c5_long_context(with_accept=False).attn
    got = G.run_attn(p).float().cpu().numpy().astype(np.float64)
    return p, got


def test_long_context_sampled_rows(long_context_run):
    """Sampled rows of every sequence of the long-context batch against the oracle."""
    p, got = long_context_run
    assert np.isfinite(got).all()
    toks, heads = G.sample_rows(p, per_seq=8)
    err = np.abs(got[toks, heads] - G.oracle_attn_rows(p, toks, heads)).max()
    G.log(f"  sampled rows: max-abs error {err:.3e}")
    assert err <= G.ATTN_TOL[p.dtype]


def test_long_context_longest_sequences_every_row(long_context_run):
    """Every output row (all block rows x all 32 query heads) of the four longest sequences of
    the long-context batch: the splits at the 4096-key cap, full splits first then the
    partial ones, compared row by row."""
    p, got = long_context_run
    longest = np.argsort(-(p.ctx_lens.astype(np.int64) + p.block_lens))[:4]
    toks, heads = [], []
    for s in longest:
        base, b = int(p.q_offsets[s]), int(p.block_lens[s])
        for i in range(b):
            for h in range(p.Hq):
                toks.append(base + i)
                heads.append(h)
    toks, heads = np.array(toks, np.int64), np.array(heads, np.int32)
    G.log(f"  sequences {longest.tolist()} (ctx {p.ctx_lens[longest].tolist()}, B {p.block_lens[longest].tolist()}): "
          f"{len(toks)} rows")
    err = np.abs(got[toks, heads] - G.oracle_attn_rows(p, toks, heads)).max()
    G.log(f"  every row of the longest sequences: max-abs error {err:.3e}")
    assert err <= G.ATTN_TOL[p.dtype]


@pytest.mark.parametrize("mode", [CAUSAL, BIDIR])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_block_dominant_mask_sensitivity(mode, dtype):
    """In-block keys scaled so in-block scores dominate: an off-by-one in the in-block mask
    moves the output by far more than the tolerance."""
    rs = W._streams(77)
    p = W.make_attn(rs, S=4, Hq=32, Hkv=8, D=128, ctx_lens=[2048, 700, 0, 1500], block_lens=[16, 9, 24, 1],
                    dtype=dtype, mask_mode=mode, block_key_gain=6.0, value_gain=0.25, name="block_dominant")
    G.check_attn(p)


EDGE = [
    # name, S, Hq, Hkv, D, ctx, B, dtype, mode
    ("ctx0", 2, 8, 2, 128, [0, 0], [5, 16], "bf16", CAUSAL),
    ("ctx0_bidir", 2, 8, 2, 128, [0, 3], [5, 16], "bf16", BIDIR),
    ("B1_decode", 3, 32, 8, 128, [100, 4095, 1], [1, 1, 1], "bf16", CAUSAL),
    ("B64_maxrows", 2, 32, 8, 128, [300, 2000], [64, 33], "bf16", CAUSAL),
    ("B64_fp32", 1, 16, 4, 128, [129], [64], "f32", CAUSAL),
    ("mha_G1", 2, 8, 8, 128, [77, 1030], [7, 12], "bf16", CAUSAL),
    ("G8", 2, 32, 4, 128, [500, 1900], [16, 32], "bf16", BIDIR),
    ("D64_bf16", 3, 16, 4, 64, [64, 65, 2000], [3, 16, 30], "bf16", CAUSAL),
    ("D64_fp32", 3, 16, 4, 64, [64, 65, 2000], [3, 16, 30], "f32", BIDIR),
    ("empty_block", 3, 8, 2, 128, [40, 50, 60], [4, 0, 6], "bf16", CAUSAL),
    ("ragged_tail_fp32", 2, 8, 2, 128, [63, 1000], [1, 17], "f32", CAUSAL),
    ("long_fp32", 1, 8, 2, 128, [9000], [12], "f32", CAUSAL),
]


@pytest.mark.parametrize("case", EDGE, ids=[c[0] for c in EDGE])
def test_edge_cases(case):
    name, S, Hq, Hkv, D, ctx, B, dtype, mode = case
    rs = W._streams(zlib.crc32(name.encode()) % 10000)
    p = W.make_attn(rs, S=S, Hq=Hq, Hkv=Hkv, D=D, ctx_lens=ctx, block_lens=B, dtype=dtype, mask_mode=mode,
                    name=name)
    G.check_attn(p)


def test_explicit_scale():
    rs = W._streams(91)
    p = W.make_attn(rs, S=2, Hq=8, Hkv=2, D=128, ctx_lens=[300, 20], block_lens=[8, 3], dtype="f32",
                    mask_mode=CAUSAL, name="scale")
    p.scale = 0.05
    G.check_attn(p)


def test_repeated_calls_reuse_workspace():
    """The merge counters return to zero after every call: a second call with the same workspace
    and a smaller batch gives the oracle's answer again, and the first call's outputs reproduce bit-exactly."""
    big = W.c3_ragged(temperatures=(), dtype="bf16").attn
    d = G.attn_to_device(big)
    import paper_2606_31315_amd as sd
    ws = torch.zeros(sd.attn_workspace_size(sd.attn_shape(d["q"], d["k"], big.max_ctx, big.max_block)),
                     dtype=torch.uint8, device=G.dev())
    o1 = G.run_attn(big, d, workspace=ws).clone()
    rs = W._streams(5)
    small = W.make_attn(rs, S=3, Hq=32, Hkv=8, D=128, ctx_lens=[3000, 10, 2500], block_lens=[5, 9, 20],
                        dtype="bf16", mask_mode=CAUSAL, name="small_after_big")
    o_small = G.run_attn(small, workspace=ws).float().cpu().numpy()
    import oracle
    ref = oracle.block_attn(small.q, small.k_cache, small.v_cache, small.ctx_lens, small.block_lens,
                            small.q_offsets, small.mask_mode)
    assert np.abs(o_small - ref).max() < 2e-2
    o2 = G.run_attn(big, d, workspace=ws)
    assert torch.equal(o1, o2)


def test_alternating_calls_arbitrary_workspace():
    """A workspace filled with arbitrary bytes, then shared by calls of different shapes in
    turn, gives the oracle's answer on every call and bit-identical outputs for repeated
    inputs (nothing is carried between calls through the workspace)."""
    import oracle
    import paper_2606_31315_amd as sd
    rs = W._streams(606)
    pa = W.make_attn(rs, S=4, Hq=32, Hkv=8, D=128, ctx_lens=[4000, 1500, 2600, 3333], block_lens=[24, 8, 13, 16],
                     dtype="bf16", mask_mode=CAUSAL, name="alt_a")
    pb = W.make_attn(rs, S=2, Hq=16, Hkv=4, D=128, ctx_lens=[5000, 700], block_lens=[32, 5], dtype="f32",
                     mask_mode=BIDIR, name="alt_b")
    da, db = G.attn_to_device(pa), G.attn_to_device(pb)
    n = max(sd.attn_workspace_size(sd.attn_shape(da["q"], da["k"], pa.max_ctx, pa.max_block)),
            sd.attn_workspace_size(sd.attn_shape(db["q"], db["k"], pb.max_ctx, pb.max_block)))
    ws = torch.randint(0, 256, (n,), dtype=torch.uint8, device=G.dev())
    refs = {}
    for p in (pa, pb):
        refs[p.name] = oracle.block_attn(p.q, p.k_cache, p.v_cache, p.ctx_lens, p.block_lens, p.q_offsets,
                                         p.mask_mode)
    first = {}
    for it in range(6):
        p, d = (pa, da) if it % 2 == 0 else (pb, db)
        o = G.run_attn(p, d, workspace=ws).float().cpu()
        err = np.abs(o.numpy().astype(np.float64) - refs[p.name]).max()
        assert err <= G.ATTN_TOL[p.dtype], (it, p.name, err)
        if p.name in first:
            assert torch.equal(first[p.name], o), (it, p.name)
        else:
            first[p.name] = o


def _many_sequences(seed, S, mode, name):
    """S sequences with ragged contexts (one empty context, some empty blocks)."""
    rs = W._streams(seed)
    ctx = rs["ctx"].integers(2000, 5000, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(0, 24, endpoint=True, size=S).astype(np.int32)
    ctx[3] = 0
    B[[0, 63, 64, 65]] = [0, 0, 7, 0]
    B[3] = max(int(B[3]), 1)
    return W.make_attn(rs, S=S, Hq=8, Hkv=2, D=128, ctx_lens=ctx, block_lens=B, dtype="bf16", mask_mode=mode,
                       name=name)


@pytest.mark.parametrize("mode", [CAUSAL, BIDIR])
def test_dense_plan_many_sequences(mode):
    """100 sequences x 2 kv heads with contexts 2k-5k: the grid is more than one wave, so the
    device numbers the existing splits densely (a prefix sum over 64 sequences per round, two
    rounds here), with empty blocks at the round's edge; every output row compared."""
    G.check_attn(_many_sequences(7301, 100, mode, "dense_many_seqs"))


def _long_split_sequences(seed, S, ctx_hi, mode, name):
    """S sequences x 4 kv heads whose plan reaches the 4096-key split cap (dense numbering of
    full splits, then the partial last splits longest first): lengths that are exact multiples
    of the split, one key past one, empty blocks and an empty context."""
    rs = W._streams(seed)
    ctx = rs["ctx"].integers(1, ctx_hi, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(1, 24, endpoint=True, size=S).astype(np.int32)
    B[[1, S - 2]] = 0
    ctx[2], B[2] = 8192 - 16, 16      # two full splits, no partial
    ctx[5], B[5] = 4096, 1            # one full split and a one-key partial
    ctx[7], B[7] = 0, 5               # no context
    ctx[9], B[9] = ctx_hi - 24, 24    # the longest sequence
    return W.make_attn(rs, S=S, Hq=8, Hkv=4, D=128, ctx_lens=ctx, block_lens=B, dtype="bf16", mask_mode=mode,
                       name=name)


@pytest.mark.parametrize("S,ctx_hi", [(40, 14000), (80, 12000)], ids=["ranked_S40", "seq_order_S80"])
@pytest.mark.parametrize("mode", [CAUSAL, BIDIR])
def test_dense_plan_long_splits(S, ctx_hi, mode):
    """Plans at the split cap: up to 64 sequences the partial splits are ranked by length on
    the device, beyond that they follow sequence order; every output row compared."""
    G.check_attn(_long_split_sequences(7400 + S, S, ctx_hi, mode, f"long_splits_S{S}"))


# ---- balanced shares: bf16 plans of more than one wave give every workgroup the same weighted
# number of key tiles, cut where a share crosses from one (sequence, kv head) pair to the next ----

def _attn_with_bounds(p, max_ctx, max_block):
    """sd_block_attn with host bounds at or above the actual lengths (they set the plan); every
    output row against the oracle."""
    import paper_2606_31315_amd as sd
    d = G.attn_to_device(p)
    G.log(f"sd_block_attn {p.name} S={p.S} Hq={p.Hq} Hkv={p.Hkv} D={p.D} host bounds ctx<={max_ctx} B<={max_block}")
    o = sd.block_attn(d["q"], d["k"], d["v"], d["ctx"], d["bl"], d["off"], p.mask_mode, max_ctx=max_ctx,
                      max_block=max_block)
    torch.cuda.synchronize()
    got = o.float().cpu().numpy().astype(np.float64)
    ref = G.oracle.block_attn(p.q, p.k_cache, p.v_cache, p.ctx_lens, p.block_lens, p.q_offsets, p.mask_mode, p.scale)
    err = np.abs(got - ref).max()
    G.log(f"  max-abs error {err:.3e}")
    assert np.isfinite(got).all() and err <= G.ATTN_TOL["bf16"], err


@pytest.mark.parametrize("mode", [CAUSAL, BIDIR])
def test_balanced_short_lengths_under_long_bound(mode):
    """Host bound 4096 keys, actual contexts 0-300 (some blocks empty): the shares shrink to
    their 16-tile minimum, so most workgroups of the grid have nothing to do; D = 64. Cache rows
    past each sequence's length hold NaN, so a tile read past a piece's end would show."""
    rs = W._streams(7501)
    S = 40
    ctx = rs["ctx"].integers(0, 300, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(0, 12, endpoint=True, size=S).astype(np.int32)
    B[[0, 17]] = 0
    B[5] = 12
    p = W.make_attn(rs, S=S, Hq=8, Hkv=4, D=64, ctx_lens=ctx, block_lens=B, dtype="bf16", mask_mode=mode,
                    Lmax=4096 + 12, name="bal_short_under_long_bound")
    _attn_with_bounds(p, 4096, 12)


@pytest.mark.parametrize("mode", [CAUSAL, BIDIR])
def test_balanced_one_long_pair_over_many_shares(mode):
    """One 30000-key sequence among short ones (50-600 keys): its pair is cut into some thirty
    pieces on consecutive workgroups, merged in several batches; short pairs share workgroups."""
    rs = W._streams(7502)
    S = 20
    ctx = rs["ctx"].integers(50, 600, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(1, 16, endpoint=True, size=S).astype(np.int32)
    ctx[6], B[6] = 30000, 16
    p = W.make_attn(rs, S=S, Hq=4, Hkv=1, D=64, ctx_lens=ctx, block_lens=B, dtype="bf16", mask_mode=mode,
                    name="bal_one_long_pair")
    _attn_with_bounds(p, p.max_ctx, p.max_block)


@pytest.mark.parametrize("mode", [CAUSAL, BIDIR])
def test_balanced_two_mtiles_per_wavefront(mode):
    """Eight query heads per kv head and blocks up to 24 rows (up to 12 m-tiles: two per
    wavefront) under the balanced plan, 48 sequences with contexts 2500-5000."""
    rs = W._streams(7503)
    S = 48
    ctx = rs["ctx"].integers(2500, 5000, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(1, 24, endpoint=True, size=S).astype(np.int32)
    B[3] = 24
    p = W.make_attn(rs, S=S, Hq=16, Hkv=2, D=64, ctx_lens=ctx, block_lens=B, dtype="bf16", mask_mode=mode,
                    name="bal_two_mtiles")
    _attn_with_bounds(p, p.max_ctx, p.max_block)
