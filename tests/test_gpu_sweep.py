"""Seeded random shapes through sd_block_attn and sd_accept, each compared with the fp64 oracle
under the same rules as the named workloads: every output row of the attention, and the
acceptance parity rule.  The shapes mix what the fixed cases test one at a time (empty
contexts and blocks, group sizes 1-8, head dims 64 and 128, both masks, both dtypes, unaligned
vocabularies, one-row blocks, every temperature path), within the documented limits
(1 <= max_block <= 64, group size x max_block <= 256 query rows)."""
import numpy as np
import pytest
import torch

import gpu_util as G
import oracle
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W
from test_gpu_append import _check as append_check

pytestmark = pytest.mark.gpu

N_ATTN = 48
N_WAVES = 16
N_ACCEPT = 48


def attn_shape(i: int) -> dict:
    """Shape of attention case i (seeded; no arithmetic of the method)."""
    r = np.random.default_rng(70000 + i)
    S = int(r.integers(1, 9))
    Hkv = int(r.choice([1, 2, 4, 8]))
    G_ = int(r.choice([1, 2, 4, 8]))
    while G_ * Hkv > 32:  # keeps the oracle's work to seconds
        G_ //= 2
    D = int(r.choice([64, 128]))
    bmax = min(48, 256 // G_)
    B = r.integers(1, bmax + 1, size=S)
    B[r.random(S) < 0.1] = 0  # empty blocks
    if B.max() == 0:
        B[0] = 1
    ctx = r.integers(1, 2501, size=S)
    ctx[r.random(S) < 0.15] = 0  # empty contexts
    dtype = "f32" if r.random() < 0.25 else "bf16"
    mode = W.MASK_BIDIR_IN_BLOCK if r.random() < 0.4 else W.MASK_CAUSAL_IN_BLOCK
    slack = int(r.integers(0, 100))
    return dict(S=S, Hq=G_ * Hkv, Hkv=Hkv, D=D, ctx_lens=ctx.astype(np.int32), block_lens=B.astype(np.int32),
                dtype=dtype, mask_mode=mode, Lmax=int(ctx.max() + B.max()) + slack)  # the host bounds' sum


@pytest.mark.parametrize("i", range(N_ATTN))
def test_attn_random_shape(i):
    sh = attn_shape(i)
    rs = W._streams(80000 + i)
    p = W.make_attn(rs, name=f"sweep{i}", **sh)
    G.log(f"  case {i}: ctx {sh['ctx_lens'].tolist()} B {sh['block_lens'].tolist()} Lmax {sh['Lmax']}")
    G.check_attn(p)


def waves_shape(i: int) -> dict:
    """Attention case i of many (sequence, kv head) pairs with long, ragged contexts: plans of more
    than one wave of even splits, which the bf16 calls serve with balanced shares and the fp32
    calls with densely numbered splits (seeded; no arithmetic of the method)."""
    r = np.random.default_rng(75000 + i)
    S = int(r.integers(16, 49))
    Hkv = int(r.choice([4, 8]))
    G_ = int(r.choice([1, 2, 4]))
    D = int(r.choice([64, 128]))
    B = r.integers(1, 33, size=S)
    B[r.random(S) < 0.05] = 0
    if B.max() == 0:
        B[0] = 1
    ctx_hi = min(7000, 50_000_000 // (S * Hkv * D) - 40)  # K and V caches of about 10^8 elements
    ctx = r.integers(0, ctx_hi + 1, size=S)
    dtype = "f32" if r.random() < 0.25 else "bf16"
    mode = W.MASK_BIDIR_IN_BLOCK if r.random() < 0.4 else W.MASK_CAUSAL_IN_BLOCK
    return dict(S=S, Hq=G_ * Hkv, Hkv=Hkv, D=D, ctx_lens=ctx.astype(np.int32), block_lens=B.astype(np.int32),
                dtype=dtype, mask_mode=mode, Lmax=int(ctx.max() + B.max()))


@pytest.mark.parametrize("i", range(N_WAVES))
def test_attn_random_multiwave(i):
    """Sampled rows of every sequence (the oracle computes them one by one)."""
    sh = waves_shape(i)
    rs = W._streams(85000 + i)
    p = W.make_attn(rs, name=f"waves{i}", **sh)
    G.log(f"  case {i}: S {sh['S']} ctx <= {int(sh['ctx_lens'].max())} B <= {int(sh['block_lens'].max())}")
    G.check_attn(p, full=False, per_seq=6)


def accept_shape(i: int) -> dict:
    """Shape of acceptance case i (seeded; no arithmetic of the method)."""
    r = np.random.default_rng(90000 + i)
    small = r.random() < 0.4
    V = int(r.integers(1, 5000)) if small else int(r.integers(5000, 200001))
    rows_budget = 40_000_000 // V  # target + draft rows the oracle reads in about a second
    S = int(r.integers(1, 25))
    bmax = int(max(1, min(64, rows_budget // (2 * S))))
    B = r.integers(1, bmax + 1, size=S)
    B[r.random(S) < 0.15] = 1  # no drafted token: the bonus draw only
    T = float(r.choice([0.0, 0.7, 1.0, 1.5]))
    dtype = "f32" if r.random() < 0.3 else "bf16"
    return dict(block_lens=B.astype(np.int32), V=V, dtype=dtype, temperature=T,
                target_sigma=float(r.choice([1.0, 3.0])), noise_sigma=float(r.choice([0.3, 1.0])))


@pytest.mark.parametrize("i", range(N_ACCEPT))
def test_accept_random_shape(i):
    sh = accept_shape(i)
    rs = W._streams(95000 + i)
    p = W.make_accept(rs, name=f"sweep{i}", **sh)
    G.log(f"  case {i}: B {sh['block_lens'].tolist()}")
    G.check_accept(p)


# ---- the paged and fused-append variants on random shapes (bf16, as those calls require) ----
N_VARIANTS = 16


def _bf16(sh: dict) -> dict:
    return dict(sh, dtype="bf16")


def _pad_caches(p, page_size):
    """The problem's caches padded with NaN keys to a whole number of pages."""
    Lp = ((p.Lmax + page_size - 1) // page_size) * page_size
    k = torch.nn.functional.pad(p.k_cache, (0, 0, 0, Lp - p.Lmax), value=float("nan"))
    v = torch.nn.functional.pad(p.v_cache, (0, 0, 0, Lp - p.Lmax), value=float("nan"))
    return k, v


def _paged_against_contiguous(p, rs, page_size, with_oracle):
    """sd_block_attn_paged over a shuffled page pool: bit-identical to sd_block_attn on the same
    keys, and (with_oracle) within the bf16 tolerance of the oracle row by row."""
    k, v = _pad_caches(p, page_size)
    kp, vp, table = W.paginate(rs, k, v, page_size)
    dev = G.dev()
    G.log(f"sd_block_attn_paged {p.name} S={p.S} page={page_size} pages={kp.shape[0]} mask={p.mask_mode}")
    got = sd.block_attn_paged(p.q.to(dev), kp.to(dev), vp.to(dev), torch.from_numpy(table).to(dev),
                              torch.from_numpy(p.ctx_lens).to(dev), torch.from_numpy(p.block_lens).to(dev),
                              torch.from_numpy(p.q_offsets).to(dev), p.mask_mode, max_ctx=p.max_ctx,
                              max_block=p.max_block)
    torch.cuda.synchronize()
    d = G.attn_to_device(p)
    d["k"], d["v"] = k.to(dev), v.to(dev)
    ref = G.run_attn(p, d)
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), "paged output differs from contiguous"
    if with_oracle:
        o = got.float().cpu().numpy().astype(np.float64)
        want = oracle.block_attn(p.q, p.k_cache, p.v_cache, p.ctx_lens, p.block_lens, p.q_offsets, p.mask_mode,
                                 p.scale)
        err = np.abs(o - want).max() if o.size else 0.0
        G.log(f"  max-abs error {err:.3e}")
        assert err <= G.ATTN_TOL["bf16"]


@pytest.mark.parametrize("i", range(N_VARIANTS))
def test_paged_random_shape(i):
    sh = _bf16(attn_shape(200 + i))
    rs = W._streams(81000 + i)
    p = W.make_attn(rs, name=f"paged_sweep{i}", **sh)
    page_size = int(np.random.default_rng(71000 + i).choice([16, 32, 64, 128, 256, 1024]))
    _paged_against_contiguous(p, rs, page_size, with_oracle=True)


@pytest.mark.parametrize("i", range(4))
def test_paged_random_multiwave(i):
    sh = _bf16(waves_shape(100 + i))
    rs = W._streams(86000 + i)
    p = W.make_attn(rs, name=f"paged_waves{i}", **sh)
    page_size = int(np.random.default_rng(76000 + i).choice([16, 64, 256]))
    _paged_against_contiguous(p, rs, page_size, with_oracle=False)


@pytest.mark.parametrize("i", range(N_VARIANTS))
def test_append_random_shape(i):
    """sd_block_attn_append: caches bit-exact, output within tolerance of the oracle and
    bit-identical to sd_block_attn (the fused-append checks of the named cases)."""
    sh = _bf16(attn_shape(300 + i))
    rs = W._streams(82000 + i)
    p = W.make_attn(rs, name=f"append_sweep{i}", **sh)
    append_check(p)


@pytest.mark.parametrize("i", range(4))
def test_append_random_multiwave(i):
    sh = _bf16(waves_shape(200 + i))
    rs = W._streams(87000 + i)
    p = W.make_attn(rs, name=f"append_waves{i}", **sh)
    append_check(p, with_oracle=False)


N_EXTREME = 12


@pytest.mark.parametrize("i", range(N_EXTREME))
def test_accept_extreme_temperature(i):
    """Very low and very high temperatures: near-one-hot and near-flat distributions (exp2
    arguments far below zero, and sums over almost the whole vocabulary)."""
    r = np.random.default_rng(99000 + i)
    sh = accept_shape(300 + i)
    sh["temperature"] = float(r.choice([0.02, 0.1, 4.0, 20.0]))
    rs = W._streams(96000 + i)
    p = W.make_accept(rs, name=f"extreme{i}", **sh)
    G.log(f"  case {i}: T {sh['temperature']} V {sh['V']} B {sh['block_lens'].tolist()}")
    G.check_accept(p)
