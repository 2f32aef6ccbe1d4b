"""GPU parity of the paged-cache variants: sd_block_attn_paged against the oracle over the
gathered caches (and bit-identical to sd_block_attn on the same keys: same arithmetic, only
the addressing differs), and sd_kv_append_paged bit-exact."""
import numpy as np
import pytest
import torch

import gpu_util as G
import oracle.paged as OPG
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu
CAUSAL, BIDIR = W.MASK_CAUSAL_IN_BLOCK, W.MASK_BIDIR_IN_BLOCK


def _paged_run(p, kp, vp, table):
    dev = G.dev()
    G.log(f"sd_block_attn_paged {p.name} S={p.S} page={kp.shape[2]} pages={kp.shape[0]} mask={p.mask_mode}")
    o = sd.block_attn_paged(p.q.to(dev), kp.to(dev), vp.to(dev), torch.from_numpy(table).to(dev),
                            torch.from_numpy(p.ctx_lens).to(dev), torch.from_numpy(p.block_lens).to(dev),
                            torch.from_numpy(p.q_offsets).to(dev), p.mask_mode, max_ctx=p.max_ctx,
                            max_block=p.max_block)
    torch.cuda.synchronize()
    return o


@pytest.mark.parametrize("page_size,mode", [(16, CAUSAL), (64, CAUSAL), (256, BIDIR), (32, BIDIR)])
def test_paged_attention_parity(page_size, mode):
    rs = W._streams(5201 + page_size)
    p = W.make_attn(rs, S=5, Hq=32, Hkv=8, D=128, ctx_lens=[3000, 17, 0, 1500, 4090], block_lens=[16, 24, 5, 1, 12],
                    dtype="bf16", mask_mode=mode, Lmax=4096 + 256, name=f"paged{page_size}")
    kp, vp, table = W.paginate(rs, p.k_cache, p.v_cache, page_size)
    got = _paged_run(p, kp, vp, table).float().cpu().numpy()
    ref = OPG.block_attn_paged(p.q, kp, vp, table, p.ctx_lens, p.block_lens, p.q_offsets, mode)
    err = np.abs(got - ref).max()
    G.log(f"  max-abs error {err:.3e}")
    assert err <= G.ATTN_TOL["bf16"]


def test_paged_equals_contiguous_bitwise_on_ragged_qwen3_batch():
    """The ragged Qwen3-4B batch with 64-key pages in a shuffled pool: the paged kernel's output
    is bit-identical to the contiguous kernel's."""
    p = W.c3_ragged(temperatures=()).attn
    rs = W._streams(5301)
    Lp = ((p.Lmax + 63) // 64) * 64
    k = torch.nn.functional.pad(p.k_cache, (0, 0, 0, Lp - p.Lmax), value=float("nan"))
    v = torch.nn.functional.pad(p.v_cache, (0, 0, 0, Lp - p.Lmax), value=float("nan"))
    kp, vp, table = W.paginate(rs, k, v, 64)
    got = _paged_run(p, kp, vp, table).cpu()
    ref = G.run_attn(p).cpu()
    assert torch.equal(got, ref)


@pytest.mark.parametrize("page_size", [16, 128])
def test_kv_append_paged_bit_exact(page_size):
    rs = W._streams(5401)
    ctx = np.array([100, 0, 250, 255], np.int32)
    B = np.array([16, 1, 6, 3], np.int32)  # the last sequence's final row lands past the table
    off = W.offsets_from_lens(B)
    k, v = W.step_caches(rs, S=4, Hkv=8, D=128, Lmax=256, ctx_lens=ctx, dtype="bf16")
    kp, vp, table = W.paginate(rs, k, v, page_size)
    blk = W.step_block_inputs(rs, total_q=int(off[-1]), Hq=8, Hkv=8, D=128, dtype="bf16")
    dev = G.dev()
    dkp, dvp = kp.to(dev), vp.to(dev)
    G.log(f"sd_kv_append_paged page={page_size}")
    sd.kv_append_paged(blk["k_new"].to(dev), blk["v_new"].to(dev), dkp, dvp, torch.from_numpy(table).to(dev),
                       torch.from_numpy(ctx).to(dev), torch.from_numpy(off).to(dev))
    torch.cuda.synchronize()
    rk, rv = OPG.kv_append_paged(kp, vp, table, blk["k_new"], blk["v_new"], ctx, off)
    assert np.array_equal(dkp.float().cpu().numpy(), rk, equal_nan=True)
    assert np.array_equal(dvp.float().cpu().numpy(), rv, equal_nan=True)


def test_kv_append_paged_many_sequences():
    """70 sequences: the owner lookup crosses a 64-sequence round, with empty blocks at its edge."""
    rs = W._streams(5402)
    S, Lmax = 70, 48
    ctx = rs["ctx"].integers(0, 40, S).astype(np.int32)
    B = rs["B"].integers(0, 6, S).astype(np.int32)
    B[[62, 63, 64, 69]] = [0, 0, 3, 0]
    off = W.offsets_from_lens(B)
    k, v = W.step_caches(rs, S=S, Hkv=8, D=128, Lmax=Lmax, ctx_lens=ctx, dtype="bf16")
    kp, vp, table = W.paginate(rs, k, v, 16)
    blk = W.step_block_inputs(rs, total_q=int(off[-1]), Hq=8, Hkv=8, D=128, dtype="bf16")
    dev = G.dev()
    dkp, dvp = kp.to(dev), vp.to(dev)
    G.log(f"sd_kv_append_paged S={S} page=16")
    sd.kv_append_paged(blk["k_new"].to(dev), blk["v_new"].to(dev), dkp, dvp, torch.from_numpy(table).to(dev),
                       torch.from_numpy(ctx).to(dev), torch.from_numpy(off).to(dev))
    torch.cuda.synchronize()
    rk, rv = OPG.kv_append_paged(kp, vp, table, blk["k_new"], blk["v_new"], ctx, off)
    assert np.array_equal(dkp.float().cpu().numpy(), rk, equal_nan=True)
    assert np.array_equal(dvp.float().cpu().numpy(), rv, equal_nan=True)


def test_paged_dense_plan_many_sequences():
    """The dense split numbering (more than one wave of splits) through page pools: bit-identical
    to the contiguous kernel on the same keys."""
    from test_gpu_attn import _many_sequences
    p = _many_sequences(7302, 100, CAUSAL, "paged_dense_many_seqs")
    rs = W._streams(7303)
    Lp = ((p.Lmax + 31) // 32) * 32
    k = torch.nn.functional.pad(p.k_cache, (0, 0, 0, Lp - p.Lmax), value=float("nan"))
    v = torch.nn.functional.pad(p.v_cache, (0, 0, 0, Lp - p.Lmax), value=float("nan"))
    kp, vp, table = W.paginate(rs, k, v, 32)
    got = _paged_run(p, kp, vp, table).cpu()
    ref = G.run_attn(p).cpu()
    assert torch.equal(got, ref)


@pytest.mark.parametrize("S,ctx_hi", [(40, 14000), (80, 12000)], ids=["ranked_S40", "seq_order_S80"])
def test_paged_dense_plan_long_splits(S, ctx_hi):
    """Plans at the 4096-key split cap (full splits, then partial splits longest first) through
    page pools of 64 keys: bit-identical to the contiguous kernel on the same keys."""
    from test_gpu_attn import _long_split_sequences
    p = _long_split_sequences(7500 + S, S, ctx_hi, CAUSAL, f"paged_long_splits_S{S}")
    rs = W._streams(7501 + S)
    Lp = ((p.Lmax + 63) // 64) * 64
    k = torch.nn.functional.pad(p.k_cache, (0, 0, 0, Lp - p.Lmax), value=float("nan"))
    v = torch.nn.functional.pad(p.v_cache, (0, 0, 0, Lp - p.Lmax), value=float("nan"))
    kp, vp, table = W.paginate(rs, k, v, 64)
    got = _paged_run(p, kp, vp, table).cpu()
    ref = G.run_attn(p).cpu()
    assert torch.equal(got, ref)
