"""Pins of the paged-cache oracle: pages scattered with torch indexing gather back to the
contiguous caches, paged attention equals contiguous attention for any page order, and the
paged append equals the contiguous append seen through the table."""
import numpy as np
import pytest

import oracle
import oracle.paged as OPG
import oracle.step as OS
from paper_2606_31315_amd import workloads as W


@pytest.mark.parametrize("page_size", [16, 64])
def test_gather_inverts_the_scatter(page_size):
    rs = W._streams(5101)
    p = W.make_attn(rs, S=3, Hq=8, Hkv=2, D=64, ctx_lens=[100, 7, 60], block_lens=[5, 9, 3], dtype="f32",
                    mask_mode=W.MASK_CAUSAL_IN_BLOCK, Lmax=128)
    kp, vp, table = W.paginate(rs, p.k_cache, p.v_cache, page_size)
    assert np.array_equal(OPG.gather(kp, table), p.k_cache.numpy(), equal_nan=True)
    assert len(np.unique(table)) == table.size  # every logical page has its own pool page


@pytest.mark.parametrize("mode", [W.MASK_CAUSAL_IN_BLOCK, W.MASK_BIDIR_IN_BLOCK])
def test_paged_attention_is_contiguous_attention(mode):
    rs = W._streams(5102)
    p = W.make_attn(rs, S=3, Hq=8, Hkv=2, D=64, ctx_lens=[100, 0, 60], block_lens=[5, 9, 3], dtype="f32",
                    mask_mode=mode, Lmax=128)
    kp, vp, table = W.paginate(rs, p.k_cache, p.v_cache, 32)
    ref = oracle.block_attn(p.q, p.k_cache, p.v_cache, p.ctx_lens, p.block_lens, p.q_offsets, mode)
    got = OPG.block_attn_paged(p.q, kp, vp, table, p.ctx_lens, p.block_lens, p.q_offsets, mode)
    assert np.array_equal(got, ref)


def test_paged_append_matches_contiguous_append():
    rs = W._streams(5103)
    ctx = np.array([30, 61, 0], np.int32)
    B = np.array([4, 3, 2], np.int32)
    off = W.offsets_from_lens(B)
    k, v = W.step_caches(rs, S=3, Hkv=2, D=64, Lmax=64, ctx_lens=ctx, dtype="f32")
    blk = W.step_block_inputs(rs, total_q=int(off[-1]), Hq=2, Hkv=2, D=64, dtype="f32")
    kp, vp, table = W.paginate(rs, k, v, 16)
    kc, vc = OS.kv_append(k, v, blk["k_new"], blk["v_new"], ctx, off)
    kp2, vp2 = OPG.kv_append_paged(kp, vp, table, blk["k_new"], blk["v_new"], ctx, off)
    assert np.array_equal(OPG.gather(kp2, table), kc, equal_nan=True)
    assert np.array_equal(OPG.gather(vp2, table), vc, equal_nan=True)
    # spare pool pages are untouched
    used = set(table.reshape(-1).tolist())
    spare = [i for i in range(kp.shape[0]) if i not in used]
    assert np.isnan(kp2[spare]).all()
