"""Pins of the step oracle (append, commit, verify step) against what does not depend on it:
attention over explicitly concatenated keys with torch's fp64 scaled_dot_product_attention,
incremental decoding for blocks of one token, and the committed-length closed form."""
import numpy as np
import pytest
import torch

import oracle
import oracle.step as OS
from paper_2606_31315_amd import workloads as W


def _sdpa_rows(q_rows, keys, vals, lims, scale):
    """fp64 SDPA of query rows [n, Hq, D] over keys/values [N, Hkv, D], row r sees keys < lims[r]."""
    n, Hq, D = q_rows.shape
    Hkv = keys.shape[1]
    G = Hq // Hkv
    k = torch.from_numpy(np.repeat(keys, G, axis=1).transpose(1, 0, 2).astype(np.float64))
    v = torch.from_numpy(np.repeat(vals, G, axis=1).transpose(1, 0, 2).astype(np.float64))
    q = torch.from_numpy(q_rows.transpose(1, 0, 2).astype(np.float64))
    mask = torch.from_numpy(np.arange(keys.shape[0])[None, :] < np.asarray(lims)[:, None])
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=scale)
    return o.numpy().transpose(1, 0, 2)


def test_append_then_attention_equals_concatenated_keys():
    """After the append, causal block attention over the cache equals attention over the
    committed keys concatenated with the block's new keys (built with np.concatenate)."""
    rs = W._streams(3101)
    S, Hq, Hkv, D = 3, 8, 2, 64
    ctx = np.array([40, 0, 17], np.int32)
    B = np.array([5, 3, 1], np.int32)
    off = W.offsets_from_lens(B)
    Lmax = 64
    k, v = W.step_caches(rs, S=S, Hkv=Hkv, D=D, Lmax=Lmax, ctx_lens=ctx, dtype="f32")
    blk = W.step_block_inputs(rs, total_q=int(off[-1]), Hq=Hq, Hkv=Hkv, D=D, dtype="f32")
    k2, v2 = OS.kv_append(k, v, blk["k_new"], blk["v_new"], ctx, off)
    got = oracle.block_attn(blk["q"].numpy(), k2, v2, ctx, B, off, W.MASK_CAUSAL_IN_BLOCK)
    for s in range(S):
        keys = np.concatenate([k[s, :, :ctx[s]].numpy().transpose(1, 0, 2), blk["k_new"][off[s]:off[s + 1]].numpy()])
        vals = np.concatenate([v[s, :, :ctx[s]].numpy().transpose(1, 0, 2), blk["v_new"][off[s]:off[s + 1]].numpy()])
        lims = ctx[s] + 1 + np.arange(B[s])
        ref = _sdpa_rows(blk["q"][off[s]:off[s + 1]].numpy(), keys, vals, lims, 1 / np.sqrt(D))
        assert np.abs(got[off[s]:off[s + 1]] - ref).max() < 1e-12


def test_append_touches_only_the_block_rows():
    rs = W._streams(3102)
    ctx = np.array([10, 20], np.int32)
    B = np.array([4, 2], np.int32)
    off = W.offsets_from_lens(B)
    k, v = W.step_caches(rs, S=2, Hkv=2, D=64, Lmax=23, ctx_lens=ctx, dtype="f32")
    blk = W.step_block_inputs(rs, total_q=6, Hq=2, Hkv=2, D=64, dtype="f32")
    k2, _ = OS.kv_append(k, v, blk["k_new"], blk["v_new"], ctx, off)
    k0 = k.numpy()
    assert np.array_equal(k2[0, :, :10], k0[0, :, :10]) and np.isnan(k2[0, :, 14:]).all()
    assert np.array_equal(k2[0, :, 10:14].transpose(1, 0, 2), blk["k_new"][0:4].numpy())
    assert np.array_equal(k2[1, :, 20:22].transpose(1, 0, 2), blk["k_new"][4:6].numpy())
    assert np.isnan(k2[1, :, 22]).all()
    # a row past the capacity is dropped
    k3, _ = OS.kv_append(k, v, blk["k_new"], blk["v_new"], np.array([21, 22], np.int32), off)
    assert np.array_equal(k3[0, :, 21:23].transpose(1, 0, 2), blk["k_new"][0:2].numpy())
    assert np.array_equal(k3[1, :, 22], blk["k_new"][4].numpy())


def test_commit_closed_form():
    assert list(OS.commit([0, 5, 100], [0, 3, 15])) == [1, 9, 116]


def _greedy_step_inputs(rs, B, V, all_accept):
    """Acceptance inputs at T=0 whose drafts are all accepted (drafts = the target argmax) or
    rejected at position 0."""
    p = W.make_accept(rs, block_lens=B, V=V, dtype="f32", temperature=0.0, target_sigma=2.0, noise_sigma=0.0)
    t = p.target.numpy()
    toks = []
    for s in range(len(B)):
        for j in range(int(B[s]) - 1):
            g = int(np.argmax(t[p.q_offsets[s] + j]))
            toks.append(g if all_accept else (g + 1) % V)
    p.draft_tokens = np.array(toks, np.int32)
    return p


@pytest.mark.parametrize("all_accept", [True, False])
def test_committed_length_over_steps(all_accept):
    """Every draft accepted: ctx grows by B_s per step; position 0 rejected: by 1."""
    rs = W._streams(3103)
    S, Hq, Hkv, D, V = 2, 4, 1, 64, 50
    B = np.array([4, 2], np.int32)
    off = W.offsets_from_lens(B)
    ctx = np.array([3, 8], np.int32)
    k, v = W.step_caches(rs, S=S, Hkv=Hkv, D=D, Lmax=40, ctx_lens=ctx, dtype="f32")
    ctx0 = ctx.copy()
    for step in range(3):
        blk = W.step_block_inputs(rs, total_q=int(off[-1]), Hq=Hq, Hkv=Hkv, D=D, dtype="f32")
        acc = _greedy_step_inputs(rs, B, V, all_accept)
        layer = dict(q=blk["q"], k_new=blk["k_new"], v_new=blk["v_new"], k_cache=k, v_cache=v)
        r = OS.verify_step([layer], ctx, B, off, W.MASK_CAUSAL_IN_BLOCK, acc.target, None, acc.draft_tokens,
                           None, 0.0)
        k, v, ctx = r.k_caches[0], r.v_caches[0], r.ctx_lens
        assert np.array_equal(ctx, ctx0 + (step + 1) * (B if all_accept else 1))


def test_single_token_blocks_are_incremental_decoding():
    """Blocks of one token (no drafts): each step's output is ordinary decode attention of the
    new token over every key so far, and the cache holds the appended keys in order."""
    rs = W._streams(3104)
    S, Hq, Hkv, D = 2, 4, 2, 64
    B = np.ones(S, np.int32)
    off = W.offsets_from_lens(B)
    ctx = np.array([6, 0], np.int32)
    k, v = W.step_caches(rs, S=S, Hkv=Hkv, D=D, Lmax=16, ctx_lens=ctx, dtype="f32")
    keys = [list(k[s, :, :ctx[s]].numpy().transpose(1, 0, 2)) for s in range(S)]
    vals = [list(v[s, :, :ctx[s]].numpy().transpose(1, 0, 2)) for s in range(S)]
    for step in range(5):
        blk = W.step_block_inputs(rs, total_q=S, Hq=Hq, Hkv=Hkv, D=D, dtype="f32")
        acc = W.make_accept(rs, block_lens=B, V=7, dtype="f32", temperature=0.0, target_sigma=1.0, noise_sigma=0.0)
        layer = dict(q=blk["q"], k_new=blk["k_new"], v_new=blk["v_new"], k_cache=k, v_cache=v)
        r = OS.verify_step([layer], ctx, B, off, W.MASK_CAUSAL_IN_BLOCK, acc.target, None, acc.draft_tokens,
                           None, 0.0)
        for s in range(S):
            keys[s].append(blk["k_new"][s].numpy())
            vals[s].append(blk["v_new"][s].numpy())
            ref = _sdpa_rows(blk["q"][s:s + 1].numpy(), np.stack(keys[s]), np.stack(vals[s]), [len(keys[s])],
                             1 / np.sqrt(D))
            assert np.abs(r.outs[0][s:s + 1] - ref).max() < 1e-12
        assert (r.accept.accept_len == 0).all()
        k, v, ctx = r.k_caches[0], r.v_caches[0], r.ctx_lens
    for s in range(S):
        assert np.array_equal(k[s, :, :ctx[s]].transpose(1, 0, 2), np.stack(keys[s]))


def test_planted_mistakes_fail_the_pins(monkeypatch):
    """A commit that forgets the anchor, or an append shifted by one row, fails a pin."""
    monkeypatch.setattr(OS, "commit", lambda c, a: (np.asarray(c) + np.asarray(a)).astype(np.int32))
    with pytest.raises(AssertionError):
        test_committed_length_over_steps(True)
    monkeypatch.undo()
    real = OS.kv_append

    def shifted(k, v, kn, vn, ctx, off):
        return real(k, v, kn, vn, np.asarray(ctx) + 1, off)
    monkeypatch.setattr(OS, "kv_append", shifted)
    with pytest.raises((AssertionError, ValueError)):
        test_append_then_attention_equals_concatenated_keys()
