"""GPU parity of the step around verification: sd_kv_append and sd_commit bit-exact against
the oracle, and sd_verify_step over several steps (every layer's attention, acceptance,
commit and caches) against the oracle run on the same inputs."""
import numpy as np
import pytest
import torch

import gpu_util as G
import oracle.step as OS
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu


def _same(t: torch.Tensor, x: np.ndarray) -> bool:
    """Bit-exact equality of a device cache with the oracle's (bf16 and fp32 widen exactly to
    fp32); NaN rows (never written) compare equal whatever their payload."""
    return np.array_equal(t.detach().float().cpu().numpy(), np.asarray(x, dtype=np.float32), equal_nan=True)


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("f32", 128), ("bf16", 64)])
def test_kv_append_bit_exact(dtype, D):
    rs = W._streams(4101)
    S, Hkv = 5, 8
    ctx = np.array([100, 0, 4000, 7, 2047], np.int32)
    B = np.array([16, 1, 24, 0, 9], np.int32)
    off = W.offsets_from_lens(B)
    Lmax = 4100
    k, v = W.step_caches(rs, S=S, Hkv=Hkv, D=D, Lmax=Lmax, ctx_lens=ctx, dtype=dtype)
    blk = W.step_block_inputs(rs, total_q=int(off[-1]), Hq=Hkv, Hkv=Hkv, D=D, dtype=dtype)
    dk, dv = k.to(G.dev()), v.to(G.dev())
    G.log(f"sd_kv_append S={S} Hkv={Hkv} D={D} dtype={dtype} total_q={int(off[-1])}")
    sd.kv_append(blk["k_new"].to(G.dev()), blk["v_new"].to(G.dev()), dk, dv, torch.from_numpy(ctx).to(G.dev()),
                 torch.from_numpy(off).to(G.dev()))
    torch.cuda.synchronize()
    rk, rv = OS.kv_append(k, v, blk["k_new"], blk["v_new"], ctx, off)
    assert _same(dk, rk)
    assert _same(dv, rv)


def test_kv_append_many_sequences_and_wide_rows():
    """150 sequences (the owner lookup takes 64 sequences per round), empty blocks on both
    sides of each round's edge, and rows of 32 heads x 128 fp32 (more 16-byte vectors per
    row than threads in the copying workgroup)."""
    rs = W._streams(4103)
    S, Hkv, D, Lmax = 150, 32, 128, 48
    ctx = rs["ctx"].integers(0, 40, S).astype(np.int32)
    B = rs["B"].integers(0, 6, S).astype(np.int32)
    B[[0, 62, 63, 64, 65, 127, 128, 149]] = [3, 0, 0, 0, 2, 0, 4, 0]
    off = W.offsets_from_lens(B)
    k, v = W.step_caches(rs, S=S, Hkv=Hkv, D=D, Lmax=Lmax, ctx_lens=ctx, dtype="f32")
    blk = W.step_block_inputs(rs, total_q=int(off[-1]), Hq=Hkv, Hkv=Hkv, D=D, dtype="f32")
    dk, dv = k.to(G.dev()), v.to(G.dev())
    G.log(f"sd_kv_append S={S} Hkv={Hkv} D={D} f32 total_q={int(off[-1])}")
    sd.kv_append(blk["k_new"].to(G.dev()), blk["v_new"].to(G.dev()), dk, dv, torch.from_numpy(ctx).to(G.dev()),
                 torch.from_numpy(off).to(G.dev()))
    torch.cuda.synchronize()
    rk, rv = OS.kv_append(k, v, blk["k_new"], blk["v_new"], ctx, off)
    assert _same(dk, rk)
    assert _same(dv, rv)


def test_kv_append_skips_rows_past_capacity():
    rs = W._streams(4102)
    ctx = np.array([30, 31], np.int32)
    B = np.array([4, 3], np.int32)
    off = W.offsets_from_lens(B)
    k, v = W.step_caches(rs, S=2, Hkv=2, D=64, Lmax=32, ctx_lens=[30, 31], dtype="bf16")
    blk = W.step_block_inputs(rs, total_q=7, Hq=2, Hkv=2, D=64, dtype="bf16")
    dk, dv = k.to(G.dev()), v.to(G.dev())
    G.log("sd_kv_append rows past Lmax")
    sd.kv_append(blk["k_new"].to(G.dev()), blk["v_new"].to(G.dev()), dk, dv, torch.from_numpy(ctx).to(G.dev()),
                 torch.from_numpy(off).to(G.dev()))
    torch.cuda.synchronize()
    rk, _ = OS.kv_append(k, v, blk["k_new"], blk["v_new"], ctx, off)
    assert _same(dk, rk)


def test_commit_exact():
    ctx = torch.tensor([0, 5, 4000, 7], dtype=torch.int32, device=G.dev())
    al = torch.tensor([0, 3, 23, 1], dtype=torch.int32, device=G.dev())
    G.log("sd_commit")
    sd.commit(al, ctx)
    torch.cuda.synchronize()
    assert ctx.cpu().tolist() == list(OS.commit([0, 5, 4000, 7], [0, 3, 23, 1]))


def _run_steps(T, steps, seed, layers=2, dtype="bf16", shape=None, mask=W.MASK_CAUSAL_IN_BLOCK):
    """`steps` verify steps of `layers` layers, each checked against the oracle's step; `shape`
    (Hq, Hkv, D, V, block_lens, ctx_lens) replaces the default four-sequence batch."""
    rs = W._streams(seed)
    sh = shape or dict(Hq=32, Hkv=8, D=128, V=32000, block_lens=[12, 16, 5, 24], ctx_lens=[1500, 3000, 40, 2200])
    Hq, Hkv, D, V = sh["Hq"], sh["Hkv"], sh["D"], sh["V"]
    B = np.asarray(sh["block_lens"], np.int32)
    S = len(B)
    off = W.offsets_from_lens(B)
    ctx = np.asarray(sh["ctx_lens"], np.int32)
    Lmax = int(ctx.max() + steps * B.max())
    caches = [W.step_caches(rs, S=S, Hkv=Hkv, D=D, Lmax=Lmax, ctx_lens=ctx, dtype=dtype) for _ in range(layers)]
    dev = G.dev()
    dcaches = [(k.to(dev), v.to(dev)) for k, v in caches]
    d_ctx = torch.from_numpy(ctx).to(dev)
    d_bl, d_off = torch.from_numpy(B).to(dev), torch.from_numpy(off).to(dev)
    max_ctx = int(ctx.max())
    for step in range(steps):
        blks = [W.step_block_inputs(rs, total_q=int(off[-1]), Hq=Hq, Hkv=Hkv, D=D, dtype=dtype)
                for _ in range(layers)]
        acc = W.make_accept(rs, block_lens=B, V=V, dtype=dtype, temperature=T, target_sigma=3.0, noise_sigma=0.7)
        dl = []
        for (dk, dv), b in zip(dcaches, blks):
            dl.append(dict(q=b["q"].to(dev), k_new=b["k_new"].to(dev), v_new=b["v_new"].to(dev), k_cache=dk,
                           v_cache=dv, out=torch.empty_like(b["q"], device=dev)))
        da = G.accept_to_device(acc)
        G.log(f"sd_verify_step step {step} T={T} layers={layers} max_ctx={max_ctx}")
        al, nt = sd.verify_step(dl, d_ctx, d_bl, d_off, mask, da["t"], da["d"], da["tok"], da["u"],
                                T, max_ctx=max_ctx, max_block=int(B.max()))
        torch.cuda.synchronize()
        ol = [dict(q=b["q"], k_new=b["k_new"], v_new=b["v_new"], k_cache=k, v_cache=v)
              for (k, v), b in zip(caches, blks)]
        ref = OS.verify_step(ol, ctx, B, off, mask, acc.target, acc.draft, acc.draft_tokens,
                             acc.uniforms, T, band=G.BAND)
        for l in range(layers):
            err = np.abs(dl[l]["out"].float().cpu().numpy() - ref.outs[l]).max()
            assert err <= G.ATTN_TOL[dtype], (step, l, err)
            assert _same(dl[l]["k_cache"], ref.k_caches[l]), (step, l)
            assert _same(dl[l]["v_cache"], ref.v_caches[l]), (step, l)
        G.compare_accept(acc, al.cpu().numpy(), nt.cpu().numpy(), ref.accept)
        # continue from the device's committed state (equal to the oracle's whenever the decisions
        # are outside the near-tie band)
        got_ctx = d_ctx.cpu().numpy()
        assert np.array_equal(got_ctx, OS.commit(ctx, al.cpu().numpy()))
        ctx = got_ctx
        caches = [(torch.from_numpy(rk).to(caches[0][0].dtype), torch.from_numpy(rv).to(caches[0][0].dtype))
                  for rk, rv in zip(ref.k_caches, ref.v_caches)]
        max_ctx += int(B.max())
    return ctx


def test_verify_step_greedy_three_steps():
    ctx = _run_steps(0.0, steps=3, seed=4201)
    assert (ctx > np.array([1500, 3000, 40, 2200])).all()


def test_verify_step_sampling_two_steps():
    _run_steps(1.0, steps=2, seed=4202)


def test_verify_step_fp32_two_steps():
    """fp32 caches and logits: the step appends with sd_kv_append and then attends (the fused
    append is bf16 only); outputs at the fp32 tolerance, caches bit-exact."""
    _run_steps(1.0, steps=2, seed=4203, dtype="f32")


def step_shape(i: int) -> dict:
    """Shape of verify-step case i (seeded; no arithmetic of the method)."""
    r = np.random.default_rng(91000 + i)
    S = int(r.integers(1, 9))
    Hkv = int(r.choice([1, 2, 8]))
    G_ = int(r.choice([1, 2, 4]))
    B = r.integers(1, min(32, 256 // G_) + 1, size=S)
    B[r.random(S) < 0.2] = 1
    return dict(Hq=G_ * Hkv, Hkv=Hkv, D=int(r.choice([64, 128])), V=int(r.integers(1000, 60001)),
                block_lens=B.tolist(), ctx_lens=r.integers(0, 3001, size=S).tolist(),
                T=float(r.choice([0.0, 1.0])), dtype="f32" if r.random() < 0.25 else "bf16",
                layers=int(r.integers(1, 4)),
                mask=W.MASK_BIDIR_IN_BLOCK if r.random() < 0.4 else W.MASK_CAUSAL_IN_BLOCK)


@pytest.mark.parametrize("i", range(8))
def test_verify_step_random_shape(i):
    """Seeded random batches through two multi-layer verify steps: group sizes, head dims,
    vocabularies, masks, dtypes and one-token blocks mixed."""
    sh = step_shape(i)
    G.log(f"  case {i}: {sh}")
    _run_steps(sh["T"], steps=2, seed=4300 + i, layers=sh["layers"], dtype=sh["dtype"], shape=sh, mask=sh["mask"])
