"""The hot path under HIP graph capture: sd_block_attn + sd_accept, and sd_verify_step, captured
once with torch.cuda.graph and replayed several times, with eager work and synchronisations
between the replays.  Every replay must equal the same calls made eagerly on identical
buffers, bit for bit (same kernels, same launch shapes, same inputs).  The calls allocate
nothing, never synchronise and clear no memory, so nothing but kernel launches is captured."""
import numpy as np
import pytest
import torch

import gpu_util as G
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu


def _bits(t: torch.Tensor) -> torch.Tensor:
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


def test_attention_and_acceptance_replays_match_eager():
    dev = G.dev()
    work = W.c3_ragged(temperatures=(1.0,))
    a, acc = work.attn, work.accept[1.0]
    q0 = a.q.to(dev)
    k, v = a.k_cache.to(dev), a.v_cache.to(dev)
    ctx, bl, off = (torch.from_numpy(x).to(dev) for x in (a.ctx_lens, a.block_lens, a.q_offsets))
    tgt, drf = acc.target.to(dev), acc.draft.to(dev)
    tok, u0 = torch.from_numpy(acc.draft_tokens).to(dev), torch.from_numpy(acc.uniforms).to(dev)
    ash = sd.attn_shape(q0, k, a.max_ctx, a.max_block)
    csh = sd.accept_shape(tgt, a.S, a.max_block)
    q, u = q0.clone(), u0.clone()                      # inputs the graph reads, refilled per replay
    bufs = {}
    for side in ("graph", "eager"):
        bufs[side] = dict(out=torch.empty_like(q0), al=torch.empty(a.S, dtype=torch.int32, device=dev),
                          nt=torch.empty(a.S, dtype=torch.int32, device=dev),
                          ws1=torch.empty(sd.attn_workspace_size(ash), dtype=torch.uint8, device=dev),
                          ws2=torch.empty(sd.accept_workspace_size(csh, 1.0), dtype=torch.uint8, device=dev))

    def step(b, q_in, u_in):
        sd.block_attn(q_in, k, v, ctx, bl, off, a.mask_mode, max_ctx=a.max_ctx, max_block=a.max_block,
                      out=b["out"], workspace=b["ws1"])
        sd.accept(tgt, drf, tok, u_in, bl, off, 1.0, max_block=a.max_block, accept_len=b["al"],
                  next_token=b["nt"], workspace=b["ws2"])

    G.log("graph capture: sd_block_attn + sd_accept (ragged Qwen3-4B batch, T=1)")
    step(bufs["graph"], q, u)                          # every kernel loaded before the capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(bufs["graph"], q, u)
    rng = np.random.default_rng(3)
    for r in range(4):
        q.copy_(q0 * (1.0 + 0.25 * r))
        u.copy_(torch.from_numpy(rng.random(u0.numel(), dtype=np.float32)).to(dev))
        step(bufs["eager"], q, u)
        torch.cuda.synchronize()
        _ = (q.float() * 2).sum().item()               # eager work between replays
        G.log(f"  replay {r}")
        graph.replay()
        torch.cuda.synchronize()
        ge, gg = bufs["eager"], bufs["graph"]
        assert torch.equal(_bits(gg["out"]), _bits(ge["out"])), r
        assert torch.equal(gg["al"], ge["al"]) and torch.equal(gg["nt"], ge["nt"]), r


def test_verify_step_replays_match_eager():
    """Two layers, T=1, four consecutive steps: the replays advance their own copy of the
    caches and context lengths exactly as the eager steps advance theirs."""
    dev = G.dev()
    rs = W._streams(4301)
    S, Hq, Hkv, D, V, layers, steps = 4, 32, 8, 128, 32000, 2, 4
    B = np.array([12, 16, 5, 24], np.int32)
    off = W.offsets_from_lens(B)
    ctx0 = np.array([1500, 3000, 40, 2200], np.int32)
    max_ctx = int(ctx0.max() + steps * B.max())       # host bound that holds for every replay
    Lmax = max_ctx + int(B.max())
    caches = [W.step_caches(rs, S=S, Hkv=Hkv, D=D, Lmax=Lmax, ctx_lens=ctx0, dtype="bf16") for _ in range(layers)]
    blks = [W.step_block_inputs(rs, total_q=int(off[-1]), Hq=Hq, Hkv=Hkv, D=D, dtype="bf16")
            for _ in range(layers)]
    acc = W.make_accept(rs, block_lens=B, V=V, dtype="bf16", temperature=1.0, target_sigma=3.0, noise_sigma=0.7)
    da = G.accept_to_device(acc)
    bl, offd = torch.from_numpy(B).to(dev), torch.from_numpy(off).to(dev)
    state = {}
    for side in ("graph", "eager", "warmup"):
        state[side] = dict(
            layers=[dict(q=b["q"].to(dev), k_new=b["k_new"].to(dev), v_new=b["v_new"].to(dev), k_cache=kc.to(dev),
                         v_cache=vc.to(dev), out=torch.empty_like(b["q"], device=dev))
                    for (kc, vc), b in zip(caches, blks)],
            ctx=torch.from_numpy(ctx0).to(dev), al=torch.empty(S, dtype=torch.int32, device=dev),
            nt=torch.empty(S, dtype=torch.int32, device=dev),
            ws=torch.empty(64 << 20, dtype=torch.uint8, device=dev))

    def step(st):
        sd.verify_step(st["layers"], st["ctx"], bl, offd, W.MASK_CAUSAL_IN_BLOCK, da["t"], da["d"], da["tok"],
                       da["u"], 1.0, max_ctx=max_ctx, max_block=int(B.max()), accept_len=st["al"],
                       next_token=st["nt"], workspace=st["ws"])

    G.log(f"graph capture: sd_verify_step, {layers} layers, {steps} replays")
    step(state["warmup"])                              # every kernel loaded before the capture
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):                      # capture only: the graph side is not advanced
        step(state["graph"])
    for r in range(steps):
        step(state["eager"])
        torch.cuda.synchronize()
        _ = state["eager"]["ctx"].sum().item()         # eager work between replays
        G.log(f"  replay {r}")
        graph.replay()
        torch.cuda.synchronize()
        e, g = state["eager"], state["graph"]
        assert torch.equal(g["ctx"], e["ctx"]) and torch.equal(g["al"], e["al"]) and torch.equal(g["nt"], e["nt"]), r
        for lg, le in zip(g["layers"], e["layers"]):
            assert torch.equal(_bits(lg["out"]), _bits(le["out"])), r
            assert torch.equal(_bits(lg["k_cache"]), _bits(le["k_cache"])), r
            assert torch.equal(_bits(lg["v_cache"]), _bits(le["v_cache"])), r
    assert (state["graph"]["ctx"].cpu().numpy() > ctx0).all()
