"""GPU tests of sd_check_attn_inputs and sd_check_accept_inputs: the error word for the
per-sequence values that sd_block_attn and sd_accept read from device memory and take on
trust.  Expected words come from the documented ranges (include/sd_block.h) applied on the
host, sequence by sequence; the check kernel must report the same bits, the same first
offending sequence and the same count.  The corrupted arrays go to the check kernel only."""
import numpy as np
import pytest
import torch

import gpu_util as G
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu

CTX, BLOCK, OFFSETS, TOKEN, UNIFORM = 1, 2, 4, 8, 16


def expect(B, off, total_q, max_block, min_block, ctx=None, max_ctx=0, tokens=None, vocab=0, uniforms=None):
    S = len(B)
    bits, first, count = 0, -1, 0
    for s in range(S):
        e = 0
        if not (min_block <= B[s] <= max_block):
            e |= BLOCK
        if ctx is not None and not (0 <= ctx[s] <= max_ctx):
            e |= CTX
        o0, o1 = int(off[s]), int(off[s + 1])
        if (s == 0 and o0 != 0) or (s == S - 1 and o1 != total_q) or o1 - o0 != B[s] or o0 < 0 or o1 > total_q:
            e |= OFFSETS
        if not e & (BLOCK | OFFSETS):
            if tokens is not None:
                d0 = o0 - s
                if d0 < 0 or d0 + B[s] - 1 > total_q - S:
                    e |= OFFSETS
                elif any(not (0 <= t < vocab) for t in tokens[d0:d0 + B[s] - 1]):
                    e |= TOKEN
            if uniforms is not None and any(not (0.0 <= u < 1.0) for u in uniforms[o0:o0 + B[s]]):
                e |= UNIFORM
        if e:
            bits |= e
            first = s if first < 0 else first
            count += 1
    return [bits, first, count]


def run_attn_check(ctx, B, off, total_q, max_ctx, max_block):
    dev = G.dev()
    t = [torch.from_numpy(np.asarray(x, np.int32)).to(dev) for x in (ctx, B, off)]
    G.log(f"sd_check_attn_inputs S={len(B)} total_q={total_q} max_ctx={max_ctx} max_block={max_block}")
    st = sd.check_attn_inputs(*t, total_q=total_q, max_ctx=max_ctx, max_block=max_block)
    torch.cuda.synchronize()
    return st.cpu().tolist()


def run_accept_check(tokens, uniforms, B, off, T, vocab, total_q, max_block):
    dev = G.dev()
    tok = torch.from_numpy(np.asarray(tokens, np.int32) if len(tokens) else np.zeros(1, np.int32)).to(dev)
    u = torch.from_numpy(np.asarray(uniforms, np.float32)).to(dev) if uniforms is not None else None
    b, o = (torch.from_numpy(np.asarray(x, np.int32)).to(dev) for x in (B, off))
    G.log(f"sd_check_accept_inputs S={len(B)} total_q={total_q} V={vocab} T={T}")
    st = sd.check_accept_inputs(tok, u, b, o, T, vocab=vocab, total_q=total_q, max_block=max_block)
    torch.cuda.synchronize()
    return st.cpu().tolist()


def test_attn_workloads_pass():
    for p in (W.c3_ragged(temperatures=()).attn, W.c4_drafter().attn):
        assert run_attn_check(p.ctx_lens, p.block_lens, p.q_offsets, p.total_q, p.max_ctx, p.max_block) == [0, -1, 0]


def test_attn_each_fault():
    B = np.array([12, 0, 20, 16, 18], np.int32)
    off = W.offsets_from_lens(B)
    ctx = np.array([4096, 0, 17, 4000, 4096], np.int32)
    tq, mc, mb = int(off[-1]), 4096, 24
    cases = []
    c = ctx.copy(); c[2] = mc + 1; cases.append((c, B, off))                  # context past max_ctx
    c = ctx.copy(); c[3] = -5; cases.append((c, B, off))                      # negative context
    b = B.copy(); b[4] = mb + 1; cases.append((ctx, b, W.offsets_from_lens(b)))  # block past max_block
    b = B.copy(); b[0] = -1; cases.append((ctx, b, off))                      # negative block, offsets then wrong
    o = off.copy(); o[0] = 1; cases.append((ctx, B, o))                       # q_offsets[0] != 0
    o = off.copy(); o[-1] += 1; cases.append((ctx, B, o))                     # q_offsets[S] != total_q
    o = off.copy(); o[2] += 3; cases.append((ctx, B, o))                      # inconsistent inside
    for c, b, o in cases:
        want = expect(b, o, tq, mb, 0, ctx=c, max_ctx=mc)
        assert want[0] != 0
        assert run_attn_check(c, b, o, tq, mc, mb) == want, (c, b, o)


def test_attn_many_sequences_random_faults():
    """1500 sequences (several passes of the 256-thread walk) with seeded random faults."""
    rng = np.random.default_rng(11)
    S, mc, mb = 1500, 8192, 32
    B = rng.integers(0, mb + 1, S).astype(np.int32)
    off = W.offsets_from_lens(B)
    ctx = rng.integers(0, mc + 1, S).astype(np.int32)
    bad = rng.choice(S, 40, replace=False)
    ctx[bad[:15]] = mc + rng.integers(1, 100, 15)
    B2 = B.copy()
    B2[bad[15:30]] = mb + 1                                                   # offsets kept: both bits
    off2 = off.copy()
    off2[bad[30:] + 1] += 1                                                   # two sequences each
    tq = int(off[-1])
    want = expect(B2, off2, tq, mb, 0, ctx=ctx, max_ctx=mc)
    assert want[2] >= 40
    assert run_attn_check(ctx, B2, off2, tq, mc, mb) == want


def test_attn_no_sequences():
    assert run_attn_check(np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(1, np.int32), 0, 10, 4) == \
        [0, -1, 0]


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_accept_workload_passes(T):
    a = W.c3_ragged(temperatures=(T,), with_attn=False).accept[T]
    u = a.uniforms if T > 0 else None
    assert run_accept_check(a.draft_tokens, u, a.block_lens, a.q_offsets, T, a.V, a.total_q, a.max_block) == \
        [0, -1, 0]


def test_accept_each_fault():
    rng = np.random.default_rng(5)
    V, mb = 1000, 16
    B = np.array([4, 1, 9, 16, 2], np.int32)
    off = W.offsets_from_lens(B)
    tq, S = int(off[-1]), len(B)
    tok = rng.integers(0, V, tq - S).astype(np.int32)
    u = rng.random(tq, dtype=np.float32)
    cases = []
    t = tok.copy(); t[3] = V; cases.append((t, u, B, off, 1.0))              # token == V
    t = tok.copy(); t[-1] = -1; cases.append((t, u, B, off, 1.0))            # negative token, last sequence
    x = u.copy(); x[0] = 1.0; cases.append((tok, x, B, off, 1.0))            # uniform == 1
    x = u.copy(); x[7] = np.nan; cases.append((tok, x, B, off, 1.0))         # NaN uniform
    x = u.copy(); x[7] = np.nan; cases.append((tok, x, B, off, 0.0))         # ignored at T = 0
    b = B.copy(); b[1] = 0; cases.append((tok, u, b, off, 1.0))              # empty block: offsets then wrong
    o = off.copy(); o[-1] -= 1; cases.append((tok, u, B, o, 1.0))
    for t, x, b, o, T in cases:
        want = expect(b, o, tq, mb, 1, tokens=t, vocab=V, uniforms=(x if T > 0 else None))
        got = run_accept_check(t, x if T > 0 else None, b, o, T, V, tq, mb)
        assert got == want, (got, want)
    assert run_accept_check(tok, u, B, off, 1.0, V, tq, mb) == [0, -1, 0]
