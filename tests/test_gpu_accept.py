"""GPU parity of sd_accept against the fp64 oracle on the same seeded inputs."""
import numpy as np
import pytest
import scipy.stats
import torch

import gpu_util as G
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_tiny(T):
    """Tiny step: V=1024 fp32, B=8; target ~ N(0,2^2), draft = target + N(0,0.5^2)."""
    G.check_accept(W.c1_tiny(temperatures=(T,)).accept[T])


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_qwen3_4b_verify(T):
    """Qwen3-4B verify: V=151936 bf16, B=16, target ~ N(0,3^2), draft = target + N(0,1)."""
    G.check_accept(W.c2_qwen3_4b_verify(temperatures=(T,)).accept[T])


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_ragged_blocks(T):
    """8 ragged blocks B in {8..24} over V=151936."""
    G.check_accept(W.c3_ragged(temperatures=(T,), with_attn=False).accept[T])


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_long_context_batch(T):
    """32 sequences, B U{4..32}, V=151936."""
    G.check_accept(W.c5_long_context(temperatures=(T,), with_attn=False).accept[T])


def _many_seq_problem(seed, S, V, bl_range, dtype, T, target_sigma=2.0, noise_sigma=0.7, name=""):
    rs = W._streams(seed)
    bl = rs["B"].integers(bl_range[0], bl_range[1], endpoint=True, size=S).astype(np.int32)
    return W.make_accept(rs, block_lens=bl, V=V, dtype=dtype, temperature=T, target_sigma=target_sigma,
                         noise_sigma=noise_sigma, name=name)


@pytest.mark.parametrize("T", [0.0, 1.0])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("V", [1, 7, 8, 1003, 4096, 50001])
def test_vocab_edges(V, dtype, T):
    """Vocabulary sizes below one vector, unaligned rows, exact multiples, many sequences and B=1 rows."""
    p = _many_seq_problem(V + (7 if dtype == "bf16" else 0), 40, V, (1, 20), dtype, T, name=f"V{V}")
    G.check_accept(p)


@pytest.mark.parametrize("V,dtype,S,bl_range,T", [
    (32768, "bf16", 3, (1, 12), 1.0),     # shares of 128 vectors: many slots per row
    (131072, "f32", 7, (1, 20), 1.0),     # fp32 rows of 32768 vectors
    (262144, "bf16", 1, (2, 2), 0.0),     # shares shorter than one round
    (262144, "bf16", 3, (4, 12), 1.0),
    (151936, "bf16", 71, (1, 24), 1.0),   # more workgroups than CUs (shares capped at 7 rows)
    (151936, "bf16", 40, (1, 40), 0.0),
])
def test_large_vocab_shapes(V, dtype, S, bl_range, T):
    """Large vocabularies (rows of 4096 to 32768 16-byte vectors) in bf16 and fp32, from one
    sequence to more sequences than a wave of workgroups covers."""
    p = _many_seq_problem(V + S + int(T), S, V, bl_range, dtype, T, target_sigma=3.0, noise_sigma=1.0,
                          name=f"large_V{V}_S{S}")
    G.check_accept(p)


@pytest.mark.parametrize("T", [1.0, 0.0])
@pytest.mark.parametrize("V,dtype", [(151936, "bf16"), (150001, "bf16"), (131075, "f32")])
def test_drafted_tokens_at_chunk_edges(V, dtype, T):
    """Drafted tokens on the elements where a row's statistics chunks meet: the first and last
    elements, the unaligned head and tail (odd vocabularies shift every row's vector boundary),
    and the first and last elements of each chunk of whole vectors; each position's acceptance
    test reads that token's logit."""
    import dataclasses
    p = _many_seq_problem(V + 17, 9, V, (8, 24), dtype, T, target_sigma=3.0, noise_sigma=0.3,
                          name=f"edges_V{V}")
    vec = 8 if dtype == "bf16" else 4
    chunk = 256 * 16 * vec  # elements in a chunk of whole vectors
    edges = [0, 1, 2, vec - 1, vec, vec + 1, V - 1, V - 2, V - vec, V - vec - 1]
    for k in range(1, V // chunk + 1):
        edges += [k * chunk + d for d in (-vec, -2, -1, 0, 1, 2, vec) if 0 <= k * chunk + d < V]
    tokens = np.array([edges[i % len(edges)] for i in range(len(p.draft_tokens))], np.int32)
    G.check_accept(dataclasses.replace(p, draft_tokens=tokens))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_greedy_ties_lowest_index(dtype):
    """Integer-valued logits at V=151936: the maximum is tied in many rows, and across vocabulary
    chunks; the lowest tied index must win, exactly as in the oracle."""
    rs = W._streams(4242)
    bl = np.array([16, 1, 9, 24, 5], dtype=np.int32)
    p = W.make_accept(rs, block_lens=bl, V=151936, dtype=dtype, temperature=0.0, target_sigma=1.0,
                      noise_sigma=0.0, name="ties")
    t = torch.round(p.target.float() * 2).clamp(-6, 6).to(p.target.dtype)
    p.target = t
    # drafts: the highest tied index (rejected) for half the positions, the lowest (accepted) otherwise
    tv = t.float().numpy()
    toks = []
    for s in range(len(bl)):
        for j in range(int(bl[s]) - 1):
            row = tv[p.q_offsets[s] + j]
            idx = np.nonzero(row == row.max())[0]
            toks.append(idx[-1] if (j % 3 == 2) else idx[0])
    p.draft_tokens = np.array(toks, dtype=np.int32)
    al, nt, ref = G.check_accept(p)
    assert (ref.accept_len > 0).any()


def test_identical_draft_accepts_everything():
    rs = W._streams(31)
    bl = np.array([12, 3, 7], dtype=np.int32)
    p = W.make_accept(rs, block_lens=bl, V=32000, dtype="bf16", temperature=1.0, target_sigma=3.0,
                      noise_sigma=0.0, name="identical")
    al, nt, ref = G.check_accept(p)
    assert (al == bl - 1).all()


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_every_block_only_its_anchor(T):
    """Blocks of one token everywhere: no drafted token and no draft row (total_q = S), so the
    call takes an empty draft_logits and the draw at T > 0 is the bonus draw from each target row."""
    rs = W._streams(4321)
    p = W.make_accept(rs, block_lens=np.ones(12, np.int32), V=151936, dtype="bf16", temperature=T,
                      target_sigma=3.0, noise_sigma=1.0, name="anchors_only")
    assert p.total_q == p.S
    al, nt, ref = G.check_accept(p)
    assert (al == 0).all()
    # the same call with no draft tensor at all
    d = G.accept_to_device(p)
    al2, nt2 = sd.accept(d["t"], None, d["tok"], d["u"], d["bl"], d["off"], T, max_block=p.max_block)
    torch.cuda.synchronize()
    assert np.array_equal(al2.cpu().numpy(), al) and np.array_equal(nt2.cpu().numpy(), nt)


def test_temperature_two():
    rs = W._streams(32)
    bl = np.array([10, 14, 4, 20], dtype=np.int32)
    p = W.make_accept(rs, block_lens=bl, V=151936, dtype="bf16", temperature=2.0, target_sigma=3.0,
                      noise_sigma=1.0, name="T2")
    G.check_accept(p)


def test_lossless_chi2_on_gpu():
    """Lossless property on the GPU's own draws (small V): committed tokens ~ target rows."""
    V, B, N = 16, 4, 8000
    rng = np.random.default_rng(99)
    t = rng.normal(0, 1.5, (B, V)).astype(np.float32)
    dl = (t[:B - 1] + rng.normal(0, 1.0, (B - 1, V))).astype(np.float32)

    def sm(x):
        e = np.exp(x - x.max())
        return e / e.sum()

    p = np.stack([sm(t[i].astype(np.float64)) for i in range(B)])
    q = np.stack([sm(dl[i].astype(np.float64)) for i in range(B - 1)])
    tok = np.stack([rng.choice(V, size=N, p=q[j]) for j in range(B - 1)], axis=1).astype(np.int32)
    u = rng.random((N, B), dtype=np.float32)
    bl = np.full(N, B, np.int32)
    prob = W.AcceptProblem(S=N, V=V, block_lens=bl, q_offsets=W.offsets_from_lens(bl),
                           target=torch.from_numpy(np.tile(t, (N, 1))), draft=torch.from_numpy(np.tile(dl, (N, 1))),
                           draft_tokens=tok.reshape(-1), uniforms=u.reshape(-1), temperature=1.0, dtype="f32",
                           name="chi2")
    al, nt = G.run_accept(prob)
    first = np.where(al >= 1, tok[:, 0], nt)
    cnt = np.bincount(first, minlength=V)
    assert scipy.stats.chisquare(cnt, p[0] * N).pvalue > 1e-3
    m = al == B - 1
    cnt = np.bincount(nt[m], minlength=V)
    assert scipy.stats.chisquare(cnt, p[B - 1] * m.sum()).pvalue > 1e-3
    alpha = np.minimum(p[:B - 1], q).sum(axis=1)
    expect = sum(np.prod(alpha[:i + 1]) for i in range(B - 1))
    assert abs(al.mean() - expect) < 4 * al.std() / np.sqrt(N)


def test_repeated_calls_reuse_workspace():
    import paper_2606_31315_amd as sd
    big = W.c3_ragged(temperatures=(1.0,), with_attn=False).accept[1.0]
    small = _many_seq_problem(8, 3, 151936, (2, 9), "bf16", 1.0, target_sigma=3.0, noise_sigma=1.0, name="small")
    d = G.accept_to_device(big)
    ws = torch.zeros(sd.accept_workspace_size(sd.accept_shape(d["t"], big.S, big.max_block), 1.0),
                     dtype=torch.uint8, device=G.dev())
    a1 = G.run_accept(big, d, workspace=ws)
    ref = G.oracle_accept(small)
    als, nts = G.run_accept(small, workspace=ws)
    G.compare_accept(small, als, nts, ref)
    a2 = G.run_accept(big, d, workspace=ws)
    assert (a1[0] == a2[0]).all() and (a1[1] == a2[1]).all()


def test_one_workspace_shared_with_attention():
    """One scratch buffer, holding arbitrary bytes on entry, serves attention and acceptance at
    T = 0 and T = 1 in turn; every acceptance result follows the parity rule."""
    import paper_2606_31315_amd as sd
    pa = W.c3_ragged(temperatures=(), dtype="bf16").attn
    da = G.attn_to_device(pa)
    probs = [_many_seq_problem(71, 12, 151936, (1, 24), "bf16", T, target_sigma=3.0, noise_sigma=1.0,
                               name=f"shared_T{T:g}") for T in (0.0, 1.0)]
    dev_p = [G.accept_to_device(p) for p in probs]
    refs = [G.oracle_accept(p) for p in probs]
    n = max([sd.attn_workspace_size(sd.attn_shape(da["q"], da["k"], pa.max_ctx, pa.max_block))] +
            [sd.accept_workspace_size(sd.accept_shape(d["t"], p.S, p.max_block), p.temperature)
             for p, d in zip(probs, dev_p)])
    ws = torch.randint(0, 256, (n,), dtype=torch.uint8, device=G.dev())
    for it in range(3):
        G.run_attn(pa, da, workspace=ws)
        for p, d, ref in zip(probs, dev_p, refs):
            al, nt = G.run_accept(p, d, workspace=ws)
            G.compare_accept(p, al, nt, ref)


# ---- the single-launch greedy path against the two-launch path ----
# At T = 0, where the shape allows it, sd_accept runs as one launch whose workgroups hand the
# per-chunk records on through tagged words; the two-launch path stays for the other shapes,
# for graph capture and for T > 0.  The same merges run in the same order, so results agree
# exactly.

_PATH_CASES = [
    ("ragged", lambda: W.c3_ragged(temperatures=(0.0,), with_attn=False).accept[0.0]),
    ("qwen3_4b", lambda: W.c2_qwen3_4b_verify(temperatures=(0.0,)).accept[0.0]),
    ("long_context", lambda: W.c5_long_context(temperatures=(0.0,), with_attn=False).accept[0.0]),
    ("V4096_f32", lambda: _many_seq_problem(5, 40, 4096, (1, 20), "f32", 0.0, name="V4096_f32")),
    ("V262144", lambda: _many_seq_problem(6, 3, 262144, (4, 12), "bf16", 0.0, target_sigma=3.0,
                                          noise_sigma=1.0, name="V262144")),
    ("V7", lambda: _many_seq_problem(7, 40, 7, (1, 20), "bf16", 0.0, name="V7")),
    ("B1_only", lambda: _many_seq_problem(8, 16, 151936, (1, 1), "bf16", 0.0, name="B1")),
    ("max_block_64", lambda: _many_seq_problem(9, 5, 32768, (60, 64), "bf16", 0.0, name="B64")),
]


# At T > 0, where the shape allows it, the mass and locate steps run as one launch whose
# workgroups hand the per-chunk mass sums on through tagged words; the three-launch path stays
# for wide chunks, grids larger than the device holds at once, graph capture and small
# workspaces.  The same sums run in the same order, so results agree exactly.
_DRAW_CASES = [
    ("ragged", lambda: W.c3_ragged(temperatures=(1.0,), with_attn=False).accept[1.0]),
    ("qwen3_4b", lambda: W.c2_qwen3_4b_verify(temperatures=(1.0,)).accept[1.0]),
    # 32 sequences x 75 chunks: more workgroups than the single launch takes (three launches)
    ("long_context", lambda: W.c5_long_context(temperatures=(1.0,), with_attn=False).accept[1.0]),
    ("V4096_f32", lambda: _many_seq_problem(15, 40, 4096, (1, 20), "f32", 1.0, name="V4096_f32_T1")),
    # fp32 rows of 37984 vectors: 149 chunks, three passes of the chunk search
    ("V151936_f32", lambda: _many_seq_problem(16, 5, 151936, (2, 12), "f32", 1.0, target_sigma=3.0,
                                              noise_sigma=1.0, name="V151936_f32_T1")),
    # draft rows not vector-aligned with their target rows (V % 8 != 0)
    ("V50001", lambda: _many_seq_problem(17, 9, 50001, (1, 16), "bf16", 1.0, target_sigma=3.0,
                                         noise_sigma=1.0, name="V50001_T1")),
    ("V7", lambda: _many_seq_problem(18, 40, 7, (1, 20), "bf16", 1.0, name="V7_T1")),
    ("V1003", lambda: _many_seq_problem(19, 40, 1003, (1, 20), "bf16", 1.0, name="V1003_T1")),
    ("B1_B2", lambda: _many_seq_problem(20, 16, 151936, (1, 2), "bf16", 1.0, target_sigma=3.0,
                                       noise_sigma=1.0, name="B1_B2_T1")),
    ("max_block_64", lambda: _many_seq_problem(21, 5, 32768, (60, 64), "bf16", 1.0, name="B64_T1")),
]


def _both_paths(p, d):
    import paper_2606_31315_amd as sd
    try:
        sd.accept_set_path(1)
        multi = G.run_accept(p, d)
        sd.accept_set_path(0)
        single = G.run_accept(p, d)
    finally:
        sd.accept_set_path(0)
    return single, multi


@pytest.mark.parametrize("name,make", _PATH_CASES, ids=[c[0] for c in _PATH_CASES])
def test_single_launch_matches_two_launches(name, make):
    """Both greedy paths give the same accept_len and next_token, bit for bit, and the single
    launch's result meets the parity rule against the oracle."""
    p = make()
    d = G.accept_to_device(p)
    (al1, nt1), (alm, ntm) = _both_paths(p, d)
    assert (al1 == alm).all() and (nt1 == ntm).all(), (name, np.nonzero(al1 != alm), np.nonzero(nt1 != ntm))
    G.compare_accept(p, al1, nt1, G.oracle_accept(p))


@pytest.mark.parametrize("name,make", _DRAW_CASES, ids=[c[0] for c in _DRAW_CASES])
def test_single_launch_draw_matches_three_launches(name, make):
    """Both sampling paths give the same accept_len and next_token, bit for bit, and the single
    launch's result meets the parity rule against the oracle."""
    p = make()
    d = G.accept_to_device(p)
    (al1, nt1), (alm, ntm) = _both_paths(p, d)
    assert (al1 == alm).all() and (nt1 == ntm).all(), (name, np.nonzero(al1 != alm), np.nonzero(nt1 != ntm))
    G.compare_accept(p, al1, nt1, G.oracle_accept(p))


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_single_launch_ignores_leftover_words(T):
    """A workspace holding an earlier call's words, random bytes, one repeated 64-bit word, or
    zeros: every call still equals the multi-launch result."""
    import paper_2606_31315_amd as sd
    p = W.c3_ragged(temperatures=(T,), with_attn=False).accept[T]
    d = G.accept_to_device(p)
    n = sd.accept_workspace_size(sd.accept_shape(d["t"], p.S, p.max_block), T)
    _, (alm, ntm) = _both_paths(p, d)
    ws = torch.empty(n, dtype=torch.uint8, device=G.dev())
    fills = [lambda: None,  # whatever the previous call left
             lambda: ws.copy_(torch.randint(0, 256, (n,), dtype=torch.uint8, device=G.dev())),
             lambda: ws.view(torch.int64).fill_(0x3F8000003F800000),
             lambda: ws.zero_()]
    for rep in range(2):
        for f in fills:
            f()
            al, nt = G.run_accept(p, d, workspace=ws)
            assert (al == alm).all() and (nt == ntm).all()


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_single_launch_gives_up_when_told_and_recovers(T):
    """With the waits cut to one poll, every output is either exact or -1 (greedy: both outputs
    of a sequence together); the next call with the default limit, on the same workspace, is
    exact."""
    import paper_2606_31315_amd as sd
    p = W.c3_ragged(temperatures=(T,), with_attn=False).accept[T]
    d = G.accept_to_device(p)
    n = sd.accept_workspace_size(sd.accept_shape(d["t"], p.S, p.max_block), T)
    ws = torch.empty(n, dtype=torch.uint8, device=G.dev())
    _, (alm, ntm) = _both_paths(p, d)
    try:
        sd.accept_set_path(0, 1)
        al, nt = G.run_accept(p, d, workspace=ws)
    finally:
        sd.accept_set_path(0)
    if T == 0:
        exact = (al == alm) & (nt == ntm)
        gave_up = (al == -1) & (nt == -1)
        assert (exact | gave_up).all(), (al, alm, nt, ntm)
    else:
        assert ((al == alm) | (al == -1)).all() and ((nt == ntm) | (nt == -1)).all(), (al, alm, nt, ntm)
    al, nt = G.run_accept(p, d, workspace=ws)
    assert (al == alm).all() and (nt == ntm).all()


@pytest.mark.parametrize("T", [0.0, 1.0])
def test_small_workspace_takes_multi_launch_path(T):
    """A workspace big enough for the multi-launch path only still gives the same results."""
    import ctypes
    import paper_2606_31315_amd as sd
    from paper_2606_31315_amd import _lib
    p = W.c3_ragged(temperatures=(T,), with_attn=False).accept[T]
    d = G.accept_to_device(p)
    shape = sd.accept_shape(d["t"], p.S, p.max_block)
    full = sd.accept_workspace_size(shape, T)
    al = torch.empty(p.S, dtype=torch.int32, device=G.dev())
    nt = torch.empty(p.S, dtype=torch.int32, device=G.dev())
    ws = torch.empty(full, dtype=torch.uint8, device=G.dev())
    L = _lib.lib()

    def call(nbytes):
        return L.sd_accept(ctypes.byref(shape), _lib._ptr(d["t"]), _lib._ptr(d["d"]), _lib._ptr(d["tok"]),
                           _lib._ptr(d["u"]), _lib._ptr(d["bl"]), _lib._ptr(d["off"]), ctypes.c_float(T),
                           _lib._ptr(al), _lib._ptr(nt), _lib._ptr(ws), nbytes, _lib._stream(None))
    # the smallest workspace the call accepts, by bisection on SD_ERR_WORKSPACE
    lo, hi = 0, full
    while hi - lo > 256:
        mid = (lo + hi) // 2 // 256 * 256
        if call(mid) == _lib.SD_OK:
            hi = mid
        else:
            lo = mid
    assert hi < full
    assert call(hi) == _lib.SD_OK
    torch.cuda.synchronize()
    _, multi = _both_paths(p, d)
    assert (al.cpu().numpy() == multi[0]).all() and (nt.cpu().numpy() == multi[1]).all()
