"""The oracle's C source under AddressSanitizer and UndefinedBehaviorSanitizer (host code only).

A second build of ``oracle/sd_oracle.c`` with ``-fsanitize=address,undefined`` and
``-fno-sanitize-recover=all`` runs in a child interpreter (the ASan runtime preloaded) over
small seeded cases that reach every branch the parity tests rely on: both masks, empty
context, single-row and empty blocks, ragged tails, GQA and MHA grouping, explicit scale and
row selection for attention; greedy and sampled acceptance with empty blocks, B = 1, vocabulary
sizes that are not a multiple of anything, tied maxima and identical draft rows.  The child
exits non-zero on the first sanitizer report; its results must equal the regular build's.
"""
import json
import os
import subprocess
import sys
import textwrap

import numpy as np
import pytest

import oracle
from paper_2606_31315_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, S, Hq, Hkv, D, ctx, B, mask)
ATTN_CASES = [
    ("causal_gqa", 2, 8, 2, 16, [0, 37], [5, 1], W.MASK_CAUSAL_IN_BLOCK),
    ("bidir_gqa", 3, 8, 2, 16, [11, 0, 64], [7, 3, 16], W.MASK_BIDIR_IN_BLOCK),
    ("empty_block", 3, 4, 4, 8, [5, 9, 3], [2, 0, 4], W.MASK_CAUSAL_IN_BLOCK),
    ("mha_bidir_ctx0", 1, 4, 4, 32, [0], [9], W.MASK_BIDIR_IN_BLOCK),
]
# (name, block_lens, V, T)
ACCEPT_CASES = [
    ("greedy", [4, 1, 0, 7], 37, 0.0),
    ("sampled", [4, 1, 0, 7], 37, 1.0),
    ("sampled_T2", [3, 6], 101, 2.0),
    ("greedy_V1", [2, 3], 1, 0.0),
]


def _attn_inputs(case):
    name, S, Hq, Hkv, D, ctx, B, mode = case
    rs = W._streams(5000 + ATTN_CASES.index(case))
    return W.make_attn(rs, S=S, Hq=Hq, Hkv=Hkv, D=D, ctx_lens=ctx, block_lens=B, dtype="f32", mask_mode=mode,
                       name=name)


def _accept_inputs(case):
    name, bl, V, T = case
    rs = W._streams(6000 + ACCEPT_CASES.index(case))
    p = W.make_accept(rs, block_lens=np.asarray(bl, np.int32), V=V, dtype="f32", temperature=T, target_sigma=2.0,
                      noise_sigma=0.5, name=name)
    t = p.target.float().numpy().copy()
    tok = p.draft_tokens.copy()
    if name == "greedy" and V > 3:  # tied maxima in every target row; draft tokens on a tie
        t[:, 1] = t[:, 3] = t.max(axis=1) + 1.0
        tok[:] = 3
    d = None if p.draft is None else p.draft.float().numpy().copy()
    if name == "sampled_T2" and d is not None:  # first draft row identical to its target row
        d[0] = t[0]
    return dict(target=t, draft=d, tokens=tok, uniforms=p.uniforms, block_lens=p.block_lens,
                q_offsets=p.q_offsets, T=T)


def _run_all(orc, store):
    """Every case through one oracle build; arrays go into ``store``."""
    for case in ATTN_CASES:
        a = _attn_inputs(case)
        store[case[0]] = orc.block_attn(a.q, a.k_cache, a.v_cache, a.ctx_lens, a.block_lens, a.q_offsets,
                                        a.mask_mode)
        tq = int(a.q_offsets[-1])
        if tq:
            tok = np.arange(tq, dtype=np.int64)
            head = (np.arange(tq) % a.q.shape[1]).astype(np.int32)
            store[case[0] + "_rows_scale"] = orc.block_attn(a.q, a.k_cache, a.v_cache, a.ctx_lens, a.block_lens,
                                                            a.q_offsets, a.mask_mode, scale=0.3, rows=(tok, head))
    for case in ACCEPT_CASES:
        x = _accept_inputs(case)
        r = orc.accept(x["target"], x["draft"], x["tokens"], x["uniforms"], x["block_lens"], x["q_offsets"], x["T"])
        for f in ("accept_len", "next_token", "accept_margin", "sample_margin", "sample_lo", "sample_hi",
                  "sample_tie_p"):
            store[f"{case[0]}_{f}"] = getattr(r, f)


def _asan_runtime():
    out = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.skipif(_asan_runtime() is None, reason="gcc has no AddressSanitizer runtime here")
def test_oracle_clean_under_asan_ubsan(tmp_path):
    lib = tmp_path / "liboracle_asan.so"
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-o", str(lib), oracle.SRC, "-lm"],
                   check=True)
    res = tmp_path / "asan.npz"
    child = textwrap.dedent(f"""
        import sys
        sys.path.insert(0, {ROOT!r})
        sys.path.insert(0, {os.path.dirname(os.path.abspath(__file__))!r})
        import numpy as np
        import oracle
        import test_oracle_sanitizers as T
        orc = oracle.Oracle({str(lib)!r})
        orc.set_threads(2)
        store = {{}}
        T._run_all(orc, store)
        np.savez({str(res)!r}, **store)
        print("child ok", len(store))
    """)
    env = dict(os.environ, LD_PRELOAD=_asan_runtime(), ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    p = subprocess.run([sys.executable, "-c", child], env=env, capture_output=True, text=True, timeout=600)
    report = (p.stdout + p.stderr)[-4000:]
    assert p.returncode == 0, report
    assert "runtime error" not in p.stderr and "AddressSanitizer" not in p.stderr, report
    got = dict(np.load(res))
    want = {}
    _run_all(oracle.default(), want)
    assert sorted(got) == sorted(want)
    for k in want:
        np.testing.assert_array_equal(got[k], want[k], err_msg=k)
    print(json.dumps({"cases": len(want)}))
