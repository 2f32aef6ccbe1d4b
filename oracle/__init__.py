"""fp64 CPU oracle for block-verify attention and speculative acceptance.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The arithmetic lives in ``sd_oracle.c``
(plain C, fp64); this module builds it with gcc and marshals arrays through
ctypes.  It imports nothing from the HIP package except the seeded workload
dataclasses, which carry inputs only.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "sd_oracle.c")
LIB = os.path.join(_HERE, "liboracle.so")


def compile_oracle(src_path: str, out_path: str) -> str:
    """gcc -O2 -fopenmp build of an oracle source file into a shared library."""
    tmp = out_path + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra",
           "-o", tmp, src_path, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out_path)
    return out_path


def build(force: bool = True) -> str:
    """Compile the oracle.  Always recompiles when ``force``."""
    if force or not os.path.exists(LIB):
        compile_oracle(SRC, LIB)
    return LIB


def _f32(x) -> np.ndarray:
    """Exact fp32 view of an input (bf16 and fp32 widen exactly)."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().to("cpu").float().numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(x, dtype=np.float32)


def _i32(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x), dtype=np.int32)


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


@dataclass
class AcceptResult:
    accept_len: np.ndarray
    next_token: np.ndarray
    accept_margin: np.ndarray
    sample_margin: np.ndarray
    sample_lo: np.ndarray
    sample_hi: np.ndarray
    sample_tie_p: np.ndarray


class Oracle:
    """ctypes handle on one build of the oracle library."""

    def __init__(self, lib_path: str):
        lib = ctypes.CDLL(lib_path)
        P = ctypes.c_void_p
        lib.oracle_block_attn.restype = ctypes.c_int
        lib.oracle_block_attn.argtypes = [ctypes.c_int] * 5 + [P] * 3 + [P] * 3 + [
            ctypes.c_int, ctypes.c_double, ctypes.c_long, P, P, P]
        lib.oracle_accept.restype = ctypes.c_int
        lib.oracle_accept.argtypes = [ctypes.c_int, ctypes.c_int, P, P, P, P, P, P,
                                      ctypes.c_double, ctypes.c_double, P, P, P, P, P, P, P]
        lib.oracle_num_threads.restype = ctypes.c_int
        lib.oracle_set_threads.argtypes = [ctypes.c_int]
        self.lib = lib
        self.path = lib_path

    def num_threads(self) -> int:
        return int(self.lib.oracle_num_threads())

    def set_threads(self, n: int) -> None:
        self.lib.oracle_set_threads(int(n))

    def block_attn(self, q, k_cache, v_cache, ctx_lens, block_lens, q_offsets, mask_mode, scale=0.0,
                   rows=None) -> np.ndarray:
        """fp64 block attention.  q [total_q,Hq,D], caches [S,Hkv,Lmax,D].

        ``rows`` = None computes everything and returns [total_q, Hq, D]; otherwise a
        pair (tok[n], head[n]) selects rows and the result is [n, D].
        """
        q = _f32(q)
        k = _f32(k_cache)
        v = _f32(v_cache)
        S, Hkv, Lmax, D = k.shape
        Hq = q.shape[1]
        ctx = _i32(ctx_lens)
        bl = _i32(block_lens)
        off = _i32(q_offsets)
        if rows is None:
            out = np.zeros((q.shape[0], Hq, D), dtype=np.float64)
            n = -1
            tok_a = head_a = np.zeros(1, dtype=np.int64)
        else:
            tok_a = np.ascontiguousarray(rows[0], dtype=np.int64)
            head_a = np.ascontiguousarray(rows[1], dtype=np.int32)
            n = len(tok_a)
            out = np.zeros((n, D), dtype=np.float64)
        rc = self.lib.oracle_block_attn(S, Hq, Hkv, D, Lmax, _p(q), _p(k), _p(v), _p(ctx), _p(bl), _p(off),
                                       int(mask_mode), float(scale), n, _p(tok_a), _p(head_a), _p(out))
        if rc != 0:
            raise ValueError("oracle_block_attn: bad arguments")
        return out

    def accept(self, target, draft, draft_tokens, uniforms, block_lens, q_offsets, temperature,
               band=1e-5) -> AcceptResult:
        """fp64 speculative acceptance (greedy at T=0, rejection sampling at T>0)."""
        t = _f32(target)
        tq, V = t.shape
        S = len(block_lens)
        d = _f32(draft) if draft is not None else np.zeros((1, 1), dtype=np.float32)
        tok = _i32(draft_tokens) if len(draft_tokens) else np.zeros(1, dtype=np.int32)
        u = _f32(uniforms) if uniforms is not None else np.zeros(max(tq, 1), dtype=np.float32)
        bl = _i32(block_lens)
        off = _i32(q_offsets)
        if temperature > 0 and draft is None:
            raise ValueError("draft logits are required at T > 0")
        al = np.zeros(S, dtype=np.int32)
        nt = np.zeros(S, dtype=np.int32)
        am = np.zeros(S, dtype=np.float64)
        sm = np.zeros(S, dtype=np.float64)
        lo = np.zeros(S, dtype=np.int32)
        hi = np.zeros(S, dtype=np.int32)
        tp = np.zeros(S, dtype=np.float64)
        rc = self.lib.oracle_accept(S, V, _p(t), _p(d), _p(tok), _p(u), _p(bl), _p(off), float(temperature),
                                   float(band), _p(al), _p(nt), _p(am), _p(sm), _p(lo), _p(hi), _p(tp))
        if rc != 0:
            raise ValueError("oracle_accept: bad arguments")
        return AcceptResult(al, nt, am, sm, lo, hi, tp)


_default = None


def default() -> Oracle:
    """The oracle built from ``sd_oracle.c`` (rebuilt when the source is newer)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        _default = Oracle(LIB)
    return _default


def block_attn(*args, **kw) -> np.ndarray:
    return default().block_attn(*args, **kw)


def accept(*args, **kw) -> "AcceptResult":
    return default().accept(*args, **kw)


def num_threads() -> int:
    return default().num_threads()


def set_threads(n: int) -> None:
    default().set_threads(n)
