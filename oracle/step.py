"""fp64 CPU oracle of the step around verification: the block's key/value append, the
commit after acceptance, and the whole verify step (append + block attention in every
layer, acceptance, commit).

TEST INFRASTRUCTURE ONLY: the test suite is the only caller.  Append and commit are
their definitions written out in numpy (a row copy and an integer update); the verify
step composes them with the fp64 attention and acceptance of ``sd_oracle.c``.

Definitions (Sec. 2.1: the drafted block is verified in parallel with its keys and
values in the cache; Fig. 1 caption and App. A.1: the longest consistent prefix is
accepted, plus one bonus or resampled token):
  append   K[s, h, ctx_s + i, :] = K_new[q_off_s + i, h, :]  (and V), i < B_s
  commit   ctx_s <- ctx_s + accept_len_s + 1   (the anchor and the accepted drafts)
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np

from . import accept as _accept
from . import block_attn as _block_attn


def _np(x, dtype=np.float32) -> np.ndarray:
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().to("cpu").float().numpy() if dtype == np.float32 else x.detach().to("cpu").numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.array(x, dtype=dtype, copy=True)


def kv_append(k_cache, v_cache, k_new, v_new, ctx_lens, q_offsets):
    """New caches (float32 copies) with the block rows written at [ctx_s, ctx_s + B_s).  A row
    that would land at or past the cache capacity is not written."""
    k = _np(k_cache)
    v = _np(v_cache)
    kn = _np(k_new)
    vn = _np(v_new)
    ctx = np.asarray(ctx_lens, dtype=np.int64)
    off = np.asarray(q_offsets, dtype=np.int64)
    Lmax = k.shape[2]
    for s in range(len(ctx)):
        for i in range(int(off[s + 1] - off[s])):
            pos = int(ctx[s]) + i
            if 0 <= pos < Lmax:
                k[s, :, pos, :] = kn[off[s] + i]
                v[s, :, pos, :] = vn[off[s] + i]
    return k, v


def commit(ctx_lens, accept_len) -> np.ndarray:
    """ctx_s + accept_len_s + 1."""
    return (np.asarray(ctx_lens, dtype=np.int64) + np.asarray(accept_len, dtype=np.int64) + 1).astype(np.int32)


@dataclass
class StepResult:
    outs: List[np.ndarray]          # per layer [total_q, Hq, D] fp64
    k_caches: List[np.ndarray]      # per layer, after the append
    v_caches: List[np.ndarray]
    accept: object                  # oracle AcceptResult
    ctx_lens: np.ndarray            # after the commit


def verify_step(layers, ctx_lens, block_lens, q_offsets, mask_mode, target, draft, draft_tokens,
                uniforms, temperature, band=1e-5, scale=0.0) -> StepResult:
    """``layers``: sequence of dicts with q, k_new, v_new, k_cache, v_cache (host arrays)."""
    outs, ks, vs = [], [], []
    for L in layers:
        k, v = kv_append(L["k_cache"], L["v_cache"], L["k_new"], L["v_new"], ctx_lens, q_offsets)
        outs.append(_block_attn(_np(L["q"]), k, v, ctx_lens, block_lens, q_offsets, mask_mode, scale))
        ks.append(k)
        vs.append(v)
    res = _accept(target, draft, draft_tokens, uniforms, block_lens, q_offsets, temperature, band=band)
    return StepResult(outs, ks, vs, res, commit(ctx_lens, res.accept_len))
