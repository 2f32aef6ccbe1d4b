"""CPU oracle of paged caches: a page pool [num_pages, Hkv, page_size, D] read through a
block table [S, max_pages] (logical key j of sequence s is row j % page_size of pool page
block_table[s, j // page_size]).

TEST INFRASTRUCTURE ONLY: the test suite is the only caller.  Paged attention is the
contiguous attention of ``sd_oracle.c`` over the caches gathered from the pool; the paged
append writes the block rows into the pool through the table.
"""
from __future__ import annotations

import numpy as np

from . import block_attn as _block_attn


def _np(x) -> np.ndarray:
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu").float().numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(x, dtype=np.float32)


def gather(pages, block_table) -> np.ndarray:
    """Contiguous [S, Hkv, max_pages * page_size, D] from a pool and its block table."""
    pool = _np(pages)
    table = np.asarray(block_table, dtype=np.int64)
    S, mp = table.shape
    _, Hkv, ps, D = pool.shape
    out = np.empty((S, Hkv, mp * ps, D), dtype=np.float32)
    for s in range(S):
        for j in range(mp):
            out[s, :, j * ps:(j + 1) * ps, :] = pool[table[s, j]]
    return out


def block_attn_paged(q, k_pages, v_pages, block_table, ctx_lens, block_lens, q_offsets, mask_mode, scale=0.0):
    return _block_attn(_np(q), gather(k_pages, block_table), gather(v_pages, block_table), ctx_lens, block_lens,
                       q_offsets, mask_mode, scale)


def kv_append_paged(k_pages, v_pages, block_table, k_new, v_new, ctx_lens, q_offsets):
    """New pools (float32 copies) with block row i of sequence s at logical key ctx_s + i; rows
    past the table's pages or with a page id outside the pool are not written."""
    kp, vp = _np(k_pages).copy(), _np(v_pages).copy()
    kn, vn = _np(k_new), _np(v_new)
    table = np.asarray(block_table, dtype=np.int64)
    off = np.asarray(q_offsets, dtype=np.int64)
    ps = kp.shape[2]
    for s in range(table.shape[0]):
        for i in range(int(off[s + 1] - off[s])):
            pos = int(ctx_lens[s]) + i
            j = pos // ps
            if pos < 0 or j >= table.shape[1]:
                continue
            pg = int(table[s, j])
            if 0 <= pg < kp.shape[0]:
                kp[pg, :, pos % ps, :] = kn[off[s] + i]
                vp[pg, :, pos % ps, :] = vn[off[s] + i]
    return kp, vp
