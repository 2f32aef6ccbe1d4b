"""ctypes binding of libsdblock.so: argument marshalling only.

Every step of the computation runs in the HIP kernels behind the C ABI declared in
include/sd_block.h.  torch is used for device memory and streams.  There is no
fallback: if the library is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsdblock.so")

SD_OK, SD_ERR_INVALID_ARG, SD_ERR_UNSUPPORTED, SD_ERR_WORKSPACE, SD_ERR_HIP = range(5)
SD_F32, SD_BF16 = 0, 1
SD_MASK_CAUSAL_IN_BLOCK, SD_MASK_BIDIR_IN_BLOCK = 0, 1

EXPORTS = ["sd_last_error", "sd_version", "sd_block_attn_workspace_size", "sd_block_attn",
           "sd_accept_workspace_size", "sd_accept", "sd_kv_append", "sd_commit", "sd_verify_step_workspace_size",
           "sd_verify_step", "sd_policy_workspace_size", "sd_block_size_policy", "sd_block_attn_paged",
           "sd_kv_append_paged", "sd_survival_tau", "sd_survival_sample", "sd_block_attn_append",
           "sd_check_attn_inputs", "sd_check_accept_inputs", "sd_accept_noalloc", "sd_accept_set_path"]

# bytes of the fixed device scratch behind sd_accept_noalloc (SD_ACCEPT_NOALLOC_SCRATCH_BYTES)
ACCEPT_NOALLOC_SCRATCH_BYTES = 4 << 20

SD_CHECK_CTX, SD_CHECK_BLOCK, SD_CHECK_OFFSETS, SD_CHECK_TOKEN, SD_CHECK_UNIFORM = 1, 2, 4, 8, 16


class SdAttnShape(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("max_kv_len", ctypes.c_int32), ("total_q", ctypes.c_int32),
                ("max_ctx", ctypes.c_int32), ("max_block", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("scale", ctypes.c_float)]


class SdAcceptShape(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("vocab", ctypes.c_int32), ("total_q", ctypes.c_int32),
                ("max_block", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class SdPolicyShape(ctypes.Structure):
    _fields_ = [("num_prompts", ctypes.c_int32), ("vocab", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("radius", ctypes.c_int32), ("base_block", ctypes.c_int32), ("logits_dtype", ctypes.c_int32)]


class SdSurvivalShape(ctypes.Structure):
    _fields_ = [("num_samples", ctypes.c_int32), ("max_pos", ctypes.c_int32), ("num_cands", ctypes.c_int32),
                ("train_block", ctypes.c_int32), ("alpha", ctypes.c_double), ("cands", ctypes.c_int32 * 64)]


class SdLayerBuffers(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p),
                ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p), ("out", ctypes.c_void_p)]


class SdError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"sdblock error {code}: {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load libsdblock.so (built in-tree by build_lib.py); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_31315_amd.build_lib` "
                               "or __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, I, Z = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.sd_last_error.restype = ctypes.c_char_p
        L.sd_last_error.argtypes = []
        L.sd_version.restype = ctypes.c_char_p
        L.sd_version.argtypes = []
        L.sd_block_attn_workspace_size.restype = ctypes.c_int
        L.sd_block_attn_workspace_size.argtypes = [ctypes.POINTER(SdAttnShape), ctypes.POINTER(Z)]
        L.sd_block_attn.restype = ctypes.c_int
        L.sd_block_attn.argtypes = [ctypes.POINTER(SdAttnShape), P, P, P, P, P, P, I, P, P, Z, P]
        L.sd_accept_workspace_size.restype = ctypes.c_int
        L.sd_accept_workspace_size.argtypes = [ctypes.POINTER(SdAcceptShape), ctypes.c_float, ctypes.POINTER(Z)]
        L.sd_accept.restype = ctypes.c_int
        L.sd_accept.argtypes = [ctypes.POINTER(SdAcceptShape), P, P, P, P, P, P, ctypes.c_float, P, P, P, Z, P]
        L.sd_accept_noalloc.restype = ctypes.c_int
        L.sd_accept_noalloc.argtypes = [ctypes.POINTER(SdAcceptShape), P, P, P, P, P, P, ctypes.c_float, P, P, P]
        L.sd_block_attn_paged.restype = ctypes.c_int
        L.sd_block_attn_paged.argtypes = [ctypes.POINTER(SdAttnShape), I, I, I, P, P, P, P, P, P, P, I, P, P, Z, P]
        L.sd_block_attn_append.restype = ctypes.c_int
        L.sd_block_attn_append.argtypes = [ctypes.POINTER(SdAttnShape), P, P, P, P, P, P, P, P, I, P, P, Z, P]
        L.sd_kv_append_paged.restype = ctypes.c_int
        L.sd_kv_append_paged.argtypes = [ctypes.POINTER(SdAttnShape), I, I, I, P, P, P, P, P, P, P, P]
        L.sd_kv_append.restype = ctypes.c_int
        L.sd_kv_append.argtypes = [ctypes.POINTER(SdAttnShape), P, P, P, P, P, P, P]
        L.sd_commit.restype = ctypes.c_int
        L.sd_commit.argtypes = [I, P, P, P]
        L.sd_verify_step_workspace_size.restype = ctypes.c_int
        L.sd_verify_step_workspace_size.argtypes = [ctypes.POINTER(SdAttnShape), ctypes.POINTER(SdAcceptShape),
                                                    ctypes.c_float, ctypes.POINTER(Z)]
        L.sd_policy_workspace_size.restype = ctypes.c_int
        L.sd_policy_workspace_size.argtypes = [ctypes.POINTER(SdPolicyShape), ctypes.POINTER(Z)]
        L.sd_block_size_policy.restype = ctypes.c_int
        L.sd_block_size_policy.argtypes = [ctypes.POINTER(SdPolicyShape), P, P, P, P, P, P, P, P, P, P, Z, P]
        L.sd_verify_step.restype = ctypes.c_int
        L.sd_verify_step.argtypes = [ctypes.POINTER(SdAttnShape), I, ctypes.POINTER(SdLayerBuffers), P, P, P, I,
                                     ctypes.POINTER(SdAcceptShape), P, P, P, P, ctypes.c_float, P, P, P, Z, P]
        L.sd_survival_tau.restype = ctypes.c_int
        L.sd_survival_tau.argtypes = [ctypes.POINTER(SdSurvivalShape), P, P, P, P, P, P, P]
        L.sd_survival_sample.restype = ctypes.c_int
        L.sd_survival_sample.argtypes = [ctypes.POINTER(SdSurvivalShape), P, ctypes.c_uint64, I, P, P, P]
        L.sd_check_attn_inputs.restype = ctypes.c_int
        L.sd_check_attn_inputs.argtypes = [ctypes.POINTER(SdAttnShape), P, P, P, P, P]
        L.sd_accept_set_path.restype = ctypes.c_int
        L.sd_accept_set_path.argtypes = [I, I]
        L.sd_check_accept_inputs.restype = ctypes.c_int
        L.sd_check_accept_inputs.argtypes = [ctypes.POINTER(SdAcceptShape), P, P, P, P, ctypes.c_float, P, P]
        _lib = L
    return _lib


def _check(rc: int) -> None:
    if rc != SD_OK:
        raise SdError(rc, lib().sd_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    """A tensor's device address for a c_void_p argument (every entry point declares its
    argument types, so ctypes converts the integer; None is NULL)."""
    return t.data_ptr() if t is not None else None


# The current stream's handle without building a torch.cuda.Stream object (about 3 us of host
# time per call otherwise); the public accessor where this torch has no raw one.
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_cur_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        if _raw_stream is not None and _cur_device is not None:
            return ctypes.c_void_p(_raw_stream(_cur_device()))
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SD_BF16
    if t.dtype == torch.float32:
        return SD_F32
    raise TypeError(f"unsupported dtype {t.dtype}; use bfloat16 or float32")


def _shape(t: Optional[torch.Tensor], name: str, *dims) -> None:
    """t must have len(dims) dimensions; an int entry must equal that size, None is free.
    Checked before any pointer reaches the library: a wrongly sized buffer would make the
    kernels read or write outside it."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    shp = t.shape
    ok = len(shp) == len(dims)
    if ok:
        for n, d in zip(shp, dims):
            if d is not None and n != d:
                ok = False
                break
    if not ok:
        want = "[" + ", ".join("*" if d is None else str(d) for d in dims) + "]"
        raise ValueError(f"{name} has shape {list(shp)}, expected {want}")


def _lens_shapes(S: int, **named) -> None:
    """Per-sequence int32 arrays: q_offsets has S + 1 entries, the others S."""
    for name, t in named.items():
        _shape(t, name, S + 1 if name == "q_offsets" else S)


def _need(t: torch.Tensor, name: str, dtype=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


class Workspace:
    """A device scratch buffer per device, grown on demand; calls sharing it must be
    ordered (one stream)."""

    def __init__(self):
        self._bufs = {}

    def get(self, nbytes: int, device: torch.device) -> torch.Tensor:
        key = device.index if device.index is not None else torch.cuda.current_device()
        buf = self._bufs.get(key)
        if buf is None or buf.numel() < nbytes:
            # 256-byte alignment comes from the caching allocator
            buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
            self._bufs[key] = buf
        return buf


_default_ws = Workspace()


def attn_shape(q: torch.Tensor, k_cache: torch.Tensor, max_ctx: int, max_block: int, scale: float = 0.0
               ) -> SdAttnShape:
    S, Hkv, Lmax, D = k_cache.shape
    return SdAttnShape(S, q.shape[1], Hkv, D, Lmax, q.shape[0], int(max_ctx), int(max_block), _dtype_code(q),
                       float(scale))


# Shape structs of the per-step calls, by their field values: the library only reads them, so
# one struct serves every call of that shape (building one costs about a microsecond of host
# time).  Bounded: cleared when it grows past _SHAPE_CACHE_MAX entries.
_SHAPE_CACHE_MAX = 256
_shape_cache: dict = {}


def _cached_shape(key, make):
    sh = _shape_cache.get(key)
    if sh is None:
        if len(_shape_cache) >= _SHAPE_CACHE_MAX:
            _shape_cache.clear()
        sh = _shape_cache[key] = make()
    return sh


def attn_workspace_size(shape: SdAttnShape) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().sd_block_attn_workspace_size(ctypes.byref(shape), ctypes.byref(n)))
    return n.value


def block_attn(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, ctx_lens: torch.Tensor,
               block_lens: torch.Tensor, q_offsets: torch.Tensor, mask_mode: int, *, max_ctx: int, max_block: int,
               scale: float = 0.0, out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
               stream=None) -> torch.Tensor:
    """Block attention (sd_block_attn).  q [total_q, Hq, D]; caches [S, Hkv, Lmax, D];
    ctx_lens, block_lens [S] and q_offsets [S+1] int32 on the device; max_ctx and
    max_block are host-known bounds of the device lengths."""
    _shape(k_cache, "k_cache", None, None, None, None)
    S, Hkv, Lmax, D = k_cache.shape
    _shape(q, "q", None, None, D)
    _shape(v_cache, "v_cache", S, Hkv, Lmax, D)
    _lens_shapes(S, ctx_lens=ctx_lens, block_lens=block_lens, q_offsets=q_offsets)
    if out is not None:
        _shape(out, "out", *q.shape)
    dev = q.device
    _need(q, "q", device=dev)
    _need(k_cache, "k_cache", q.dtype, dev)
    _need(v_cache, "v_cache", q.dtype, dev)
    for name, t in (("ctx_lens", ctx_lens), ("block_lens", block_lens), ("q_offsets", q_offsets)):
        _need(t, name, torch.int32, dev)
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", q.dtype, dev)
    shape = _cached_shape(("attn", S, q.shape[1], Hkv, D, Lmax, q.shape[0], int(max_ctx), int(max_block), q.dtype,
                           float(scale)), lambda: attn_shape(q, k_cache, max_ctx, max_block, scale))
    if workspace is None:  # a caller's workspace is checked against the need by the library
        workspace = _default_ws.get(attn_workspace_size(shape), dev)
    _check(lib().sd_block_attn(ctypes.byref(shape), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(ctx_lens),
                               _ptr(block_lens), _ptr(q_offsets), int(mask_mode), _ptr(out), _ptr(workspace),
                               workspace.numel() * workspace.element_size(), _stream(stream)))
    return out


def block_attn_append(q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor, k_cache: torch.Tensor,
                      v_cache: torch.Tensor, ctx_lens: torch.Tensor, block_lens: torch.Tensor, q_offsets: torch.Tensor,
                      mask_mode: int, *, max_ctx: int, max_block: int, scale: float = 0.0,
                      out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    """Block attention with the block's keys/values read from k_new, v_new [total_q, Hkv, D] and
    written into the caches by the same launch (sd_block_attn_append); bf16."""
    _shape(k_cache, "k_cache", None, None, None, None)
    S, Hkv, Lmax, D = k_cache.shape
    _shape(q, "q", None, None, D)
    _shape(v_cache, "v_cache", S, Hkv, Lmax, D)
    _shape(k_new, "k_new", q.shape[0], Hkv, D)
    _shape(v_new, "v_new", q.shape[0], Hkv, D)
    _lens_shapes(S, ctx_lens=ctx_lens, block_lens=block_lens, q_offsets=q_offsets)
    if out is not None:
        _shape(out, "out", *q.shape)
    dev = q.device
    _need(q, "q", torch.bfloat16, dev)
    for name, t in (("k_new", k_new), ("v_new", v_new), ("k_cache", k_cache), ("v_cache", v_cache)):
        _need(t, name, torch.bfloat16, dev)
    for name, t in (("ctx_lens", ctx_lens), ("block_lens", block_lens), ("q_offsets", q_offsets)):
        _need(t, name, torch.int32, dev)
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", q.dtype, dev)
    shape = attn_shape(q, k_cache, max_ctx, max_block, scale)
    nbytes = attn_workspace_size(shape)
    if workspace is None:
        workspace = _default_ws.get(nbytes, dev)
    _check(lib().sd_block_attn_append(ctypes.byref(shape), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache),
                                      _ptr(v_cache), _ptr(ctx_lens), _ptr(block_lens), _ptr(q_offsets),
                                      int(mask_mode), _ptr(out), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), _stream(stream)))
    return out


def block_attn_paged(q: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor, block_table: torch.Tensor,
                     ctx_lens: torch.Tensor, block_lens: torch.Tensor, q_offsets: torch.Tensor, mask_mode: int, *,
                     max_ctx: int, max_block: int, scale: float = 0.0, out: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Block attention over paged caches (sd_block_attn_paged).  k_pages, v_pages
    [num_pages, Hkv, page_size, D] bf16; block_table [S, max_pages] int32 on the device."""
    _shape(k_pages, "k_pages", None, None, None, None)
    _shape(v_pages, "v_pages", *k_pages.shape)
    _shape(q, "q", None, None, k_pages.shape[3])
    _shape(block_table, "block_table", None, None)
    _lens_shapes(block_table.shape[0], ctx_lens=ctx_lens, block_lens=block_lens, q_offsets=q_offsets)
    if out is not None:
        _shape(out, "out", *q.shape)
    dev = q.device
    _need(q, "q", torch.bfloat16, dev)
    _need(k_pages, "k_pages", torch.bfloat16, dev)
    _need(v_pages, "v_pages", torch.bfloat16, dev)
    for name, t in (("block_table", block_table), ("ctx_lens", ctx_lens), ("block_lens", block_lens),
                    ("q_offsets", q_offsets)):
        _need(t, name, torch.int32, dev)
    num_pages, Hkv, page_size, D = k_pages.shape
    S, max_pages = block_table.shape
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", q.dtype, dev)
    shape = SdAttnShape(S, q.shape[1], Hkv, D, max_pages * page_size, q.shape[0], int(max_ctx), int(max_block),
                        SD_BF16, float(scale))
    nbytes = attn_workspace_size(shape)
    if workspace is None:
        workspace = _default_ws.get(nbytes, dev)
    _check(lib().sd_block_attn_paged(ctypes.byref(shape), page_size, num_pages, max_pages, _ptr(block_table), _ptr(q),
                                     _ptr(k_pages), _ptr(v_pages), _ptr(ctx_lens), _ptr(block_lens), _ptr(q_offsets),
                                     int(mask_mode), _ptr(out), _ptr(workspace),
                                     workspace.numel() * workspace.element_size(), _stream(stream)))
    return out


def kv_append_paged(k_new: torch.Tensor, v_new: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor,
                    block_table: torch.Tensor, ctx_lens: torch.Tensor, q_offsets: torch.Tensor, stream=None) -> None:
    """sd_kv_append into page pools [num_pages, Hkv, page_size, D] through block_table [S, max_pages]."""
    _shape(k_pages, "k_pages", None, None, None, None)
    _shape(v_pages, "v_pages", *k_pages.shape)
    _shape(k_new, "k_new", None, k_pages.shape[1], k_pages.shape[3])
    _shape(v_new, "v_new", *k_new.shape)
    _shape(block_table, "block_table", None, None)
    _lens_shapes(block_table.shape[0], ctx_lens=ctx_lens, q_offsets=q_offsets)
    dev = k_new.device
    _need(k_new, "k_new", device=dev)
    _need(v_new, "v_new", k_new.dtype, dev)
    _need(k_pages, "k_pages", k_new.dtype, dev)
    _need(v_pages, "v_pages", k_new.dtype, dev)
    for name, t in (("block_table", block_table), ("ctx_lens", ctx_lens), ("q_offsets", q_offsets)):
        _need(t, name, torch.int32, dev)
    num_pages, Hkv, page_size, D = k_pages.shape
    S, max_pages = block_table.shape
    shape = SdAttnShape(S, Hkv, Hkv, D, max_pages * page_size, k_new.shape[0], 0, 1, _dtype_code(k_new), 0.0)
    _check(lib().sd_kv_append_paged(ctypes.byref(shape), page_size, num_pages, max_pages, _ptr(block_table),
                                    _ptr(k_new), _ptr(v_new), _ptr(k_pages), _ptr(v_pages), _ptr(ctx_lens),
                                    _ptr(q_offsets), _stream(stream)))


def accept_shape(target_logits: torch.Tensor, num_seqs: int, max_block: int) -> SdAcceptShape:
    return SdAcceptShape(int(num_seqs), target_logits.shape[1], target_logits.shape[0], int(max_block),
                         _dtype_code(target_logits))


def accept_workspace_size(shape: SdAcceptShape, temperature: float) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().sd_accept_workspace_size(ctypes.byref(shape), float(temperature), ctypes.byref(n)))
    return n.value


def _accept_checks(target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets, temperature,
                   accept_len, next_token) -> int:
    """Shape, dtype and device checks of an acceptance call; returns S."""
    _shape(block_lens, "block_lens", None)
    S = block_lens.shape[0]
    _shape(target_logits, "target_logits", None, None)
    total_q, V = target_logits.shape
    _lens_shapes(S, q_offsets=q_offsets)
    _shape(draft_tokens, "draft_tokens", None)
    if draft_tokens.shape[0] < total_q - S:
        raise ValueError(f"draft_tokens has {draft_tokens.shape[0]} entries, needs total_q - S = {total_q - S}")
    # no draft row exists where every block holds only its anchor (total_q = S): then
    # draft_logits may be None
    need_draft = temperature > 0 and (draft_logits is not None or total_q > S)
    if need_draft:
        _shape(draft_logits, "draft_logits", total_q - S, V)
    if temperature > 0:
        _shape(uniforms, "uniforms", total_q)
    for name, t in (("accept_len", accept_len), ("next_token", next_token)):
        if t is not None:
            _shape(t, name, S)
    dev = target_logits.device
    _need(target_logits, "target_logits", device=dev)
    if need_draft:
        _need(draft_logits, "draft_logits", target_logits.dtype, dev)
    if temperature > 0:
        _need(uniforms, "uniforms", torch.float32, dev)
    for name, t in (("draft_tokens", draft_tokens), ("block_lens", block_lens), ("q_offsets", q_offsets)):
        _need(t, name, torch.int32, dev)
    for name, t in (("accept_len", accept_len), ("next_token", next_token)):
        if t is not None:
            _need(t, name, torch.int32, dev)
    return S


def accept(target_logits: torch.Tensor, draft_logits: Optional[torch.Tensor], draft_tokens: torch.Tensor,
           uniforms: Optional[torch.Tensor], block_lens: torch.Tensor, q_offsets: torch.Tensor, temperature: float,
           *, max_block: int, accept_len: Optional[torch.Tensor] = None, next_token: Optional[torch.Tensor] = None,
           workspace: Optional[torch.Tensor] = None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Speculative acceptance (sd_accept).  Returns device int32 (accept_len[S], next_token[S])."""
    S = _accept_checks(target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets, temperature,
                       accept_len, next_token)
    dev = target_logits.device
    if accept_len is None:
        accept_len = torch.empty(S, dtype=torch.int32, device=dev)
    if next_token is None:
        next_token = torch.empty(S, dtype=torch.int32, device=dev)
    shape = _cached_shape(("accept", S, target_logits.shape[1], target_logits.shape[0], int(max_block),
                           target_logits.dtype), lambda: accept_shape(target_logits, S, max_block))
    if workspace is None:  # a caller's workspace is checked against the need by the library
        workspace = _default_ws.get(accept_workspace_size(shape, temperature), dev)
    _check(lib().sd_accept(ctypes.byref(shape), _ptr(target_logits),
                           _ptr(draft_logits if temperature > 0 else None), _ptr(draft_tokens),
                           _ptr(uniforms if temperature > 0 else None), _ptr(block_lens), _ptr(q_offsets),
                           float(temperature), _ptr(accept_len), _ptr(next_token), _ptr(workspace),
                           workspace.numel() * workspace.element_size(), _stream(stream)))
    return accept_len, next_token


def accept_noalloc(target_logits: torch.Tensor, draft_logits: Optional[torch.Tensor], draft_tokens: torch.Tensor,
                   uniforms: Optional[torch.Tensor], block_lens: torch.Tensor, q_offsets: torch.Tensor,
                   temperature: float, *, max_block: int, accept_len: torch.Tensor, next_token: torch.Tensor,
                   stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """sd_accept_noalloc: acceptance into caller-given accept_len[S], next_token[S], with the
    library's fixed device scratch instead of a workspace (the call allocates nothing)."""
    S = _accept_checks(target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets, temperature,
                       accept_len, next_token)
    shape = accept_shape(target_logits, S, max_block)
    _check(lib().sd_accept_noalloc(ctypes.byref(shape), _ptr(target_logits),
                                   _ptr(draft_logits if temperature > 0 else None), _ptr(draft_tokens),
                                   _ptr(uniforms if temperature > 0 else None), _ptr(block_lens), _ptr(q_offsets),
                                   float(temperature), _ptr(accept_len), _ptr(next_token), _stream(stream)))
    return accept_len, next_token


def accept_set_path(mode: int, spin_limit: int = 0) -> None:
    """sd_accept_set_path (a test hook): mode 0 lets acceptance run as one launch where the
    shape, workspace and stream allow it, mode 1 always uses the multi-launch path; spin_limit
    bounds the single launch's waits (<= 0: the library default)."""
    _check(lib().sd_accept_set_path(int(mode), int(spin_limit)))


def check_attn_inputs(ctx_lens: torch.Tensor, block_lens: torch.Tensor, q_offsets: torch.Tensor, *, total_q: int,
                      max_ctx: int, max_block: int, status: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    """sd_check_attn_inputs: device int32 [3] = (OR of SD_CHECK_* bits, first offending
    sequence or -1, number of offending sequences)."""
    _shape(block_lens, "block_lens", None)
    _lens_shapes(block_lens.shape[0], ctx_lens=ctx_lens, q_offsets=q_offsets)
    if status is not None:
        _shape(status, "status", 3)
    dev = block_lens.device
    for name, t in (("ctx_lens", ctx_lens), ("block_lens", block_lens), ("q_offsets", q_offsets)):
        _need(t, name, torch.int32, dev)
    if status is None:
        status = torch.empty(3, dtype=torch.int32, device=dev)
    _need(status, "status", torch.int32, dev)
    shape = SdAttnShape(num_seqs=block_lens.shape[0], num_q_heads=1, num_kv_heads=1, head_dim=128,
                        max_kv_len=max_ctx + max_block, total_q=total_q, max_ctx=max_ctx, max_block=max_block,
                        dtype=SD_BF16, scale=0.0)
    _check(lib().sd_check_attn_inputs(ctypes.byref(shape), _ptr(ctx_lens), _ptr(block_lens), _ptr(q_offsets),
                                      _ptr(status), _stream(stream)))
    return status


def check_accept_inputs(draft_tokens: torch.Tensor, uniforms: Optional[torch.Tensor], block_lens: torch.Tensor,
                        q_offsets: torch.Tensor, temperature: float, *, vocab: int, total_q: int, max_block: int,
                        status: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """sd_check_accept_inputs: device int32 [3], as check_attn_inputs."""
    _shape(block_lens, "block_lens", None)
    S = block_lens.shape[0]
    _lens_shapes(S, q_offsets=q_offsets)
    _shape(draft_tokens, "draft_tokens", None)
    if draft_tokens.shape[0] < total_q - S:
        raise ValueError(f"draft_tokens has {draft_tokens.shape[0]} entries, needs total_q - S = {total_q - S}")
    if temperature > 0:
        _shape(uniforms, "uniforms", total_q)
    if status is not None:
        _shape(status, "status", 3)
    dev = block_lens.device
    for name, t in (("draft_tokens", draft_tokens), ("block_lens", block_lens), ("q_offsets", q_offsets)):
        _need(t, name, torch.int32, dev)
    if temperature > 0:
        _need(uniforms, "uniforms", torch.float32, dev)
    if status is None:
        status = torch.empty(3, dtype=torch.int32, device=dev)
    _need(status, "status", torch.int32, dev)
    shape = SdAcceptShape(num_seqs=block_lens.shape[0], vocab=vocab, total_q=total_q, max_block=max_block,
                          dtype=SD_BF16)
    _check(lib().sd_check_accept_inputs(ctypes.byref(shape), _ptr(draft_tokens),
                                        _ptr(uniforms if temperature > 0 else None), _ptr(block_lens),
                                        _ptr(q_offsets), float(temperature), _ptr(status), _stream(stream)))
    return status


def kv_append(k_new: torch.Tensor, v_new: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
              ctx_lens: torch.Tensor, q_offsets: torch.Tensor, stream=None) -> None:
    """Write the block's keys and values into the caches at rows [ctx_s, ctx_s + B_s) (sd_kv_append).
    k_new, v_new [total_q, Hkv, D]; caches [S, Hkv, Lmax, D]; ctx_lens [S], q_offsets [S+1] int32."""
    _shape(k_cache, "k_cache", None, None, None, None)
    S, Hkv, Lmax, D = k_cache.shape
    _shape(v_cache, "v_cache", S, Hkv, Lmax, D)
    _shape(k_new, "k_new", None, Hkv, D)
    _shape(v_new, "v_new", *k_new.shape)
    _lens_shapes(S, ctx_lens=ctx_lens, q_offsets=q_offsets)
    dev = k_new.device
    _need(k_new, "k_new", device=dev)
    _need(v_new, "v_new", k_new.dtype, dev)
    _need(k_cache, "k_cache", k_new.dtype, dev)
    _need(v_cache, "v_cache", k_new.dtype, dev)
    _need(ctx_lens, "ctx_lens", torch.int32, dev)
    _need(q_offsets, "q_offsets", torch.int32, dev)
    S, Hkv, Lmax, D = k_cache.shape
    shape = SdAttnShape(S, Hkv, Hkv, D, Lmax, k_new.shape[0], 0, 1, _dtype_code(k_new), 0.0)
    _check(lib().sd_kv_append(ctypes.byref(shape), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
                              _ptr(ctx_lens), _ptr(q_offsets), _stream(stream)))


def commit(accept_len: torch.Tensor, ctx_lens: torch.Tensor, stream=None) -> None:
    """ctx_lens += accept_len + 1 on the device (sd_commit)."""
    _shape(ctx_lens, "ctx_lens", None)
    _shape(accept_len, "accept_len", ctx_lens.shape[0])
    _need(accept_len, "accept_len", torch.int32)
    _need(ctx_lens, "ctx_lens", torch.int32, accept_len.device)
    _check(lib().sd_commit(int(ctx_lens.shape[0]), _ptr(accept_len), _ptr(ctx_lens), _stream(stream)))


def verify_step(layers, ctx_lens: torch.Tensor, block_lens: torch.Tensor, q_offsets: torch.Tensor, mask_mode: int,
                target_logits: torch.Tensor, draft_logits: Optional[torch.Tensor], draft_tokens: torch.Tensor,
                uniforms: Optional[torch.Tensor], temperature: float, *, max_ctx: int, max_block: int,
                scale: float = 0.0, accept_len: Optional[torch.Tensor] = None,
                next_token: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """One verify step (sd_verify_step): per layer append + block attention, then acceptance,
    then commit.  `layers` is a sequence of dicts with q, k_new, v_new, k_cache, v_cache, out."""
    if len(layers) < 1:
        raise ValueError("at least one layer")
    l0 = layers[0]
    _shape(l0["k_cache"], "layers[0].k_cache", None, None, None, None)
    S, Hkv, Lmax, D = l0["k_cache"].shape
    _shape(l0["q"], "layers[0].q", None, None, D)
    total_q, Hq = l0["q"].shape[0], l0["q"].shape[1]
    for i, L_ in enumerate(layers):
        _shape(L_["q"], f"layers[{i}].q", total_q, Hq, D)
        _shape(L_["out"], f"layers[{i}].out", total_q, Hq, D)
        for key in ("k_new", "v_new"):
            _shape(L_[key], f"layers[{i}].{key}", total_q, Hkv, D)
        for key in ("k_cache", "v_cache"):
            _shape(L_[key], f"layers[{i}].{key}", S, Hkv, Lmax, D)
    _lens_shapes(S, ctx_lens=ctx_lens, block_lens=block_lens, q_offsets=q_offsets)
    _shape(target_logits, "target_logits", total_q, None)
    V = target_logits.shape[1]
    _shape(draft_tokens, "draft_tokens", None)
    if draft_tokens.shape[0] < total_q - S:
        raise ValueError(f"draft_tokens has {draft_tokens.shape[0]} entries, needs total_q - S = {total_q - S}")
    # no draft row exists where every block holds only its anchor (total_q = S): then
    # draft_logits may be None
    need_draft = temperature > 0 and (draft_logits is not None or total_q > S)
    if need_draft:
        _shape(draft_logits, "draft_logits", total_q - S, V)
    if temperature > 0:
        _shape(uniforms, "uniforms", total_q)
    for name, t in (("accept_len", accept_len), ("next_token", next_token)):
        if t is not None:
            _shape(t, name, S)
    dev = l0["q"].device
    for i, L_ in enumerate(layers):
        _need(L_["q"], f"layers[{i}].q", l0["q"].dtype, dev)
        for key in ("k_new", "v_new", "k_cache", "v_cache", "out"):
            _need(L_[key], f"layers[{i}].{key}", l0["q"].dtype, dev)
    for name, t in (("ctx_lens", ctx_lens), ("block_lens", block_lens), ("q_offsets", q_offsets),
                    ("draft_tokens", draft_tokens)):
        _need(t, name, torch.int32, dev)
    _need(target_logits, "target_logits", device=dev)
    S = block_lens.shape[0]
    ash = attn_shape(l0["q"], l0["k_cache"], max_ctx, max_block, scale)
    csh = accept_shape(target_logits, S, max_block)
    n = ctypes.c_size_t(0)
    _check(lib().sd_verify_step_workspace_size(ctypes.byref(ash), ctypes.byref(csh), float(temperature),
                                               ctypes.byref(n)))
    if workspace is None:
        workspace = _default_ws.get(n.value, dev)
    if accept_len is None:
        accept_len = torch.empty(S, dtype=torch.int32, device=dev)
    if next_token is None:
        next_token = torch.empty(S, dtype=torch.int32, device=dev)
    arr = (SdLayerBuffers * len(layers))(*[SdLayerBuffers(L_["q"].data_ptr(), L_["k_new"].data_ptr(),
                                                          L_["v_new"].data_ptr(), L_["k_cache"].data_ptr(),
                                                          L_["v_cache"].data_ptr(), L_["out"].data_ptr())
                                           for L_ in layers])
    _check(lib().sd_verify_step(ctypes.byref(ash), len(layers), arr, _ptr(ctx_lens), _ptr(block_lens), _ptr(q_offsets),
                                int(mask_mode), ctypes.byref(csh), _ptr(target_logits),
                                _ptr(draft_logits if temperature > 0 else None), _ptr(draft_tokens),
                                _ptr(uniforms if temperature > 0 else None), float(temperature), _ptr(accept_len),
                                _ptr(next_token), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                _stream(stream)))
    return accept_len, next_token


def policy_shape(last_logits: torch.Tensor, w1: torch.Tensor, w3: torch.Tensor, base_block: int) -> SdPolicyShape:
    C = w3.shape[0]
    return SdPolicyShape(last_logits.shape[0], last_logits.shape[1], w1.shape[0], (C - 1) // 2, int(base_block),
                         _dtype_code(last_logits))


def block_size_policy(last_logits: torch.Tensor, w1: torch.Tensor, b1: torch.Tensor, w2: torch.Tensor,
                      b2: torch.Tensor, w3: torch.Tensor, b3: torch.Tensor, base_block: int, *,
                      scores: Optional[torch.Tensor] = None, block_size: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Block-size policy (sd_block_size_policy): last-token logits [P, V] -> (scores [P, 2k+1] fp32,
    block sizes [P] int32).  Weights bf16 [out, in], biases fp32; 2k+1 = w3.shape[0]."""
    _shape(last_logits, "last_logits", None, None)
    P, V = last_logits.shape
    _shape(w1, "w1", None, V)
    H = w1.shape[0]
    _shape(b1, "b1", H)
    _shape(w2, "w2", H, H)
    _shape(b2, "b2", H)
    _shape(w3, "w3", None, H)
    C = w3.shape[0]
    _shape(b3, "b3", C)
    if scores is not None:
        _shape(scores, "scores", P, C)
    if block_size is not None:
        _shape(block_size, "block_size", P)
    dev = last_logits.device
    _need(last_logits, "last_logits", device=dev)
    for name, t in (("w1", w1), ("w2", w2), ("w3", w3)):
        _need(t, name, torch.bfloat16, dev)
    for name, t in (("b1", b1), ("b2", b2), ("b3", b3)):
        _need(t, name, torch.float32, dev)
    if w3.shape[0] % 2 != 1:
        raise ValueError("w3 must have 2k+1 rows")
    shape = policy_shape(last_logits, w1, w3, base_block)
    n = ctypes.c_size_t(0)
    _check(lib().sd_policy_workspace_size(ctypes.byref(shape), ctypes.byref(n)))
    if workspace is None:
        workspace = _default_ws.get(n.value, dev)
    P = last_logits.shape[0]
    if scores is None:
        scores = torch.empty(P, w3.shape[0], dtype=torch.float32, device=dev)
    if block_size is None:
        block_size = torch.empty(P, dtype=torch.int32, device=dev)
    _check(lib().sd_block_size_policy(ctypes.byref(shape), _ptr(last_logits), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2),
                                      _ptr(w3), _ptr(b3), _ptr(scores), _ptr(block_size), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), _stream(stream)))
    return scores, block_size


def survival_shape(gamma: torch.Tensor, cands, train_block: int, alpha: float) -> SdSurvivalShape:
    cands = [int(b) for b in cands]
    if not 1 <= len(cands) <= 64:
        raise ValueError("between 1 and 64 candidates")
    sh = SdSurvivalShape(gamma.shape[0], gamma.shape[1], len(cands), int(train_block), float(alpha))
    for i, b in enumerate(cands):
        sh.cands[i] = b
    return sh


def survival_tau(gamma: torch.Tensor, cands, train_block: int, alpha: float, b_hat: Optional[torch.Tensor] = None,
                 *, lipschitz: bool = True, stream=None):
    """Prefix-survival model (sd_survival_tau): gamma [N, P] fp32 -> (tau [N, C] fp64, B* [N] int32,
    regret [N] fp64 or None, L_tau [N] fp64 or None)."""
    _shape(gamma, "gamma", None, None)
    if b_hat is not None:
        _shape(b_hat, "b_hat", gamma.shape[0])
    dev = gamma.device
    _need(gamma, "gamma", torch.float32)
    if b_hat is not None:
        _need(b_hat, "b_hat", torch.int32, dev)
    shape = survival_shape(gamma, cands, train_block, alpha)
    N, C = gamma.shape[0], shape.num_cands
    tau = torch.empty(N, C, dtype=torch.float64, device=dev)
    b_star = torch.empty(N, dtype=torch.int32, device=dev)
    regret = torch.empty(N, dtype=torch.float64, device=dev) if b_hat is not None else None
    lip = torch.empty(N, dtype=torch.float64, device=dev) if lipschitz else None
    _check(lib().sd_survival_tau(ctypes.byref(shape), _ptr(gamma), _ptr(b_hat), _ptr(tau), _ptr(b_star), _ptr(regret),
                                 _ptr(lip), _stream(stream)))
    return tau, b_star, regret, lip


def survival_sample(gamma: torch.Tensor, cands, train_block: int, alpha: float, seed: int, trials: int, *,
                    hist: bool = True, stream=None):
    """Monte Carlo of the accepted length (sd_survival_sample): -> (mean [N, C] fp64,
    histogram [N, C, P + 1] int32 or None)."""
    _shape(gamma, "gamma", None, None)
    dev = gamma.device
    _need(gamma, "gamma", torch.float32)
    shape = survival_shape(gamma, cands, train_block, alpha)
    N, P, C = gamma.shape[0], gamma.shape[1], shape.num_cands
    mean = torch.empty(N, C, dtype=torch.float64, device=dev)
    h = torch.empty(N, C, P + 1, dtype=torch.int32, device=dev) if hist else None
    _check(lib().sd_survival_sample(ctypes.byref(shape), _ptr(gamma), ctypes.c_uint64(int(seed) % 2**64),
                                    int(trials), _ptr(mean), _ptr(h), _stream(stream)))
    return mean, h


def version() -> str:
    return lib().sd_version().decode()
