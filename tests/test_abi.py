"""The C ABI on the host: the library loads, exports what include/sd_block.h declares,
and rejects bad arguments with the documented status codes before touching a device."""
import ctypes
import os
import re

import pytest

from paper_2606_31315_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sd_block.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sd_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = L.lib()
    names = declared_functions()
    assert set(names) == set(L.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), f"missing export {n}"
    assert L.version().startswith("sdblock")


def good_attn_shape(**kw):
    sh = L.SdAttnShape(num_seqs=2, num_q_heads=32, num_kv_heads=8, head_dim=128, max_kv_len=4200, total_q=20,
                       max_ctx=4096, max_block=16, dtype=L.SD_BF16, scale=0.0)
    for k, v in kw.items():
        setattr(sh, k, v)
    return sh


def attn_ws(sh):
    n = ctypes.c_size_t(0)
    rc = L.lib().sd_block_attn_workspace_size(ctypes.byref(sh), ctypes.byref(n))
    return rc, n.value


def test_attn_workspace_size_valid():
    rc, n = attn_ws(good_attn_shape())
    assert rc == L.SD_OK and n > 0
    rc2, n2 = attn_ws(good_attn_shape(num_seqs=4, total_q=40))
    assert rc2 == L.SD_OK and n2 >= n


@pytest.mark.parametrize("field,value,code", [
    ("num_seqs", -1, L.SD_ERR_INVALID_ARG),
    ("num_q_heads", 0, L.SD_ERR_INVALID_ARG),
    ("num_kv_heads", 5, L.SD_ERR_INVALID_ARG),       # 32 % 5 != 0
    ("head_dim", 96, L.SD_ERR_UNSUPPORTED),
    ("max_block", 0, L.SD_ERR_INVALID_ARG),
    ("max_block", 65, L.SD_ERR_INVALID_ARG),
    ("max_kv_len", 4000, L.SD_ERR_INVALID_ARG),      # max_ctx + max_block > Lmax
    ("total_q", 33, L.SD_ERR_INVALID_ARG),           # > S * max_block
    ("dtype", 7, L.SD_ERR_INVALID_ARG),
    ("scale", float("nan"), L.SD_ERR_INVALID_ARG),
    ("scale", -1.0, L.SD_ERR_INVALID_ARG),
])
def test_attn_shape_errors(field, value, code):
    rc, _ = attn_ws(good_attn_shape(**{field: value}))
    assert rc == code
    assert L.lib().sd_last_error().decode()


def test_attn_group_too_large():
    rc, _ = attn_ws(good_attn_shape(num_q_heads=64, num_kv_heads=1, max_block=8, total_q=16))  # 64*8 > 256 rows
    assert rc == L.SD_ERR_UNSUPPORTED


def call_attn(sh, ptrs=None, mask=0, ws_bytes=None, ws_ptr=256):
    P = ctypes.c_void_p
    p = dict(q=4096, k=8192, v=12288, ctx=16, bl=32, off=48, out=16384)
    if ptrs:
        p.update(ptrs)
    if ws_bytes is None:
        ws_bytes = attn_ws(sh)[1]
    return L.lib().sd_block_attn(ctypes.byref(sh) if sh is not None else None, P(p["q"]), P(p["k"]), P(p["v"]),
                                 P(p["ctx"]), P(p["bl"]), P(p["off"]), mask, P(p["out"]), P(ws_ptr), ws_bytes, None)


def test_attn_call_errors_without_device():
    # every one of these is rejected on the host: the fake addresses are never dereferenced
    assert L.lib().sd_block_attn(None, *([None] * 6), 0, None, None, 0, None) == L.SD_ERR_INVALID_ARG
    sh = good_attn_shape()
    assert call_attn(sh, mask=2) == L.SD_ERR_INVALID_ARG
    assert call_attn(sh, ptrs=dict(q=0)) == L.SD_ERR_INVALID_ARG
    assert call_attn(sh, ptrs=dict(k=8200)) == L.SD_ERR_INVALID_ARG        # misaligned cache
    assert call_attn(sh, ws_ptr=300) == L.SD_ERR_INVALID_ARG               # misaligned workspace
    assert call_attn(sh, ws_bytes=1024) == L.SD_ERR_WORKSPACE
    # empty batches succeed without any device work
    assert call_attn(good_attn_shape(num_seqs=0, total_q=0)) == L.SD_OK
    assert call_attn(good_attn_shape(total_q=0)) == L.SD_OK


def call_attn_append(sh, ptrs=None, mask=0):
    P = ctypes.c_void_p
    p = dict(q=4096, kn=20480, vn=24576, k=8192, v=12288, ctx=16, bl=32, off=48, out=16384)
    if ptrs:
        p.update(ptrs)
    return L.lib().sd_block_attn_append(ctypes.byref(sh), P(p["q"]), P(p["kn"]), P(p["vn"]), P(p["k"]), P(p["v"]),
                                        P(p["ctx"]), P(p["bl"]), P(p["off"]), mask, P(p["out"]), P(256),
                                        attn_ws(sh)[1], None)


def test_attn_append_call_errors_without_device():
    sh = good_attn_shape()
    assert call_attn_append(good_attn_shape(dtype=L.SD_F32)) == L.SD_ERR_UNSUPPORTED
    assert call_attn_append(sh, ptrs=dict(kn=0)) == L.SD_ERR_INVALID_ARG
    assert call_attn_append(sh, ptrs=dict(vn=0)) == L.SD_ERR_INVALID_ARG
    assert call_attn_append(sh, ptrs=dict(kn=20488)) == L.SD_ERR_INVALID_ARG     # misaligned new rows
    assert call_attn_append(sh, ptrs=dict(q=0)) == L.SD_ERR_INVALID_ARG
    assert call_attn_append(sh, mask=2) == L.SD_ERR_INVALID_ARG
    assert call_attn_append(good_attn_shape(total_q=0), mask=2) == L.SD_ERR_INVALID_ARG
    assert call_attn_append(good_attn_shape(total_q=0)) == L.SD_OK


def test_verify_step_checks_everything_before_enqueueing():
    """Bad acceptance or commit arguments are reported before any layer is enqueued: every
    call below returns its status on the host (the fake addresses are never dereferenced)."""
    P = ctypes.c_void_p
    ash = good_attn_shape()
    csh = L.SdAcceptShape(num_seqs=2, vocab=151936, total_q=20, max_block=16, dtype=L.SD_BF16)
    layers = (L.SdLayerBuffers * 2)(*[L.SdLayerBuffers(1 << 20, 2 << 20, 3 << 20, 4 << 20, 5 << 20, 6 << 20)
                                      for _ in range(2)])
    n = ctypes.c_size_t(0)
    assert L.lib().sd_verify_step_workspace_size(ctypes.byref(ash), ctypes.byref(csh), ctypes.c_float(1.0),
                                                 ctypes.byref(n)) == L.SD_OK

    def call(ctx=16, target=1 << 24, draft=2 << 24, tok=48, u=64, al=80, nt=96, T=1.0):
        return L.lib().sd_verify_step(ctypes.byref(ash), 2, layers, P(ctx), P(32), P(112), 0, ctypes.byref(csh),
                                      P(target), P(draft), P(tok), P(u), ctypes.c_float(T), P(al), P(nt),
                                      P(1 << 28), n.value, None)
    assert call(draft=0) == L.SD_ERR_INVALID_ARG          # T > 0 needs the draft logits
    assert call(u=0) == L.SD_ERR_INVALID_ARG
    assert call(al=0) == L.SD_ERR_INVALID_ARG
    assert call(target=(1 << 24) + 8) == L.SD_ERR_INVALID_ARG   # misaligned logits
    assert call(ctx=0) == L.SD_ERR_INVALID_ARG
    assert "ctx_lens" in L.lib().sd_last_error().decode()


def test_check_calls_errors_without_device():
    P = ctypes.c_void_p
    f = L.lib().sd_check_attn_inputs
    sh = good_attn_shape()
    assert f(None, P(16), P(32), P(48), P(64), None) == L.SD_ERR_INVALID_ARG
    assert f(ctypes.byref(good_attn_shape(max_block=65)), P(16), P(32), P(48), P(64), None) == L.SD_ERR_INVALID_ARG
    assert f(ctypes.byref(good_attn_shape(max_ctx=-1)), P(16), P(32), P(48), P(64), None) == L.SD_ERR_INVALID_ARG
    assert f(ctypes.byref(sh), P(16), P(32), P(48), None, None) == L.SD_ERR_INVALID_ARG      # no status
    assert f(ctypes.byref(sh), None, P(32), P(48), P(64), None) == L.SD_ERR_INVALID_ARG
    g = L.lib().sd_check_accept_inputs
    ash = L.SdAcceptShape(num_seqs=8, vocab=151936, total_q=124, max_block=24, dtype=L.SD_BF16)
    assert g(None, P(16), P(32), P(48), P(64), ctypes.c_float(1.0), P(80), None) == L.SD_ERR_INVALID_ARG
    assert g(ctypes.byref(ash), P(16), None, P(48), P(64), ctypes.c_float(1.0), P(80), None) == L.SD_ERR_INVALID_ARG
    assert g(ctypes.byref(ash), P(16), P(32), P(48), P(64), ctypes.c_float(-1.0), P(80), None) == L.SD_ERR_INVALID_ARG
    assert g(ctypes.byref(ash), P(16), P(32), P(48), P(64), ctypes.c_float(float("nan")), P(80), None) == \
        L.SD_ERR_INVALID_ARG
    assert g(ctypes.byref(ash), None, P(32), P(48), P(64), ctypes.c_float(0.0), P(80), None) == L.SD_ERR_INVALID_ARG
    bad_v = L.SdAcceptShape(num_seqs=8, vocab=0, total_q=124, max_block=24, dtype=L.SD_BF16)
    assert g(ctypes.byref(bad_v), P(16), P(32), P(48), P(64), ctypes.c_float(0.0), P(80), None) == \
        L.SD_ERR_INVALID_ARG
    assert L.lib().sd_last_error().decode()


def good_accept_shape(**kw):
    sh = L.SdAcceptShape(num_seqs=8, vocab=151936, total_q=124, max_block=24, dtype=L.SD_BF16)
    for k, v in kw.items():
        setattr(sh, k, v)
    return sh


def accept_ws(sh, T):
    n = ctypes.c_size_t(0)
    rc = L.lib().sd_accept_workspace_size(ctypes.byref(sh), ctypes.c_float(T), ctypes.byref(n))
    return rc, n.value


def test_accept_workspace_size_valid():
    rc0, n0 = accept_ws(good_accept_shape(), 0.0)
    rc1, n1 = accept_ws(good_accept_shape(), 1.0)
    assert rc0 == rc1 == L.SD_OK and n1 >= n0 > 0


@pytest.mark.parametrize("field,value,T,code", [
    ("num_seqs", -1, 1.0, L.SD_ERR_INVALID_ARG),
    ("vocab", 0, 1.0, L.SD_ERR_INVALID_ARG),
    ("max_block", 0, 1.0, L.SD_ERR_INVALID_ARG),
    ("max_block", 65, 0.0, L.SD_ERR_INVALID_ARG),
    ("total_q", 7, 0.0, L.SD_ERR_INVALID_ARG),        # fewer rows than sequences
    ("total_q", 8 * 24 + 1, 0.0, L.SD_ERR_INVALID_ARG),
    ("dtype", 3, 0.0, L.SD_ERR_INVALID_ARG),
    ("vocab", 1000, -1.0, L.SD_ERR_INVALID_ARG),
    ("vocab", 1000, float("inf"), L.SD_ERR_INVALID_ARG),
    ("vocab", 1000, float("nan"), L.SD_ERR_INVALID_ARG),
])
def test_accept_shape_errors(field, value, T, code):
    rc, _ = accept_ws(good_accept_shape(**{field: value}), T)
    assert rc == code


def call_accept(sh, T, ptrs=None, ws_bytes=None, ws_ptr=256):
    P = ctypes.c_void_p
    p = dict(t=4096, d=8192, tok=16, u=32, bl=48, off=64, al=80, nt=96)
    if ptrs:
        p.update(ptrs)
    if ws_bytes is None:
        ws_bytes = accept_ws(sh, T)[1]
    return L.lib().sd_accept(ctypes.byref(sh), P(p["t"]), P(p["d"]), P(p["tok"]), P(p["u"]), P(p["bl"]),
                             P(p["off"]), ctypes.c_float(T), P(p["al"]), P(p["nt"]), P(ws_ptr), ws_bytes, None)


def test_accept_call_errors_without_device():
    sh = good_accept_shape()
    assert call_accept(sh, 1.0, ptrs=dict(d=0)) == L.SD_ERR_INVALID_ARG    # T>0 needs draft logits
    assert call_accept(sh, 1.0, ptrs=dict(u=0)) == L.SD_ERR_INVALID_ARG    # and uniforms
    assert call_accept(sh, 0.0, ptrs=dict(tok=0)) == L.SD_ERR_INVALID_ARG
    assert call_accept(sh, 0.0, ptrs=dict(t=4100)) == L.SD_ERR_INVALID_ARG
    assert call_accept(sh, 1.0, ws_bytes=100) == L.SD_ERR_WORKSPACE
    assert call_accept(good_accept_shape(num_seqs=0, total_q=0), 1.0) == L.SD_OK


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(L, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        L.lib()


def good_survival_shape(**kw):
    sh = L.SdSurvivalShape(num_samples=100, max_pos=32, num_cands=5, train_block=16, alpha=0.01)
    for i, b in enumerate([14, 15, 16, 17, 18]):
        sh.cands[i] = b
    for k, v in kw.items():
        setattr(sh, k, v)
    return sh


def call_survival_tau(sh, gamma=4096, b_hat=0, regret=0, tau=8192, b_star=16384, lip=0):
    P = ctypes.c_void_p
    return L.lib().sd_survival_tau(ctypes.byref(sh) if sh is not None else None, P(gamma), P(b_hat), P(tau),
                                   P(b_star), P(regret), P(lip), None)


def call_survival_sample(sh, gamma=4096, trials=100, mean=8192, hist=0):
    P = ctypes.c_void_p
    return L.lib().sd_survival_sample(ctypes.byref(sh), P(gamma), ctypes.c_uint64(1), trials, P(mean), P(hist), None)


@pytest.mark.parametrize("field,value", [
    ("num_samples", -1), ("max_pos", 0), ("max_pos", 129), ("num_cands", 0), ("num_cands", 65),
    ("alpha", -0.5), ("alpha", float("inf")), ("alpha", float("nan")),
])
def test_survival_shape_errors(field, value):
    sh = good_survival_shape(**{field: value})
    assert call_survival_tau(sh) == L.SD_ERR_INVALID_ARG
    assert call_survival_sample(sh) == L.SD_ERR_INVALID_ARG
    assert L.lib().sd_last_error().decode()


def test_survival_call_errors_without_device():
    assert call_survival_tau(None) == L.SD_ERR_INVALID_ARG
    sh = good_survival_shape()
    sh.cands[2] = 15                                                   # not strictly ascending
    assert call_survival_tau(sh) == L.SD_ERR_INVALID_ARG
    sh = good_survival_shape()
    sh.cands[4] = 33                                                   # past max_pos
    assert call_survival_tau(sh) == L.SD_ERR_INVALID_ARG
    sh = good_survival_shape()
    assert call_survival_tau(sh, gamma=0) == L.SD_ERR_INVALID_ARG
    assert call_survival_tau(sh, gamma=4100) == L.SD_ERR_INVALID_ARG   # misaligned
    assert call_survival_tau(sh, b_hat=64) == L.SD_ERR_INVALID_ARG     # b_hat without regret
    assert call_survival_tau(sh, regret=64) == L.SD_ERR_INVALID_ARG    # regret without b_hat
    assert call_survival_tau(sh, tau=0) == L.SD_ERR_INVALID_ARG
    assert call_survival_sample(sh, trials=0) == L.SD_ERR_INVALID_ARG
    assert call_survival_sample(sh, trials=(1 << 30) + 1) == L.SD_ERR_INVALID_ARG
    assert call_survival_sample(sh, mean=0) == L.SD_ERR_INVALID_ARG
    # no samples: nothing to do, no device work
    assert call_survival_tau(good_survival_shape(num_samples=0), gamma=0) == L.SD_OK
    assert call_survival_sample(good_survival_shape(num_samples=0), gamma=0) == L.SD_OK


def test_accept_noalloc_rejects_shapes_beyond_its_scratch():
    """The allocation-free acceptance call refuses, before touching a device, a shape whose
    workspace exceeds the fixed scratch, and says so; a shape that fits passes its host checks."""
    big = L.SdAcceptShape(num_seqs=64, vocab=1 << 26, total_q=64 * 64, max_block=64, dtype=L.SD_BF16)
    n = ctypes.c_size_t(0)
    assert L.lib().sd_accept_workspace_size(ctypes.byref(big), 1.0, ctypes.byref(n)) == L.SD_OK
    assert n.value > L.ACCEPT_NOALLOC_SCRATCH_BYTES
    z = ctypes.c_void_p(0)
    rc = L.lib().sd_accept_noalloc(ctypes.byref(big), z, z, z, z, z, z, 1.0, z, z, z)
    assert rc == L.SD_ERR_WORKSPACE
    assert "scratch" in L.lib().sd_last_error().decode()
    # a zero-sequence call needs no device and returns SD_OK
    empty = L.SdAcceptShape(num_seqs=0, vocab=151936, total_q=0, max_block=16, dtype=L.SD_BF16)
    assert L.lib().sd_accept_noalloc(ctypes.byref(empty), z, z, z, z, z, z, 1.0, z, z, z) == L.SD_OK
    # bad arguments are reported as for sd_accept
    bad = L.SdAcceptShape(num_seqs=2, vocab=151936, total_q=1, max_block=16, dtype=L.SD_BF16)
    assert L.lib().sd_accept_noalloc(ctypes.byref(bad), z, z, z, z, z, z, 1.0, z, z, z) == L.SD_ERR_INVALID_ARG
