"""The Python binding checks every tensor's shape against the shape it passes to the C ABI
and raises before any pointer reaches the library (host only: meta tensors carry shapes and
no memory, so nothing is launched).  A correctly shaped set of meta tensors gets past the
shape checks and stops at the device check instead."""
import pytest
import torch

from paper_2606_31315_amd import _lib as L

S, HQ, HKV, D, LMAX, V = 3, 8, 2, 128, 64, 50
BL = [4, 2, 5]
TQ = sum(BL)


def meta(*shape, dtype=torch.bfloat16):
    return torch.empty(*shape, dtype=dtype, device="meta")


def i32(n):
    return meta(n, dtype=torch.int32)


def attn_args():
    return dict(q=meta(TQ, HQ, D), k_cache=meta(S, HKV, LMAX, D), v_cache=meta(S, HKV, LMAX, D),
                ctx_lens=i32(S), block_lens=i32(S), q_offsets=i32(S + 1), mask_mode=0, max_ctx=32, max_block=8)


def call_attn(**over):
    a = attn_args()
    a.update(over)
    return L.block_attn(a.pop("q"), a.pop("k_cache"), a.pop("v_cache"), a.pop("ctx_lens"), a.pop("block_lens"),
                        a.pop("q_offsets"), a.pop("mask_mode"), **a)


def expect_device_error(fn, **kw):
    with pytest.raises(ValueError, match="device tensor"):
        fn(**kw)


def expect_shape_error(fn, name, **kw):
    with pytest.raises(ValueError, match=rf"^{name} has shape|^{name} has \d+ entries"):
        fn(**kw)


def test_attn_good_shapes_reach_the_device_check():
    expect_device_error(call_attn)


@pytest.mark.parametrize("name,bad", [
    ("q", meta(TQ, HQ, 64)),                 # head_dim differs from the cache
    ("q", meta(TQ, HQ * D)),                 # wrong rank
    ("v_cache", meta(S, HKV, LMAX + 1, D)),  # v cache differs from k cache
    ("v_cache", meta(S, HKV + 1, LMAX, D)),
    ("ctx_lens", i32(S - 1)),
    ("block_lens", i32(S + 1)),
    ("q_offsets", i32(S)),                   # S + 1 entries needed
    ("out", meta(TQ - 1, HQ, D)),
])
def test_attn_rejects_bad_shapes(name, bad):
    expect_shape_error(call_attn, name, **{name: bad})


def call_append(**over):
    a = dict(q=meta(TQ, HQ, D), k_new=meta(TQ, HKV, D), v_new=meta(TQ, HKV, D), k_cache=meta(S, HKV, LMAX, D),
             v_cache=meta(S, HKV, LMAX, D), ctx_lens=i32(S), block_lens=i32(S), q_offsets=i32(S + 1))
    a.update(over)
    return L.block_attn_append(a["q"], a["k_new"], a["v_new"], a["k_cache"], a["v_cache"], a["ctx_lens"],
                               a["block_lens"], a["q_offsets"], 0, max_ctx=32, max_block=8)


def test_append_shapes():
    expect_device_error(call_append)
    expect_shape_error(call_append, "k_new", k_new=meta(TQ + 1, HKV, D))
    expect_shape_error(call_append, "v_new", v_new=meta(TQ, HKV, 64))
    expect_shape_error(call_append, "v_cache", v_cache=meta(S, HKV, LMAX, 64))


def call_paged(**over):
    a = dict(q=meta(TQ, HQ, D), k_pages=meta(20, HKV, 16, D), v_pages=meta(20, HKV, 16, D),
             block_table=meta(S, 4, dtype=torch.int32), ctx_lens=i32(S), block_lens=i32(S), q_offsets=i32(S + 1))
    a.update(over)
    return L.block_attn_paged(a["q"], a["k_pages"], a["v_pages"], a["block_table"], a["ctx_lens"], a["block_lens"],
                              a["q_offsets"], 0, max_ctx=32, max_block=8)


def test_paged_shapes():
    expect_device_error(call_paged)
    expect_shape_error(call_paged, "v_pages", v_pages=meta(19, HKV, 16, D))
    expect_shape_error(call_paged, "q", q=meta(TQ, HQ, 64))
    expect_shape_error(call_paged, "ctx_lens", ctx_lens=i32(S + 2))
    expect_shape_error(call_paged, "block_table", block_table=meta(S * 4, dtype=torch.int32))


def test_kv_append_shapes():
    def call(**over):
        a = dict(k_new=meta(TQ, HKV, D), v_new=meta(TQ, HKV, D), k_cache=meta(S, HKV, LMAX, D),
                 v_cache=meta(S, HKV, LMAX, D), ctx_lens=i32(S), q_offsets=i32(S + 1))
        a.update(over)
        return L.kv_append(**a)
    expect_device_error(call)
    expect_shape_error(call, "k_new", k_new=meta(TQ, HKV + 1, D))
    expect_shape_error(call, "v_new", v_new=meta(TQ - 1, HKV, D))
    expect_shape_error(call, "q_offsets", q_offsets=i32(S))

    def call_p(**over):
        a = dict(k_new=meta(TQ, HKV, D), v_new=meta(TQ, HKV, D), k_pages=meta(20, HKV, 16, D),
                 v_pages=meta(20, HKV, 16, D), block_table=meta(S, 4, dtype=torch.int32), ctx_lens=i32(S),
                 q_offsets=i32(S + 1))
        a.update(over)
        return L.kv_append_paged(**a)
    expect_device_error(call_p)
    expect_shape_error(call_p, "k_new", k_new=meta(TQ, HKV, 64))
    expect_shape_error(call_p, "ctx_lens", ctx_lens=i32(S - 1))


def call_accept(T=1.0, **over):
    a = dict(target_logits=meta(TQ, V), draft_logits=meta(TQ - S, V), draft_tokens=i32(TQ - S),
             uniforms=meta(TQ, dtype=torch.float32), block_lens=i32(S), q_offsets=i32(S + 1))
    a.update(over)
    return L.accept(a["target_logits"], a["draft_logits"], a["draft_tokens"], a["uniforms"], a["block_lens"],
                    a["q_offsets"], T, max_block=8, accept_len=a.get("accept_len"), next_token=a.get("next_token"))


def test_accept_shapes():
    expect_device_error(call_accept)
    expect_device_error(call_accept, T=0.0, draft_logits=None, uniforms=None)
    # T > 0: the draft tensor may be left out only where no block holds a drafted token
    expect_device_error(call_accept, target_logits=meta(S, V), draft_logits=None, draft_tokens=i32(0),
                        uniforms=meta(S, dtype=torch.float32))
    with pytest.raises(TypeError, match="draft_logits"):
        call_accept(draft_logits=None)
    expect_shape_error(call_accept, "draft_logits", draft_logits=meta(TQ, V))       # one row per draft
    expect_shape_error(call_accept, "draft_logits", draft_logits=meta(TQ - S, V + 1))
    expect_shape_error(call_accept, "uniforms", uniforms=meta(TQ - 1, dtype=torch.float32))
    expect_shape_error(call_accept, "draft_tokens", draft_tokens=i32(TQ - S - 1))
    expect_shape_error(call_accept, "q_offsets", q_offsets=i32(S))
    expect_shape_error(call_accept, "accept_len", accept_len=i32(S + 1))
    expect_shape_error(call_accept, "next_token", next_token=i32(S - 1))
    expect_shape_error(call_accept, "target_logits", target_logits=meta(TQ * V))


def test_check_inputs_shapes():
    with pytest.raises(ValueError, match="^ctx_lens has shape"):
        L.check_attn_inputs(i32(S + 1), i32(S), i32(S + 1), total_q=TQ, max_ctx=32, max_block=8)
    with pytest.raises(ValueError, match="^status has shape"):
        L.check_attn_inputs(i32(S), i32(S), i32(S + 1), total_q=TQ, max_ctx=32, max_block=8, status=i32(2))
    with pytest.raises(ValueError, match="^uniforms has shape"):
        L.check_accept_inputs(i32(TQ - S), meta(TQ + 1, dtype=torch.float32), i32(S), i32(S + 1), 1.0, vocab=V,
                              total_q=TQ, max_block=8)
    with pytest.raises(ValueError, match="device tensor"):
        L.check_accept_inputs(i32(TQ - S), meta(TQ, dtype=torch.float32), i32(S), i32(S + 1), 1.0, vocab=V,
                              total_q=TQ, max_block=8)


def test_commit_shapes():
    with pytest.raises(ValueError, match="^accept_len has shape"):
        L.commit(i32(S + 1), i32(S))


def layer(**over):
    d = dict(q=meta(TQ, HQ, D), k_new=meta(TQ, HKV, D), v_new=meta(TQ, HKV, D), k_cache=meta(S, HKV, LMAX, D),
             v_cache=meta(S, HKV, LMAX, D), out=meta(TQ, HQ, D))
    d.update(over)
    return d


def call_step(layers, **over):
    a = dict(ctx_lens=i32(S), block_lens=i32(S), q_offsets=i32(S + 1), target_logits=meta(TQ, V),
             draft_logits=meta(TQ - S, V), draft_tokens=i32(TQ - S), uniforms=meta(TQ, dtype=torch.float32))
    a.update(over)
    return L.verify_step(layers, a["ctx_lens"], a["block_lens"], a["q_offsets"], 0, a["target_logits"],
                         a["draft_logits"], a["draft_tokens"], a["uniforms"], 1.0, max_ctx=32, max_block=8)


def test_verify_step_shapes():
    expect_device_error(call_step, layers=[layer(), layer()])
    expect_shape_error(call_step, r"layers\[1\]\.out", layers=[layer(), layer(out=meta(TQ, HQ, 64))])
    expect_shape_error(call_step, r"layers\[1\]\.k_cache", layers=[layer(), layer(k_cache=meta(S, HKV, LMAX + 16, D))])
    expect_shape_error(call_step, r"layers\[0\]\.v_new", layers=[layer(v_new=meta(TQ, HKV, 64))])
    expect_shape_error(call_step, "target_logits", layers=[layer()], target_logits=meta(TQ + 1, V))
    expect_shape_error(call_step, "draft_logits", layers=[layer()], draft_logits=meta(TQ - S, V - 1))


def test_policy_shapes():
    P, VV, H, C = 2, 64, 16, 5

    def call(**over):
        a = dict(last_logits=meta(P, VV), w1=meta(H, VV), b1=meta(H, dtype=torch.float32), w2=meta(H, H),
                 b2=meta(H, dtype=torch.float32), w3=meta(C, H), b3=meta(C, dtype=torch.float32))
        a.update(over)
        return L.block_size_policy(a["last_logits"], a["w1"], a["b1"], a["w2"], a["b2"], a["w3"], a["b3"], 16,
                                   scores=a.get("scores"))
    expect_device_error(call)
    expect_shape_error(call, "w1", w1=meta(H, VV + 8))
    expect_shape_error(call, "w2", w2=meta(H, H + 8))
    expect_shape_error(call, "b3", b3=meta(C + 2, dtype=torch.float32))
    expect_shape_error(call, "scores", scores=meta(P, C + 1, dtype=torch.float32))


def test_survival_shapes():
    with pytest.raises(ValueError, match="^gamma has shape"):
        L.survival_tau(meta(32, dtype=torch.float32), [15, 16, 17], 16, 0.01)
    with pytest.raises(ValueError, match="^b_hat has shape"):
        L.survival_tau(meta(10, 32, dtype=torch.float32), [15, 16, 17], 16, 0.01, b_hat=i32(11))
