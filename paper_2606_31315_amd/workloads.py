"""Seeded synthetic inputs for block-verify attention and speculative acceptance.

This module only draws random numbers and lays them out; it holds none of the
arithmetic of the method (no attention, no softmax, no acceptance test).  Both
the HIP path and the CPU oracle read the inputs it produces.

Shapes follow the workloads the speculative step runs on: a diffusion drafter
proposes a block of B tokens per sequence in one pass and the target model
verifies the block in parallel (Sec. 2.1); the block size is picked once per
prompt from a small window around the training block size (Sec. 2.2, Finding II;
Sec. 2.4, Eq. 9), so the per-step kernels see ragged B across a batch.

Random streams: numpy PCG64 with ``SeedSequence(seed).spawn(9)`` sub-streams in
the order [ctx, B, q, K, V, target logits, draft noise, draft sampling,
uniforms].  fp32 draws are rounded to bf16 with round-to-nearest-even (torch's
cast) when the workload is bf16; both sides read the same rounded values.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

MASK_CAUSAL_IN_BLOCK = 0
MASK_BIDIR_IN_BLOCK = 1

_STREAMS = ["ctx", "B", "q", "K", "V", "target", "noise", "draft", "uniforms"]


def _streams(seed: int) -> dict:
    kids = np.random.SeedSequence(seed).spawn(len(_STREAMS))
    return {name: np.random.Generator(np.random.PCG64(k)) for name, k in zip(_STREAMS, kids)}


def _to_dtype(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    if dtype == "bf16":
        return t.to(torch.bfloat16)
    if dtype == "f32":
        return t
    raise ValueError(f"unknown dtype {dtype!r}")


def offsets_from_lens(block_lens: np.ndarray) -> np.ndarray:
    """Exclusive prefix sum of the block lengths: row range of sequence s is [off[s], off[s+1])."""
    off = np.zeros(len(block_lens) + 1, dtype=np.int32)
    off[1:] = np.cumsum(block_lens, dtype=np.int64).astype(np.int32)
    return off


@dataclass
class AttnProblem:
    """One block-attention call.

    q, out: [sum(B), Hq, D] packed ragged rows; k_cache, v_cache: [S, Hkv, Lmax, D]
    with the block's own keys/values already written at [ctx_s, ctx_s + B_s).
    Cache rows at or beyond ctx_s + B_s hold ``tail_fill`` (NaN by default) so a
    read past the valid region poisons the output instead of passing silently.
    """
    S: int
    Hq: int
    Hkv: int
    D: int
    Lmax: int
    ctx_lens: np.ndarray
    block_lens: np.ndarray
    q_offsets: np.ndarray
    q: torch.Tensor
    k_cache: torch.Tensor
    v_cache: torch.Tensor
    dtype: str
    mask_mode: int
    scale: float = 0.0  # 0 means 1/sqrt(D)
    name: str = ""

    @property
    def total_q(self) -> int:
        return int(self.q_offsets[-1])

    @property
    def max_ctx(self) -> int:
        return int(self.ctx_lens.max()) if self.S else 0

    @property
    def max_block(self) -> int:
        return int(self.block_lens.max()) if self.S else 0

    def kv_bytes(self) -> int:
        """Algorithmic K+V bytes: one read of every key/value row a query can see."""
        e = 2 if self.dtype == "bf16" else 4
        rows = int((self.ctx_lens.astype(np.int64) + self.block_lens).sum())
        return rows * self.Hkv * self.D * 2 * e

    def qo_bytes(self) -> int:
        e = 2 if self.dtype == "bf16" else 4
        return 2 * self.total_q * self.Hq * self.D * e

    def flops(self) -> int:
        """Upper bound 4*D flop per (query row, visible-or-masked key) pair, as priced in the roofline."""
        return int(sum(self.Hq * int(b) * (int(c) + int(b)) * 4 * self.D
                       for c, b in zip(self.ctx_lens, self.block_lens)))


@dataclass
class AcceptProblem:
    """One acceptance call.

    target: [sum(B), V] -- row off[s]+i is the target's next-token logits after block position i.
    draft:  [sum(B)-S, V] -- row off[s]-s+j is the drafter's logits for block position j+1 (j < B_s-1).
    draft_tokens: [sum(B)-S] int32, the drafted tokens, paired with target row j.
    uniforms: [sum(B)] fp32 in [0,1): slot off[s]+j drives acceptance test j, slot off[s]+B_s-1 the final sample.
    """
    S: int
    V: int
    block_lens: np.ndarray
    q_offsets: np.ndarray
    target: torch.Tensor
    draft: Optional[torch.Tensor]
    draft_tokens: np.ndarray
    uniforms: np.ndarray
    temperature: float
    dtype: str
    name: str = ""

    @property
    def total_q(self) -> int:
        return int(self.q_offsets[-1])

    @property
    def max_block(self) -> int:
        return int(self.block_lens.max()) if self.S else 0

    def logit_bytes(self) -> int:
        """Algorithmic bytes: one read of every target row, plus every draft row when T > 0."""
        e = 2 if self.dtype == "bf16" else 4
        rows = self.total_q + ((self.total_q - self.S) if self.temperature > 0 else 0)
        return rows * self.V * e


@dataclass
class Workload:
    name: str
    attn: Optional[AttnProblem]
    accept: dict = field(default_factory=dict)  # temperature -> AcceptProblem

    def verified_draft_tokens(self) -> int:
        p = self.attn
        return int((p.block_lens.astype(np.int64) - 1).clip(min=0).sum())


# --------------------------------------------------------------------------- #
# generic builders
# --------------------------------------------------------------------------- #

def make_attn(rs: dict, *, S, Hq, Hkv, D, ctx_lens, block_lens, dtype, mask_mode, Lmax=None,
              tail_fill=float("nan"), block_key_gain=1.0, q_gain=1.0, value_gain=1.0, name="") -> AttnProblem:
    """Attention inputs: q, K, V ~ N(0,1) (times the optional gains), rounded to ``dtype``.

    ``block_key_gain`` scales the in-block keys [ctx, ctx+B) and ``q_gain`` the
    queries; gains > 1 make in-block scores dominate so that an off-by-one in the
    in-block mask moves the output by far more than the bf16 tolerance.
    """
    ctx_lens = np.asarray(ctx_lens, dtype=np.int32)
    block_lens = np.asarray(block_lens, dtype=np.int32)
    if Lmax is None:  # capacity for the longest context plus the largest block
        Lmax = int(ctx_lens.max() + block_lens.max()) if S else 1
    off = offsets_from_lens(block_lens)
    tq = int(off[-1])
    q = rs["q"].standard_normal((tq, Hq, D), dtype=np.float32) * np.float32(q_gain)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    if dtype not in ("bf16", "f32"):
        raise ValueError(f"unknown dtype {dtype!r}")
    k = torch.full((S, Hkv, Lmax, D), tail_fill, dtype=tdt)
    v = torch.full((S, Hkv, Lmax, D), tail_fill, dtype=tdt)
    for s in range(S):
        n = int(ctx_lens[s] + block_lens[s])
        ks = rs["K"].standard_normal((Hkv, n, D), dtype=np.float32)
        vs = rs["V"].standard_normal((Hkv, n, D), dtype=np.float32)
        if block_key_gain != 1.0:
            c = int(ctx_lens[s])
            ks[:, c:n] *= np.float32(block_key_gain)
        if value_gain != 1.0:
            vs *= np.float32(value_gain)
        k[s, :, :n] = torch.from_numpy(ks).to(tdt)
        v[s, :, :n] = torch.from_numpy(vs).to(tdt)
    return AttnProblem(S=S, Hq=Hq, Hkv=Hkv, D=D, Lmax=Lmax, ctx_lens=ctx_lens, block_lens=block_lens,
                       q_offsets=off, q=_to_dtype(q, dtype), k_cache=k,
                       v_cache=v, dtype=dtype, mask_mode=mask_mode, name=name)


def _gumbel_argmax(rs_draft, logits: np.ndarray, temperature: float) -> np.ndarray:
    """Sample one token per row from the drafter: argmax at T=0 (lowest index on ties),
    else the Gumbel-max draw argmax(logits/T + G), which is distributed as the drafter's
    softmax at temperature T without forming the softmax."""
    if temperature == 0:
        return np.argmax(logits, axis=1).astype(np.int32)
    out = np.empty(logits.shape[0], dtype=np.int32)
    for r in range(logits.shape[0]):
        g = rs_draft.gumbel(size=logits.shape[1])
        out[r] = int(np.argmax(logits[r].astype(np.float64) / temperature + g))
    return out


def make_accept(rs: dict, *, block_lens, V, dtype, temperature, target_sigma, noise_sigma,
                name="", draft_logits_needed=None) -> AcceptProblem:
    """Acceptance inputs: target ~ N(0, target_sigma^2); draft row j = target row j + N(0, noise_sigma^2);
    draft tokens drawn from the drafter at ``temperature``; fp32 uniforms in [0,1)."""
    block_lens = np.asarray(block_lens, dtype=np.int32)
    S = len(block_lens)
    off = offsets_from_lens(block_lens)
    tq = int(off[-1])
    nd = tq - S
    target = rs["target"].standard_normal((tq, V), dtype=np.float32) * np.float32(target_sigma)
    t_dt = _to_dtype(target, dtype)
    t_vals = t_dt.float().numpy()
    draft = np.empty((nd, V), dtype=np.float32)
    for s in range(S):
        for j in range(int(block_lens[s]) - 1):
            draft[off[s] - s + j] = t_vals[off[s] + j] + \
                rs["noise"].standard_normal(V, dtype=np.float32) * np.float32(noise_sigma)
    d_dt = _to_dtype(draft, dtype)
    d_vals = d_dt.float().numpy()
    tokens = _gumbel_argmax(rs["draft"], d_vals, temperature)
    uniforms = rs["uniforms"].random(tq, dtype=np.float32)
    if draft_logits_needed is None:
        draft_logits_needed = temperature > 0
    return AcceptProblem(S=S, V=V, block_lens=block_lens, q_offsets=off, target=t_dt,
                         draft=d_dt if draft_logits_needed else None, draft_tokens=tokens,
                         uniforms=uniforms, temperature=float(temperature), dtype=dtype, name=name)


# --------------------------------------------------------------------------- #
# the five workloads
# --------------------------------------------------------------------------- #

RAGGED_BLOCK_SET = np.array([8, 10, 12, 14, 16, 18, 20, 24], dtype=np.int32)


def _nearest_in_set(draws: np.ndarray, allowed: np.ndarray) -> np.ndarray:
    """Element of ``allowed`` nearest to each draw; ties go to the smaller element."""
    d = np.abs(draws[:, None] - allowed[None, :].astype(np.float64))
    return allowed[np.argmin(d, axis=1)]  # argmin keeps the first (smaller) on ties


def c1_tiny(temperatures=(0.0, 1.0), seed=1001) -> Workload:
    """Tiny CPU-checkable step: 1 sequence, 4 q heads / 1 kv head, D=64, fp32, ctx 256, B=8,
    causal-in-block; acceptance over V=1024 with target ~ N(0,2^2), draft = target + N(0,0.5^2)."""
    out = Workload(name="tiny_fp32_ctx256_B8_V1024", attn=None)
    rs = _streams(seed)
    out.attn = make_attn(rs, S=1, Hq=4, Hkv=1, D=64, ctx_lens=[256], block_lens=[8], dtype="f32",
                         mask_mode=MASK_CAUSAL_IN_BLOCK, name=out.name)
    for T in temperatures:
        rs = _streams(seed)
        out.accept[T] = make_accept(rs, block_lens=[8], V=1024, dtype="f32", temperature=T,
                                    target_sigma=2.0, noise_sigma=0.5, name=out.name)
    return out


def c2_qwen3_4b_verify(temperatures=(1.0,), seed=1002, dtype="bf16") -> Workload:
    """Qwen3-4B-shaped verify step: 1 sequence, 32/8 heads, D=128, bf16, ctx 2048, B=16, causal;
    acceptance over V=151936 with target ~ N(0,3^2), draft = target + N(0,1)."""
    out = Workload(name="qwen3_4b_verify_S1_ctx2048_B16", attn=None)
    rs = _streams(seed)
    out.attn = make_attn(rs, S=1, Hq=32, Hkv=8, D=128, ctx_lens=[2048], block_lens=[16], dtype=dtype,
                         mask_mode=MASK_CAUSAL_IN_BLOCK, name=out.name)
    for T in temperatures:
        rs = _streams(seed)
        out.accept[T] = make_accept(rs, block_lens=[16], V=151936, dtype=dtype, temperature=T,
                                    target_sigma=3.0, noise_sigma=1.0, name=out.name)
    return out


def c3_block_lens(seed=1003, S=8) -> np.ndarray:
    rs = _streams(seed)
    draws = rs["B"].normal(16.0, 3.0, size=S)
    return _nearest_in_set(draws, RAGGED_BLOCK_SET).astype(np.int32)


def c3_ragged(temperatures=(0.0, 1.0), seed=1003, dtype="bf16", S=8, ctx=4096, vocab=151936,
              with_attn=True) -> Workload:
    """Instance-adaptive ragged blocks: 8 sequences, Qwen3-4B attention shape (32/8/128), bf16,
    ctx 4096 each, B_s from {8,..,24} nearest to N(16,3^2); causal; acceptance over V=151936."""
    out = Workload(name="qwen3_4b_ragged_S8_ctx4096_B8-24", attn=None)
    B = c3_block_lens(seed, S)
    if with_attn:
        rs = _streams(seed)
        out.attn = make_attn(rs, S=S, Hq=32, Hkv=8, D=128, ctx_lens=[ctx] * S, block_lens=B, dtype=dtype,
                             mask_mode=MASK_CAUSAL_IN_BLOCK, Lmax=ctx + int(RAGGED_BLOCK_SET.max()),
                             name=out.name)
    for T in temperatures:
        rs = _streams(seed)
        out.accept[T] = make_accept(rs, block_lens=B, V=vocab, dtype=dtype, temperature=T,
                                    target_sigma=3.0, noise_sigma=1.0, name=out.name)
    return out


def c4_drafter(seed=1004, dtype="bf16", S=16) -> Workload:
    """Drafter block-diffusion pass: 16 sequences, 32/8/128, bf16, ctx ~ U{1024..8192},
    B ~ U{8..32}, bidirectional-in-block; no acceptance."""
    rs = _streams(seed)
    ctx = rs["ctx"].integers(1024, 8192, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(8, 32, endpoint=True, size=S).astype(np.int32)
    out = Workload(name="drafter_bidir_S16_ctx1k-8k_B8-32", attn=None)
    out.attn = make_attn(rs, S=S, Hq=32, Hkv=8, D=128, ctx_lens=ctx, block_lens=B, dtype=dtype,
                         mask_mode=MASK_BIDIR_IN_BLOCK, Lmax=8192 + 32, name=out.name)
    return out


def c5_long_context(temperatures=(1.0,), seed=1005, dtype="bf16", S=32, with_attn=True,
                    with_accept=True) -> Workload:
    """Long-context serving step: 32 sequences, Qwen3-8B attention shape (32/8/128), bf16,
    ctx ~ U{8192..32768}, B ~ U{4..32}, causal; acceptance over V=151936 at T=1."""
    rs = _streams(seed)
    ctx = rs["ctx"].integers(8192, 32768, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(4, 32, endpoint=True, size=S).astype(np.int32)
    out = Workload(name="qwen3_8b_long_S32_ctx8k-32k_B4-32", attn=None)
    if with_attn:
        out.attn = make_attn(rs, S=S, Hq=32, Hkv=8, D=128, ctx_lens=ctx, block_lens=B, dtype=dtype,
                             mask_mode=MASK_CAUSAL_IN_BLOCK, Lmax=32768 + 32, name=out.name)
    if with_accept:
        for T in temperatures:
            rs = _streams(seed)
            out.accept[T] = make_accept(rs, block_lens=B, V=151936, dtype=dtype, temperature=T,
                                        target_sigma=3.0, noise_sigma=1.0, name=out.name)
    return out


def c4_lens(seed=1004, S=16):
    rs = _streams(seed)
    ctx = rs["ctx"].integers(1024, 8192, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(8, 32, endpoint=True, size=S).astype(np.int32)
    return ctx, B


def c5_lens(seed=1005, S=32):
    rs = _streams(seed)
    ctx = rs["ctx"].integers(8192, 32768, endpoint=True, size=S).astype(np.int32)
    B = rs["B"].integers(4, 32, endpoint=True, size=S).astype(np.int32)
    return ctx, B


# --------------------------------------------------------------------------- #
# inputs of the step around verification (append, verify in every layer, commit)
# --------------------------------------------------------------------------- #

def step_caches(rs: dict, *, S, Hkv, D, Lmax, ctx_lens, dtype, tail_fill=float("nan")):
    """One layer's caches [S, Hkv, Lmax, D]: committed rows [0, ctx_s) ~ N(0,1), the rest
    ``tail_fill`` (NaN), so a read of an unwritten row poisons the output."""
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    k = torch.full((S, Hkv, Lmax, D), tail_fill, dtype=tdt)
    v = torch.full((S, Hkv, Lmax, D), tail_fill, dtype=tdt)
    for s in range(S):
        n = int(ctx_lens[s])
        k[s, :, :n] = torch.from_numpy(rs["K"].standard_normal((Hkv, n, D), dtype=np.float32)).to(tdt)
        v[s, :, :n] = torch.from_numpy(rs["V"].standard_normal((Hkv, n, D), dtype=np.float32)).to(tdt)
    return k, v


def step_block_inputs(rs: dict, *, total_q, Hq, Hkv, D, dtype) -> dict:
    """One layer's block inputs of one step: q [total_q, Hq, D] and the block's new keys and
    values [total_q, Hkv, D], all ~ N(0,1)."""
    return dict(q=_to_dtype(rs["q"].standard_normal((total_q, Hq, D), dtype=np.float32), dtype),
                k_new=_to_dtype(rs["K"].standard_normal((total_q, Hkv, D), dtype=np.float32), dtype),
                v_new=_to_dtype(rs["V"].standard_normal((total_q, Hkv, D), dtype=np.float32), dtype))


# --------------------------------------------------------------------------- #
# block-size policy inputs: last-token logits and random MLP weights
# --------------------------------------------------------------------------- #

@dataclass
class PolicyProblem:
    """Last-token logits [P, V] and the MLP's weights (bf16, [out, in]) and biases (fp32).

    The trained predictor weights are not available; the weights here are seeded random
    draws: W1 ~ N(0, 1) (its input p sums to one), W2, W3 ~ N(0, 1/H), biases ~ N(0, 0.05^2).
    """
    logits: torch.Tensor
    w1: torch.Tensor
    b1: np.ndarray
    w2: torch.Tensor
    b2: np.ndarray
    w3: torch.Tensor
    b3: np.ndarray
    base_block: int
    radius: int
    dtype: str
    name: str = ""

    @property
    def P(self) -> int:
        return int(self.logits.shape[0])

    @property
    def V(self) -> int:
        return int(self.logits.shape[1])

    @property
    def H(self) -> int:
        return int(self.w1.shape[0])

    def weight_bytes(self) -> int:
        return 2 * (self.w1.numel() + self.w2.numel() + self.w3.numel())


def make_policy(seed: int, *, P, V, H=2048, radius=2, base_block=16, dtype="bf16", logit_sigma=3.0,
                name="") -> PolicyProblem:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    C = 2 * radius + 1
    logits = _to_dtype(g.standard_normal((P, V), dtype=np.float32) * np.float32(logit_sigma), dtype)
    w1 = torch.from_numpy(g.standard_normal((H, V), dtype=np.float32)).to(torch.bfloat16)
    w2 = torch.from_numpy(g.standard_normal((H, H), dtype=np.float32) / np.float32(np.sqrt(H))).to(torch.bfloat16)
    w3 = torch.from_numpy(g.standard_normal((C, H), dtype=np.float32) / np.float32(np.sqrt(H))).to(torch.bfloat16)
    b1 = (g.standard_normal(H, dtype=np.float32) * np.float32(0.05)).astype(np.float32)
    b2 = (g.standard_normal(H, dtype=np.float32) * np.float32(0.05)).astype(np.float32)
    b3 = (g.standard_normal(C, dtype=np.float32) * np.float32(0.05)).astype(np.float32)
    return PolicyProblem(logits, w1, b1, w2, b2, w3, b3, base_block, radius, dtype, name)


# --------------------------------------------------------------------------- #
# paged caches: the same keys and values scattered over a pool of pages
# --------------------------------------------------------------------------- #

def paginate(rs: dict, k_cache: torch.Tensor, v_cache: torch.Tensor, page_size: int, spare_pages: int = 3,
             fill=float("nan")):
    """Scatter contiguous caches [S, Hkv, Lmax, D] (Lmax a multiple of page_size) into pools
    [num_pages, Hkv, page_size, D] in a seeded random page order, with ``spare_pages`` unused
    pool pages holding ``fill``.  Returns (k_pages, v_pages, block_table [S, Lmax/page_size])."""
    S, Hkv, Lmax, D = k_cache.shape
    if Lmax % page_size:
        raise ValueError("Lmax must be a multiple of page_size")
    mp = Lmax // page_size
    num_pages = S * mp + spare_pages
    perm = rs["ctx"].permutation(num_pages)[:S * mp].astype(np.int32)
    table = perm.reshape(S, mp)
    kp = torch.full((num_pages, Hkv, page_size, D), fill, dtype=k_cache.dtype)
    vp = torch.full((num_pages, Hkv, page_size, D), fill, dtype=v_cache.dtype)
    kv = k_cache.reshape(S, Hkv, mp, page_size, D).permute(0, 2, 1, 3, 4)  # [S, mp, Hkv, ps, D]
    vv = v_cache.reshape(S, Hkv, mp, page_size, D).permute(0, 2, 1, 3, 4)
    idx = torch.from_numpy(table.reshape(-1).astype(np.int64))
    kp[idx] = kv.reshape(S * mp, Hkv, page_size, D)
    vp[idx] = vv.reshape(S * mp, Hkv, page_size, D)
    return kp, vp, table


# --------------------------------------------------------------------------- #
# prefix-survival model: per-sample, per-position predictability
# --------------------------------------------------------------------------- #

@dataclass
class SurvivalProblem:
    gamma: np.ndarray      # [N, P] fp32 in (0, 1]: predictability gamma_j(x) of drafted position j
    cands: np.ndarray      # [C] int32, strictly ascending candidate block sizes (<= P)
    train_block: int       # B, the drafter's training block size
    alpha: float           # retention sharpness
    b_hat: np.ndarray      # [N] int32: a predicted block size per sample, drawn from the candidates
    name: str = ""

    @property
    def N(self) -> int:
        return int(self.gamma.shape[0])

    @property
    def P(self) -> int:
        return int(self.gamma.shape[1])


def make_survival(seed: int, *, N, P=32, train_block=16, radius=2, alpha=0.01, gamma_lo=0.6, gamma_hi=0.97,
                  jitter=0.03, name="") -> SurvivalProblem:
    """Samples whose predictability is near-constant across positions: gamma_x ~ U(lo, hi) per
    sample, gamma_j(x) = gamma_x + N(0, jitter^2) clipped to [0.01, 1]; candidates are the local
    interval {B - k, ..., B + k}; b_hat is uniform over the candidates."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    base = g.uniform(gamma_lo, gamma_hi, size=(N, 1))
    gamma = np.clip(base + jitter * g.standard_normal((N, P)), 0.01, 1.0).astype(np.float32)
    cands = np.arange(train_block - radius, train_block + radius + 1, dtype=np.int32)
    b_hat = g.choice(cands, size=N).astype(np.int32)
    return SurvivalProblem(gamma, cands, int(train_block), float(alpha), b_hat, name)
