"""sd_accept_noalloc (the acceptance call that allocates nothing, for callers that cannot
allocate) against sd_accept with its own workspace: the same kernels, so every result must be
identical.  Two calls in a row per temperature, the second on a smaller input, so the second
runs on scratch that still holds the first call's contents."""
import numpy as np
import pytest
import torch

import gpu_util as G
import paper_2606_31315_amd as sd
from paper_2606_31315_amd import workloads as W

pytestmark = pytest.mark.gpu


def _small(T):
    rs = W._streams(8080 + int(T))
    bl = np.array([3, 1, 7], dtype=np.int32)
    return W.make_accept(rs, block_lens=bl, V=50001, dtype="bf16", temperature=T, target_sigma=3.0,
                         noise_sigma=1.0, name=f"small_T{T:g}")


@pytest.mark.parametrize("T", [1.0, 0.0])
def test_noalloc_matches_sd_accept(T):
    big = W.c3_ragged(temperatures=(T,), with_attn=False).accept[T]
    for p in (big, _small(T)):
        d = G.accept_to_device(p)
        G.log(f"sd_accept_noalloc {p.name} S={p.S} V={p.V} total_q={p.total_q} T={T}")
        al_ref, nt_ref = sd.accept(d["t"], d["d"], d["tok"], d["u"], d["bl"], d["off"], T, max_block=p.max_block)
        al = torch.full((p.S,), -7, dtype=torch.int32, device=G.dev())
        nt = torch.full((p.S,), -7, dtype=torch.int32, device=G.dev())
        sd.accept_noalloc(d["t"], d["d"], d["tok"], d["u"], d["bl"], d["off"], T, max_block=p.max_block,
                          accept_len=al, next_token=nt)
        torch.cuda.synchronize()
        assert torch.equal(al, al_ref) and torch.equal(nt, nt_ref), (al.cpu(), al_ref.cpu(), nt.cpu(), nt_ref.cpu())
        # and the results follow the parity rule against the oracle
        G.compare_accept(p, al.cpu().numpy(), nt.cpu().numpy(), G.oracle_accept(p))
