"""MI355X-native hot path of BlockPilot's speculative step (arXiv 2606.31315).

Two operations, both hand-written HIP for gfx950 behind the C ABI in
include/sd_block.h:

  block_attn  block-verify / block-diffusion attention of ragged blocks over a GQA
              KV cache (causal-in-block or bidirectional-in-block mask);
  accept      vocabulary-wide speculative acceptance (greedy at T=0, lossless
              rejection sampling at T>0) returning accept_len and the next token.

and the step around them: kv_append (the block's keys and values into the cache;
block_attn_append fuses it into the attention launch),
commit (ctx += accept_len + 1) and verify_step (append + attention per layer,
acceptance, commit, in one native call); block_attn_paged and kv_append_paged over
page pools with a block table; and the once-per-prompt block-size policy
(block_size_policy: softmax of the last-token logits through a two-hidden-layer MLP);
survival_tau and survival_sample: the prefix-survival model of the accepted length
(expected length per candidate block size, the best size, regret, Monte Carlo);
check_attn_inputs and check_accept_inputs: an error word for the per-sequence device
values the calls above take on trust.
"""
from ._lib import (SD_BF16, SD_F32, SD_MASK_BIDIR_IN_BLOCK, SD_MASK_CAUSAL_IN_BLOCK, SdError, Workspace,
                   accept, accept_noalloc, accept_set_path, accept_shape, accept_workspace_size, attn_shape, attn_workspace_size, block_attn,
                   block_attn_append, block_attn_paged, block_size_policy, check_accept_inputs, check_attn_inputs,
                   commit, kv_append_paged,
                   kv_append, lib, survival_sample, survival_tau, verify_step, version)

__all__ = ["block_attn", "block_attn_append", "check_attn_inputs", "check_accept_inputs", "block_attn_paged", "kv_append_paged", "accept", "accept_noalloc", "accept_set_path", "kv_append", "commit", "verify_step", "block_size_policy", "survival_tau", "survival_sample", "attn_shape", "accept_shape",
           "attn_workspace_size", "accept_workspace_size",
           "Workspace", "SdError", "lib", "version", "SD_BF16", "SD_F32", "SD_MASK_CAUSAL_IN_BLOCK",
           "SD_MASK_BIDIR_IN_BLOCK"]
