// check.hpp -- validation of the per-sequence values that the hot calls read from device
// memory and take on trust (context and block lengths, row offsets, drafted tokens,
// uniforms).  One workgroup walks the sequences and files an error word; it reads an array
// element only where the values checked before it keep the index inside the array.
#pragma once

#include <limits.h>

#include "common.hpp"

namespace sdb {

enum : int {
  kCheckCtx = 1,       // ctx_s outside [0, max_ctx]
  kCheckBlock = 2,     // B_s outside [min_block, max_block]
  kCheckOffsets = 4,   // q_offsets not the exclusive prefix sum of block_lens ending at total_q
  kCheckToken = 8,     // a drafted token outside [0, V)
  kCheckUniform = 16,  // a uniform outside [0, 1) (NaN included)
};

struct CheckArgs {
  const int *ctx_lens;      // [S] or null (acceptance)
  const int *block_lens;    // [S]
  const int *q_offsets;     // [S + 1]
  const int *draft_tokens;  // [total_q - S] or null (attention)
  const float *uniforms;    // [total_q] or null (attention, or acceptance at T = 0)
  int *status;              // [3]: OR of the bits, first offending sequence or -1, count
  int S, total_q, max_ctx, min_block, max_block, vocab;
};

__global__ __launch_bounds__(256) void check_inputs_kernel(CheckArgs a) {
  __shared__ int sh_bits, sh_first, sh_count;
  const int tid = threadIdx.x;
  if (tid == 0) {
    sh_bits = 0;
    sh_first = INT_MAX;
    sh_count = 0;
  }
  __syncthreads();
  int bits = 0, first = INT_MAX, count = 0;
  for (int s = tid; s < a.S; s += 256) {
    int e = 0;
    const int B = a.block_lens[s];
    if (B < a.min_block || B > a.max_block) e |= kCheckBlock;
    if (a.ctx_lens) {
      const int c = a.ctx_lens[s];
      if (c < 0 || c > a.max_ctx) e |= kCheckCtx;
    }
    const int o0 = a.q_offsets[s], o1 = a.q_offsets[s + 1];
    if ((s == 0 && o0 != 0) || (s == a.S - 1 && o1 != a.total_q) || o1 - o0 != B || o0 < 0 || o1 > a.total_q)
      e |= kCheckOffsets;
    if (!(e & (kCheckBlock | kCheckOffsets))) {  // rows [o0, o1) lie inside [0, total_q)
      if (a.draft_tokens) {
        const int d0 = o0 - s;  // draft rows of s: [d0, d0 + B - 1)
        if (d0 < 0 || d0 + B - 1 > a.total_q - a.S) {
          e |= kCheckOffsets;
        } else {
          for (int j = 0; j < B - 1; ++j) {
            const int t = a.draft_tokens[d0 + j];
            if (t < 0 || t >= a.vocab) e |= kCheckToken;
          }
        }
      }
      if (a.uniforms)
        for (int j = 0; j < B; ++j) {
          const float u = a.uniforms[o0 + j];
          if (!(u >= 0.f && u < 1.f)) e |= kCheckUniform;
        }
    }
    if (e) {
      bits |= e;
      first = min(first, s);
      ++count;
    }
  }
  atomicOr(&sh_bits, bits);
  atomicMin(&sh_first, first);
  atomicAdd(&sh_count, count);
  __syncthreads();
  if (tid == 0) {
    a.status[0] = sh_bits;
    a.status[1] = sh_first == INT_MAX ? -1 : sh_first;
    a.status[2] = sh_count;
  }
}

}  // namespace sdb
