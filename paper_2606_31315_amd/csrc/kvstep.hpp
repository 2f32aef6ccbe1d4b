// kvstep.hpp -- the two small steps on either side of verification.
//
//   kv_append_kernel  before the verify pass of a layer: the block's new keys and values go to
//                     cache rows [ctx_s, ctx_s + B_s) of every kv head of sequence s, where the
//                     block attention reads them (the block is verified in parallel, Sec. 2.1).
//   commit_kernel     after acceptance: the anchor and the accepted drafts are now cached,
//                     ctx_s += accept_len_s + 1.  Rows of rejected drafts stay in the cache past
//                     the new length and are overwritten by the next step's append (the accepted
//                     prefix is the longest consistent one, Fig. 1 caption).
//
// Both are copies or integer updates; they move B_s * Hkv * D elements per sequence and layer.
#pragma once

#include "common.hpp"

namespace sdb {

struct AppendArgs {
  const void *k_new;   // [total_q, Hkv, D]
  const void *v_new;   // [total_q, Hkv, D]
  void *k_cache;       // [S, Hkv, Lmax, D]
  void *v_cache;
  const int *ctx_lens;
  const int *q_offsets;
  int S, Hkv, Lmax, total_q;
  int row_vecs;        // 16-byte vectors per (token, head) row: D * element bytes / 16
  // page pools only: caches are [num_pages, Hkv, page_size, D], logical page j of sequence s is
  // pool page block_table[s * max_pages + j]
  const int *block_table;
  int page_log2, max_pages, num_pages;
};

// The sequence s that owns packed row r (the largest s with off[s] <= r; r < off[S]) and the
// row's cache position ctx[s] + r - off[s], in every lane of the wavefront.  Lane k loads
// off[k] and ctx[k] together, so one round of loads (64 sequences per round) settles both;
// offsets ascend, so the first round that has a lane past r is the last one needed.
__device__ __forceinline__ void row_owner_pos(const int *off, const int *ctx, int S, int r, int &s_out,
                                              int &pos_out) {
  const int lane = threadIdx.x & 63;
  int s = 0, pos = 0;
  for (int k0 = 0; k0 < S; k0 += 64) {
    const int k = min(k0 + lane, S - 1);  // clamped: no per-load branch
    const int o = off[k], c = ctx[k];
    const unsigned long long valid = __ballot(k0 + lane < S);
    const unsigned long long le = __ballot(k0 + lane < S && o <= r);
    if (le) {
      const int last = 63 - __clzll((long long)le);
      s = k0 + last;
      pos = __shfl(c, last, 64) + (r - __shfl(o, last, 64));
    }
    if (le != valid) break;
  }
  s_out = s;
  pos_out = pos;
}

// grid = (total_q, 2): block (r, kv) copies token row r of K (kv = 0) or V (kv = 1) for every
// kv head; threads stride over the Hkv * row_vecs 16-byte vectors.  The first vectors are
// loaded before the owner lookup (they do not depend on it), so the copy costs one round of
// loads.  A destination row at or past Lmax (a ctx_len beyond the cache) is skipped rather
// than written out of bounds.
__global__ __launch_bounds__(256) void kv_append_kernel(AppendArgs a) {
  const int r = blockIdx.x;
  const int kv = blockIdx.y;
  const int n = a.Hkv * a.row_vecs;
  const u32x4 *src = reinterpret_cast<const u32x4 *>(kv ? a.v_new : a.k_new) + (size_t)r * n;
  const int i0 = threadIdx.x;
  const u32x4 first = src[min(i0, n - 1)];
  int s, pos;
  row_owner_pos(a.q_offsets, a.ctx_lens, a.S, r, s, pos);
  if (pos < 0 || pos >= a.Lmax) return;
  u32x4 *dst = reinterpret_cast<u32x4 *>(kv ? a.v_cache : a.k_cache);
  for (int i = i0; i < n; i += blockDim.x) {
    const int h = i / a.row_vecs, c = i - h * a.row_vecs;
    dst[(((size_t)s * a.Hkv + h) * a.Lmax + pos) * a.row_vecs + c] = (i == i0) ? first : src[i];
  }
}

// The same copy into page pools.  A row past the sequence's pages, or whose page id lies
// outside the pool, is skipped rather than written.
__global__ __launch_bounds__(256) void kv_append_paged_kernel(AppendArgs a) {
  const int r = blockIdx.x;
  const int kv = blockIdx.y;
  const int n = a.Hkv * a.row_vecs;
  const u32x4 *src = reinterpret_cast<const u32x4 *>(kv ? a.v_new : a.k_new) + (size_t)r * n;
  const int i0 = threadIdx.x;
  const u32x4 first = src[min(i0, n - 1)];
  int s, pos;
  row_owner_pos(a.q_offsets, a.ctx_lens, a.S, r, s, pos);
  if (pos < 0 || pos >= a.Lmax) return;
  const int pg = ld_uniform(a.block_table, (long long)s * a.max_pages + (pos >> a.page_log2));
  if (pg < 0 || pg >= a.num_pages) return;
  const size_t row0 = (((size_t)pg * a.Hkv) << a.page_log2) + (pos & ((1 << a.page_log2) - 1));
  u32x4 *dst = reinterpret_cast<u32x4 *>(kv ? a.v_cache : a.k_cache);
  for (int i = i0; i < n; i += blockDim.x) {
    const int h = i / a.row_vecs, c = i - h * a.row_vecs;
    dst[(row0 + ((size_t)h << a.page_log2)) * a.row_vecs + c] = (i == i0) ? first : src[i];
  }
}

// ctx_lens[s] += accept_len[s] + 1 for every sequence.
__global__ __launch_bounds__(256) void commit_kernel(const int *accept_len, int *ctx_lens, int S) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s < S) ctx_lens[s] += accept_len[s] + 1;
}

}  // namespace sdb
