// attn.hpp -- block attention over a GQA KV cache with ragged per-sequence blocks.
//
// Operation (Sec. 2.1): the B_s block rows of sequence s attend to their committed
// context and to the block itself, causally for target verification or
// bidirectionally for the block-diffusion drafter.  Query head h reads kv head
// h / G with G = Hq / Hkv.
//
// Kernel design (gfx950):
//   * One workgroup (4 wavefronts) per (sequence, kv head, KV split).  All G*B_s
//     query rows of the sequence's kv-head group are packed into 16-row MFMA tiles,
//     so each K/V byte is read from HBM once for the whole group.
//   * K tile staged in LDS row-major; V tile written to LDS transposed
//     (d-major, 4 consecutive keys per 8-byte word) so the P.V contraction over keys
//     reads its operand with 8-byte LDS loads.
//   * S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (16x16x4_f32 for fp32 inputs): each lane
//     then owns four keys of one query row, which is exactly the B-operand layout the
//     O^T += V^T P^T MFMA needs, so P never leaves registers.
//   * Online softmax in the log2 domain (scale * log2 e folded into one FMA), with
//     per-lane partial row sums reduced once at the end.
//   * A sequence whose keys fit one split writes its output directly.  Otherwise each
//     split writes fp32 partials (unnormalised O, row max, row sum) and a second launch,
//     block_attn_merge_kernel, combines them.  The kernel boundary is the only
//     cross-workgroup synchronisation: an in-kernel "last workgroup merges" scheme needs
//     agent-scope release fences, which on gfx950 write back the XCD's L2 and cost far
//     more than the second launch.
#pragma once

#include "common.hpp"

namespace sdb {

struct AttnArgs {
  const void *q;
  const void *k;
  const void *v;
  void *out;
  const int *ctx_lens;
  const int *block_lens;
  const int *q_offsets;
  float *part_o;      // [n_work, Mpad, D] unnormalised partial outputs
  float2 *part_ml;    // [n_work, Mpad]    (row max in log2 units, row sum)
  int S, Hq, Hkv, G, Lmax;
  int split_len;      // longest split (keys), a multiple of gran
  int gran;           // split lengths are multiples of gran keys
  int max_splits;     // splits per (sequence, kv head) at the host-known maximum length
  int Mpad;           // rows reserved per work item in the partial buffers
  int n_work;         // S * Hkv * max_splits
  int per_xcd;        // ceil(n_work / 8): the XCD-grouped deal of a one-wave grid
  int dense;          // more than one wave: work items numbered densely on the device
  float scale_log2;   // softmax scale * log2(e)
  int causal;
  // paged caches only: k, v are page pools [num_pages, Hkv, page_size, D]; logical page j of
  // sequence s is pool page block_table[s * max_pages + j]
  const int *block_table;
  int page_log2, max_pages, num_pages;
  // fused append only: the block's new keys and values [total_q, Hkv, D]
  const void *k_new;
  const void *v_new;
  // balanced plan (bf16, plain caches; bal_share): bal_grid workgroups, shares of at least
  // bal_min_tiles key tiles of bal_kt keys
  int bal, bal_grid, bal_min_tiles, bal_kt;
};

// ---- work items ----------------------------------------------------------------
// Each (sequence, kv head) pair of L keys is cut into nsplit = ceil(L / split_len) splits of
// even length (ceil(L / nsplit) rounded up to gran keys, never more than split_len, so every
// split is non-empty).  One work item per split.
//   One-wave grid (n_work <= one workgroup per CU): workgroup w owns slot w = pair *
//     max_splits + split, dealt so that a pair's splits share an XCD; slots past a pair's
//     nsplit have no work.
//   Larger grids: the items that exist are numbered densely on the device, sequence by
//     sequence, pair by pair, split by split (a prefix sum of Hkv * nsplit over the
//     sequences, 64 per round), and workgroup i takes item i; round-robin dispatch over the
//     XCDs then spreads every long sequence over all of them, and no workgroup is spent on an
//     empty slot.
//   Dense grids whose splits are at the length cap (kLongSplit) instead cut each pair into
//     full splits of split_len keys plus one partial last split, and number all full splits
//     first and then the partial ones, longest first, so the shortest items fill the tail
//     (32 sequences, contexts 8k-32k: 537 -> 513 us).  Shorter capped-below plans keep even
//     splits: there the partial items would be tiny workgroups (16 sequences, contexts 1k-8k:
//     96.0 us even, 100.3 us full + partial).
// Partial slots are the workgroup's slot (one wave) or the pair's slot base + split (dense).
struct AttnItem {
  int s, g, split, nsplit, k0, k1, slot, ctx, B, qoff;
};

// Longest split the planner makes (keys); dense plans at this length order their items
// longest first.
constexpr int kLongSplit = 4096;

__device__ __forceinline__ bool attn_item(const AttnArgs &a, int b, AttnItem &it) {
  if (!a.dense) {
    const int w = xcd_logical_id(b, a.per_xcd);
    if (w >= a.n_work) return false;
    it.split = w % a.max_splits;
    const int sg = w / a.max_splits;
    it.g = sg % a.Hkv;
    it.s = sg / a.Hkv;
    it.ctx = a.ctx_lens[it.s];
    it.B = a.block_lens[it.s];
    it.qoff = a.q_offsets[it.s];
    if (it.B <= 0) return false;
    it.nsplit = (it.ctx + it.B + a.split_len - 1) / a.split_len;
    if (it.split >= it.nsplit) return false;
    it.slot = w;
  } else if (a.split_len >= kLongSplit) {
    // Splits at the length cap (long contexts, several waves): full splits of split_len keys
    // first, sequence by sequence; then each sequence's partial last split, longest first
    // (in sequence order beyond 64 sequences), so the shortest items run last and fill the
    // tail.  Slots stay in the per-pair order the merge reads.
    const int lane = threadIdx.x & 63;
    const int sl = a.split_len;
    int before = 0, sbefore = 0;
    bool found = false;
    for (int c0 = 0; c0 < a.S && !found; c0 += 64) {
      const int k = min(c0 + lane, a.S - 1);  // clamped: no per-load branch
      const int ctx = a.ctx_lens[k], B = a.block_lens[k], off = a.q_offsets[k];
      const bool live = c0 + lane < a.S && B > 0;
      const int n = live ? (ctx + B + sl - 1) / sl : 0;
      const int nf = live ? (ctx + B) / sl : 0;
      const int items = nf * a.Hkv;
      const int incl = before + wave_scan_i(items);
      const int sincl = sbefore + wave_scan_i(n * a.Hkv);
      const unsigned long long hit = __ballot(incl > b && incl - items <= b);
      if (hit) {
        const int l = __ffsll((long long)hit) - 1;  // wave-uniform
        it.s = c0 + l;
        it.ctx = __builtin_amdgcn_readlane(ctx, l);
        it.B = __builtin_amdgcn_readlane(B, l);
        it.qoff = __builtin_amdgcn_readlane(off, l);
        it.nsplit = __builtin_amdgcn_readlane(n, l);
        const int nfl = __builtin_amdgcn_readlane(nf, l);
        const int r = b - __builtin_amdgcn_readlane(incl - items, l);
        it.g = r / nfl;
        it.split = r - it.g * nfl;
        it.slot = __builtin_amdgcn_readlane(sincl - n * a.Hkv, l) + it.g * it.nsplit + it.split;
        found = true;
      }
      before = __builtin_amdgcn_readlane(incl, 63);
      sbefore = __builtin_amdgcn_readlane(sincl, 63);
    }
    if (!found) {
      const int p = b - before;  // index among the partial items
      const int rank = p / a.Hkv;
      const int g = p - rank * a.Hkv;
      int pb = 0;
      sbefore = 0;
      for (int c0 = 0; c0 < a.S && !found; c0 += 64) {
        const int k = min(c0 + lane, a.S - 1);  // clamped: no per-load branch
        const int ctx = a.ctx_lens[k], B = a.block_lens[k], off = a.q_offsets[k];
        const bool live = c0 + lane < a.S && B > 0;
        const int n = live ? (ctx + B + sl - 1) / sl : 0;
        const int part = live ? (ctx + B) % sl : 0;
        const int sincl = sbefore + wave_scan_i(n * a.Hkv);
        int key;  // this lane's position among the partial items (valid where part > 0)
        if (a.S <= 64) {
          key = 0;
          for (int t = 0; t < a.S; ++t) {
            const int pt = __builtin_amdgcn_readlane(part, t);
            key += (pt > part) || (pt == part && t < lane);
          }
        } else {
          const int has = part > 0 ? 1 : 0;
          key = pb + wave_scan_i(has) - has;
          pb = __builtin_amdgcn_readlane(pb + wave_scan_i(has), 63);
        }
        const unsigned long long hit = __ballot(part > 0 && key == rank);
        if (hit) {
          const int l = __ffsll((long long)hit) - 1;  // wave-uniform
          it.s = c0 + l;
          it.ctx = __builtin_amdgcn_readlane(ctx, l);
          it.B = __builtin_amdgcn_readlane(B, l);
          it.qoff = __builtin_amdgcn_readlane(off, l);
          it.nsplit = __builtin_amdgcn_readlane(n, l);
          it.g = g;
          it.split = it.nsplit - 1;
          it.slot = __builtin_amdgcn_readlane(sincl - n * a.Hkv, l) + g * it.nsplit + it.split;
          found = true;
        }
        sbefore = __builtin_amdgcn_readlane(sincl, 63);
      }
      if (!found) return false;  // past the last item
    }
    it.k0 = it.split * sl;
    it.k1 = min(it.k0 + sl, it.ctx + it.B);
    return true;
  } else {
    const int lane = threadIdx.x & 63;
    int before = 0;
    bool found = false;
    for (int c0 = 0; c0 < a.S && !found; c0 += 64) {
      const int k = min(c0 + lane, a.S - 1);  // clamped: no per-load branch
      const int ctx = a.ctx_lens[k], B = a.block_lens[k], off = a.q_offsets[k];
      const int n = (c0 + lane < a.S && B > 0) ? (ctx + B + a.split_len - 1) / a.split_len : 0;
      const int items = n * a.Hkv;
      const int incl = before + wave_scan_i(items);
      const unsigned long long hit = __ballot(incl > b && incl - items <= b);
      if (hit) {
        const int l = __ffsll((long long)hit) - 1;  // wave-uniform
        it.s = c0 + l;
        it.ctx = __builtin_amdgcn_readlane(ctx, l);
        it.B = __builtin_amdgcn_readlane(B, l);
        it.qoff = __builtin_amdgcn_readlane(off, l);
        it.nsplit = __builtin_amdgcn_readlane(n, l);
        const int r = b - __builtin_amdgcn_readlane(incl - items, l);
        it.g = r / it.nsplit;
        it.split = r - it.g * it.nsplit;
        it.slot = b;
        found = true;
      }
      before = __builtin_amdgcn_readlane(incl, 63);
    }
    if (!found) return false;  // past the last item
  }
  const int L = it.ctx + it.B;
  const int slen = (((L + it.nsplit - 1) / it.nsplit + a.gran - 1) / a.gran) * a.gran;
  it.k0 = it.split * slen;
  it.k1 = min(it.k0 + slen, L);
  return true;
}

// ---- balanced plan ---------------------------------------------------------------
// Pair (s, g) holds n = ceil((ctx_s + B_s) / kt) key tiles (none when B_s = 0), each weighing
// w = bal_weight(m-tiles of its block) units; the pairs line up in (sequence, kv head) order,
// W units in all.  Workgroup w takes the tiles whose first unit lies in [w * per, (w + 1) * per),
// per = max(ceil(W / bal_grid), bal_min_tiles * the lightest weight), so every workgroup gets
// about the same work whatever the lengths are; its share is cut where it crosses from one pair
// to the next, one work item per piece.  The piece of workgroup w in pair q = s * Hkv + g files
// its partial at slot w + q, so a pair's pieces hold consecutive slots from (first workgroup) + q.
// (Even splits per pair leave ragged batches with fractional waves: 16 sequences, contexts
// 1k-8k, about 350 splits of up to 2064 keys on 256 CUs.)
#ifndef SDB_BAL_WEIGHTS
#define SDB_BAL_WEIGHTS 1
#endif
// Relative time of one key tile by the block's m-tiles (16-row query tiles): up to 3 m-tiles
// the split kernel streams a tile at the memory's pace; beyond that the wavefronts' LDS reads
// and arithmetic add to it (8 sequences x 8 kv heads, contexts 4096, one wave, MI355X: 33.1 us
// per call at 2 m-tiles, 33.7 at 3, 34.5 at 4, 35.5 at 5, 37.9 at 6, 40.0 at 7, 41.6 at 8).
// Chosen by A/B on the multi-wave batches: against the steeper table measured before the
// kernel's lane swaps (20, 23, 25, 28, 32, 33 for 1-3 ... 8 m-tiles), 16 sequences with contexts
// 1k-8k 82.75 -> 81.14 us per call, 32 sequences with contexts 8k-32k 472.9 -> 452.1 us.
constexpr int kBalWeightMax8 = 31;  // the weight at 8 m-tiles; 4 more per m-tile past 8
__device__ __forceinline__ int bal_weight(int nmt) {
  if (!SDB_BAL_WEIGHTS) return 1;
  constexpr int kw[9] = {20, 20, 20, 20, 22, 24, 26, 29, kBalWeightMax8};
  return nmt <= 8 ? kw[nmt] : kBalWeightMax8 + 4 * (nmt - 8);
}

struct BalShare {
  int per, u0, u1;  // units per share; this workgroup's unit range [u0, u1)
};

// Lanes hold sequence values; per-pair tiles and weight of that sequence (0 past a.S / empty).
__device__ __forceinline__ int bal_seq_tiles(bool live, int ctx, int B, int kt) {
  return (live && B > 0) ? (ctx + B + kt - 1) / kt : 0;
}
__device__ __forceinline__ int bal_seq_weight(const AttnArgs &a, int B) {
  return bal_weight((a.G * max(B, 0) + 15) / 16);
}

__device__ __forceinline__ int bal_per(const AttnArgs &a, int W) {
  return max((W + a.bal_grid - 1) / a.bal_grid, a.bal_min_tiles * bal_weight(1));
}

// First tile of a pair (start unit p0, weight w) whose first unit is at or after unit u.
__device__ __forceinline__ int bal_tile_at(int u, int p0, int w) {
  return u <= p0 ? 0 : (u - p0 + w - 1) / w;
}

// This workgroup's share: the total W, one round of loads per 64 sequences.
__device__ __forceinline__ BalShare bal_share(const AttnArgs &a, int w, int kt) {
  const int lane = threadIdx.x & 63;
  int W = 0;
  for (int c0 = 0; c0 < a.S; c0 += 64) {
    const int k = min(c0 + lane, a.S - 1);  // clamped: no per-load branch
    const int B = a.block_lens[k];
    const int u = bal_seq_tiles(c0 + lane < a.S, a.ctx_lens[k], B, kt) * bal_seq_weight(a, B) * a.Hkv;
    W += __builtin_amdgcn_readlane(wave_scan_i(u), 63);
  }
  BalShare sh;
  sh.per = bal_per(a, W);
  sh.u0 = min(w * sh.per, W);
  sh.u1 = min(sh.u0 + sh.per, W);
  return sh;
}

// The next piece of the share: u0 is a cursor, the first unit not yet handed out.  The first
// tile whose first unit is at or after u0 starts the piece, if that unit lies before u1; the
// piece runs to the last tile of the same pair whose first unit lies before u1, and the cursor
// moves to the first unit of the tile after it.  Every piece moves the cursor forward, so the
// loop over pieces ends.  False when the share is done.
__device__ __forceinline__ bool bal_item(const AttnArgs &a, BalShare &sh, int kt, AttnItem &it) {
  const int lane = threadIdx.x & 63;
  // Two rounds at most: when u0 lies inside a pair's last tile past its first unit, the next
  // tile is the first of the next pair with tiles, whose first unit is that pair's start.
  for (int round = 0; round < 2; ++round) {
    if (sh.u0 >= sh.u1) return false;
    int before = 0;
    bool next_pair = false;
    for (int c0 = 0; c0 < a.S; c0 += 64) {
      const int k = min(c0 + lane, a.S - 1);  // clamped: no per-load branch
      const int ctx = a.ctx_lens[k], B = a.block_lens[k], off = a.q_offsets[k];
      const int t = bal_seq_tiles(c0 + lane < a.S, ctx, B, kt);
      const int wt = bal_seq_weight(a, B);
      const int sequ = t * wt * a.Hkv;
      const int incl = before + wave_scan_i(sequ);
      const unsigned long long hit = __ballot(incl > sh.u0 && incl - sequ <= sh.u0);  // holds unit u0
      if (hit) {
        const int l = __ffsll((long long)hit) - 1;  // wave-uniform
        const int ts = __builtin_amdgcn_readlane(t, l), w = __builtin_amdgcn_readlane(wt, l);
        const int pu = ts * w;  // units of each of the sequence's pairs
        const int pre = __builtin_amdgcn_readlane(incl - sequ, l);
        const int g = (sh.u0 - pre) / pu;
        const int p0 = pre + g * pu;  // first unit of pair (s, g)
        const int j0 = bal_tile_at(sh.u0, p0, w);
        if (j0 >= ts) {  // past the first unit of the pair's last tile: the next pair
          sh.u0 = p0 + pu;
          next_pair = true;
          break;
        }
        if (p0 + j0 * w >= sh.u1) {  // the next tile belongs to the next share
          sh.u0 = sh.u1;
          return false;
        }
        const int j1 = min(bal_tile_at(sh.u1, p0, w), ts);  // > j0
        it.s = c0 + l;
        it.g = g;
        it.ctx = __builtin_amdgcn_readlane(ctx, l);
        it.B = __builtin_amdgcn_readlane(B, l);
        it.qoff = __builtin_amdgcn_readlane(off, l);
        it.k0 = j0 * kt;
        it.k1 = min(j1 * kt, it.ctx + it.B);
        const int wf = p0 / sh.per, wl = (p0 + (ts - 1) * w) / sh.per;
        const int wme = (p0 + j0 * w) / sh.per;  // this workgroup
        it.nsplit = wl - wf + 1;
        it.split = wme - wf;
        it.slot = wme + it.s * a.Hkv + g;
        sh.u0 = p0 + j1 * w;
        return true;
      }
      before = __builtin_amdgcn_readlane(incl, 63);
    }
    if (!next_pair) return false;  // no sequence holds u0: past the last tile
  }
  return false;
}

// Partial slot of split 0 of pair (s, g) and the pair's split count (0: no block).
__device__ __forceinline__ int2 attn_pair_slots(const AttnArgs &a, int s, int g, int &B) {
  if (a.bal) {
    const int lane = threadIdx.x & 63;
    int W = 0, pre = 0, ts = 0, Bs = 0;
    for (int c0 = 0; c0 < a.S; c0 += 64) {
      const int k = min(c0 + lane, a.S - 1);  // clamped: no per-load branch
      const int Bk = a.block_lens[k];
      const int t = bal_seq_tiles(c0 + lane < a.S, a.ctx_lens[k], Bk, a.bal_kt);
      const int sequ = t * bal_seq_weight(a, Bk) * a.Hkv;
      const int incl = wave_scan_i(sequ);
      if (s >= c0 && s < c0 + 64) {  // wave-uniform
        const int l = s - c0;
        pre = W + __builtin_amdgcn_readlane(incl - sequ, l);
        ts = __builtin_amdgcn_readlane(t, l);
        Bs = __builtin_amdgcn_readlane(Bk, l);
      }
      W += __builtin_amdgcn_readlane(incl, 63);
    }
    B = Bs;
    if (Bs <= 0) return int2{0, 0};
    const int per = bal_per(a, W), w = bal_seq_weight(a, Bs);
    const int p0 = pre + g * ts * w;
    const int wf = p0 / per, wl = (p0 + (ts - 1) * w) / per;
    return int2{wf + s * a.Hkv + g, wl - wf + 1};
  }
  if (!a.dense) {
    // both lengths in one round of scalar loads: one use of both before the branch on B, so the
    // context length's load is not sunk behind it
    B = ld_uniform(a.block_lens, s);
    int ctx = ld_uniform(a.ctx_lens, s);
    asm volatile("" : "+s"(B), "+s"(ctx));
    if (B <= 0) return int2{0, 0};
    return int2{(s * a.Hkv + g) * a.max_splits, (ctx + B + a.split_len - 1) / a.split_len};
  }
  const int lane = threadIdx.x & 63;
  int before = 0;
  for (int c0 = 0; c0 <= s; c0 += 64) {
    const int k = min(c0 + lane, a.S - 1);  // clamped: no per-load branch
    const int ctx = a.ctx_lens[k], Bk = a.block_lens[k];
    const int n = (c0 + lane < a.S && Bk > 0) ? (ctx + Bk + a.split_len - 1) / a.split_len : 0;
    const int incl = before + wave_scan_i(n * a.Hkv);
    if (s < c0 + 64) {
      const int l = s - c0;
      B = __builtin_amdgcn_readlane(Bk, l);
      const int ns = __builtin_amdgcn_readlane(n, l);
      if (B <= 0) return int2{0, 0};
      return int2{__builtin_amdgcn_readlane(incl, l) - ns * a.Hkv + g * ns, ns};
    }
    before = __builtin_amdgcn_readlane(incl, 63);
  }
  B = 0;
  return int2{0, 0};
}

template <bool BF16>
struct AttnCfg {
  static constexpr int EB = BF16 ? 2 : 4;    // element bytes
  static constexpr int KT = BF16 ? 64 : 32;  // keys per tile
  static constexpr int NSUB = KT / 16;       // 16-key sub-tiles
  static constexpr int KPAD = 16 / EB;       // K row padding (elements)
  static constexpr int VPAD = BF16 ? 4 : 4;  // V^T row padding (keys)
};

// ---- operand loads -------------------------------------------------------
// K rows: chunk c (16 bytes) of the tile is row c / CPR, column chunk c % CPR.
template <bool BF16, int D>
__device__ __forceinline__ void load_k_tile(u32x4 (&kr)[(AttnCfg<BF16>::KT * D * AttnCfg<BF16>::EB / 16) / 256],
                                            const char *kbase, int key0, int key_end, int tid) {
  constexpr int CPR = D * AttnCfg<BF16>::EB / 16;
  constexpr int N = (AttnCfg<BF16>::KT * CPR) / 256;
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const int c = tid + 256 * j;
    const int row = c / CPR, col = c % CPR;
    // keys past the split end re-read the last valid key: finite data whose score the
    // mask removes, and no branch around the load
    const int key = min(key0 + row, key_end - 1);
    kr[j] = *reinterpret_cast<const u32x4 *>(kbase + ((size_t)key * D) * AttnCfg<BF16>::EB + col * 16);
  }
}

template <bool BF16, int D>
__device__ __forceinline__ void store_k_tile(char *ks, const u32x4 (&kr)[(AttnCfg<BF16>::KT * D * AttnCfg<BF16>::EB / 16) / 256],
                                             int tid) {
  using C = AttnCfg<BF16>;
  constexpr int CPR = D * C::EB / 16;
  constexpr int N = (C::KT * CPR) / 256;
  constexpr int PITCH = (D + C::KPAD) * C::EB;
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const int c = tid + 256 * j;
    const int row = c / CPR, col = c % CPR;
    *reinterpret_cast<u32x4 *>(ks + row * PITCH + col * 16) = kr[j];
  }
}

// V rows: item (kg, col) = 4 consecutive keys 4*kg.. x 8 consecutive dims col*8..
template <bool BF16, int D>
struct VItem {
  static constexpr int VEC_PER_KEY = 8 * AttnCfg<BF16>::EB / 16;  // 16-byte loads per key
  u32x4 r[4 * VEC_PER_KEY];
};

template <bool BF16, int D>
__device__ __forceinline__ void load_v_tile(VItem<BF16, D> &vi, const char *vbase, int key0, int key_end,
                                            int tid) {
  using C = AttnCfg<BF16>;
  constexpr int NITEMS = (C::KT / 4) * (D / 8);
  constexpr int VPK = VItem<BF16, D>::VEC_PER_KEY;
  if (tid >= NITEMS) return;
  const int kg = tid / (D / 8), col = tid % (D / 8);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int key = min(key0 + kg * 4 + r, key_end - 1);  // masked keys get weight 0
#pragma unroll
    for (int h = 0; h < VPK; ++h)
      vi.r[r * VPK + h] = *reinterpret_cast<const u32x4 *>(vbase + ((size_t)key * D + col * 8) * C::EB + h * 16);
  }
}

__device__ __forceinline__ uint32_t u32x4_get(const u32x4 &v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

template <bool BF16, int D>
__device__ __forceinline__ void store_v_tile(char *vts, const VItem<BF16, D> &vi, int tid) {
  using C = AttnCfg<BF16>;
  constexpr int NITEMS = (C::KT / 4) * (D / 8);
  constexpr int PITCH = (C::KT + C::VPAD) * C::EB;  // bytes per d row of V^T
  if (tid >= NITEMS) return;
  const int kg = tid / (D / 8), col = tid % (D / 8);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    char *dst = vts + (col * 8 + e) * PITCH + kg * 4 * C::EB;
    if constexpr (BF16) {
      // element e of key r sits in 32-bit word e/2, half e%2
      const int w = e >> 1, sh = (e & 1) * 16;
      const uint32_t k0 = (u32x4_get(vi.r[0], w) >> sh) & 0xffffu;
      const uint32_t k1 = (u32x4_get(vi.r[1], w) >> sh) & 0xffffu;
      const uint32_t k2 = (u32x4_get(vi.r[2], w) >> sh) & 0xffffu;
      const uint32_t k3 = (u32x4_get(vi.r[3], w) >> sh) & 0xffffu;
      *reinterpret_cast<uint2 *>(dst) = uint2{k0 | (k1 << 16), k2 | (k3 << 16)};
    } else {
      // fp32: element e of key r is word e%4 of 16-byte load r*2 + e/4
      const int h = e >> 2, w = e & 3;
      *reinterpret_cast<u32x4 *>(dst) = u32x4{u32x4_get(vi.r[0 * 2 + h], w), u32x4_get(vi.r[1 * 2 + h], w),
                                              u32x4_get(vi.r[2 * 2 + h], w), u32x4_get(vi.r[3 * 2 + h], w)};
    }
  }
}

// ---- the kernel -------------------------------------------------------------
// Query operand per 16-row m-tile:
//   bf16: D/32 bf16x8 values, element e of step t is dim t*32 + (lane/16)*8 + e
//   fp32: D/16 float4 values, element e of vector t4 is dim t4*16 + (lane/16)*4 + e
template <bool BF16, int D>
struct QOperand {
  static constexpr int N = BF16 ? D / 32 : D / 16;
  typename std::conditional<BF16, bf16x8, f32x4>::type v[N];
};

template <bool BF16, int D, int MT>
__global__ __launch_bounds__(256) void block_attn_kernel(AttnArgs a) {
  using C = AttnCfg<BF16>;
  constexpr int KT = C::KT, NSUB = C::NSUB, EB = C::EB;
  constexpr int KPITCH = (D + C::KPAD) * EB;   // bytes per K row in LDS
  constexpr int VPITCH = (KT + C::VPAD) * EB;  // bytes per V^T row in LDS
  constexpr int NDT = D / 16;                  // 16-wide output column tiles
  __shared__ __attribute__((aligned(16))) char ks[KT * KPITCH];
  __shared__ __attribute__((aligned(16))) char vts[D * VPITCH];

  AttnItem it;
  if (!attn_item(a, blockIdx.x, it)) return;
  const int s = it.s, g = it.g, k0 = it.k0, k1 = it.k1, nsplit = it.nsplit;
  const int ctx = it.ctx, B = it.B, qoff = it.qoff;
  const int M = a.G * B;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l16 = lane & 15;   // query row inside an m-tile / key row inside a sub-tile
  const int kgrp = lane >> 4;  // 0..3

  const char *kbase = reinterpret_cast<const char *>(a.k) + ((size_t)(s * a.Hkv + g) * a.Lmax) * D * EB;
  const char *vbase = reinterpret_cast<const char *>(a.v) + ((size_t)(s * a.Hkv + g) * a.Lmax) * D * EB;

  // ---- query operand and per-row state for this wave's m-tiles ----
  const int nmt = (M + 15) >> 4;
  QOperand<BF16, D> qop[MT];
  f32x4 oacc[MT][NDT];
  float m_run[MT], l_run[MT];
  int row_i[MT];  // block position of this lane's query row (or a large value for padding rows)
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    const int mt = wave + 4 * j;
    const int m = mt * 16 + l16;
    m_run[j] = -INFINITY;
    l_run[j] = 0.f;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) oacc[j][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bool valid = (mt < nmt) && (m < M);
    row_i[j] = valid ? m / a.G : 0;
    const char *qrow = valid ? reinterpret_cast<const char *>(a.q) +
                                   ((size_t)(qoff + m / a.G) * a.Hq + g * a.G + m % a.G) * D * EB
                             : nullptr;
#pragma unroll
    for (int t = 0; t < QOperand<BF16, D>::N; ++t) {
      if constexpr (BF16) {
        u32x4 raw = valid ? *reinterpret_cast<const u32x4 *>(qrow + (t * 32 + kgrp * 8) * EB) : u32x4{0, 0, 0, 0};
        qop[j].v[t] = __builtin_bit_cast(bf16x8, raw);
      } else {
        qop[j].v[t] = valid ? *reinterpret_cast<const f32x4 *>(qrow + (t * 16 + kgrp * 4) * EB)
                            : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  }

  // ---- stream the split's keys in tiles of KT ----
  constexpr int NKR = (KT * D * EB / 16) / 256;
  u32x4 kr[NKR];
  VItem<BF16, D> vi;
  const int ntiles = (k1 - k0 + KT - 1) / KT;
  load_k_tile<BF16, D>(kr, kbase, k0, k1, tid);
  load_v_tile<BF16, D>(vi, vbase, k0, k1, tid);

  for (int t = 0; t < ntiles; ++t) {
    const int kt = k0 + t * KT;
    if (t > 0) __syncthreads();
    store_k_tile<BF16, D>(ks, kr, tid);
    store_v_tile<BF16, D>(vts, vi, tid);
    __syncthreads();
    if (t + 1 < ntiles) {
      load_k_tile<BF16, D>(kr, kbase, kt + KT, k1, tid);
      load_v_tile<BF16, D>(vi, vbase, kt + KT, k1, tid);
    }

    // S^T = K Q^T for every active m-tile: sacc[j][sub] holds keys kt+sub*16+kgrp*4+r, row l16
    f32x4 sacc[MT][NSUB];
#pragma unroll
    for (int j = 0; j < MT; ++j)
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb) sacc[j][sb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int sb = 0; sb < NSUB; ++sb) {
      const char *krow = ks + (sb * 16 + l16) * KPITCH;
      if constexpr (BF16) {
#pragma unroll
        for (int st = 0; st < D / 32; ++st) {
          const bf16x8 av = *reinterpret_cast<const bf16x8 *>(krow + (st * 32 + kgrp * 8) * EB);
#pragma unroll
          for (int j = 0; j < MT; ++j)
            sacc[j][sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, qop[j].v[st], sacc[j][sb], 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int t4 = 0; t4 < D / 16; ++t4) {
          const f32x4 av = *reinterpret_cast<const f32x4 *>(krow + (t4 * 16 + kgrp * 4) * EB);
#pragma unroll
          for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int j = 0; j < MT; ++j)
              sacc[j][sb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], qop[j].v[t4][e], sacc[j][sb], 0, 0, 0);
        }
      }
    }

    // mask + online softmax (log2 domain); P kept in registers
    // every m-tile slot runs the same code; slots past the sequence's rows hold zero
    // queries and are never written out
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int lim = a.causal ? min(k1, ctx + row_i[j] + 1) : k1;  // keys < lim are visible
      float tmax = -INFINITY;
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt + sb * 16 + kgrp * 4 + r;
          const float sv = (key < lim) ? sacc[j][sb][r] * a.scale_log2 : -INFINITY;
          sacc[j][sb][r] = sv;
          tmax = fmaxf(tmax, sv);
        }
      tmax = fmaxf(tmax, shfl_xor_f(tmax, 16));
      tmax = fmaxf(tmax, shfl_xor_f(tmax, 32));
      const float mnew = fmaxf(m_run[j], tmax);
      const float muse = (mnew == -INFINITY) ? 0.f : mnew;
      const float alpha = fast_exp2(m_run[j] - muse);
      m_run[j] = mnew;
      float psum = 0.f;
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = fast_exp2(sacc[j][sb][r] - muse);
          sacc[j][sb][r] = p;
          psum += p;
        }
      l_run[j] = l_run[j] * alpha + psum;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) oacc[j][dt] *= alpha;
    }

    // O^T += V^T P^T
    if constexpr (BF16) {
#pragma unroll
      for (int kk = 0; kk < NSUB / 2; ++kk) {
        bf16x8 pb[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
          u32x4 raw{pack_bf16x2(sacc[j][2 * kk][0], sacc[j][2 * kk][1]),
                    pack_bf16x2(sacc[j][2 * kk][2], sacc[j][2 * kk][3]),
                    pack_bf16x2(sacc[j][2 * kk + 1][0], sacc[j][2 * kk + 1][1]),
                    pack_bf16x2(sacc[j][2 * kk + 1][2], sacc[j][2 * kk + 1][3])};
          pb[j] = __builtin_bit_cast(bf16x8, raw);
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const char *vrow = vts + (dt * 16 + l16) * VPITCH;
          const uint2 lo = *reinterpret_cast<const uint2 *>(vrow + (kk * 32 + kgrp * 4) * EB);
          const uint2 hi = *reinterpret_cast<const uint2 *>(vrow + (kk * 32 + 16 + kgrp * 4) * EB);
          const bf16x8 av = __builtin_bit_cast(bf16x8, (u32x4{lo.x, lo.y, hi.x, hi.y}));
#pragma unroll
          for (int j = 0; j < MT; ++j)
            oacc[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pb[j], oacc[j][dt], 0, 0, 0);
        }
      }
    } else {
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const f32x4 av = *reinterpret_cast<const f32x4 *>(vts + (dt * 16 + l16) * VPITCH + (sb * 16 + kgrp * 4) * EB);
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int j = 0; j < MT; ++j)
              oacc[j][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[r], sacc[j][sb][r], oacc[j][dt], 0, 0, 0);
        }
    }
  }

  // ---- row sums: reduce the per-lane partials over the four key groups ----
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    l_run[j] += shfl_xor_f(l_run[j], 16);
    l_run[j] += shfl_xor_f(l_run[j], 32);
  }

  auto out_row_ptr = [&](int m) -> char * {
    return reinterpret_cast<char *>(a.out) + ((size_t)(qoff + m / a.G) * a.Hq + g * a.G + m % a.G) * D * EB;
  };

  if (nsplit == 1) {
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int mt = wave + 4 * j;
      const int m = mt * 16 + l16;
      if (mt >= nmt || m >= M) continue;
      const float inv = 1.f / l_run[j];
      char *orow = out_row_ptr(m);
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const int d = dt * 16 + kgrp * 4;
        const f32x4 o = oacc[j][dt] * inv;
        if constexpr (BF16)
          *reinterpret_cast<uint2 *>(orow + d * EB) = uint2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
        else
          *reinterpret_cast<f32x4 *>(orow + d * EB) = o;
      }
    }
    return;
  }

  // ---- several splits: write this split's partials for the merge launch ----
  const size_t wrow = (size_t)it.slot * a.Mpad;
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    const int mt = wave + 4 * j;
    const int m = mt * 16 + l16;
    if (mt >= nmt || m >= M) continue;
    float *prow = a.part_o + (wrow + m) * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) *reinterpret_cast<f32x4 *>(prow + dt * 16 + kgrp * 4) = oacc[j][dt];
    if (kgrp == 0) a.part_ml[wrow + m] = float2{m_run[j], l_run[j]};
  }
}

// Merge of the split partials: workgroup (s, g, row block) combines
//   O = sum_sp 2^(m_sp - M) O_sp / sum_sp 2^(m_sp - M) l_sp,  M = max_sp m_sp
// for RB rows of the (sequence, kv head) group, D/4 threads per row, one float4 each.
// SB: splits whose loads are issued together (the host sizes it to the plan's split count).
template <bool BF16, int D, int SB>
__global__ __launch_bounds__(256) void block_attn_merge_kernel(AttnArgs a) {
  constexpr int EB = BF16 ? 2 : 4;
  constexpr int TPR = D / 4;       // threads per row
  constexpr int RB = 256 / TPR;    // rows per workgroup
  const int nrb = a.Mpad / RB + ((a.Mpad % RB) ? 1 : 0);
  const int rb = blockIdx.x % nrb;
  const int sg = blockIdx.x / nrb;
  const int s = sg / a.Hkv, g = sg % a.Hkv;
  const int qoff = ld_uniform(a.q_offsets, s);  // issued with the lengths, not after the merge
  int B;
  const int2 ps = attn_pair_slots(a, s, g, B);
  const int nsplit = ps.y;
  if (nsplit <= 1) return;  // no block, or written directly by the split kernel
  const int M = a.G * B;
  const int m = rb * RB + threadIdx.x / TPR;
  if (m >= M) return;
  const int d = (threadIdx.x % TPR) * 4;
  const size_t wbase = (size_t)ps.x * a.Mpad + m;  // row m of split 0
  // online merge over batches of SB splits whose loads are issued together (clamped, no
  // per-load branch): one memory round trip per batch instead of one per split
  float mx = -INFINITY, lsum = 0.f;
  f32x4 acc{0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < nsplit; s0 += SB) {
    float2 ml[SB];
    f32x4 po[SB];
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const size_t r = wbase + (size_t)min(s0 + k, nsplit - 1) * a.Mpad;
      ml[k] = a.part_ml[r];
      po[k] = *reinterpret_cast<const f32x4 *>(a.part_o + r * D + d);
    }
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      if (s0 + k >= nsplit || ml[k].x == -INFINITY) continue;  // a split with no visible key
      const float mn = fmaxf(mx, ml[k].x);
      const float wo = (mx == -INFINITY) ? 0.f : fast_exp2(mx - mn);
      const float wn = fast_exp2(ml[k].x - mn);
      lsum = lsum * wo + ml[k].y * wn;
      acc = acc * wo + po[k] * wn;
      mx = mn;
    }
  }
  const f32x4 o = acc * (1.f / lsum);
  char *orow = reinterpret_cast<char *>(a.out) + ((size_t)(qoff + m / a.G) * a.Hq + g * a.G + m % a.G) * D * EB;
  if constexpr (BF16)
    *reinterpret_cast<uint2 *>(orow + d * EB) = uint2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
  else
    *reinterpret_cast<f32x4 *>(orow + d * EB) = o;
}

}  // namespace sdb
