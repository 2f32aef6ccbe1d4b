// accept.hpp -- vocabulary-wide speculative acceptance for a ragged batch of blocks.
//
// Operation: verification accepts the longest consistent prefix of the drafted block
// (Fig. 1 caption; App. A.1) without changing the target's output distribution
// (Sec. 1; Sec. 3.1 "Metrics"): greedy matching at T = 0, and at T > 0 the standard
// lossless rule -- accept draft j with probability min(1, p_j(d_j)/q_j(d_j)); on the
// first rejection draw the token from max(0, p_j - q_j); if every draft is accepted
// draw the bonus token from the last target row.
//
// Kernels (gfx950).  An agent-scope fence per workgroup costs an L2 write-back on gfx950
// and one workgroup streams a row far below HBM speed, so every phase that needs a whole
// row spreads it over many workgroups and hands results on across a kernel boundary, or
// through tagged words that need no fence (the single launches below).  (Measured on the
// ragged Qwen3-4B batch at T = 1: drawing the token in the mass kernel's last workgroup per
// sequence, found by a counter behind a release fence, made the call 35.9 us against 29.7 us
// with the separate locate kernel.)
//   accept_stats_kernel     persistent grid over (row, vocab chunk) items of every target
//                           row, and every draft row when T > 0.  One streaming pass of
//                           16-byte loads: T = 0 keeps (max value, lowest index); T > 0 keeps
//                           an online (max, sum of exp2((x - max) log2e / T)) with one
//                           rescale per batch of loads.  Each item's record is filed under
//                           (sequence, block position) with the drafted token's logit (or
//                           the token itself at T = 0) and the position's uniform, so the
//                           decision needs one parallel round of loads.
//   accept_greedy_kernel    T = 0, one wavefront per sequence: lane i merges the records of
//                           position i, a ballot finds the first rejection.
//   accept_mass_kernel      T > 0, grid = (sequence, vocab chunk): every workgroup makes the
//                           small per-sequence decision, then sums the residual
//                           max(0, p_j - q_j) and p_j over its chunk of the selected row.
//   accept_locate_kernel    T > 0, one workgroup per sequence: scans the chunk sums for the
//                           chunk holding u* times the total mass, then scans that chunk in
//                           vocabulary order.
//   accept_fused_kernel     T = 0 in one launch: the statistics items, then one workgroup per
//                           sequence that waits for its records (tagged words) and decides.
//   accept_draw_kernel      T > 0, the mass and locate steps in one launch: the chunk sums are
//                           handed between the workgroups of a sequence as tagged words.
// The single launches run where the shape, the workspace and the stream allow them; the
// launches above stay for the other cases and give the same results bit for bit.
#pragma once

#include <limits.h>

#include <type_traits>

#include "common.hpp"

namespace sdb {

struct AcceptArgs {
  const void *target;
  const void *draft;
  const int *draft_tokens;
  const float *uniforms;
  const int *block_lens;
  const int *q_offsets;
  int *accept_len;
  int *next_token;
  // Records [kinds * S * mb, nch], kind 0 = target position, kind 1 = draft position (T > 0),
  // index (kind * S + s) * mb + j:
  //   T > 0: (max, sum, logit at the drafted token or NaN, uniform u_j)
  //   T = 0: (max value, index bits, drafted token bits or -1, -)
  float4 *stats;
  double2 *samp;      // [S, nch2]: (residual mass, p mass) per sampling chunk (T > 0)
  float4 *seqinfo;    // [S, 2]: (accept_len bits, residual?, target max, 1/target sum),
                      //         (draft max, 1/draft sum, u*, -)   (T > 0)
  int S, V, total_q, rows, mb, nch, nch2;
  float c;            // log2(e) / T (T > 0)
  // Single-launch greedy path (accept_fused_kernel): records handed between workgroups as
  // tagged words, (tag << 32) | payload bits, each written and read by one 64-bit agent-scope
  // atomic access.  Word k of a record carries tag + k * kTagStep, and a record counts only
  // when all three words carry their tags.  The block position is the last index, so that a
  // wavefront polling one word of every position touches one or two cache lines.
  unsigned long long *trec;  // [S, nch, 3, mb] record words (the T = 0 records above)
  unsigned tag;              // this call's tag (a bijective hash of a per-process call counter)
  int n_items;               // statistics workgroups; workgroups past them run the tail
  int spin_limit;            // polls before a waiting workgroup gives up
  // Single-launch draw (accept_draw_kernel, T > 0): the residual and p mass sums of every
  // sampling chunk (floats) as tagged words, word k (0 residual, 1 p) carrying tag + k * kTagStep,
  // in kSumReplicas copies, at index ((s * kSumReplicas + r) * 2 + k) * nch2 + chunk.
  unsigned long long *csum;
};

// Copies of the draw kernel's chunk sums: the workgroups of chunk c poll copy c mod
// kSumReplicas, so each cache line of sums serves a few pollers instead of all of a sequence's
// (ragged Qwen3-4B batch at T = 1, 75 chunks per row: sd_accept 22.76 us with one copy, 21.96
// with 16; 22.07 with 8, 21.99 with 32).
#ifndef SDB_SUM_REPLICAS
#define SDB_SUM_REPLICAS 16
#endif
constexpr int kSumReplicas = SDB_SUM_REPLICAS;
static_assert(kSumReplicas >= 1 && 2 * kSumReplicas <= 256, "one word of one copy per thread of the filing workgroup");

// ---- tagged words: one relaxed 64-bit atomic store or load at agent scope each ----
// A relaxed atomic access is single-copy atomic and coherent across the XCDs' L2 caches, so
// the payload read with this call's tag is the one written with it; no fence orders one word
// after another, and none is needed, since every word carries its own tag.
__device__ __forceinline__ void tag_put(unsigned long long *p, unsigned tag, uint32_t bits) {
  __hip_atomic_store(p, ((unsigned long long)tag << 32) | bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long tag_get(const unsigned long long *p) {
  return __hip_atomic_load(const_cast<unsigned long long *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool tag_is(unsigned long long w, unsigned tag) { return (unsigned)(w >> 32) == tag; }
// Tag step between the words of a record: leftover contents pass for a record only if every
// word's upper half matches its own tag -- about 2^-96 for a record of any earlier data, and
// never for memory filled with one repeated word.
constexpr unsigned kTagStep = 0x9e3779b9u;
__device__ __forceinline__ float tag_f(unsigned long long w) { return __uint_as_float((uint32_t)w); }

// Chunk `c` of `nch` of a row that starts at absolute element a0 and holds V elements.
// Elements are grouped in 16-byte vectors of VEC elements on absolute boundaries, spread
// evenly over the chunks (sizes differ by at most one, so no chunk is empty while the row
// has at least nch whole vectors); the unaligned head goes to chunk 0 and the tail to the
// last chunk.  Every chunk is a contiguous element range [e0, e1) of the row.
struct RowChunk {
  long long vb, ve;  // absolute vector range
  int hb, he;        // scalar head (relative elements)
  int tb, te;        // scalar tail (relative elements)
  int e0, e1;        // the chunk's contiguous relative range
};

template <int VEC>
__device__ __forceinline__ RowChunk row_chunk(long long a0, int V, int c, int nch) {
  RowChunk r;
  const long long o0 = (a0 + VEC - 1) / VEC, o1 = (a0 + V) / VEC;
  if (o1 <= o0) {  // no whole vector: chunk 0 takes every element
    r.vb = r.ve = 0;
    r.hb = 0;
    r.he = (c == 0) ? V : 0;
    r.tb = r.te = 0;
    r.e0 = 0;
    r.e1 = (c == 0) ? V : 0;
    if (c != 0) r.e0 = r.e1 = V;
    return r;
  }
  const long long nv = o1 - o0;
  r.vb = o0 + nv * c / nch;
  r.ve = o0 + nv * (c + 1) / nch;
  r.hb = 0;
  r.he = (c == 0) ? (int)(o0 * VEC - a0) : 0;
  r.tb = (int)(o1 * VEC - a0);
  r.te = (c == nch - 1) ? V : r.tb;
  r.e0 = (c == 0) ? 0 : (int)(r.vb * VEC - a0);
  r.e1 = (c == nch - 1) ? V : (int)(r.ve * VEC - a0);
  return r;
}

template <bool BF16>
__device__ __forceinline__ float load_elem(const void *base, long long idx) {
  if constexpr (BF16)
    return __uint_as_float(((uint32_t)reinterpret_cast<const uint16_t *>(base)[idx]) << 16);
  else
    return reinterpret_cast<const float *>(base)[idx];
}

// Unpack one 16-byte vector into VEC floats.
template <bool BF16>
__device__ __forceinline__ void unpack(const u32x4 &v, float *x) {
  if constexpr (BF16) {
    x[0] = bf16_lo(v.x); x[1] = bf16_hi(v.x); x[2] = bf16_lo(v.y); x[3] = bf16_hi(v.y);
    x[4] = bf16_lo(v.z); x[5] = bf16_hi(v.z); x[6] = bf16_lo(v.w); x[7] = bf16_hi(v.w);
  } else {
    x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y);
    x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
  }
}

// Largest s with key(s) <= r, where key(s) = q_offsets[s] - s*draft (non-decreasing);
// r is uniform across the workgroup.
__device__ __forceinline__ int owner_of_row(const int *off, int S, int r, int draft) {
  int lo = 0, hi = S - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (ld_uniform(off, mid) - mid * draft <= r) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// max(a, b, c) in one instruction.  Written as an instruction so that the compiler's IEEE-mode
// lowering of fmaxf, which first quiets each operand with an extra v_max_f32 x, x (one per
// unpacked element here), is not applied; logits are never signalling NaNs.
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// ---- greedy (T = 0) helpers: (value, index) with ties to the lower index ----
__device__ __forceinline__ void argmax_merge(float &bv, int &bi, float v, int i) {
  if (v > bv || (v == bv && i < bi)) { bv = v; bi = i; }
}

// ---- sampling helpers: (max, sum) pairs of sum exp2((x - max) c) ----
__device__ __forceinline__ void lse_merge(float &m, float &sum, float m2, float s2, float c) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;  // both empty
  sum = ((m == -INFINITY) ? 0.f : sum * fast_exp2((m - mn) * c)) +
        ((m2 == -INFINITY) ? 0.f : s2 * fast_exp2((m2 - mn) * c));
  m = mn;
}

// Vectors per fold of the T > 0 statistics (one maximum and one rescale per group): 4 against 2
// measured 21.72 against 21.92 us per sd_accept call at T = 1 on the ragged Qwen3-4B batch; 8
// needs 104 VGPRs, which leaves a second wave of workgroups.
#ifndef SDB_STATS_GROUP
#define SDB_STATS_GROUP 4
#endif
constexpr int kStatsVecs = 16;    // 16-byte vectors per thread per stats item (8, 10, 12, 14: 0.1-0.4 us slower per call at T = 1)
constexpr int kLocThreads = 256;  // locate kernel workgroup
constexpr int kMaxChunks2 = 4096; // sampling chunks per sequence
// Sampling chunks hold at most 256 whole vectors, so one vector per thread of the mass and
// locate kernels covers a chunk, unless the vocabulary needs more than kMaxChunks2 such
// chunks; then both kernels run with kTailVecsWide vectors per thread per round and the
// locate kernel recomputes runs longer than that element by element.
constexpr int kTailVecsWide = 8;

// One stats item in flight: its loads, issued together, and what processing it needs.  A
// statistics chunk is kStatsChunk whole vectors of the row (the last chunk holds the rest
// and may be empty), plus the row's unaligned head (chunk 0) and tail (last chunk).
constexpr int kStatsChunk = 256 * kStatsVecs;

template <int NV>
struct StatsItem {
  u32x4 v[NV];   // this thread's vectors (clamped loads; padding applied when processed)
  float xh, xt;  // head and tail element (or element tid of a tiny row)
  float uj;      // uniform of the position (target rows, T > 0)
  float xd;      // T > 0: the drafted token's logit where this chunk holds it, else NaN
  int rec, tok;  // record index (-1: not recorded), drafted token or -1
  int c;         // chunk index
  int e0;        // row-relative element of the chunk's first whole vector
  int nvc;       // whole vectors in the chunk
  int nh, ntl;   // head / tail elements handled by this chunk
  int tb;        // row-relative start of the tail
};

// Issue every load of `item`: this thread's vectors (uniform chunk base, 32-bit offsets) and
// one head and one tail element, first and unconditionally -- loads past the end are clamped
// onto valid addresses and replaced by padding when the item is processed, because a load
// under a branch makes the compiler wait for it.  Then the row's (sequence, position), its
// drafted token and uniform, through scalar loads, which do not wait for the vectors in
// flight.  VECS: every row holds a whole vector (V >= 2 VEC - 1);
// otherwise the vocabulary is below 256 elements, there is one chunk, and each thread loads
// element tid of the row.
template <bool BF16, bool SAMPLE, bool VECS>
__device__ __forceinline__ void stats_issue(const AcceptArgs &a, int item, StatsItem<kStatsVecs> &it) {
  constexpr int VEC = BF16 ? 8 : 4;
  const int tid = threadIdx.x;
  const int row = item / a.nch;
  it.c = item - row * a.nch;
  const bool is_draft = row >= a.total_q;
  const int rr = is_draft ? row - a.total_q : row;
  const char *base = reinterpret_cast<const char *>(is_draft ? a.draft : a.target);
  const unsigned long long a0 = (unsigned long long)rr * (unsigned)a.V;
  const int h = (int)((VEC - (unsigned)(a0 % VEC)) % VEC);  // head elements before the first whole vector
  const int nv = (a.V - h) / VEC;                           // whole vectors in the row
  const int v0 = it.c * kStatsChunk;
  it.nvc = max(0, min(kStatsChunk, nv - v0));
  it.e0 = h + v0 * VEC;
  it.tb = h + nv * VEC;
  const bool last = it.c == a.nch - 1;
  it.nh = (it.c == 0) ? h : 0;
  it.ntl = last ? a.V - it.tb : 0;
  if constexpr (VECS) {
    // the chunk's vectors; an empty chunk reads the row's last whole vector and discards it
    const char *cb = base + (a0 + h) * (BF16 ? 2 : 4) + (unsigned)min(v0, nv - 1) * 16u;
    const unsigned lastv = (unsigned)max(it.nvc, 1) - 1u;
    // non-temporal: each logit is read once by this pass (measured on the ragged Qwen3-4B batch
    // at T = 1: sd_accept 25.4 -> 24.5 us)
#pragma unroll
    for (int u = 0; u < kStatsVecs; ++u) {
      const v4u32 w = __builtin_nontemporal_load(reinterpret_cast<const v4u32 *>(cb + min((unsigned)tid + 256u * u, lastv) * 16u));
      it.v[u] = u32x4{w.x, w.y, w.z, w.w};
    }
    it.xh = load_elem<BF16>(base, a0 + min(tid, a.V - 1));
    it.xt = load_elem<BF16>(base, a0 + min(it.tb + tid, a.V - 1));
  } else {
    it.xh = load_elem<BF16>(base, a0 + min(tid, a.V - 1));
    it.xt = 0.f;
  }

  int sq, j, tok = -1;
  it.uj = 0.f;
  if (is_draft) {
    sq = owner_of_row(a.q_offsets, a.S, rr, 1);
    j = rr - (ld_uniform(a.q_offsets, sq) - sq);
    if (SAMPLE) tok = ld_uniform(a.draft_tokens, rr);
  } else {
    sq = owner_of_row(a.q_offsets, a.S, rr, 0);
    j = rr - ld_uniform(a.q_offsets, sq);
    if (rr + 1 < ld_uniform(a.q_offsets, sq + 1)) tok = ld_uniform(a.draft_tokens, rr - sq);
    if (SAMPLE) it.uj = ld_uniform(a.uniforms, rr);
  }
  it.rec = (j >= 0 && j < a.mb) ? ((is_draft ? a.S : 0) + sq) * a.mb + j : -1;
  it.tok = tok;
  // T > 0: the drafted token's logit by a scalar load of its own, in the chunk whose elements
  // hold it (head and tail included), so that no lane's registers are searched for it and no
  // wait on the vectors in flight comes before the arithmetic
  it.xd = NAN;
  if (SAMPLE && tok >= 0) {
    const int cs = (it.c == 0) ? 0 : it.e0;
    const int ce = last ? a.V : it.e0 + it.nvc * VEC;
    if (tok >= cs && tok < ce) {
      const unsigned long long e = a0 + (unsigned)tok;
      if constexpr (BF16) {
        const uint32_t w = ld_uniform(reinterpret_cast<const uint32_t *>(base), (long long)(e >> 1));
        it.xd = __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
      } else {
        it.xd = ld_uniform(reinterpret_cast<const float *>(base), (long long)e);
      }
    }
  }
}

// Reduce one landed item to its record: T > 0 (max, sum of exp2((x - max) c)) with one
// rescale per item, and the drafted token's logit as loaded at issue; T = 0 (max, lowest index).
template <bool BF16, bool SAMPLE, bool VECS, bool FUSED = false>
__device__ __forceinline__ void stats_process(const AcceptArgs &a, StatsItem<kStatsVecs> &it, float *sh_v,
                                              float *sh_s, int *sh_i) {
  constexpr int VEC = BF16 ? 8 : 4;
  constexpr uint32_t kPad = BF16 ? 0xff80ff80u : 0xff800000u;  // -inf in every element
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // head / tail elements this thread holds (row-relative index), or -inf
  const bool hv = VECS ? tid < it.nh : tid < a.V;
  const bool tv = VECS && tid < it.ntl;
  const int eh = tid, et = it.tb + tid;
  const float xh = hv ? it.xh : -INFINITY;
  const float xt = tv ? it.xt : -INFINITY;
  float bv = -INFINITY;  // greedy: best value / SAMPLE: the wavefront's max
  int bi = INT_MAX;      // greedy: index of best
  float sum = 0.f;       // SAMPLE: sum of exp2((x - bv) c)
  // Vectors past the end of a partial chunk were loaded from a clamped address; they become
  // padding in place (a full chunk skips this), so one reduction serves every chunk and the
  // registers hold one copy of the data.
  if (!VECS || it.nvc < kStatsChunk) {
#pragma unroll
    for (int u = 0; u < kStatsVecs; ++u)
      if (!(VECS && tid + 256 * u < it.nvc)) it.v[u] = u32x4{kPad, kPad, kPad, kPad};
  }
  auto vec_at = [&](int u) { return it.v[u]; };
  auto reduce = [&]() {
    if constexpr (SAMPLE) {
      // One pass over the elements, each unpacked once: a running (m, sum of exp2((x - m) c))
      // per thread, folded SDB_STATS_GROUP vectors at a time -- the group's maximum by v_max3,
      // one rescale of the running sum when the maximum moved, then exp2 per element.  About
      // five VALU instructions per element (unpack, max3/2, fma, exp2, add) against ten for a
      // max pass and an exp pass that each unpack.
      float m = -INFINITY;
      auto fold = [&](const float *x, auto nc) {
        constexpr int N = decltype(nc)::value;
        float mv = m;
#pragma unroll
        for (int e = 0; e < N; e += 2) mv = max3f(mv, x[e], x[e + 1]);
        // m = -inf: exp2(-inf) = 0 clears the empty sum; an unchanged maximum keeps it
        sum *= (mv > m) ? fast_exp2((m - mv) * a.c) : 1.f;
        m = mv;
        const float off = (mv == -INFINITY) ? 0.f : -mv * a.c;  // all padding so far: terms are 0
#pragma unroll
        for (int e = 0; e < N; ++e) sum += fast_exp2(fmaf(x[e], a.c, off));
      };
      constexpr int G = SDB_STATS_GROUP;  // vectors per group
      static_assert(kStatsVecs % G == 0, "whole groups");
#pragma unroll
      for (int u = 0; u < kStatsVecs; u += G) {
        float x[G * VEC];
#pragma unroll
        for (int g = 0; g < G; ++g) unpack<BF16>(vec_at(u + g), x + g * VEC);
        fold(x, std::integral_constant<int, G * VEC>{});
      }
      const float ht[2] = {xh, xt};
      fold(ht, std::integral_constant<int, 2>{});
      // the wavefront's reference maximum, and this thread's sum rescaled to it
      bv = wave_max_f(m);
      sum = (m == -INFINITY) ? 0.f : sum * fast_exp2((m - bv) * a.c);
      return;
    }
    // One pass: each vector's maximum (v_max3 over its elements), then the thread's maximum,
    // the first vector that holds it, and the first element of that vector equal to it --
    // about 2.3 VALU instructions per element against 7-8 for a compare and select on every
    // element (measured on MI355X).
    float vm[kStatsVecs];
#pragma unroll
    for (int u = 0; u < kStatsVecs; ++u) {
      float x[VEC];
      unpack<BF16>(vec_at(u), x);
      float m = max3f(x[0], x[1], x[2]);
#pragma unroll
      for (int e = 3; e + 1 < VEC; e += 2) m = max3f(m, x[e], x[e + 1]);
      if constexpr (VEC % 2 == 0) m = max3f(m, x[VEC - 1], x[VEC - 1]);
      vm[u] = m;
    }
    float bm = max3f(xh, xt, xt);
#pragma unroll
    for (int u = 0; u < kStatsVecs; u += 2) bm = max3f(bm, vm[u], vm[u + 1]);
    static_assert(kStatsVecs % 2 == 0, "vector maxima are merged in pairs");
    if (bm != -INFINITY) {  // first index of the maximum among this thread's elements
      int su = -1;
      u32x4 sel = vec_at(0);
#pragma unroll
      for (int u = kStatsVecs - 1; u >= 0; --u) {  // selects, not branches
        const bool hit = vm[u] == bm;
        const u32x4 w = vec_at(u);
        su = hit ? u : su;
        sel.x = hit ? w.x : sel.x;
        sel.y = hit ? w.y : sel.y;
        sel.z = hit ? w.z : sel.z;
        sel.w = hit ? w.w : sel.w;
      }
      int idx = INT_MAX;
      if (su >= 0) {
        float x[VEC];
        unpack<BF16>(sel, x);
        const int eb = it.e0 + (tid + 256 * su) * VEC;
#pragma unroll
        for (int e = VEC - 1; e >= 0; --e)
          if (x[e] == bm) idx = eb + e;
      }
      if (tv && xt == bm) idx = min(idx, et);
      if (hv && xh == bm) idx = min(idx, eh);
      bv = bm;
      bi = idx;
    }
  };

  float xd = it.xd;  // T > 0: uniform over the workgroup

  reduce();
  if constexpr (SAMPLE) {
    sum = wave_sum_f(sum);
  } else {
    // the wavefront's largest value (NaN never wins), then the lowest index holding it: the
    // argmax_merge order, by DPP lane moves instead of a butterfly of LDS shuffles
    const float wmax = wave_max_f(bv);
    bi = wave_min_i(bv == wmax ? bi : INT_MAX);
    bv = wmax;
  }

  if (lane == 0) { sh_v[wave] = bv; sh_s[wave] = sum; sh_i[wave] = bi; }
  __syncthreads();
  if (tid == 0) {
    for (int w2 = 1; w2 < 4; ++w2) {
      if constexpr (SAMPLE) {
        lse_merge(bv, sum, sh_v[w2], sh_s[w2], a.c);
      } else {
        argmax_merge(bv, bi, sh_v[w2], sh_i[w2]);
      }
    }
    if (it.rec >= 0) {
      if constexpr (FUSED) {  // (max, sum, drafted logit) or (max, index, drafted token); u_j is an input
        const int ks = it.rec / a.mb, j = it.rec - ks * a.mb;
        unsigned long long *w = a.trec + ((size_t)ks * a.nch + it.c) * 3 * a.mb + j;
        tag_put(w, a.tag, __float_as_uint(bv));
        tag_put(w + a.mb, a.tag + kTagStep, SAMPLE ? __float_as_uint(sum) : (uint32_t)bi);
        tag_put(w + 2 * a.mb, a.tag + 2 * kTagStep, SAMPLE ? __float_as_uint(xd) : (uint32_t)it.tok);
      } else {
        a.stats[(size_t)it.rec * a.nch + it.c] =
            SAMPLE ? float4{bv, sum, xd, it.uj} : float4{bv, __int_as_float(bi), __int_as_float(it.tok), 0.f};
      }
    }
  }
}

// One (row, vocab chunk) item per workgroup.  Measured on MI355X, this beats keeping a
// second item's loads in flight per workgroup: the pass is as much arithmetic as traffic,
// and more resident workgroups hide both.
template <bool BF16, bool SAMPLE, bool VECS>
#ifndef SDB_STATS_MINW
#define SDB_STATS_MINW 1
#endif
__global__ __launch_bounds__(256, SDB_STATS_MINW) void accept_stats_kernel(AcceptArgs a) {
  __shared__ float sh_v[8];
  __shared__ float sh_s[4];
  __shared__ int sh_i[4];
  StatsItem<kStatsVecs> it;
  stats_issue<BF16, SAMPLE, VECS>(a, blockIdx.x, it);
  stats_process<BF16, SAMPLE, VECS>(a, it, sh_v, sh_s, sh_i);
}

// Greedy decision for sequence s on one wavefront: lane i merges the records of block
// position i into its lowest-index argmax and tests the drafted token there.
__global__ __launch_bounds__(64) void accept_greedy_kernel(AcceptArgs a) {
  const int s = blockIdx.x;
  const int lane = threadIdx.x;
  const int B = ld_uniform(a.block_lens, s);
  const int n = B - 1;
  int gi = INT_MAX, tok = -1;
  if (lane < a.mb) {  // issued before B arrives; positions >= B are ignored below
    const float4 *st = a.stats + (size_t)(s * a.mb + lane) * a.nch;
    float gv = -INFINITY;
    for (int c0 = 0; c0 < a.nch; c0 += 8) {
      float4 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = st[min(c0 + k, a.nch - 1)];  // clamped: no per-load branch
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (c0 + k >= a.nch) v[k] = float4{-INFINITY, __int_as_float(INT_MAX), __int_as_float(-1), 0.f};
      if (c0 == 0) tok = __float_as_int(v[0].z);
#pragma unroll
      for (int k = 0; k < 8; ++k) argmax_merge(gv, gi, v[k].x, __float_as_int(v[k].y));
    }
    if (gi == INT_MAX) gi = 0;  // every logit -inf: all tie, lowest index
  }
  const bool rejects = (lane < n) && (tok != gi);
  const unsigned long long rej = __ballot(rejects);
  const int acc = rej ? (__ffsll((long long)rej) - 1) : max(n, 0);
  const int next = __builtin_amdgcn_readlane(gi, acc);  // wave-uniform lane
  if (lane == 0) {
    a.accept_len[s] = acc;
    a.next_token[s] = next;
  }
}

// Merge the chunk records (max, sum, captured logit, u) of one target position and one
// draft position: every load of a batch of kRecBatch chunks of both issued together, then
// the maximum over chunks and one exp2 per chunk against it.  Exactly one chunk holds the
// captured logit; the others carry NaN, which fmaxf drops.
constexpr int kRecBatch = 8;

__device__ __forceinline__ void merge_one(const float4 *v, int k0, int nch, float c, float &m, float &sum,
                                          float &x) {
  float bm = -INFINITY;
#pragma unroll
  for (int k = 0; k < kRecBatch; ++k) bm = fmaxf(bm, v[k].x);
  const float mn = fmaxf(m, bm);
  if (mn == -INFINITY) return;
  float acc = (m == -INFINITY) ? 0.f : sum * fast_exp2((m - mn) * c);
#pragma unroll
  for (int k = 0; k < kRecBatch; ++k) {
    if (k0 + k < nch) acc += v[k].y * fast_exp2((v[k].x - mn) * c);  // exp2(-inf) = 0
    x = fmaxf(x, v[k].z);
  }
  m = mn;
  sum = acc;
}

__device__ __forceinline__ void merge_records2(const float4 *st, const float4 *sd, int nch, float c, float &tm,
                                               float &ts, float &td, float &u, float &qm, float &qs, float &dd) {
  for (int c0 = 0; c0 < nch; c0 += kRecBatch) {
    float4 v[kRecBatch], w[kRecBatch];
#pragma unroll
    for (int k = 0; k < kRecBatch; ++k) {  // clamped: no per-load branch
      v[k] = st[min(c0 + k, nch - 1)];
      w[k] = sd[min(c0 + k, nch - 1)];
    }
#pragma unroll
    for (int k = 0; k < kRecBatch; ++k)
      if (c0 + k >= nch) v[k] = w[k] = float4{-INFINITY, 0.f, NAN, 0.f};
    if (c0 == 0) u = v[0].w;
    merge_one(v, c0, nch, c, tm, ts, td);
    merge_one(w, c0, nch, c, qm, qs, dd);
  }
}

// Sampling decision for sequence s on one wavefront (lane i = block position i).  Every
// lane returns the accepted length, the normalisers of the selected row and u*.
struct SampleSel {
  int acc;
  bool residual;
  float tm, ts, qm, qs, ustar;
};

// The decision from the merged records of lane i's block position: target (tm, ts, td),
// draft (qm, qs, dd), uniform u.
__device__ __forceinline__ SampleSel sample_select(const AcceptArgs &a, int B, float tm, float ts, float td, float u,
                                                   float qm, float qs, float dd) {
  const int lane = threadIdx.x & 63;
  const int n = B - 1;
  bool rejects = false;
  if (lane < n) {
    // rho = p(d) / q(d) = exp2((td - tm) c - (dd - qm) c) * qs / ts; q(d) = 0 accepts.  A token
    // outside the vocabulary leaves td, dd NaN and is rejected.
    const double lr = (double)((td - tm) * a.c) - (double)((dd - qm) * a.c);
    const double rho = (dd != -INFINITY) ? exp2(lr) * (double)qs / (double)ts : INFINITY;
    rejects = !((double)u < rho);
  }
  const unsigned long long rej = __ballot(rejects);
  SampleSel r;
  r.acc = rej ? (__ffsll((long long)rej) - 1) : max(n, 0);
  r.residual = r.acc < n;
  r.tm = lane_f(tm, r.acc);  // wave-uniform lanes: scalar reads
  r.ts = lane_f(ts, r.acc);
  r.qm = lane_f(qm, r.acc);
  r.qs = lane_f(qs, r.acc);
  r.ustar = lane_f(u, B - 1);
  return r;
}

__device__ SampleSel sampling_decision(const AcceptArgs &a, int s, int B) {
  const int lane = threadIdx.x & 63;
  float tm = -INFINITY, ts = 0.f, qm = -INFINITY, qs = 0.f, td = NAN, dd = NAN, u = 0.f;
  if (lane < a.mb)  // issued before B arrives; positions >= B are ignored below
    merge_records2(a.stats + (size_t)(s * a.mb + lane) * a.nch, a.stats + (size_t)((a.S + s) * a.mb + lane) * a.nch,
                   a.nch, a.c, tm, ts, td, u, qm, qs, dd);
  return sample_select(a, B, tm, ts, td, u, qm, qs, dd);
}

// Normalised sampling mass of one element: p = exp2((t - tm) c) / ts, and at a rejection the
// residual max(0, p - q) with q = exp2((d - qm) c) / qs.  Both sampling kernels call this one
// function, so a chunk's mass and its rescan agree.
struct SampleParams {
  float tm, inv_ts, qm, inv_qs, c;
};

__device__ __forceinline__ void elem_masses(float t, float q, const SampleParams &sp, bool residual, float &r,
                                            float &p) {
  p = fast_exp2((t - sp.tm) * sp.c) * sp.inv_ts;
  if (residual) {
    const float qq = fast_exp2((q - sp.qm) * sp.c) * sp.inv_qs;
    r = fmaxf(p - qq, 0.f);
  } else {
    r = p;
  }
}

// Sampling masses, grid = (sequence, vocab chunk).  Every workgroup makes the decision,
// then sums the residual (or p at the bonus row) and p over its chunk of the selected row.
// NV: vectors per thread per round; the plan sizes chunks so that one round of NV = 1 covers
// a chunk, which keeps the dependent chain at one round of row loads after the decision.
// Wavefront 0 of a workgroup of sequence s decides and leaves the selection in sh_si:
// (accept_len bits, residual?, target max, 1/target sum), (draft max, 1/draft sum, u*, -).
// With publish set it also writes accept_len and the selection for the locate kernel.
__device__ __forceinline__ void mass_decide(const AcceptArgs &a, int s, int B, float4 *sh_si, bool publish) {
  if (threadIdx.x >= 64) return;
  const SampleSel sel = sampling_decision(a, s, B);
  if (threadIdx.x == 0) {
    const float4 s0{__int_as_float(sel.acc), sel.residual ? 1.f : 0.f, sel.tm, 1.f / sel.ts};
    const float4 s1{sel.residual ? sel.qm : 0.f, sel.residual ? 1.f / sel.qs : 0.f, sel.ustar, 0.f};
    sh_si[0] = s0;
    sh_si[1] = s1;
    if (publish) {
      a.accept_len[s] = sel.acc;
      a.seqinfo[2 * s] = s0;
      a.seqinfo[2 * s + 1] = s1;
    }
  }
}

template <bool BF16, int NV>
__global__ __launch_bounds__(256) void accept_mass_kernel(AcceptArgs a) {
  constexpr int VEC = BF16 ? 8 : 4;
  __shared__ float4 sh_si[2];
  __shared__ double sh_r[4], sh_p[4];
  const int s = blockIdx.x / a.nch2;
  const int c = blockIdx.x % a.nch2;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int B = ld_uniform(a.block_lens, s);
  const int off = ld_uniform(a.q_offsets, s);
  mass_decide(a, s, B, sh_si, c == 0);
  __syncthreads();
  const float4 si0 = sh_si[0], si1 = sh_si[1];
  const int j = __float_as_int(si0.x);
  const bool residual = si0.y != 0.f;
  const SampleParams sp{si0.z, si0.w, si1.x, si1.y, a.c};
  const long long ta0 = (long long)(off + j) * a.V;
  const long long da0 = (long long)(off - s + j) * a.V;  // read only at a rejection
  const RowChunk ch = row_chunk<VEC>(ta0, a.V, c, a.nch2);
  // the draft row shares the target row's vector alignment iff (ta0 - da0) % VEC == 0
  const bool dvec = ((ta0 - da0) % VEC) == 0;

  float sr = 0.f, spm = 0.f;
  const char *tbase = reinterpret_cast<const char *>(a.target) + ch.vb * 16;
  const char *dbase = reinterpret_cast<const char *>(a.draft) + (ch.vb + (da0 - ta0) / VEC) * 16;
  const unsigned nvc = (unsigned)(ch.ve - ch.vb);
  for (unsigned r0 = tid; r0 < nvc; r0 += 256u * NV) {
    u32x4 tb[NV], qb[NV];
#pragma unroll
    for (int u = 0; u < NV; ++u) {  // clamped: no per-load branch (r0 < nvc here)
      const unsigned r = min(r0 + 256u * u, nvc - 1u);
      tb[u] = *reinterpret_cast<const u32x4 *>(tbase + r * 16u);
      qb[u] = u32x4{0u, 0u, 0u, 0u};
    }
    if (residual && dvec) {
#pragma unroll
      for (int u = 0; u < NV; ++u)
        qb[u] = *reinterpret_cast<const u32x4 *>(dbase + min(r0 + 256u * u, nvc - 1u) * 16u);
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const unsigned r = r0 + 256u * u;
      float t[VEC], q[VEC];
      unpack<BF16>(tb[u], t);
      unpack<BF16>(qb[u], q);
      if (residual && !dvec && r < nvc) {
        const long long e = (ch.vb + r) * VEC - ta0 + da0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) q[i] = load_elem<BF16>(a.draft, e + i);
      }
      float vr = 0.f, vp = 0.f;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        float er, ep;
        elem_masses(t[i], q[i], sp, residual, er, ep);
        vr += er;
        vp += ep;
      }
      if (r < nvc) {
        sr += vr;
        spm += vp;
      }
    }
  }
  // scalar head (chunk 0) and tail (last chunk): fewer than 2 * VEC elements each
  for (int e = ch.hb + tid; e < ch.he; e += 256) {
    float er, ep;
    elem_masses(load_elem<BF16>(a.target, ta0 + e), residual ? load_elem<BF16>(a.draft, da0 + e) : 0.f, sp,
                residual, er, ep);
    sr += er;
    spm += ep;
  }
  for (int e = ch.tb + tid; e < ch.te; e += 256) {
    float er, ep;
    elem_masses(load_elem<BF16>(a.target, ta0 + e), residual ? load_elem<BF16>(a.draft, da0 + e) : 0.f, sp,
                residual, er, ep);
    sr += er;
    spm += ep;
  }
  const float wr = wave_sum_f(sr), wp = wave_sum_f(spm);
  if (lane == 0) { sh_r[wave] = wr; sh_p[wave] = wp; }
  __syncthreads();
  if (tid == 0)  // rounded to float, as accept_draw_kernel files them
    a.samp[(size_t)s * a.nch2 + c] = double2{(double)(float)(sh_r[0] + sh_r[1] + sh_r[2] + sh_r[3]),
                                             (double)(float)(sh_p[0] + sh_p[1] + sh_p[2] + sh_p[3])};
}

// Final draw for sequence s (T > 0), one workgroup per sequence.  Wavefront 0 scans the
// chunk sums for the chunk whose cumulative-mass interval holds u* times the total; then each
// thread takes a contiguous run of that chunk's vectors (thread 0 also the unaligned head,
// the last thread the tail), the runs' masses are scanned across the workgroup, and the one
// thread whose interval holds the target walks its run in vocabulary order.  A residual with
// no mass (rounding only) draws from p instead.  NV: the longest run kept in registers (runs
// of the planned chunk sizes fit; longer ones are recomputed element by element).
constexpr int kLocSums = 4;  // chunk sums per lane held in registers by the chunk search

// cm[k] for a wave-uniform k < kLocSums, by selects (no indexed register access).
__device__ __forceinline__ double2 pick_sums(const double2 *cm, int k) {
  double2 r = cm[0];
#pragma unroll
  for (int q = 1; q < kLocSums; ++q)
    if (q == k) r = cm[q];
  return r;
}

// Chunk search of the final draw on one wavefront: chunk_sums(k) gives lane l the (residual,
// p) sums of chunk 64k + l (zero past the last chunk).  The total is u* times the summed mass;
// the chosen chunk is the one whose cumulative interval [lo, hi) holds it, consecutive
// intervals meeting exactly across passes.  A residual with no mass (rounding only) draws from
// p; a target past every interval (rounding) takes the last chunk with mass (cex = INFINITY:
// its last token with mass).
struct ChunkPick {
  int kc;
  double cex, tgt;
  bool use_p;
};

template <typename F>
__device__ __forceinline__ ChunkPick chunk_search(F chunk_sums, int passes, double ustar) {
  bool any_r = false;
  for (int k = 0; k < passes; ++k) any_r |= __ballot(chunk_sums(k).x > 0.0) != 0;
  const bool use_p = !any_r;
  double carry = 0.0;
  for (int k = 0; k < passes; ++k) {
    const double2 c2 = chunk_sums(k);
    double ex;
    const double in = wave_scan_d(use_p ? c2.y : c2.x, &ex);
    carry += readlane_d(in, 63);
  }
  const double tgt = ustar * carry;
  int kc = -1, klast = -1;
  double cex = 0.0;
  carry = 0.0;
  for (int k = 0; k < passes; ++k) {
    const double2 c2 = chunk_sums(k);
    const double m = use_p ? c2.y : c2.x;
    double ex;
    const double in = wave_scan_d(m, &ex);
    const double lo = carry + ex, hi = carry + in;
    const unsigned long long hit = __ballot(m > 0.0 && lo <= tgt && tgt < hi);
    if (hit && kc < 0) {
      const int l = __ffsll((long long)hit) - 1;
      kc = 64 * k + l;
      cex = readlane_d(lo, l);
    }
    const unsigned long long pos = __ballot(m > 0.0);
    if (pos) klast = 64 * k + 63 - __clzll((long long)pos);
    carry = carry + readlane_d(in, 63);
  }
  ChunkPick r;
  r.kc = kc >= 0 ? kc : max(klast, 0);
  r.cex = kc >= 0 ? cex : INFINITY;
  r.tgt = tgt;
  r.use_p = use_p;
  return r;
}

template <bool BF16, int NV>
__global__ __launch_bounds__(kLocThreads) void accept_locate_kernel(AcceptArgs a) {
  constexpr int VEC = BF16 ? 8 : 4;
  constexpr int NW = kLocThreads / 64;
  __shared__ double sh_w[NW];
  __shared__ double sh_cex, sh_tgt;
  __shared__ int sh_kc, sh_usep, sh_hit;
  __shared__ int sh_last[NW];
  const int s = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float4 si0 = ld_uniform4(a.seqinfo, 2 * s), si1 = ld_uniform4(a.seqinfo, 2 * s + 1);
  const int off = ld_uniform(a.q_offsets, s);
  const int j = __float_as_int(si0.x);
  const bool residual = si0.y != 0.f;
  const SampleParams sp{si0.z, si0.w, si1.x, si1.y, a.c};
  const double ustar = (double)si1.z;

  if (wave == 0) {
    // chunk search, 64 chunks per pass.  Up to 64 * kLocSums chunk sums are loaded in one
    // round; more are loaded pass by pass.
    const double2 *cs = a.samp + (size_t)s * a.nch2;
    const int passes = (a.nch2 + 63) / 64;
    double2 cm[kLocSums];
#pragma unroll
    for (int k = 0; k < kLocSums; ++k) {  // clamped: no per-load branch
      cm[k] = cs[min(64 * k + lane, a.nch2 - 1)];
      if (64 * k + lane >= a.nch2) cm[k] = double2{0.0, 0.0};
    }
    auto chunk_sums = [&](int k) {
      if (k < kLocSums) return pick_sums(cm, k);
      double2 r = cs[min(64 * k + lane, a.nch2 - 1)];
      if (64 * k + lane >= a.nch2) r = double2{0.0, 0.0};
      return r;
    };
    const ChunkPick cp = chunk_search(chunk_sums, passes, ustar);
    if (lane == 0) {
      sh_kc = cp.kc;
      sh_cex = cp.cex;
      sh_tgt = cp.tgt;
      sh_usep = cp.use_p;
      sh_hit = 0;
    }
  }
  __syncthreads();
  const int kc = sh_kc;
  const double cex = sh_cex, tgt = sh_tgt;
  const bool use_q = residual && !sh_usep;

  // this thread's run of chunk kc: vectors [v0, v1) relative to the chunk, plus the head
  // (thread 0) and the tail (last thread) elements
  const long long ta0 = (long long)(off + j) * a.V;
  const long long da0 = (long long)(off - s + j) * a.V;
  const RowChunk cc = row_chunk<VEC>(ta0, a.V, kc, a.nch2);
  const int nvc = (int)(cc.ve - cc.vb);
  const int rv = (nvc + kLocThreads - 1) / kLocThreads;
  const int v0 = min(tid * rv, nvc), v1 = min(v0 + rv, nvc);
  const bool dvec = ((ta0 - da0) % VEC) == 0;
  auto mass_at = [&](float t, float q) {
    float r, p;
    elem_masses(t, q, sp, use_q, r, p);
    return use_q ? r : p;
  };
  auto scalar_mass = [&](int e) {
    return mass_at(load_elem<BF16>(a.target, ta0 + e), use_q ? load_elem<BF16>(a.draft, da0 + e) : 0.f);
  };
  double own = 0.0;
  int elast = -1;
  if (tid == 0)
    for (int e = cc.hb; e < cc.he; ++e) {
      const float m = scalar_mass(e);
      own += (double)m;
      if (m > 0.f) elast = e;
    }
  float mreg[NV * VEC];
  const char *tb = reinterpret_cast<const char *>(a.target) + cc.vb * 16;
  const char *db = reinterpret_cast<const char *>(a.draft) + (cc.vb + (da0 - ta0) / VEC) * 16;
  if (rv <= NV) {
    u32x4 tv[NV], qv[NV];
#pragma unroll
    for (int u = 0; u < NV; ++u) tv[u] = qv[u] = u32x4{0u, 0u, 0u, 0u};
    if (nvc > 0) {  // clamped: no per-load branch
      const bool ld_q = use_q && dvec;
#pragma unroll
      for (int u = 0; u < NV; ++u) {
        const unsigned r = (unsigned)min(v0 + u, nvc - 1);
        tv[u] = *reinterpret_cast<const u32x4 *>(tb + r * 16u);
        if (ld_q) qv[u] = *reinterpret_cast<const u32x4 *>(db + r * 16u);
      }
    }
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      float t[VEC], q[VEC];
      unpack<BF16>(tv[u], t);
      unpack<BF16>(qv[u], q);
      const int eb = (int)((cc.vb + v0 + u) * VEC - ta0);
      if (use_q && !dvec && v0 + u < v1) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) q[i] = load_elem<BF16>(a.draft, da0 + eb + i);
      }
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const float m = (v0 + u < v1) ? mass_at(t[i], q[i]) : 0.f;
        mreg[u * VEC + i] = m;
        own += (double)m;
        if (m > 0.f) elast = eb + i;
      }
    }
  } else {  // runs longer than the register window: masses recomputed by the walk below
    for (int v = v0; v < v1; ++v) {
      const int eb = (int)((cc.vb + v) * VEC - ta0);
      for (int i = 0; i < VEC; ++i) {
        const float m = scalar_mass(eb + i);
        own += (double)m;
        if (m > 0.f) elast = eb + i;
      }
    }
  }
  if (tid == kLocThreads - 1)
    for (int e = cc.tb; e < cc.te; ++e) {
      const float m = scalar_mass(e);
      own += (double)m;
      if (m > 0.f) elast = e;
    }

  // workgroup scan of the run masses; consecutive intervals meet exactly
  double ex;
  const double in = wave_scan_d(own, &ex);
  if (lane == 63) sh_w[wave] = in;
  __syncthreads();
  double before = 0.0;
  for (int w2 = 0; w2 < wave; ++w2) before += sh_w[w2];
  const double lo = cex + (before + ex), hi = cex + (before + in);
  if (own > 0.0 && lo <= tgt && tgt < hi) {  // at most one thread: walk its run
    double cum = lo;
    int found = -1;
    auto step = [&](int e, float m) {
      if (found < 0 && m > 0.f) {
        if (cum + (double)m > tgt) found = e;
        cum += (double)m;
      }
    };
    if (tid == 0)
      for (int e = cc.hb; e < cc.he; ++e) step(e, scalar_mass(e));
    if (rv <= NV) {
#pragma unroll
      for (int u = 0; u < NV; ++u)
#pragma unroll
        for (int i = 0; i < VEC; ++i)
          if (v0 + u < v1) step((int)((cc.vb + v0 + u) * VEC - ta0) + i, mreg[u * VEC + i]);
    } else {
      for (int v = v0; v < v1; ++v) {
        const int eb = (int)((cc.vb + v) * VEC - ta0);
        for (int i = 0; i < VEC; ++i) step(eb + i, scalar_mass(eb + i));
      }
    }
    if (tid == kLocThreads - 1)
      for (int e = cc.tb; e < cc.te; ++e) step(e, scalar_mass(e));
    a.next_token[s] = found >= 0 ? found : elast;  // rounding: the run's last token with mass
    sh_hit = 1;
  }
  const int wl = wave_max_i(elast);
  if (lane == 0) sh_last[wave] = wl;
  __syncthreads();
  if (tid == 0 && !sh_hit) {  // rounding: the chunk's last token with mass (0 if none)
    int t = -1;
    for (int w2 = 0; w2 < NW; ++w2) t = max(t, sh_last[w2]);
    a.next_token[s] = max(t, 0);
  }
}

// ===========================================================================================
// Single-launch greedy acceptance (T = 0).  The statistics items above run as the first
// n_items workgroups and file their records as tagged words; one workgroup per sequence after
// them waits for its sequence's records and decides as accept_greedy_kernel does.  Only those
// tail workgroups wait, and only for words that statistics workgroups (which never wait)
// write, so the launch completes whenever the tail workgroups can be resident at once (the
// host launches it only then).  A wait gives up after spin_limit polls and the sequence
// reports -1; a fresh tag per call makes a call ignore whatever an earlier call (or any other
// use of the workspace) left behind.  Results equal the two-kernel path's bit for bit.
// Measured on the ragged Qwen3-4B batch: 15.0 us per call against 17.2 us for two launches.
// At T > 0 a launch holding the statistics too needs two waits in a row (records, then every
// sampling chunk's sums); each poll round is a trip to memory (about 1.5 us) and the
// workgroups of a sequence see the records up to a round apart, so that single launch
// measured 26.8 us against 24.1 us for three launches.  The statistics stay a launch of their
// own at T > 0, and accept_draw_kernel below joins the mass and locate steps.
// ===========================================================================================
constexpr int kFusedMaxNch = 8;  // statistics chunks per row (one batch of records)
static_assert(kFusedMaxNch == kRecBatch, "a position's records merge as one batch");

// Polls until every word a lane needs carries this call's tag (the loop is wavefront-uniform),
// sleeping between rounds; false after spin_limit rounds.  poll() issues one round of loads
// and returns whether this lane has everything.
template <typename F>
__device__ __forceinline__ bool spin_until(const AcceptArgs &a, F poll) {
  for (int it = 0;; ++it) {
    if (__all(poll())) return true;
    if (it >= a.spin_limit) return false;
    __builtin_amdgcn_s_sleep(2);
  }
}

// One lane waits for one word: the record a sequence's last statistics workgroup files, so
// that the full poll rarely needs a second round.
__device__ __forceinline__ bool wait_word(const AcceptArgs &a, const unsigned long long *w) {
  return spin_until(a, [&]() { return tag_is(tag_get(w), a.tag); });
}

// The tagged records of block position `lane` of sequence s, NCH chunks of three words; pay
// receives the payloads.  Every round loads every word (no load sits under a branch) and keeps
// those that carry their tag.
template <int NCH>
__device__ __forceinline__ bool poll_records(const AcceptArgs &a, int s, bool need, uint32_t (&pay)[3 * kFusedMaxNch]) {
  const int lane = threadIdx.x & 63;
  const unsigned long long *base = a.trec + (size_t)s * NCH * 3 * a.mb + min(lane, a.mb - 1);
  unsigned miss = need ? ((1u << (3 * NCH)) - 1u) : 0u;
#pragma unroll
  for (int i = 0; i < 3 * kFusedMaxNch; ++i) pay[i] = 0u;
  return spin_until(a, [&]() {
    unsigned long long w[3 * NCH];
#pragma unroll
    for (int i = 0; i < 3 * NCH; ++i) w[i] = tag_get(base + (size_t)i * a.mb);
#pragma unroll
    for (int i = 0; i < 3 * NCH; ++i)
      if (((miss >> i) & 1u) && tag_is(w[i], a.tag + (unsigned)(i % 3) * kTagStep)) {
        pay[i] = (uint32_t)w[i];
        miss &= ~(1u << i);
      }
    return miss == 0u;
  });
}

// poll_records with the chunk count as a constant (nch <= kFusedMaxNch, checked by the host).
__device__ __forceinline__ bool poll_records_n(const AcceptArgs &a, int s, bool need,
                                               uint32_t (&pay)[3 * kFusedMaxNch]) {
  switch (a.nch) {
    case 1: return poll_records<1>(a, s, need, pay);
    case 2: return poll_records<2>(a, s, need, pay);
    case 3: return poll_records<3>(a, s, need, pay);
    case 4: return poll_records<4>(a, s, need, pay);
    case 5: return poll_records<5>(a, s, need, pay);
    case 6: return poll_records<6>(a, s, need, pay);
    case 7: return poll_records<7>(a, s, need, pay);
    default: return poll_records<8>(a, s, need, pay);
  }
}

// The records of chunks [0, nch) as the two-kernel path pads them for its one batch.
__device__ __forceinline__ void records_batch(const AcceptArgs &a, const uint32_t (&pay)[3 * kFusedMaxNch],
                                              float4 (&v)[kRecBatch], float4 pad) {
#pragma unroll
  for (int k = 0; k < kRecBatch; ++k)
    v[k] = (k < a.nch) ? float4{__uint_as_float(pay[3 * k]), __uint_as_float(pay[3 * k + 1]),
                                __uint_as_float(pay[3 * k + 2]), 0.f}
                       : pad;
}

// Word 0 of the record that sequence s's highest-numbered statistics item files: the last
// chunk of its last row.
__device__ __forceinline__ const unsigned long long *last_record(const AcceptArgs &a, int s, int Bc) {
  return a.trec + ((size_t)s * a.nch + (a.nch - 1)) * 3 * a.mb + (Bc - 1);
}

// T = 0: one workgroup per sequence; wavefront 0 merges and decides as accept_greedy_kernel.
__device__ void fused_greedy_tail(const AcceptArgs &a, int s) {
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  const int B = ld_uniform(a.block_lens, s);
  const int Bc = min(max(B, 1), a.mb);
  const int n = B - 1;
  bool ok = true;
  if (lane == 0) ok = wait_word(a, last_record(a, s, Bc));
  ok = __builtin_amdgcn_readlane(ok ? 1 : 0, 0) != 0;
  uint32_t pay[3 * kFusedMaxNch];
  if (ok) ok = poll_records_n(a, s, lane < Bc, pay);
  if (!ok) {
    if (lane == 0) {
      a.accept_len[s] = -1;
      a.next_token[s] = -1;
    }
    return;
  }
  int gi = INT_MAX, tok = -1;
  {
    float gv = -INFINITY;
    float4 v[kRecBatch];
    records_batch(a, pay, v, float4{-INFINITY, __int_as_float(INT_MAX), __int_as_float(-1), 0.f});
    tok = __float_as_int(v[0].z);
#pragma unroll
    for (int k = 0; k < kRecBatch; ++k) argmax_merge(gv, gi, v[k].x, __float_as_int(v[k].y));
    if (gi == INT_MAX) gi = 0;  // every logit -inf: all tie, lowest index
  }
  const bool rejects = (lane < n) && (tok != gi);
  const unsigned long long rej = __ballot(rejects);
  const int acc = rej ? (__ffsll((long long)rej) - 1) : max(n, 0);
  const int next = __builtin_amdgcn_readlane(gi, acc);  // wave-uniform lane
  if (lane == 0) {
    a.accept_len[s] = acc;
    a.next_token[s] = next;
  }
}

// At most 128 VGPRs: four workgroups per CU, so that the tail's workgroups fit at once.
template <bool BF16, bool VECS>
__global__ __launch_bounds__(256, 4) void accept_fused_kernel(AcceptArgs a) {
  if ((int)blockIdx.x < a.n_items) {
    __shared__ float sh_v[8];
    __shared__ float sh_s[4];
    __shared__ int sh_i[4];
    StatsItem<kStatsVecs> it;
    stats_issue<BF16, false, VECS>(a, blockIdx.x, it);
    stats_process<BF16, false, VECS, true>(a, it, sh_v, sh_s, sh_i);
    return;
  }
  fused_greedy_tail(a, (int)blockIdx.x - a.n_items);
}

// ===========================================================================================
// Sampling draw in one launch (T > 0, sampling chunks of at most 256 vectors).  Grid =
// (sequence, sampling chunk), as accept_mass_kernel: every workgroup decides and sums its chunk
// of the selected row as that kernel does, keeping its elements' masses in registers, and files
// the chunk's two sums as tagged words.  While wavefront 0 waits for every chunk sum of the
// sequence, the workgroup scans its own chunk as accept_locate_kernel would (run masses and
// their prefixes over the chunk).  Every workgroup of a sequence then runs the locate kernel's
// chunk search on the same words, so all agree on the chunk that holds u* times the total, and
// only that chunk's workgroup goes on: the thread whose interval holds the target walks its run
// and writes the outputs.  The sums are the mass kernel's, rounded to float as that kernel files
// them, and the scans are the locate kernel's, so results agree bit for bit with the two
// launches.  Every workgroup waits for all workgroups of its sequence, so the host launches it
// only when the whole grid fits on the device at once with a quarter to spare.  A wait that
// gives up after spin_limit polls writes -1 to both outputs of its sequence; the chosen chunk's
// workgroup, once its wait has succeeded, writes the exact values, so an output that is not -1
// is exact.  Measured on the ragged Qwen3-4B batch at T = 1: 22.7 us per call against 24.3 us
// for the statistics, mass and locate launches (A/B, same box): the wait for the last chunk sum
// (one round trip, about 1.5 us) replaces a kernel boundary and the locate kernel's two rounds
// of loads.
// ===========================================================================================

// Poll the chunk sums of sequence s: lane l receives chunk 64k + l in cm[k] for k < P (zero
// past the last chunk).  Rounds load only the residual sums, one word per chunk, until each
// carries its tag: every workgroup of a sequence polls the same lines.  The p sums matter only
// when no chunk has residual mass (the chunk search then draws from p); only then are they
// polled too.  No load sits under a per-lane branch.  (Measured on the ragged Qwen3-4B batch:
// polling all four halves of two double sums per chunk, 25.4 us per call; one float word,
// 24.3 us; keeping two rounds in flight, a new one every half round trip, 23.9 us against
// 22.7 us with one round at a time, since every extra load lands on the lines the sequence's
// other workgroups poll.)
template <int P>
__device__ __forceinline__ bool poll_chunk_sums(const AcceptArgs &a, int s, int copy, double2 (&cm)[kLocSums]) {
  static_assert(P >= 1 && P <= kLocSums, "chunk sums held in registers");
  const int lane = threadIdx.x & 63;
  const unsigned long long *base = a.csum + (size_t)(s * kSumReplicas + copy) * 2 * a.nch2;
  float r[P], pm[P];
  unsigned miss = 0u;
#pragma unroll
  for (int k = 0; k < P; ++k) {
    r[k] = pm[k] = 0.f;
    if (64 * k + lane < a.nch2) miss |= 1u << k;
  }
  auto poll = [&](int kind, float (&dst)[P]) {
    const unsigned tag = a.tag + (unsigned)kind * kTagStep;
    unsigned m = miss;
    auto issue = [&](unsigned long long (&w)[P]) {
#pragma unroll
      for (int k = 0; k < P; ++k) w[k] = tag_get(base + (size_t)kind * a.nch2 + min(64 * k + lane, a.nch2 - 1));
    };
    auto take = [&](const unsigned long long (&w)[P]) {
#pragma unroll
      for (int k = 0; k < P; ++k)
        if (((m >> k) & 1u) && tag_is(w[k], tag)) {
          dst[k] = tag_f(w[k]);
          m &= ~(1u << k);
        }
      return m == 0u;
    };
    return spin_until(a, [&]() {
      unsigned long long w[P];
      issue(w);
      return take(w);
    });
  };
  bool ok = poll(0, r);
  bool any_r = false;
#pragma unroll
  for (int k = 0; k < P; ++k) any_r |= __ballot(r[k] > 0.f) != 0;
  if (ok && !any_r) ok = poll(1, pm);
#pragma unroll
  for (int k = 0; k < kLocSums; ++k) cm[k] = double2{0.0, 0.0};
#pragma unroll
  for (int k = 0; k < P; ++k) cm[k] = double2{(double)r[k], (double)pm[k]};
  return ok;
}

__device__ __forceinline__ bool poll_chunk_sums_n(const AcceptArgs &a, int s, int copy, double2 (&cm)[kLocSums]) {
  static_assert(kLocSums == 4, "one case per pass count");
  switch ((a.nch2 + 63) / 64) {
    case 1: return poll_chunk_sums<1>(a, s, copy, cm);
    case 2: return poll_chunk_sums<2>(a, s, copy, cm);
    case 3: return poll_chunk_sums<3>(a, s, copy, cm);
    default: return poll_chunk_sums<4>(a, s, copy, cm);
  }
}

template <bool BF16>
__global__ __launch_bounds__(256, 4) void accept_draw_kernel(AcceptArgs a) {
  constexpr int VEC = BF16 ? 8 : 4;
  constexpr int NW = 4;
  static_assert(kLocThreads == 64 * NW, "the chunk scan runs on the whole workgroup");
  __shared__ float4 sh_si[2];
  __shared__ double sh_r[NW], sh_p[NW], sh_w[NW];
  __shared__ float sh_em[2][2][2 * VEC];  // [head, tail][residual, p] masses of the scalar elements
  __shared__ double sh_cex, sh_tgt;
  __shared__ int sh_kc, sh_usep, sh_ok, sh_hit, sh_last[NW];
  const int s = blockIdx.x / a.nch2;
  const int c = blockIdx.x % a.nch2;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int B = ld_uniform(a.block_lens, s);
  const int off = ld_uniform(a.q_offsets, s);
  mass_decide(a, s, B, sh_si, false);
  __syncthreads();
  const float4 si0 = sh_si[0], si1 = sh_si[1];
  const int j = __float_as_int(si0.x);
  const bool residual = si0.y != 0.f;
  const SampleParams sp{si0.z, si0.w, si1.x, si1.y, a.c};
  const long long ta0 = (long long)(off + j) * a.V;
  const long long da0 = (long long)(off - s + j) * a.V;  // read only at a rejection
  const RowChunk ch = row_chunk<VEC>(ta0, a.V, c, a.nch2);
  const bool dvec = ((ta0 - da0) % VEC) == 0;
  const int nvc = (int)(ch.ve - ch.vb);  // <= 256: one vector per thread
  const bool has = tid < nvc;

  // ---- the chunk's masses: accept_mass_kernel's sums, element by element ----
  float mr[VEC], mp[VEC];
  float sr = 0.f, spm = 0.f;
  {
    u32x4 tb{0u, 0u, 0u, 0u}, qb{0u, 0u, 0u, 0u};
    if (nvc > 0) {  // clamped: no per-load branch
      const unsigned r = (unsigned)min(tid, nvc - 1);
      tb = *reinterpret_cast<const u32x4 *>(reinterpret_cast<const char *>(a.target) + (ch.vb + r) * 16);
      if (residual && dvec)
        qb = *reinterpret_cast<const u32x4 *>(reinterpret_cast<const char *>(a.draft) +
                                              (ch.vb + r + (da0 - ta0) / VEC) * 16);
    }
    float t[VEC], q[VEC];
    unpack<BF16>(tb, t);
    unpack<BF16>(qb, q);
    if (residual && !dvec && has) {
      const long long e = (ch.vb + tid) * VEC - ta0 + da0;
#pragma unroll
      for (int i = 0; i < VEC; ++i) q[i] = load_elem<BF16>(a.draft, e + i);
    }
    float vr = 0.f, vp = 0.f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      elem_masses(t[i], q[i], sp, residual, mr[i], mp[i]);
      vr += mr[i];
      vp += mp[i];
    }
    if (has) {
      sr += vr;
      spm += vp;
    }
  }
  // scalar head (chunk 0) and tail (last chunk): fewer than 2 * VEC elements each, one per thread
  for (int e = ch.hb + tid; e < ch.he; e += 256) {
    float er, ep;
    elem_masses(load_elem<BF16>(a.target, ta0 + e), residual ? load_elem<BF16>(a.draft, da0 + e) : 0.f, sp,
                residual, er, ep);
    sr += er;
    spm += ep;
    if (e - ch.hb < 2 * VEC) { sh_em[0][0][e - ch.hb] = er; sh_em[0][1][e - ch.hb] = ep; }
  }
  for (int e = ch.tb + tid; e < ch.te; e += 256) {
    float er, ep;
    elem_masses(load_elem<BF16>(a.target, ta0 + e), residual ? load_elem<BF16>(a.draft, da0 + e) : 0.f, sp,
                residual, er, ep);
    sr += er;
    spm += ep;
    if (e - ch.tb < 2 * VEC) { sh_em[1][0][e - ch.tb] = er; sh_em[1][1][e - ch.tb] = ep; }
  }
  const float wr = wave_sum_f(sr), wp = wave_sum_f(spm);
  if (lane == 0) { sh_r[wave] = wr; sh_p[wave] = wp; }
  __syncthreads();
  if (tid < 2 * kSumReplicas) {  // the chunk's sums, rounded to float as accept_mass_kernel files
    // them; one word of one copy per lane
    const float cr = (float)(sh_r[0] + sh_r[1] + sh_r[2] + sh_r[3]), cp = (float)(sh_p[0] + sh_p[1] + sh_p[2] + sh_p[3]);
    const int k = tid & 1, r = tid >> 1;
    tag_put(a.csum + ((size_t)(s * kSumReplicas + r) * 2 + k) * a.nch2 + c, a.tag + (unsigned)k * kTagStep,
            __float_as_uint(k ? cp : cr));
  }

  // ---- the chunk's scan, ahead of the chunk search: accept_locate_kernel's run masses
  // (residual masses at a rejection) and their prefixes over the chunk.  Only where no chunk
  // of the sequence has residual mass (rounding only) is it redone with p. ----
  const int eb = (int)((ch.vb + tid) * VEC - ta0);
  float mm[VEC];
  double pre_lo, pre_hi, own;
  int elast;
  auto chunk_scan = [&](bool use_q) {
    own = 0.0;
    elast = -1;
    if (tid == 0)
      for (int e = ch.hb; e < ch.he; ++e) {
        const float m = use_q ? sh_em[0][0][e - ch.hb] : sh_em[0][1][e - ch.hb];
        own += (double)m;
        if (m > 0.f) elast = e;
      }
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      const float m = has ? (use_q ? mr[i] : mp[i]) : 0.f;
      mm[i] = m;
      own += (double)m;
      if (m > 0.f) elast = eb + i;
    }
    if (tid == kLocThreads - 1)
      for (int e = ch.tb; e < ch.te; ++e) {
        const float m = use_q ? sh_em[1][0][e - ch.tb] : sh_em[1][1][e - ch.tb];
        own += (double)m;
        if (m > 0.f) elast = e;
      }
    double ex;
    const double in = wave_scan_d(own, &ex);
    const int wl = wave_max_i(elast);
    if (lane == 63) sh_w[wave] = in;
    if (lane == 0) sh_last[wave] = wl;
    __syncthreads();
    double before = 0.0;
    for (int w2 = 0; w2 < wave; ++w2) before += sh_w[w2];
    pre_lo = before + ex;
    pre_hi = before + in;
  };
  chunk_scan(residual);

  // ---- every chunk sum of the sequence, then the chunk search ----
  if (wave == 0) {
    double2 cm[kLocSums];
    const bool ok = poll_chunk_sums_n(a, s, c % kSumReplicas, cm);
    if (ok) {
      const ChunkPick cp = chunk_search([&](int k) { return pick_sums(cm, k); }, (a.nch2 + 63) / 64,
                                        (double)si1.z);
      if (lane == 0) {
        sh_kc = cp.kc;
        sh_cex = cp.cex;
        sh_tgt = cp.tgt;
        sh_usep = cp.use_p;
      }
    }
    if (lane == 0) {
      sh_ok = ok;
      sh_hit = 0;
    }
  }
  __syncthreads();
  if (!sh_ok) {
    if (tid == 0) {
      a.accept_len[s] = -1;
      a.next_token[s] = -1;
    }
    return;
  }
  if (sh_kc != c) return;

  // ---- the chosen chunk: the thread whose interval holds the target walks its run ----
  const bool use_q = residual && !sh_usep;
  if (use_q != residual) {  // workgroup-uniform
    __syncthreads();        // every read of sh_w and sh_last above is done
    chunk_scan(use_q);
  }
  const double cex = sh_cex, tgt = sh_tgt;
  const double lo = cex + pre_lo, hi = cex + pre_hi;
  if (own > 0.0 && lo <= tgt && tgt < hi) {  // at most one thread: walk its run
    double cum = lo;
    int found = -1;
    auto step = [&](int e, float m) {
      if (found < 0 && m > 0.f) {
        if (cum + (double)m > tgt) found = e;
        cum += (double)m;
      }
    };
    if (tid == 0)
      for (int e = ch.hb; e < ch.he; ++e) step(e, use_q ? sh_em[0][0][e - ch.hb] : sh_em[0][1][e - ch.hb]);
#pragma unroll
    for (int i = 0; i < VEC; ++i)
      if (has) step(eb + i, mm[i]);
    if (tid == kLocThreads - 1)
      for (int e = ch.tb; e < ch.te; ++e) step(e, use_q ? sh_em[1][0][e - ch.tb] : sh_em[1][1][e - ch.tb]);
    a.next_token[s] = found >= 0 ? found : elast;  // rounding: the run's last token with mass
    a.accept_len[s] = j;
    sh_hit = 1;
  }
  __syncthreads();
  if (tid == 0 && !sh_hit) {  // rounding: the chunk's last token with mass (0 if none)
    int t = -1;
    for (int w2 = 0; w2 < NW; ++w2) t = max(t, sh_last[w2]);
    a.next_token[s] = max(t, 0);
    a.accept_len[s] = j;
  }
}

}  // namespace sdb
