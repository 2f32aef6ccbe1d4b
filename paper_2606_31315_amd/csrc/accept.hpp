// accept.hpp -- vocabulary-wide speculative acceptance for a ragged batch of blocks.
//
// Operation: verification accepts the longest consistent prefix of the drafted block
// (Fig. 1 caption; App. A.1) without changing the target's output distribution
// (Sec. 1; Sec. 3.1 "Metrics"): greedy matching at T = 0, and at T > 0 the standard
// lossless rule -- accept draft j with probability min(1, p_j(d_j)/q_j(d_j)); on the
// first rejection draw the token from max(0, p_j - q_j); if every draft is accepted
// draw the bonus token from the last target row.
//
// Kernels (gfx950); kernel boundaries are the only cross-workgroup synchronisation
// (an agent-scope fence per workgroup costs an L2 writeback on gfx950):
//   accept_stats_kernel     grid = (row, vocab chunk) over every target row, and every
//                           draft row when T > 0.  One streaming pass of 16-byte loads:
//                           T = 0 keeps (max value, lowest index); T > 0 keeps an online
//                           (max, sum of exp2((x - max) log2e / T)) with one rescale per
//                           batch of loads, never per element.
//   accept_greedy_kernel    T = 0, one wavefront per sequence: merge the chunk partials,
//                           lane i tests drafted position i, a ballot finds the first
//                           rejection; writes accept_len and the next token.
//   accept_sample_kernel    T > 0, grid = (sequence, vocab chunk): every workgroup redoes
//                           the small per-sequence decision (lane i tests position i,
//                           ballot), then sums the residual max(0, p - q) (or p at the
//                           bonus row) over its chunk.
//   accept_scan_kernel      T > 0, one workgroup per sequence: locate the chunk holding
//                           u* times the total mass and scan it in vocabulary order.
#pragma once

#include <limits.h>

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
  float2 *stats;      // [rows, nch]: (max, sum) at T > 0; (max value, index bits) at T = 0
  float4 *seqinfo;    // [S, 2]: (row, residual?, target max, 1/target sum), (draft max, 1/draft sum, 0, 0)
  double2 *samp;      // [S, nch2]: (residual mass, p mass) per chunk
  int S, V, total_q, nch, nch2;
  float c;            // log2(e) / T (T > 0)
};

// Chunk `c` of `nch` of a row that starts at absolute element a0 and holds V elements.
// Elements are grouped in 16-byte vectors of VEC elements on absolute boundaries; the
// unaligned head goes to chunk 0 and the tail to the last chunk.  Every chunk is a
// contiguous element range [e0, e1) of the row.
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
  const long long per = (nv + nch - 1) / nch;
  r.vb = min(o0 + per * c, o1);
  r.ve = min(r.vb + per, o1);
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

// Largest s with key(s) <= r, where key(s) = q_offsets[s] - s*draft (non-decreasing).
__device__ __forceinline__ int owner_of_row(const int *off, int S, int r, int draft) {
  int lo = 0, hi = S - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (off[mid] - mid * draft <= r) lo = mid; else hi = mid - 1;
  }
  return lo;
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

constexpr int kUnroll = 4;  // 16-byte vectors in flight per thread per batch

template <bool BF16, bool SAMPLE>
__global__ __launch_bounds__(256) void accept_stats_kernel(AcceptArgs a) {
  constexpr int VEC = BF16 ? 8 : 4;
  __shared__ float sh_v[4];
  __shared__ float sh_s[4];
  __shared__ int sh_i[4];

  const int row = blockIdx.x / a.nch;
  const int c = blockIdx.x % a.nch;
  const bool is_draft = row >= a.total_q;
  const int rr = is_draft ? row - a.total_q : row;
  const void *base = is_draft ? a.draft : a.target;
  const long long a0 = (long long)rr * a.V;
  const RowChunk ch = row_chunk<VEC>(a0, a.V, c, a.nch);
  const int tid = threadIdx.x;

  float bv = -INFINITY;  // greedy: best value / SAMPLE: running max
  int bi = INT_MAX;      // greedy: index of best
  float sum = 0.f;       // SAMPLE: sum of exp2((x - bv) c)

  // scalar head and tail
  for (int e = ch.hb + tid; e < ch.he; e += 256) {
    const float x = load_elem<BF16>(base, a0 + e);
    if constexpr (SAMPLE) lse_merge(bv, sum, x, 1.f, a.c);
    else if (x > bv) { bv = x; bi = e; }
  }
  // vectors: full batches of kUnroll loads in flight per thread, then single vectors
  const u32x4 *vbase = reinterpret_cast<const u32x4 *>(base);
  long long v = ch.vb + tid;
  for (; v + 256LL * (kUnroll - 1) < ch.ve; v += 256LL * kUnroll) {
    u32x4 buf[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) buf[u] = vbase[v + 256LL * u];
    float x[kUnroll][VEC];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) unpack<BF16>(buf[u], x[u]);
    if constexpr (SAMPLE) {
      float bm = -INFINITY;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
#pragma unroll
        for (int e = 0; e < VEC; ++e) bm = fmaxf(bm, x[u][e]);
      if (bm > bv) {
        sum = (bv == -INFINITY) ? 0.f : sum * fast_exp2((bv - bm) * a.c);
        bv = bm;
      }
      if (bv != -INFINITY) {
        const float off = -bv * a.c;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
#pragma unroll
          for (int e = 0; e < VEC; ++e) sum += fast_exp2(fmaf(x[u][e], a.c, off));
      }
    } else {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int e0 = (int)((v + 256LL * u) * VEC - a0);
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          if (x[u][e] > bv) { bv = x[u][e]; bi = e0 + e; }
      }
    }
  }
  for (; v < ch.ve; v += 256) {
    float x[VEC];
    unpack<BF16>(vbase[v], x);
    const int e0 = (int)(v * VEC - a0);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      if constexpr (SAMPLE) lse_merge(bv, sum, x[e], 1.f, a.c);
      else if (x[e] > bv) { bv = x[e]; bi = e0 + e; }
    }
  }
  if (ch.tb < ch.te) {
    for (int e = ch.tb + tid; e < ch.te; e += 256) {
      const float x = load_elem<BF16>(base, a0 + e);
      if constexpr (SAMPLE) lse_merge(bv, sum, x, 1.f, a.c);
      else argmax_merge(bv, bi, x, e);
    }
  }

  // wavefront then workgroup reduction
  const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
  for (int msk = 1; msk < 64; msk <<= 1) {
    const float ov = __shfl_xor(bv, msk, 64);
    if constexpr (SAMPLE) {
      const float os = __shfl_xor(sum, msk, 64);
      lse_merge(bv, sum, ov, os, a.c);
    } else {
      const int oi = __shfl_xor(bi, msk, 64);
      argmax_merge(bv, bi, ov, oi);
    }
  }
  if (lane == 0) { sh_v[wave] = bv; sh_s[wave] = sum; sh_i[wave] = bi; }
  __syncthreads();
  if (tid == 0) {
    for (int w2 = 1; w2 < 4; ++w2) {
      if constexpr (SAMPLE) lse_merge(bv, sum, sh_v[w2], sh_s[w2], a.c);
      else argmax_merge(bv, bi, sh_v[w2], sh_i[w2]);
    }
    a.stats[(size_t)row * a.nch + c] = SAMPLE ? float2{bv, sum} : float2{bv, __int_as_float(bi)};
  }

}

// Greedy decision for sequence s on one wavefront: lane i merges the chunk partials of
// target row i into its lowest-index argmax and tests drafted position i.
template <bool BF16>
__global__ __launch_bounds__(64) void accept_greedy_kernel(AcceptArgs a) {
  const int s = blockIdx.x;
  const int lane = threadIdx.x;
  const int B = a.block_lens[s];
  const int n = B - 1;
  const int off = a.q_offsets[s];
  const int tok = (lane < n) ? a.draft_tokens[off - s + lane] : 0;
  int gi = INT_MAX;
  if (lane < B) {
    const float2 *st = a.stats + (size_t)(off + lane) * a.nch;
    float gv = -INFINITY;
    for (int c0 = 0; c0 < a.nch; c0 += 8) {
      float2 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = (c0 + k < a.nch) ? st[c0 + k] : float2{-INFINITY, __int_as_float(INT_MAX)};
#pragma unroll
      for (int k = 0; k < 8; ++k) argmax_merge(gv, gi, v[k].x, __float_as_int(v[k].y));
    }
    if (gi == INT_MAX) gi = 0;  // every logit -inf: all tie, lowest index
  }
  const bool rejects = (lane < n) && (tok != gi);
  const unsigned long long rej = __ballot(rejects);
  const int acc = rej ? (__ffsll((long long)rej) - 1) : max(n, 0);
  const int next = __shfl(gi, acc, 64);
  if (lane == 0) {
    a.accept_len[s] = acc;
    a.next_token[s] = next;
  }
}

// Merge a row's chunk partials (max, sum) with the loads issued in batches of 8.
__device__ __forceinline__ void merge_lse_partials(const float2 *st, int nch, float c, float &m, float &sum) {
  for (int c0 = 0; c0 < nch; c0 += 8) {
    float2 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = (c0 + k < nch) ? st[c0 + k] : float2{-INFINITY, 0.f};
#pragma unroll
    for (int k = 0; k < 8; ++k) lse_merge(m, sum, v[k].x, v[k].y, c);
  }
}

// Sampling decision for sequence s on one wavefront (lane i = block position i).
// Returns, in every lane, the accepted length and the normalisers of the selected row.
struct SampleSel {
  int acc;
  bool residual;
  float tm, ts, qm, qs;
};

template <bool BF16>
__device__ SampleSel sampling_decision(const AcceptArgs &a, int s) {
  const int lane = threadIdx.x & 63;
  const int B = a.block_lens[s];
  const int n = B - 1;
  const int off = a.q_offsets[s];
  const int doff = off - s;
  float tm = -INFINITY, ts = 0.f, qm = -INFINITY, qs = 0.f;
  bool rejects = false;
  // issue the draft token load first: the two logit gathers depend on it
  const int d = (lane < n) ? a.draft_tokens[doff + lane] : 0;
  if (lane < B) merge_lse_partials(a.stats + (size_t)(off + lane) * a.nch, a.nch, a.c, tm, ts);
  if (lane < n) {
    merge_lse_partials(a.stats + (size_t)(a.total_q + doff + lane) * a.nch, a.nch, a.c, qm, qs);
    const float td = load_elem<BF16>(a.target, (long long)(off + lane) * a.V + d);
    const float dd = load_elem<BF16>(a.draft, (long long)(doff + lane) * a.V + d);
    // rho = p(d) / q(d) = exp2((td - tm) c - (dd - qm) c) * qs / ts; q(d) = 0 accepts
    const double lr = (double)((td - tm) * a.c) - (double)((dd - qm) * a.c);
    const double rho = (dd != -INFINITY) ? exp2(lr) * (double)qs / (double)ts : INFINITY;
    rejects = !((double)a.uniforms[off + lane] < rho);
  }
  const unsigned long long rej = __ballot(rejects);
  SampleSel r;
  r.acc = rej ? (__ffsll((long long)rej) - 1) : max(n, 0);
  r.residual = r.acc < n;
  r.tm = __shfl(tm, r.acc, 64);
  r.ts = __shfl(ts, r.acc, 64);
  r.qm = __shfl(qm, r.acc, 64);
  r.qs = __shfl(qs, r.acc, 64);
  return r;
}

// Residual / target mass of one element in the sampling pass.  si0 = (row, residual?,
// target max, 1/target sum), si1 = (draft max, 1/draft sum, -, -).
__device__ __forceinline__ void sample_masses(float t, float q, const float4 &si0, const float4 &si1, float c,
                                              float &r, float &p) {
  p = fast_exp2((t - si0.z) * c) * si0.w;
  if (si0.y != 0.f) {
    const float qq = fast_exp2((q - si1.x) * c) * si1.y;
    r = fmaxf(p - qq, 0.f);
  } else {
    r = p;
  }
}

template <bool BF16>
__global__ __launch_bounds__(256) void accept_sample_kernel(AcceptArgs a) {
  constexpr int VEC = BF16 ? 8 : 4;
  __shared__ double sh_r[4], sh_p[4];
  __shared__ float4 sh_si[2];

  const int s = blockIdx.x / a.nch2;
  const int c = blockIdx.x % a.nch2;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (wave == 0) {
    const SampleSel sel = sampling_decision<BF16>(a, s);
    if (lane == 0) {
      const float4 si0{__int_as_float(sel.acc), sel.residual ? 1.f : 0.f, sel.tm, 1.f / sel.ts};
      const float4 si1{sel.residual ? sel.qm : 0.f, sel.residual ? 1.f / sel.qs : 0.f, 0.f, 0.f};
      sh_si[0] = si0;
      sh_si[1] = si1;
      if (c == 0) {
        a.accept_len[s] = sel.acc;
        a.seqinfo[2 * s] = si0;
        a.seqinfo[2 * s + 1] = si1;
      }
    }
  }
  __syncthreads();
  const float4 si0 = sh_si[0], si1 = sh_si[1];
  const int j = __float_as_int(si0.x);
  const int off = a.q_offsets[s];
  const long long ta0 = (long long)(off + j) * a.V;
  const long long da0 = (long long)(off - s + j) * a.V;  // read only for a residual draw
  const bool residual = si0.y != 0.f;
  const RowChunk ch = row_chunk<VEC>(ta0, a.V, c, a.nch2);

  float sr = 0.f, sp = 0.f;
  auto scalar_range = [&](int e0, int e1) {
    for (int e = e0 + tid; e < e1; e += 256) {
      const float t = load_elem<BF16>(a.target, ta0 + e);
      const float q = residual ? load_elem<BF16>(a.draft, da0 + e) : 0.f;
      float r, p;
      sample_masses(t, q, si0, si1, a.c, r, p);
      sr += r;
      sp += p;
    }
  };
  scalar_range(ch.hb, ch.he);
  // The draft row shares the target row's vector alignment only when (ta0 - da0) is a
  // multiple of VEC; otherwise its elements are read one by one.
  const bool draft_vec = ((ta0 - da0) % VEC) == 0;
  const u32x4 *tv = reinterpret_cast<const u32x4 *>(a.target);
  for (long long v = ch.vb + tid; v < ch.ve; v += 256) {
    float t8[VEC], q8[VEC];
    unpack<BF16>(tv[v], t8);
    const long long rel = v * VEC - ta0;
    if (residual) {
      if (draft_vec) {
        unpack<BF16>(reinterpret_cast<const u32x4 *>(a.draft)[(da0 + rel) / VEC], q8);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) q8[e] = load_elem<BF16>(a.draft, da0 + rel + e);
      }
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) q8[e] = 0.f;
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      float r, p;
      sample_masses(t8[e], q8[e], si0, si1, a.c, r, p);
      sr += r;
      sp += p;
    }
  }
  scalar_range(ch.tb, ch.te);

  double dr = sr, dp = sp;
#pragma unroll
  for (int msk = 1; msk < 64; msk <<= 1) {
    dr += __shfl_xor(dr, msk, 64);
    dp += __shfl_xor(dp, msk, 64);
  }
  if (lane == 0) { sh_r[wave] = dr; sh_p[wave] = dp; }
  __syncthreads();
  if (tid == 0)
    a.samp[(size_t)s * a.nch2 + c] =
        double2{sh_r[0] + sh_r[1] + sh_r[2] + sh_r[3], sh_p[0] + sh_p[1] + sh_p[2] + sh_p[3]};
}

constexpr int kScanRun = 24;  // elements per thread in the final scan (chunks hold <= 4096 + 7)

// Block-wide inclusive scan of one double per thread (256 threads): wavefront shuffles,
// then the wavefront totals through LDS.  Returns the inclusive prefix; *total gets the sum.
__device__ __forceinline__ double block_scan_incl(double v, double *sh4, double *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  if (lane == 63) sh4[wave] = v;
  __syncthreads();
  double before = 0.0;
  for (int w2 = 0; w2 < wave; ++w2) before += sh4[w2];
  *total = sh4[0] + sh4[1] + sh4[2] + sh4[3];
  __syncthreads();
  return v + before;
}

// Final inverse-CDF draw for sequence s: locate the chunk holding u* times the total
// mass (block-wide scan of the chunk masses), then scan that chunk in vocabulary order
// with a contiguous run of elements per thread, held in registers.
template <bool BF16>
__global__ __launch_bounds__(256) void accept_scan_kernel(AcceptArgs a) {
  constexpr int VEC = BF16 ? 8 : 4;
  __shared__ double sh4[4];
  __shared__ int s_chunk, s_lastpos, s_found;

  const int s = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int B = a.block_lens[s];
  const int off = a.q_offsets[s];
  const float4 si0 = a.seqinfo[2 * s], si1 = a.seqinfo[2 * s + 1];
  const int j = __float_as_int(si0.x);
  const bool residual = si0.y != 0.f;
  const long long ta0 = (long long)(off + j) * a.V;
  const long long da0 = (long long)(off - s + j) * a.V;
  const double2 *cs = a.samp + (size_t)s * a.nch2;
  const double ustar = (double)a.uniforms[off + B - 1];

  // totals of the residual and of p (p is the fallback when the residual has no mass)
  double tr = 0.0, tp = 0.0;
  for (int k = tid; k < a.nch2; k += 256) {
    const double2 c = cs[k];
    tr += c.x;
    tp += c.y;
  }
  double tot_r, tot_p;
  block_scan_incl(tr, sh4, &tot_r);
  block_scan_incl(tp, sh4, &tot_p);
  const bool use_p = !(tot_r > 0.0);
  const double tot = use_p ? tot_p : tot_r;
  const double tgt = ustar * tot;
  if (tid == 0) {
    s_chunk = INT_MAX;
    s_lastpos = 0;
    s_found = INT_MAX;
  }
  __syncthreads();
  // locate the chunk: first k whose cumulative mass exceeds tgt
  double carry = 0.0, chunk_excl = 0.0;
  for (int base = 0; base < a.nch2; base += 256) {
    const int k = base + tid;
    const double m = (k < a.nch2) ? (use_p ? cs[k].y : cs[k].x) : 0.0;
    double seg;
    const double incl = block_scan_incl(m, sh4, &seg) + carry;
    if (m > 0.0) {
      atomicMax(&s_lastpos, k);
      if (incl - m <= tgt && tgt < incl) atomicMin(&s_chunk, k);
    }
    carry += seg;
  }
  __syncthreads();
  const bool found_chunk = s_chunk != INT_MAX;
  const int cstar = found_chunk ? s_chunk : s_lastpos;  // rounding: last chunk with mass
  // mass before chunk cstar (recomputed the same way by every thread)
  {
    double before = 0.0;
    for (int k = tid; k < cstar; k += 256) before += use_p ? cs[k].y : cs[k].x;
    double t;
    block_scan_incl(before, sh4, &t);
    chunk_excl = t;
  }
  const double ctgt = found_chunk ? tgt - chunk_excl : INFINITY;

  // scan chunk cstar: this thread's contiguous run, masses kept in registers
  const bool use_q = residual && !use_p;
  const RowChunk cc = row_chunk<VEC>(ta0, a.V, cstar, a.nch2);
  const int len = cc.e1 - cc.e0;
  const int run = (len + 255) / 256;  // <= kScanRun for chunks of at most 4096 + 7 elements
  const int e_beg = min(cc.e0 + tid * run, cc.e1), e_end = min(e_beg + run, cc.e1);
  float mass[kScanRun];
  double own = 0.0;
  int last_pos_own = -1;
#pragma unroll
  for (int k = 0; k < kScanRun; ++k) {
    const int e = e_beg + k;
    float t = 0.f, q = 0.f;
    if (e < e_end) {
      t = load_elem<BF16>(a.target, ta0 + e);
      if (use_q) q = load_elem<BF16>(a.draft, da0 + e);
    }
    float r, p;
    sample_masses(t, q, si0, si1, a.c, r, p);
    mass[k] = (e < e_end) ? (use_q ? r : p) : 0.f;
    own += (double)mass[k];
    if (mass[k] > 0.f) last_pos_own = e;
  }
  double dummy;
  const double incl = block_scan_incl(own, sh4, &dummy);
  const double excl = incl - own;
  if (ctgt != INFINITY && excl <= ctgt && ctgt < incl) {
    double cum = excl;
    int found = -1;
#pragma unroll
    for (int k = 0; k < kScanRun; ++k) {
      cum += (double)mass[k];
      if (found < 0 && cum > ctgt && e_beg + k < e_end) found = e_beg + k;
    }
    if (found < 0) found = last_pos_own;  // rounding: the run's last token with mass
    if (found >= 0) atomicMin(&s_found, found);
  }
  int lp = last_pos_own;
#pragma unroll
  for (int msk = 1; msk < 64; msk <<= 1) lp = max(lp, __shfl_xor(lp, msk, 64));
  if (lane == 0) sh4[wave] = (double)lp;
  __syncthreads();
  if (tid == 0) {
    int tok = s_found;
    if (tok == INT_MAX) tok = (int)fmax(fmax(sh4[0], sh4[1]), fmax(sh4[2], sh4[3]));
    a.next_token[s] = tok;
  }
}

}  // namespace sdb
