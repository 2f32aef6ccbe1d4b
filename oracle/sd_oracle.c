/*
 * sd_oracle.c -- plain, slow, fp64 CPU oracle for block-verify attention and
 * speculative acceptance.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  It shares no code, header,
 * table or helper with the HIP library; the two meet only through the seeded
 * inputs of the workload generator.
 *
 * Everything is computed in double precision from the exact values of the
 * inputs (bf16 and fp32 both widen to fp64 without rounding), with no blocking,
 * fusion or reordering beyond what the definitions state.
 *
 * Method (BlockPilot, arXiv 2606.31315):
 *   - A speculative step drafts a block of B tokens with a block-diffusion
 *     drafter in one forward pass and the target verifies the whole block in
 *     one parallel forward pass (Sec. 2.1; Fig. 1 caption).
 *   - The block size is fixed per prompt (Sec. 2.4, Eq. 9), hence ragged B
 *     across a batch.
 *   - Verification accepts the longest consistent prefix of the drafted block
 *     (Fig. 1 caption; App. A.1, prefix-survival view) and keeps the target's
 *     output distribution unchanged (Sec. 1; Sec. 3.1 "Metrics"), i.e. standard
 *     lossless speculative sampling: greedy matching at T=0, rejection sampling
 *     against min(1, p/q) with a residual resample at T>0.
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes of the repository):
 *   R1 block = [anchor, d_1 .. d_{B-1}]: B target rows, B-1 draft rows,
 *      accept_len in [0, B-1], one bonus/resampled token.
 *   R2 softmax scale 1/sqrt(D) unless overridden.
 *   R3 GQA: query head h reads kv head floor(h / (Hq/Hkv)).
 *   R4 causal-in-block: block row i sees keys [0, ctx+i]; bidirectional-in-block:
 *      every block row sees keys [0, ctx+B).
 *   R5 p = softmax(t/T), q = softmax(delta/T); T = 0 is greedy.
 *   R6 argmax ties go to the lowest index.
 *   R7 accept test i is u_i < p_i(d_i)/q_i(d_i) (strict), u_i in [0,1).
 *   R8 uniform slot j drives test j; the last slot of the block drives the one
 *      final sample.
 *   R9 a residual with total mass <= 0 (rounding only) falls back to p_j.
 *   R10 inverse CDF in ascending vocabulary order: the first x whose inclusive
 *      cumulative mass exceeds u*S; if rounding leaves none, the last x with
 *      nonzero mass.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_MASK_CAUSAL 0
#define ORC_MASK_BIDIR 1

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* Sequence that owns packed query row `tok`: off[s] <= tok < off[s+1]. */
static int owner_seq(int S, const int *q_offsets, long tok) {
  for (int s = 0; s < S; ++s)
    if (tok >= q_offsets[s] && tok < q_offsets[s + 1]) return s;
  return -1;
}

/*
 * Attention for one output row: query row `tok` (block position i of sequence
 * s), query head h.  Softmax attention over the keys the mask lets it see
 * (Sec. 2.1: the target verifies the block in parallel with causal attention;
 * the block-diffusion drafter attends bidirectionally inside the block).
 */
static void attn_row(int Hq, int Hkv, int D, int Lmax, const float *q, const float *k_cache,
                     const float *v_cache, int s, int ctx, int B, long tok, int i, int h,
                     int mask_mode, double scale, double *o, double *score) {
  const int G = Hq / Hkv;
  const int g = h / G;                                  /* R3 */
  const int n_keys = (mask_mode == ORC_MASK_CAUSAL) ? ctx + i + 1 : ctx + B; /* R4 */
  const float *qr = q + ((size_t)tok * Hq + h) * D;
  const float *kb = k_cache + ((size_t)s * Hkv + g) * (size_t)Lmax * D;
  const float *vb = v_cache + ((size_t)s * Hkv + g) * (size_t)Lmax * D;

  double mx = -INFINITY;
  for (int j = 0; j < n_keys; ++j) {
    double acc = 0.0;
    for (int d = 0; d < D; ++d) acc += (double)qr[d] * (double)kb[(size_t)j * D + d];
    score[j] = scale * acc;
    if (score[j] > mx) mx = score[j];
  }
  double den = 0.0;
  for (int d = 0; d < D; ++d) o[d] = 0.0;
  for (int j = 0; j < n_keys; ++j) {
    double w = exp(score[j] - mx);
    den += w;
    for (int d = 0; d < D; ++d) o[d] += w * (double)vb[(size_t)j * D + d];
  }
  for (int d = 0; d < D; ++d) o[d] /= den;
}

/*
 * Block attention over a ragged batch.
 *
 *   q       [total_q, Hq, D]       packed block rows, row q_offsets[s]+i is block position i of s
 *   k_cache [S, Hkv, Lmax, D]      keys; block keys already at [ctx_s, ctx_s + B_s)
 *   v_cache [S, Hkv, Lmax, D]
 *   scale   softmax scale; <= 0 means 1/sqrt(D) (R2)
 *
 * If n_rows < 0 every row is computed and `out` is [total_q, Hq, D].
 * Otherwise only the listed rows (row_tok[r], row_head[r]) are computed and
 * `out` is [n_rows, D].  Returns 0, or -1 on a bad argument.
 */
int oracle_block_attn(int S, int Hq, int Hkv, int D, int Lmax, const float *q, const float *k_cache,
                      const float *v_cache, const int *ctx_lens, const int *block_lens,
                      const int *q_offsets, int mask_mode, double scale, long n_rows,
                      const long *row_tok, const int *row_head, double *out) {
  if (S < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || D <= 0) return -1;
  if (mask_mode != ORC_MASK_CAUSAL && mask_mode != ORC_MASK_BIDIR) return -1;
  if (scale <= 0) scale = 1.0 / sqrt((double)D);
  const long total_q = q_offsets[S];
  const long jobs = (n_rows < 0) ? total_q * Hq : n_rows;
  int bad = 0;
#pragma omp parallel
  {
    double *score = (double *)malloc(sizeof(double) * (size_t)(Lmax > 0 ? Lmax : 1));
#pragma omp for schedule(dynamic, 1)
    for (long r = 0; r < jobs; ++r) {
      long tok;
      int h;
      double *o;
      if (n_rows < 0) {
        tok = r / Hq;
        h = (int)(r % Hq);
        o = out + (size_t)r * D;
      } else {
        tok = row_tok[r];
        h = row_head[r];
        o = out + (size_t)r * D;
      }
      int s = owner_seq(S, q_offsets, tok);
      if (s < 0 || h < 0 || h >= Hq || ctx_lens[s] + block_lens[s] > Lmax) {
        bad = 1;
        continue;
      }
      attn_row(Hq, Hkv, D, Lmax, q, k_cache, v_cache, s, ctx_lens[s], block_lens[s], tok,
               (int)(tok - q_offsets[s]), h, mask_mode, scale, o, score);
    }
    free(score);
  }
  return bad ? -1 : 0;
}

/* Smallest index attaining the maximum of row x[0..V) (R6). */
static int argmax_lowest(const float *x, int V) {
  int best = 0;
  for (int v = 1; v < V; ++v)
    if (x[v] > x[best]) best = v;
  return best;
}

/* p = softmax(x / T) in fp64 with the maximum subtracted (R5). */
static void softmax_T(const float *x, int V, double T, double *p) {
  double mx = -INFINITY;
  for (int v = 0; v < V; ++v)
    if ((double)x[v] > mx) mx = (double)x[v];
  double z = 0.0;
  for (int v = 0; v < V; ++v) {
    p[v] = exp(((double)x[v] - mx) / T);
    z += p[v];
  }
  for (int v = 0; v < V; ++v) p[v] /= z;
}

/*
 * Inverse-CDF draw from unnormalised masses r[0..V) with total S at position
 * u*S (R10).  Returns the token.
 */
static int inverse_cdf(const double *r, int V, double target) {
  double c = 0.0;
  int last_pos = -1;
  for (int v = 0; v < V; ++v) {
    if (r[v] > 0) last_pos = v;
    c += r[v];
    if (c > target) return v;
  }
  return last_pos;
}

/*
 * Speculative acceptance for a ragged batch.
 *
 *   target   [total_q, V]      row q_offsets[s]+i: target logits after block position i
 *   draft    [total_q - S, V]  row q_offsets[s]-s+j: drafter logits for position j+1 (T > 0 only)
 *   draft_tokens [total_q - S] token j+1 of the block, paired with target row j
 *   uniforms [total_q]         slot q_offsets[s]+j drives test j; slot +B_s-1 the final sample (R8)
 *
 * Outputs per sequence: accept_len (leading accepted drafts), next_token (bonus or
 * resampled token), and for the parity harness
 *   accept_margin  min over the tested positions of |u_i - min(1, rho_i)| (+inf at T = 0 or none)
 *   sample_margin  distance of u*S to the nearer edge of the chosen token's CDF interval, over S
 *   sample_lo/hi   tokens an inverse-CDF draw picks at (u* -/+ band)*S, clamped into [0, S]
 *   sample_tie_p   probability, over a uniform u*, that the final draw lands within band*S of
 *                  an edge of its token's interval: sum over x of min(r(x)/S, 2 band); the
 *                  expected rate of final-draw near-ties (0 at T = 0)
 * Block length 0 yields accept_len 0, next_token -1.
 */
int oracle_accept(int S, int V, const float *target, const float *draft, const int *draft_tokens,
                  const float *uniforms, const int *block_lens, const int *q_offsets,
                  double temperature, double band, int *accept_len, int *next_token,
                  double *accept_margin, double *sample_margin, int *sample_lo, int *sample_hi,
                  double *sample_tie_p) {
  if (S < 0 || V <= 0 || !(temperature >= 0) || isinf(temperature)) return -1;
  int bad = 0;
#pragma omp parallel
  {
    double *p = (double *)malloc(sizeof(double) * (size_t)V);
    double *qd = (double *)malloc(sizeof(double) * (size_t)V);
    double *r = (double *)malloc(sizeof(double) * (size_t)V);
#pragma omp for schedule(dynamic, 1)
    for (int s = 0; s < S; ++s) {
      const int B = block_lens[s];
      const long off = q_offsets[s];
      const long doff = off - s;
      accept_margin[s] = INFINITY;
      sample_margin[s] = INFINITY;
      sample_tie_p[s] = 0.0;
      if (B <= 0) {
        accept_len[s] = 0;
        next_token[s] = -1;
        sample_lo[s] = sample_hi[s] = -1;
        continue;
      }
      const int n = B - 1; /* drafted tokens (R1) */
      for (int j = 0; j < n; ++j)
        if (draft_tokens[doff + j] < 0 || draft_tokens[doff + j] >= V) bad = 1;
      if (temperature == 0.0) {
        /* Greedy: the drafted token must equal the target's argmax. */
        int a = 0;
        while (a < n && draft_tokens[doff + a] == argmax_lowest(target + (size_t)(off + a) * V, V)) ++a;
        accept_len[s] = a;
        next_token[s] = argmax_lowest(target + (size_t)(off + a) * V, V);
        sample_lo[s] = sample_hi[s] = next_token[s];
        continue;
      }
      /* T > 0: test positions in order until the first rejection. */
      int a = 0;
      for (; a < n; ++a) {
        const int d = draft_tokens[doff + a];
        softmax_T(target + (size_t)(off + a) * V, V, temperature, p);
        softmax_T(draft + (size_t)(doff + a) * V, V, temperature, qd);
        const double rho = (qd[d] > 0) ? p[d] / qd[d] : INFINITY;
        const double u = (double)uniforms[off + a];
        const double m = fabs(u - (rho < 1.0 ? rho : 1.0));
        if (m < accept_margin[s]) accept_margin[s] = m;
        if (!(u < rho)) break; /* R7 */
      }
      accept_len[s] = a;
      /* Final sample: residual max(0, p_a - q_a) after a rejection, p_n at the bonus row. */
      double tot = 0.0;
      softmax_T(target + (size_t)(off + a) * V, V, temperature, p);
      if (a < n) {
        softmax_T(draft + (size_t)(doff + a) * V, V, temperature, qd);
        for (int v = 0; v < V; ++v) {
          r[v] = p[v] - qd[v];
          if (r[v] < 0) r[v] = 0;
          tot += r[v];
        }
        if (!(tot > 0)) { /* R9 */
          for (int v = 0; v < V; ++v) r[v] = p[v];
          tot = 1.0;
        }
      } else {
        for (int v = 0; v < V; ++v) r[v] = p[v];
        tot = 1.0;
      }
      const double ustar = (double)uniforms[off + n];
      const double tgt = ustar * tot;
      const int x = inverse_cdf(r, V, tgt);
      next_token[s] = x;
      double below = 0.0; /* cumulative mass strictly before x */
      for (int v = 0; v < x; ++v) below += r[v];
      double m1 = (tgt - below) / tot, m2 = (below + r[x] - tgt) / tot;
      sample_margin[s] = m1 < m2 ? m1 : m2;
      double lo_t = tgt - band * tot, hi_t = tgt + band * tot;
      if (lo_t < 0) lo_t = 0;
      if (hi_t > tot) hi_t = tot;
      sample_lo[s] = inverse_cdf(r, V, lo_t);
      sample_hi[s] = inverse_cdf(r, V, hi_t);
      /* Token x owns [below_x, below_x + r(x)) of [0, S); the near-tie part of it is the
       * band*S next to each edge, or all of it when the interval is narrower than 2 band S. */
      double ptie = 0.0;
      for (int v = 0; v < V; ++v) {
        const double w = r[v] / tot;
        ptie += w < 2.0 * band ? w : 2.0 * band;
      }
      sample_tie_p[s] = ptie;
    }
    free(p);
    free(qd);
    free(r);
  }
  return bad ? -1 : 0;
}
