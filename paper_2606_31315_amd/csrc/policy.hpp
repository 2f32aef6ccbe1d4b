// policy.hpp -- the block-size policy on the GPU, run once per prompt after prefill.
//
// Sec. 2.3-2.4: the predictive distribution of the prompt's last token, p = softmax(z) over the
// vocabulary, is the input of a small MLP (two hidden layers of width 2048 by default, Sec. 3.1)
// whose outputs score the 2k+1 candidate block sizes {B-k, ..., B+k}; the block size is the
// argmax of the scores (Eq. 9).  Here:
//   h1 = relu(W1 p + b1),  h2 = relu(W2 h1 + b2),  o = W3 h2 + b3,  B_hat = B - k + argmax o.
//
// Kernels (gfx950).  The W1 product dominates: W1 is [hidden, V] bf16 (622 MB for Qwen3's
// vocabulary), read once, so the policy is HBM-bound.
//   policy_stats_kernel   grid (prompt, chunk): (max, sum exp(z - max)) of one vocabulary chunk.
//   policy_prob_kernel    grid (prompt, chunk): merges the chunk records, writes p in fp32.
//   policy_dense_kernel   y = act(W x + b) for every prompt: a workgroup owns R rows of W and
//                         streams them once with 16-byte loads, all prompts' FMAs per element
//                         (p stays L2-resident: 4 bytes per element per prompt).
//   policy_head_kernel    one workgroup per prompt: the 2k+1 scores and their argmax.
#pragma once

#include "common.hpp"

namespace sdb {

constexpr int kPolicyChunks = 64;   // vocabulary chunks of the softmax passes
constexpr int kPolicyMaxPrompts = 8;  // prompts per dense pass (accumulators per thread)
constexpr int kDenseRows = 2;       // rows of W per dense workgroup

struct PolicyArgs {
  const void *logits;   // [P, V] bf16 or fp32
  float2 *stats;        // [P, kPolicyChunks] (max, sum exp(z - max))
  float *prob;          // [P, V]
  int P, V, logits_bf16;
};

template <bool BF16>
__device__ __forceinline__ float ld_logit(const void *base, long long i) {
  if constexpr (BF16) return __uint_as_float(((uint32_t)reinterpret_cast<const uint16_t *>(base)[i]) << 16);
  else return reinterpret_cast<const float *>(base)[i];
}

__device__ __forceinline__ void chunk_range(int V, int c, int &e0, int &e1) {
  e0 = (int)((long long)V * c / kPolicyChunks);
  e1 = (int)((long long)V * (c + 1) / kPolicyChunks);
}

template <bool BF16>
__global__ __launch_bounds__(256) void policy_stats_kernel(PolicyArgs a) {
  __shared__ float sh_m[4], sh_s[4];
  const int pr = blockIdx.x / kPolicyChunks, c = blockIdx.x % kPolicyChunks;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int e0, e1;
  chunk_range(a.V, c, e0, e1);
  const long long row = (long long)pr * a.V;
  float m = -INFINITY;
  for (int e = e0 + tid; e < e1; e += 256) m = fmaxf(m, ld_logit<BF16>(a.logits, row + e));
  m = wave_max_f(m);
  if (lane == 0) sh_m[wave] = m;
  __syncthreads();
  m = fmaxf(fmaxf(sh_m[0], sh_m[1]), fmaxf(sh_m[2], sh_m[3]));
  float s = 0.f;
  if (m != -INFINITY)
    for (int e = e0 + tid; e < e1; e += 256) s += fast_exp2((ld_logit<BF16>(a.logits, row + e) - m) * 1.4426950408889634f);
  s = wave_sum_f(s);
  if (lane == 0) sh_s[wave] = s;
  __syncthreads();
  if (tid == 0) a.stats[blockIdx.x] = float2{m, (sh_s[0] + sh_s[1]) + (sh_s[2] + sh_s[3])};
}

template <bool BF16>
__global__ __launch_bounds__(256) void policy_prob_kernel(PolicyArgs a) {
  const int pr = blockIdx.x / kPolicyChunks, c = blockIdx.x % kPolicyChunks;
  const int tid = threadIdx.x;
  // every thread merges the prompt's chunk records (64 loads, the same for all threads)
  const float2 *st = a.stats + (size_t)pr * kPolicyChunks;
  float M = -INFINITY;
  for (int k = 0; k < kPolicyChunks; ++k) M = fmaxf(M, st[k].x);
  double Z = 0.0;
  for (int k = 0; k < kPolicyChunks; ++k)
    if (st[k].x != -INFINITY) Z += (double)st[k].y * (double)fast_exp2((st[k].x - M) * 1.4426950408889634f);
  const float inv = (float)(1.0 / Z);
  int e0, e1;
  chunk_range(a.V, c, e0, e1);
  const long long row = (long long)pr * a.V;
  for (int e = e0 + tid; e < e1; e += 256)
    a.prob[row + e] = fast_exp2((ld_logit<BF16>(a.logits, row + e) - M) * 1.4426950408889634f) * inv;
}

// y[p, n] = act(sum_i W[n, i] x[p, i] + b[n]) for rows n of this workgroup and every prompt p.
// W [rows, cols] bf16 row-major (cols % 8 == 0), x [P, cols] fp32, y [P, rows] fp32.
struct DenseArgs {
  const uint16_t *w;
  const float *x;
  const float *b;
  float *y;
  int rows, cols, P;
};

// U vectors per row are loaded before any is used (clamped indices, no per-load branch), so a
// thread keeps U * (R + 2 NP) 16-byte loads in flight.
template <int NP, bool RELU>
__global__ __launch_bounds__(256) void policy_dense_kernel(DenseArgs a) {
  constexpr int R = kDenseRows;
  constexpr int U = NP <= 2 ? 4 : (NP <= 4 ? 2 : 1);
  __shared__ float sh[4][R][NP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.x * R;
  const int nv = a.cols / 8;  // 16-byte vectors of bf16 per row
  float acc[R][NP];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int p = 0; p < NP; ++p) acc[r][p] = 0.f;
  const u32x4 *wr[R];
#pragma unroll
  for (int r = 0; r < R; ++r) wr[r] = reinterpret_cast<const u32x4 *>(a.w + (size_t)min(n0 + r, a.rows - 1) * a.cols);
  const f32x4 *xr[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) xr[p] = reinterpret_cast<const f32x4 *>(a.x + (size_t)min(p, a.P - 1) * a.cols);
  for (int v0 = tid; v0 < nv; v0 += 256 * U) {
    u32x4 wv[U][R];
    f32x4 xv[U][NP][2];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = min(v0 + 256 * u, nv - 1);
#pragma unroll
      for (int r = 0; r < R; ++r) wv[u][r] = wr[r][v];
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        xv[u][p][0] = xr[p][2 * v];
        xv[u][p][1] = xr[p][2 * v + 1];
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (v0 + 256 * u >= nv) break;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const float w[8] = {bf16_lo(wv[u][r].x), bf16_hi(wv[u][r].x), bf16_lo(wv[u][r].y), bf16_hi(wv[u][r].y),
                            bf16_lo(wv[u][r].z), bf16_hi(wv[u][r].z), bf16_lo(wv[u][r].w), bf16_hi(wv[u][r].w)};
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[r][p] = fmaf(w[e], xv[u][p][e >> 2][e & 3], acc[r][p]);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const float s = wave_sum_f(acc[r][p]);
      if (lane == 0) sh[wave][r][p] = s;
    }
  __syncthreads();
  if (tid < R * NP) {
    const int r = tid / NP, p = tid % NP;
    const int n = n0 + r;
    if (n < a.rows && p < a.P) {
      float y = (sh[0][r][p] + sh[1][r][p]) + (sh[2][r][p] + sh[3][r][p]) + a.b[n];
      if (RELU) y = fmaxf(y, 0.f);
      a.y[(size_t)p * a.rows + n] = y;
    }
  }
}

// Scores of the C candidates for prompt p and their argmax (lowest index on ties):
// o = W3 h2 + b3, W3 [C, H] bf16, h2 [P, H] fp32.
struct HeadArgs {
  const uint16_t *w;
  const float *x;
  const float *b;
  float *scores;      // [P, C]
  int *block_size;    // [P]
  int C, H, base, radius;
};

__global__ __launch_bounds__(256) void policy_head_kernel(HeadArgs a) {
  __shared__ float sh[4];
  __shared__ float sc[64];
  const int pr = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float *x = a.x + (size_t)pr * a.H;
  for (int c = 0; c < a.C; ++c) {
    const uint16_t *w = a.w + (size_t)c * a.H;
    float s = 0.f;
    for (int i = tid; i < a.H; i += 256) s = fmaf(__uint_as_float(((uint32_t)w[i]) << 16), x[i], s);
    s = wave_sum_f(s);
    if (lane == 0) sh[wave] = s;
    __syncthreads();
    if (tid == 0) sc[c] = (sh[0] + sh[1]) + (sh[2] + sh[3]) + a.b[c];
    __syncthreads();
  }
  if (tid == 0) {
    int best = 0;
    for (int c = 0; c < a.C; ++c) {
      a.scores[(size_t)pr * a.C + c] = sc[c];
      if (sc[c] > sc[best]) best = c;
    }
    a.block_size[pr] = a.base - a.radius + best;
  }
}

}  // namespace sdb
