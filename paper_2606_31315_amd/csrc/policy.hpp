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
//   policy_stats_kernel   grid (prompt, chunk): (max, sum exp(z - max)) of one vocabulary chunk,
//                         one online pass per thread.
//   policy_dense_kernel   y = act(W x + b) for every prompt: a workgroup owns R rows of W and
//                         streams them once with 16-byte loads, all prompts' FMAs per element.
//                         For the first layer x is p = softmax(z), made on the fly from the
//                         logits and the merged chunk records (p is never written out; the
//                         logits stay L2-resident: 2 or 4 bytes per element per prompt).
//   policy_head_kernel    one workgroup per prompt, one wavefront per candidate in turn: the
//                         2k+1 scores and their argmax.
#pragma once

#include "common.hpp"

namespace sdb {

constexpr int kPolicyChunks = 64;   // vocabulary chunks of the softmax passes
constexpr int kPolicyMaxPrompts = 8;  // prompts per dense pass (accumulators per thread)
constexpr int kDenseRows = 2;       // rows of W per dense workgroup

struct PolicyArgs {
  const void *logits;   // [P, V] bf16 or fp32
  float2 *stats;        // [P, kPolicyChunks] (max, sum exp(z - max))
  int P, V, logits_bf16;
};

constexpr float kLog2e = 1.4426950408889634f;

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
  // online (max, sum) per thread: one rescale when the maximum moves
  float m = -INFINITY, s = 0.f;
  for (int e = e0 + tid; e < e1; e += 256) {
    const float z = ld_logit<BF16>(a.logits, row + e);
    if (z > m) {
      s = (m == -INFINITY) ? 0.f : s * fast_exp2((m - z) * kLog2e);
      m = z;
    }
    if (m != -INFINITY) s += fast_exp2((z - m) * kLog2e);  // a -inf logit adds 0
  }
  const float wm = wave_max_f(m);
  float ws = (m == -INFINITY) ? 0.f : s * fast_exp2((m - wm) * kLog2e);
  ws = wave_sum_f(ws);
  if (lane == 0) {
    sh_m[wave] = wm;
    sh_s[wave] = ws;
  }
  __syncthreads();
  if (tid == 0) {
    const float M = fmaxf(fmaxf(sh_m[0], sh_m[1]), fmaxf(sh_m[2], sh_m[3]));
    float S = 0.f;
    for (int w = 0; w < 4; ++w)
      if (sh_m[w] != -INFINITY) S += sh_s[w] * fast_exp2((sh_m[w] - M) * kLog2e);
    a.stats[blockIdx.x] = float2{M, S};
  }
}

// y[p, n] = act(sum_i W[n, i] x[p, i] + b[n]) for rows n of this workgroup and every prompt p.
// W [rows, cols] bf16 row-major (cols % 8 == 0), y [P, rows] fp32.  x [P, cols] is
//   XM = 0: fp32 activations;
//   XM = 1, 2: bf16 (1) or fp32 (2) logits z, and the layer's input is p = softmax(z), made here
//   from z and the prompt's kPolicyChunks chunk records: p_i = 2^((z_i - M) log2 e) / Z.
struct DenseArgs {
  const uint16_t *w;
  const void *x;
  const float *b;
  float *y;
  int rows, cols, P;
  const float2 *stats;  // XM != 0: [P, kPolicyChunks]
};

// U vectors per row are loaded before any is used (clamped indices, no per-load branch), so a
// thread keeps U * (R + NP * (1 or 2)) 16-byte loads in flight.
template <int NP, bool RELU, int XM>
__global__ __launch_bounds__(256) void policy_dense_kernel(DenseArgs a) {
  constexpr int R = kDenseRows;
  constexpr int U = NP <= 2 ? 4 : (NP <= 4 ? 2 : 1);
  constexpr int XV = (XM == 1) ? 1 : 2;  // 16-byte x loads per 8 elements
  static_assert(kPolicyChunks == kWave, "one chunk record per lane");
  __shared__ float sh[4][R][NP];
  __shared__ float sh_norm[2][NP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.x * R;
  const int nv = a.cols / 8;  // 16-byte vectors of bf16 per row
  float mx[NP], inv[NP];
  if constexpr (XM != 0) {
    // merge the prompt's chunk records: M = max of the chunk maxima, Z = sum of the rescaled sums
    if (wave == 0) {
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        const float2 r = a.stats[(size_t)min(p, a.P - 1) * kPolicyChunks + lane];
        const float M = wave_max_f(r.x);
        const double z = wave_sum_d(r.x != -INFINITY ? (double)r.y * (double)fast_exp2((r.x - M) * kLog2e) : 0.0);
        if (lane == 0) {
          sh_norm[0][p] = M;
          sh_norm[1][p] = (float)(1.0 / z);
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      mx[p] = sh_norm[0][p];
      inv[p] = sh_norm[1][p];
    }
  }
  float acc[R][NP];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int p = 0; p < NP; ++p) acc[r][p] = 0.f;
  const u32x4 *wr[R];
#pragma unroll
  for (int r = 0; r < R; ++r) wr[r] = reinterpret_cast<const u32x4 *>(a.w + (size_t)min(n0 + r, a.rows - 1) * a.cols);
  const u32x4 *xr[NP];
  const size_t xrow = (size_t)a.cols * (XM == 1 ? 2 : 4) / 16;  // 16-byte vectors per x row
#pragma unroll
  for (int p = 0; p < NP; ++p) xr[p] = reinterpret_cast<const u32x4 *>(a.x) + (size_t)min(p, a.P - 1) * xrow;
  for (int v0 = tid; v0 < nv; v0 += 256 * U) {
    u32x4 wv[U][R];
    u32x4 xv[U][NP][XV];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = min(v0 + 256 * u, nv - 1);
#pragma unroll
      for (int r = 0; r < R; ++r) wv[u][r] = wr[r][v];
#pragma unroll
      for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int k = 0; k < XV; ++k) xv[u][p][k] = xr[p][XV * v + k];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (v0 + 256 * u >= nv) break;
      float x[NP][8];
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        if constexpr (XM == 1) {
          const u32x4 z = xv[u][p][0];
          const float zz[8] = {bf16_lo(z.x), bf16_hi(z.x), bf16_lo(z.y), bf16_hi(z.y),
                               bf16_lo(z.z), bf16_hi(z.z), bf16_lo(z.w), bf16_hi(z.w)};
#pragma unroll
          for (int e = 0; e < 8; ++e) x[p][e] = fast_exp2((zz[e] - mx[p]) * kLog2e) * inv[p];
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const u32x4 h = xv[u][p][e >> 2];
            const uint32_t bits = (e & 3) == 0 ? h.x : (e & 3) == 1 ? h.y : (e & 3) == 2 ? h.z : h.w;
            const float f = __uint_as_float(bits);
            x[p][e] = (XM == 2) ? fast_exp2((f - mx[p]) * kLog2e) * inv[p] : f;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const float w[8] = {bf16_lo(wv[u][r].x), bf16_hi(wv[u][r].x), bf16_lo(wv[u][r].y), bf16_hi(wv[u][r].y),
                            bf16_lo(wv[u][r].z), bf16_hi(wv[u][r].z), bf16_lo(wv[u][r].w), bf16_hi(wv[u][r].w)};
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[r][p] = fmaf(w[e], x[p][e], acc[r][p]);
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

// One workgroup per prompt; wavefront w scores candidates w, w + 4, ...: each lane takes
// 8-element slices of the candidate's W3 row (one 16-byte load) and of h2 (two 16-byte
// loads), four slices in flight, then a wavefront sum.  W3 rows are 16-byte aligned (H % 8 == 0).
__global__ __launch_bounds__(256) void policy_head_kernel(HeadArgs a) {
  __shared__ float sc[64];
  const int pr = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const f32x4 *x4 = reinterpret_cast<const f32x4 *>(a.x + (size_t)pr * a.H);
  const int nv = a.H / 8;  // 8-element slices per row
  for (int c = wave; c < a.C; c += 4) {
    const u32x4 *w4 = reinterpret_cast<const u32x4 *>(a.w + (size_t)c * a.H);
    float s = 0.f;
    for (int v0 = lane; v0 < nv; v0 += 64 * 4) {
      u32x4 wv[4];
      f32x4 xv[4][2];
#pragma unroll
      for (int u = 0; u < 4; ++u) {  // clamped: no per-load branch
        const int v = min(v0 + 64 * u, nv - 1);
        wv[u] = w4[v];
        xv[u][0] = x4[2 * v];
        xv[u][1] = x4[2 * v + 1];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (v0 + 64 * u >= nv) break;
        const float w[8] = {bf16_lo(wv[u].x), bf16_hi(wv[u].x), bf16_lo(wv[u].y), bf16_hi(wv[u].y),
                            bf16_lo(wv[u].z), bf16_hi(wv[u].z), bf16_lo(wv[u].w), bf16_hi(wv[u].w)};
#pragma unroll
        for (int e = 0; e < 8; ++e) s = fmaf(w[e], xv[u][e >> 2][e & 3], s);
      }
    }
    s = wave_sum_f(s);
    if (lane == 0) sc[c] = s + a.b[c];
  }
  __syncthreads();
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
