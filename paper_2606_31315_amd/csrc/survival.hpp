// survival.hpp -- the prefix-survival model of acceptance length, on the GPU.
//
// App. A.1: with q_j(x, b) the probability that drafted position j is accepted once positions
// 1..j-1 were, the expected accepted length is tau(b; x) = sum_{i<=b} prod_{j<=i} q_j(x, b).
// App. A.2: q_j(x, b) = gamma_j(x) r(b; B), r(b; B) = exp(-alpha (b - B)^2), B the drafter's
// training block size; the best block size of sample x is B*(x) = argmax over the candidates.
// App. A.3: the regret of a predicted size is R(x) = tau(B*(x)) - tau(B_hat(x)), bounded by
// L_tau |B* - B_hat| for the discrete Lipschitz constant L_tau of tau over the candidates.
//
//   survival_tau_kernel     one thread per sample: tau for every candidate, B*, the regret of
//                           B_hat and L_tau.  A workgroup stages its samples' gamma rows
//                           through LDS so the HBM reads are contiguous 16-byte vectors.
//   survival_sample_kernel  Monte Carlo of L_b(x): one wavefront per (sample, candidate), one
//                           lane per trial in turn.  Uniforms come from Philox4x64-10 (Salmon
//                           et al., SC'11) keyed by (seed, 0) at counter ((i-1)/4, t, c, n), word
//                           (i-1) mod 4 for drafted position i, as the top 53 bits over 2^53, so
//                           every trial's draws are fixed by its indices alone.
//
// fp64 throughout: gamma (fp32) widens exactly, the products and sums are fp64.
#pragma once

#include "common.hpp"

namespace sdb {

constexpr int kSurvMaxCands = 64;
constexpr int kSurvMaxPos = 128;
constexpr int kSurvLdsBytes = 65536;  // staging budget of survival_tau_kernel

struct SurvivalArgs {
  const float *gamma;   // [N, P]
  const int *b_hat;     // [N] or null
  double *tau;          // [N, C]
  int *b_star;          // [N]
  double *regret;       // [N] or null
  double *lipschitz;    // [N] or null
  double *mean_len;     // [N, C]   (sampler)
  int *len_hist;        // [N, C, P + 1] or null (sampler)
  unsigned long long seed;
  int N, P, C, train_block, trials;
  double alpha;
  int cands[kSurvMaxCands];
};

__device__ __forceinline__ double retention(int b, int B, double alpha) {
  const double d = (double)(b - B);
  return exp(-alpha * d * d);
}

// One thread per sample, blockDim.x samples per workgroup (64, 128 or 256, so that the
// staged rows fit 64 KB of LDS).  Dynamic LDS: C retention factors (doubles), then the gamma
// rows, row stride P + 1 floats (odd, so a wavefront's per-thread row reads fall in distinct
// banks).
__global__ __launch_bounds__(256) void survival_tau_kernel(SurvivalArgs a) {
  extern __shared__ __attribute__((aligned(16))) double r_lds[];
  const int P = a.P, C = a.C, stride = P + 1;
  float *lds = reinterpret_cast<float *>(r_lds + kSurvMaxCands);
  const int tid = threadIdx.x, spw = blockDim.x;
  const long long n0 = (long long)blockIdx.x * spw;
  const int rows = (int)min((long long)spw, (long long)a.N - n0);
  // the workgroup's rows are one contiguous run of rows * P floats; 16-byte loads when P % 4 == 0
  const float *src = a.gamma + n0 * P;
  const int total = rows * P;
  if ((P & 3) == 0) {
    // batches of 8 vectors per thread, every load of a batch issued before any LDS store
    const float4 *s4 = reinterpret_cast<const float4 *>(src);
    const int nvec = total / 4;
    for (int v0 = tid; v0 < nvec; v0 += 8 * spw) {
      float4 x[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) x[k] = s4[min(v0 + k * spw, nvec - 1)];  // clamped: no per-load branch
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int v = v0 + k * spw;
        if (v < nvec) {
          const int e = 4 * v, row = e / P, col = e % P;  // P % 4 == 0: the 4 floats share a row
          float *d = lds + row * stride + col;
          d[0] = x[k].x;
          d[1] = x[k].y;
          d[2] = x[k].z;
          d[3] = x[k].w;
        }
      }
    }
  } else {
    for (int e = tid; e < total; e += spw) lds[(e / P) * stride + e % P] = src[e];
  }
  if (tid < C) r_lds[tid] = retention(a.cands[tid], a.train_block, a.alpha);
  __syncthreads();
  if (tid >= rows) return;
  const long long n = n0 + tid;
  const float *g = lds + tid * stride;
  double best_tau = -1.0, prev_tau = 0.0, lip = 0.0, hat_tau = 0.0;
  int best_b = a.cands[0], prev_b = 0;
  const int bh = a.b_hat ? a.b_hat[n] : -1;
  bool hat_found = false;
  for (int c = 0; c < C; ++c) {
    const int b = a.cands[c];
    const double r = r_lds[c];
    double prod = 1.0, t = 0.0;
    for (int i = 0; i < b; ++i) {
      prod *= (double)g[i] * r;  // prod_{j<=i+1} q_j
      t += prod;
    }
    a.tau[n * C + c] = t;
    if (t > best_tau) {  // strict: ties keep the smaller block size
      best_tau = t;
      best_b = b;
    }
    // A chord's slope over non-adjacent candidates is a weighted mean of the adjacent slopes
    // it spans, so the largest slope over all pairs is the largest over adjacent pairs.
    if (c > 0) lip = fmax(lip, fabs(t - prev_tau) / (double)(b - prev_b));
    if (b == bh) {
      hat_tau = t;
      hat_found = true;
    }
    prev_tau = t;
    prev_b = b;
  }
  a.b_star[n] = best_b;
  if (a.lipschitz) a.lipschitz[n] = lip;
  if (a.regret) a.regret[n] = hat_found ? best_tau - hat_tau : __builtin_nan("");
}

// ---- Philox4x64-10 ----
struct Philox4x64 {
  unsigned long long v[4];
};

__device__ __forceinline__ Philox4x64 philox4x64_10(unsigned long long c0, unsigned long long c1,
                                                    unsigned long long c2, unsigned long long c3,
                                                    unsigned long long k0, unsigned long long k1) {
  constexpr unsigned long long M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  constexpr unsigned long long W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const unsigned long long hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
    const unsigned long long hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
    const unsigned long long n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += W0;
    k1 += W1;
  }
  return Philox4x64{{c0, c1, c2, c3}};
}

__device__ __forceinline__ double u53(unsigned long long w) {
  return (double)(w >> 11) * (1.0 / 9007199254740992.0);
}

constexpr int kSurvWavesPerWg = 4;

// Dynamic LDS per wavefront: q_1..q_b (doubles), then the histogram of L (P + 1 ints).
__global__ __launch_bounds__(256) void survival_sample_kernel(SurvivalArgs a) {
  extern __shared__ __attribute__((aligned(16))) double slds[];
  const int P = a.P, C = a.C;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int per_wave = P + (P + 2) / 2;  // P doubles of q, then P + 1 ints (rounded up to doubles)
  double *q = slds + wave * per_wave;
  int *hist = reinterpret_cast<int *>(q + P);
  const long long pair = (long long)blockIdx.x * kSurvWavesPerWg + wave;
  if (pair >= (long long)a.N * C) return;  // wave-uniform; no workgroup barrier follows
  const long long n = pair / C;
  const int c = (int)(pair % C);
  const int b = a.cands[c];
  const double r = retention(b, a.train_block, a.alpha);
  for (int i = lane; i < b; i += 64) q[i] = (double)a.gamma[n * P + i] * r;
  for (int i = lane; i <= P; i += 64) hist[i] = 0;
  // the wavefront's own LDS writes, visible to all of its lanes
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  unsigned long long sum = 0;
  for (int t = lane; t < a.trials; t += 64) {
    int L = 0;
    bool alive = true;
    for (int blk = 0; alive && 4 * blk < b; ++blk) {
      const Philox4x64 w = philox4x64_10((unsigned long long)blk, (unsigned long long)t, (unsigned long long)c,
                                         (unsigned long long)n, a.seed, 0ull);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int i = 4 * blk + k;
        if (!alive || i >= b) break;
        if (u53(w.v[k]) < q[i]) ++L;
        else alive = false;
      }
    }
    sum += (unsigned long long)L;
    if (a.len_hist) atomicAdd(&hist[L], 1);
  }
  // wavefront sum of the lengths (exact integers)
  for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
  if (lane == 0) a.mean_len[pair] = (double)sum / (double)a.trials;
  if (a.len_hist) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    int *out = a.len_hist + pair * (P + 1);
    for (int i = lane; i <= P; i += 64) out[i] = hist[i];
  }
}

}  // namespace sdb
