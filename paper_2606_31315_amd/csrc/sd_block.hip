// sd_block.hip -- C ABI of libsdblock.so (declared in include/sd_block.h).
//
// Host side only: argument validation, workspace layout, launch planning and kernel
// dispatch.  The arithmetic lives in attn.hpp and accept.hpp.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <random>
#include <string>

#include "accept.hpp"
#include "attn.hpp"
#include "attn_bf16.hpp"
#include "check.hpp"
#include "kvstep.hpp"
#include "policy.hpp"
#include "sd_block.h"
#include "survival.hpp"

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return SD_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int check_launch(const char *what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(SD_ERR_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
  return ok();
}

// bf16 key tile and LDS ring depth: KT keys of K and of V per stage, NS stages.  Measured on
// the ragged Qwen3-4B batch (sd_block_attn call, 5 interleaved rounds): 3 stages 37.0 us,
// 4 stages 37.5-37.9, 2 stages 37.8, 5 stages 38.7; 128-key tiles in 2 stages 39.0.  HBM is
// saturated by 256 workgroups with two tiles in flight each; more in flight only adds queueing.
#ifndef SDB_BF16_KT
#define SDB_BF16_KT 64
#define SDB_BF16_NS 3
#endif
constexpr int kBf16KT = SDB_BF16_KT, kBf16NS = SDB_BF16_NS;

// ---------------------------------------------------------------------------
// attention planning
// ---------------------------------------------------------------------------
struct AttnPlan {
  int G, KT, split_len, max_splits, Mpad, n_work, per_xcd, grid, dense, MT;
  int bal;  // balanced shares (bf16; see bal_share)
  int ve;   // bf16 with one m-tile per wavefront and blocks of 7-8 m-tiles: early V^T reads (VE)
  size_t off_ml, off_o, total;
};

// Balanced plan: one workgroup per CU of the MI355X (the bf16 split kernel holds a CU), each
// share at least 16 key tiles (1024 keys), like the shortest split of the other multi-wave plans.
constexpr int kBalGrid = 256;
constexpr int kBalMinTiles = 16;

int attn_plan(const sd_attn_shape *sh, AttnPlan *p) {
  if (!sh) return fail(SD_ERR_INVALID_ARG, "sd_block_attn: shape is NULL");
  const int S = sh->num_seqs, Hq = sh->num_q_heads, Hkv = sh->num_kv_heads, D = sh->head_dim;
  if (S < 0) return fail(SD_ERR_INVALID_ARG, "num_seqs must be >= 0 (got %d)", S);
  if (Hq < 1 || Hkv < 1) return fail(SD_ERR_INVALID_ARG, "head counts must be >= 1 (Hq=%d, Hkv=%d)", Hq, Hkv);
  if (Hq % Hkv) return fail(SD_ERR_INVALID_ARG, "num_q_heads %d is not a multiple of num_kv_heads %d", Hq, Hkv);
  if (sh->dtype != SD_BF16 && sh->dtype != SD_F32) return fail(SD_ERR_INVALID_ARG, "unknown dtype %d", sh->dtype);
  if (D != 64 && D != 128) return fail(SD_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", D);
  if (sh->max_block < 1 || sh->max_block > 64)
    return fail(SD_ERR_INVALID_ARG, "max_block must be in [1, 64] (got %d)", sh->max_block);
  if (sh->max_ctx < 0) return fail(SD_ERR_INVALID_ARG, "max_ctx must be >= 0 (got %d)", sh->max_ctx);
  if (sh->max_kv_len < 1 || (long long)sh->max_ctx + sh->max_block > sh->max_kv_len)
    return fail(SD_ERR_INVALID_ARG, "max_ctx + max_block (%d + %d) exceeds max_kv_len %d", sh->max_ctx,
                sh->max_block, sh->max_kv_len);
  if (sh->total_q < 0 || (long long)sh->total_q > (long long)S * sh->max_block)
    return fail(SD_ERR_INVALID_ARG, "total_q %d outside [0, num_seqs * max_block]", sh->total_q);
  const int G = Hq / Hkv;
  if ((long long)G * sh->max_block > 256)
    return fail(SD_ERR_UNSUPPORTED, "group size %d times max_block %d exceeds 256 query rows", G, sh->max_block);
  if (!(sh->scale >= 0.f) || isinf(sh->scale)) return fail(SD_ERR_INVALID_ARG, "scale must be finite and >= 0");

  p->G = G;
  p->KT = (sh->dtype == SD_BF16) ? kBf16KT : 32;
  const long long max_L = (long long)sh->max_ctx + sh->max_block;
  const long long pairs = (long long)S * Hkv;
  // Split the keys so that, at the maximum length, the grid is one wave: one workgroup per
  // CU for the bf16 kernel (one 512-thread workgroup fills a CU's LDS ring), two for the fp32
  // kernel.  A grid just over one wave runs its last workgroups as a tail (measured on the
  // ragged Qwen3-4B batch: 5 splits of 1024 keys, 48.3 us; 4 splits of 1088, 40.4 us).
  // Splits stay at most 4096 keys so long ragged contexts still spread over several waves.
  // Rounding the split to 16 keys rather than a whole 64-key tile keeps the splits even
  // (same batch: 4 x 1040 keys, split kernel 31.8 us; 4 x 1088, 32.6 us).
  const long long target_wgs = (sh->dtype == SD_BF16) ? 256 : 512;
  long long want = pairs > 0 ? target_wgs / pairs : 1;
  if (want < 1) want = 1;
  // Split lengths are multiples of 16 keys for bf16 (a split's last key tile may be
  // partial) and of the key tile for fp32.
  const int gran = (sh->dtype == SD_BF16) ? 16 : p->KT;
  long long sl = (max_L + want - 1) / want;
  sl = ((sl + gran - 1) / gran) * gran;
  // bf16 splits longer than 2048 keys: size them for two waves at the maximum length instead.
  // One wave of long workgroups ends with the slowest CU, and ragged lengths leave CUs idle;
  // two or more waves let the dispatcher rebalance (16 sequences x 8 kv heads, bidirectional:
  // contexts 1k-8k 98.7 -> 94.8 us, all at 8k 123.1 -> 109.4 us; three or more waves at the
  // maximum length measured slower on the uniform batch, 116.5-133.0 us).
  if (sh->dtype == SD_BF16 && sl > 2048) {
    sl = (max_L * pairs + 2 * target_wgs - 1) / (2 * target_wgs);
    sl = ((sl + gran - 1) / gran) * gran;
    if (sl < 1024) sl = 1024;
  }
  if (sl > sdb::kLongSplit) sl = sdb::kLongSplit;
  // At least 256 keys per split: below that a workgroup's fixed start-up and the merge of many
  // partials outweigh the spread (Qwen3-4B verify at batch 1, ctx 2048, 8 kv heads: minimum 64
  // keys 20.15 us per call, 256 18.17, 512 18.13, 1024 21.30).
  if (sl < 256) sl = 256;
  if (sl < p->KT) sl = p->KT;
  p->split_len = (int)sl;
  p->max_splits = (int)((max_L + sl - 1) / sl);
  p->Mpad = ((G * sh->max_block + 15) / 16) * 16;
  const long long nw = pairs * p->max_splits;
  if (nw > (1LL << 30)) return fail(SD_ERR_INVALID_ARG, "problem too large");
  p->n_work = (int)nw;
  // One wave: one workgroup per slot, the splits of a pair dealt to one XCD (measured slightly
  // faster on the ragged Qwen3-4B batch than round-robin).  More than one wave: the device
  // numbers the existing splits densely (attn_item), so no workgroup is spent on an empty slot
  // and round-robin dispatch spreads long sequences over every XCD (long-context batch, 32
  // sequences with contexts 8k-32k: 677-714 us with one workgroup per slot, about 600 dense).
  p->dense = nw > target_wgs;
  p->per_xcd = (int)((nw + sdb::kNumXcd - 1) / sdb::kNumXcd);
  p->grid = p->dense ? (int)nw : p->per_xcd * sdb::kNumXcd;
  // Where even splits would need more than one wave (bf16), every workgroup gets an equal share
  // of all the pairs' (weighted) key tiles instead (bal_share), in the plain, paged and
  // fused-append calls alike.  Partial slots: one per workgroup and pair a share touches, at
  // most kBalGrid + pairs.
  p->bal = sh->dtype == SD_BF16 && p->dense && p->max_splits > 1;
  {  // the device sums tile weights (at most kBalWeightMax8 + 4 per m-tile past 8) in 32-bit integers
    const long long nmt_max = (G * (long long)sh->max_block + 15) / 16;
    const long long wmax = sdb::kBalWeightMax8 + 4 * std::max(0LL, nmt_max - 8);
    if (pairs * ((max_L + kBf16KT - 1) / kBf16KT) * wmax > (1LL << 30)) p->bal = 0;
  }
  const long long slots = p->bal ? std::max(nw, (long long)kBalGrid + pairs) : nw;
  const int nmt = p->Mpad / 16;
  if (sh->dtype == SD_BF16) p->MT = nmt <= 8 ? 1 : 2;  // 8 wavefronts, 1 or 2 m-tiles each
  else p->MT = nmt <= 4 ? 1 : nmt <= 8 ? 2 : 4;      // 4 wavefronts
  p->ve = sh->dtype == SD_BF16 && nmt >= 7 && nmt <= 8;
  size_t off = 0;
  p->off_ml = off;
  if (p->max_splits > 1) off = align256(off + (size_t)slots * p->Mpad * sizeof(float2));
  p->off_o = off;
  if (p->max_splits > 1) off = align256(off + (size_t)slots * p->Mpad * D * sizeof(float));
  p->total = off > 0 ? off : 256;
  return ok();
}

template <bool BF16, int D, int MT>
void launch_attn(const sdb::AttnArgs &a, int grid, hipStream_t st) {
  hipLaunchKernelGGL((sdb::block_attn_kernel<BF16, D, MT>), dim3(grid), dim3(256), 0, st, a);
}

// The balanced plan (bf16): kBalGrid workgroups, then the merge.
template <int D, bool PAGED = false, bool APPEND = false>
void launch_attn_bal(sdb::AttnArgs a, int MT, hipStream_t st, bool ve) {
  a.bal = 1;
  if (ve)
    hipLaunchKernelGGL((sdb::block_attn_bf16_kernel<D, 1, kBf16KT, kBf16NS, PAGED, APPEND, true, true>),
                       dim3(a.bal_grid), dim3(512), 0, st, a);
  else if (MT == 1)
    hipLaunchKernelGGL((sdb::block_attn_bf16_kernel<D, 1, kBf16KT, kBf16NS, PAGED, APPEND, true>), dim3(a.bal_grid),
                       dim3(512), 0, st, a);
  else
    hipLaunchKernelGGL((sdb::block_attn_bf16_kernel<D, 2, kBf16KT, kBf16NS, PAGED, APPEND, true>), dim3(a.bal_grid),
                       dim3(512), 0, st, a);
  constexpr int RB = 256 / (D / 4);
  const int nrb = (a.Mpad + RB - 1) / RB;
  hipLaunchKernelGGL((sdb::block_attn_merge_kernel<true, D, 8>), dim3(a.S * a.Hkv * nrb), dim3(256), 0, st, a);
}

template <bool BF16, int D, bool PAGED = false, bool APPEND = false>
void launch_attn_all(const sdb::AttnArgs &a, int grid, int MT, hipStream_t st, bool ve = false) {
  if constexpr (BF16) {
    if (ve)
      hipLaunchKernelGGL((sdb::block_attn_bf16_kernel<D, 1, kBf16KT, kBf16NS, PAGED, APPEND, false, true>), dim3(grid),
                         dim3(512), 0, st, a);
    else if (MT == 1)
      hipLaunchKernelGGL((sdb::block_attn_bf16_kernel<D, 1, kBf16KT, kBf16NS, PAGED, APPEND>), dim3(grid), dim3(512), 0,
                         st, a);
    else
      hipLaunchKernelGGL((sdb::block_attn_bf16_kernel<D, 2, kBf16KT, kBf16NS, PAGED, APPEND>), dim3(grid), dim3(512), 0,
                         st, a);
  } else {
    if (MT == 1) launch_attn<BF16, D, 1>(a, grid, st);
    else if (MT == 2) launch_attn<BF16, D, 2>(a, grid, st);
    else launch_attn<BF16, D, 4>(a, grid, st);
  }
  if (a.max_splits > 1) {
    constexpr int RB = 256 / (D / 4);  // rows per merge workgroup
    const int nrb = (a.Mpad + RB - 1) / RB;
    const dim3 g(a.S * a.Hkv * nrb);
    // every split's loads in one round where the plan allows up to 16 splits (Qwen3-4B verify at
    // batch 1, 9 splits per pair: merge kernel 5.34 -> 4.51 us)
    if (a.max_splits <= 4) hipLaunchKernelGGL((sdb::block_attn_merge_kernel<BF16, D, 4>), g, dim3(256), 0, st, a);
    else if (a.max_splits <= 8) hipLaunchKernelGGL((sdb::block_attn_merge_kernel<BF16, D, 8>), g, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((sdb::block_attn_merge_kernel<BF16, D, 16>), g, dim3(256), 0, st, a);
  }
}

// ---------------------------------------------------------------------------
// acceptance planning
// ---------------------------------------------------------------------------
struct AcceptPlan {
  int rows, nch, nch2, stats_grid, tail_wide;
  size_t off_stats, off_samp, off_seq, total;
  // single launch at T = 0 (accept_fused_kernel): possible for this shape, its tail
  // workgroups (one per sequence), and its workspace (tagged records)
  int fused_ok, n_tail;
  size_t total_fused;
  // single-launch draw at T > 0 (accept_draw_kernel): possible for this shape, and its
  // workspace (the two-launch layout, then the tagged chunk sums)
  int draw_ok;
  size_t off_draw, total_draw;
};

// Sequences of one single-launch call, at most (the launch also checks them against the
// device's resident capacity for the kernel).
constexpr int kFusedMaxTail = 1024;

int accept_plan(const sd_accept_shape *sh, float temperature, AcceptPlan *p) {
  if (!sh) return fail(SD_ERR_INVALID_ARG, "sd_accept: shape is NULL");
  const int S = sh->num_seqs, V = sh->vocab;
  if (S < 0) return fail(SD_ERR_INVALID_ARG, "num_seqs must be >= 0 (got %d)", S);
  if (V < 1 || V > (1 << 28)) return fail(SD_ERR_INVALID_ARG, "vocab must be in [1, 2^28] (got %d)", V);
  if (sh->dtype != SD_BF16 && sh->dtype != SD_F32) return fail(SD_ERR_INVALID_ARG, "unknown dtype %d", sh->dtype);
  if (sh->max_block < 1 || sh->max_block > 64)
    return fail(SD_ERR_INVALID_ARG, "max_block must be in [1, 64] (got %d)", sh->max_block);
  if (sh->total_q < S || (long long)sh->total_q > (long long)S * sh->max_block)
    return fail(SD_ERR_INVALID_ARG, "total_q %d outside [num_seqs, num_seqs * max_block]", sh->total_q);
  if (!(temperature >= 0.f) || isinf(temperature))
    return fail(SD_ERR_INVALID_ARG, "temperature must be finite and >= 0");
  const bool sample = temperature > 0.f;
  const long long rows = (long long)sh->total_q + (sample ? (long long)sh->total_q - S : 0);
  if (rows * (long long)V > (1LL << 46)) return fail(SD_ERR_INVALID_ARG, "problem too large");
  const int VEC = (sh->dtype == SD_BF16) ? 8 : 4;
  const long long vecs = V / VEC;
  // statistics chunks: kStatsChunk whole vectors each (one load of kStatsVecs vectors per
  // thread); a row holds vecs or vecs - 1 whole vectors, the last chunk takes the rest
  long long nch = (vecs + sdb::kStatsChunk - 1) / sdb::kStatsChunk;
  if (nch < 1) nch = 1;
  // sampling chunks: at most 256 whole vectors each, so the mass and locate kernels hold one
  // vector per thread and reach the selected row in one round of loads (ragged Qwen3-4B batch
  // at T = 1); vocabularies that would need
  // more than kMaxChunks2 chunks take wider chunks and the kernels' multi-vector rounds
  long long nch2 = (vecs + sdb::kLocThreads - 1) / sdb::kLocThreads;
  int tail_wide = 0;
  if (nch2 > sdb::kMaxChunks2) {
    tail_wide = 1;
    const long long per = (long long)sdb::kLocThreads * sdb::kTailVecsWide;
    nch2 = (vecs + per - 1) / per;
    if (nch2 > sdb::kMaxChunks2) nch2 = sdb::kMaxChunks2;
  }
  if (nch2 < 1) nch2 = 1;
  if (rows * nch > (1LL << 30)) return fail(SD_ERR_INVALID_ARG, "problem too large");
  const long long items = rows * nch;
  p->rows = (int)rows;
  p->nch = (int)nch;
  p->nch2 = (int)nch2;
  p->tail_wide = tail_wide;
  p->stats_grid = (int)(items > 0 ? items : 1);
  const size_t kinds = sample ? 2 : 1;
  size_t off = 0;
  p->off_stats = off;
  off = align256(off + kinds * (size_t)S * sh->max_block * nch * sizeof(float4));
  p->off_samp = off;
  if (sample) off = align256(off + (size_t)S * nch2 * sizeof(double2));
  p->off_seq = off;
  if (sample) off = align256(off + (size_t)S * 2 * sizeof(float4));
  p->total = off > 0 ? off : 256;
  // the single launch (greedy only): one batch of records per position
  p->n_tail = S;
  p->fused_ok = !sample && S >= 1 && nch <= sdb::kFusedMaxNch && S <= kFusedMaxTail && items + S <= INT_MAX;
  p->total_fused =
      p->fused_ok ? align256((size_t)S * sh->max_block * nch * 3 * sizeof(unsigned long long)) : 0;
  // the single-launch draw (sampling): chunks of one vector per thread, whose sums a
  // wavefront holds in registers
  p->draw_ok = sample && S >= 1 && !tail_wide && nch2 <= 64LL * sdb::kLocSums && (long long)S * nch2 <= INT_MAX;
  p->off_draw = p->total;
  p->total_draw =
      p->draw_ok ? p->total + align256((size_t)S * sdb::kSumReplicas * 2 * nch2 * sizeof(unsigned long long)) : 0;
  return ok();
}

int check_cache_shape(const sd_attn_shape *sh, const char *what) {
  if (!sh) return fail(SD_ERR_INVALID_ARG, "%s: shape is NULL", what);
  if (sh->num_seqs < 0) return fail(SD_ERR_INVALID_ARG, "num_seqs must be >= 0 (got %d)", sh->num_seqs);
  if (sh->num_q_heads < 1 || sh->num_kv_heads < 1 || sh->num_q_heads % sh->num_kv_heads)
    return fail(SD_ERR_INVALID_ARG, "head counts must be >= 1 with Hq %% Hkv == 0 (Hq=%d, Hkv=%d)",
                sh->num_q_heads, sh->num_kv_heads);
  if (sh->dtype != SD_BF16 && sh->dtype != SD_F32) return fail(SD_ERR_INVALID_ARG, "unknown dtype %d", sh->dtype);
  if (sh->head_dim != 64 && sh->head_dim != 128)
    return fail(SD_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", sh->head_dim);
  if (sh->max_kv_len < 1) return fail(SD_ERR_INVALID_ARG, "max_kv_len must be >= 1 (got %d)", sh->max_kv_len);
  if (sh->total_q < 0) return fail(SD_ERR_INVALID_ARG, "total_q must be >= 0 (got %d)", sh->total_q);
  return ok();
}

struct PolicyPlan {
  size_t off_stats, off_h1, off_h2, total;
};

int policy_plan(const sd_policy_shape *sh, PolicyPlan *p) {
  if (!sh) return fail(SD_ERR_INVALID_ARG, "sd_block_size_policy: shape is NULL");
  if (sh->num_prompts < 0) return fail(SD_ERR_INVALID_ARG, "num_prompts must be >= 0 (got %d)", sh->num_prompts);
  if (sh->vocab < 8 || sh->vocab % 8 || sh->vocab > (1 << 28))
    return fail(SD_ERR_UNSUPPORTED, "vocab must be a multiple of 8 in [8, 2^28] (got %d)", sh->vocab);
  if (sh->hidden < 8 || sh->hidden % 8 || sh->hidden > (1 << 20))
    return fail(SD_ERR_UNSUPPORTED, "hidden must be a multiple of 8 in [8, 2^20] (got %d)", sh->hidden);
  if (sh->radius < 0 || 2 * sh->radius + 1 > 64)
    return fail(SD_ERR_INVALID_ARG, "radius must give at most 64 candidates (got %d)", sh->radius);
  if (sh->base_block - sh->radius < 1)
    return fail(SD_ERR_INVALID_ARG, "candidate block sizes must be >= 1 (base %d, radius %d)", sh->base_block,
                sh->radius);
  if (sh->logits_dtype != SD_BF16 && sh->logits_dtype != SD_F32)
    return fail(SD_ERR_INVALID_ARG, "unknown dtype %d", sh->logits_dtype);
  const size_t P = (size_t)sh->num_prompts;
  size_t off = 0;
  p->off_stats = off;
  off = align256(off + P * sdb::kPolicyChunks * sizeof(float2));
  p->off_h1 = off;
  off = align256(off + P * sh->hidden * sizeof(float));
  p->off_h2 = off;
  off = align256(off + P * sh->hidden * sizeof(float));
  p->total = off > 0 ? off : 256;
  return ok();
}

template <bool RELU, int XM>
void launch_dense(const sdb::DenseArgs &d, hipStream_t st) {
  const dim3 grid((d.rows + sdb::kDenseRows - 1) / sdb::kDenseRows);
  if (d.P <= 1) hipLaunchKernelGGL((sdb::policy_dense_kernel<1, RELU, XM>), grid, dim3(256), 0, st, d);
  else if (d.P <= 2) hipLaunchKernelGGL((sdb::policy_dense_kernel<2, RELU, XM>), grid, dim3(256), 0, st, d);
  else if (d.P <= 4) hipLaunchKernelGGL((sdb::policy_dense_kernel<4, RELU, XM>), grid, dim3(256), 0, st, d);
  else hipLaunchKernelGGL((sdb::policy_dense_kernel<8, RELU, XM>), grid, dim3(256), 0, st, d);
}

}  // namespace

extern "C" {

const char *sd_last_error(void) { return g_err.c_str(); }

const char *sd_version(void) { return "sdblock 0.1 gfx950"; }

int sd_block_attn_workspace_size(const sd_attn_shape *shape, size_t *bytes) {
  if (!bytes) return fail(SD_ERR_INVALID_ARG, "bytes is NULL");
  AttnPlan p;
  int rc = attn_plan(shape, &p);
  if (rc) return rc;
  *bytes = p.total;
  return ok();
}

namespace {

int attn_args(const sd_attn_shape *sh, const AttnPlan &p, const void *q, const void *k_cache, const void *v_cache,
              const int32_t *ctx_lens, const int32_t *block_lens, const int32_t *q_offsets, int32_t mask_mode,
              void *out, void *workspace, size_t workspace_bytes, sdb::AttnArgs *a) {
  if (mask_mode != SD_MASK_CAUSAL_IN_BLOCK && mask_mode != SD_MASK_BIDIR_IN_BLOCK)
    return fail(SD_ERR_INVALID_ARG, "unknown mask_mode %d", mask_mode);
  if (!q || !k_cache || !v_cache || !out || !ctx_lens || !block_lens || !q_offsets || !workspace)
    return fail(SD_ERR_INVALID_ARG, "sd_block_attn: NULL pointer argument");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out))
    return fail(SD_ERR_INVALID_ARG, "q, caches and out must be 16-byte aligned");
  if (((uintptr_t)workspace & 255u) != 0) return fail(SD_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (workspace_bytes < p.total)
    return fail(SD_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, p.total);
  a->q = q;
  a->k = k_cache;
  a->v = v_cache;
  a->out = out;
  a->ctx_lens = ctx_lens;
  a->block_lens = block_lens;
  a->q_offsets = q_offsets;
  char *ws = (char *)workspace;
  a->part_ml = (float2 *)(ws + p.off_ml);
  a->part_o = (float *)(ws + p.off_o);
  a->S = sh->num_seqs;
  a->Hq = sh->num_q_heads;
  a->Hkv = sh->num_kv_heads;
  a->G = p.G;
  a->Lmax = sh->max_kv_len;
  a->split_len = p.split_len;
  a->gran = sh->dtype == SD_BF16 ? 16 : p.KT;
  a->max_splits = p.max_splits;
  a->Mpad = p.Mpad;
  a->n_work = p.n_work;
  a->per_xcd = p.per_xcd;
  a->dense = p.dense;
  const float scale = sh->scale > 0.f ? sh->scale : 1.0f / sqrtf((float)sh->head_dim);
  a->scale_log2 = scale * 1.4426950408889634f;
  a->causal = mask_mode == SD_MASK_CAUSAL_IN_BLOCK;
  a->block_table = nullptr;
  a->page_log2 = a->max_pages = a->num_pages = 0;
  a->k_new = a->v_new = nullptr;
  a->bal = 0;  // sd_block_attn turns it on where its plan says so
  a->bal_grid = kBalGrid;
  a->bal_min_tiles = kBalMinTiles;
  a->bal_kt = kBf16KT;
  return ok();
}

}  // namespace

int sd_block_attn(const sd_attn_shape *sh, const void *q, const void *k_cache, const void *v_cache,
                  const int32_t *ctx_lens, const int32_t *block_lens, const int32_t *q_offsets,
                  int32_t mask_mode, void *out, void *workspace, size_t workspace_bytes, void *stream) {
  AttnPlan p;
  int rc = attn_plan(sh, &p);
  if (rc) return rc;
  if (sh->num_seqs == 0 || sh->total_q == 0) {
    if (mask_mode != SD_MASK_CAUSAL_IN_BLOCK && mask_mode != SD_MASK_BIDIR_IN_BLOCK)
      return fail(SD_ERR_INVALID_ARG, "unknown mask_mode %d", mask_mode);
    return ok();
  }
  sdb::AttnArgs a;
  rc = attn_args(sh, p, q, k_cache, v_cache, ctx_lens, block_lens, q_offsets, mask_mode, out, workspace,
                 workspace_bytes, &a);
  if (rc) return rc;
  const int grid = p.grid;
  hipStream_t st = (hipStream_t)stream;
  const bool bf = sh->dtype == SD_BF16;
  if (p.bal) {
    if (sh->head_dim == 128) launch_attn_bal<128>(a, p.MT, st, p.ve);
    else launch_attn_bal<64>(a, p.MT, st, p.ve);
    return check_launch("sd_block_attn");
  }
  if (sh->head_dim == 128) {
    if (bf) launch_attn_all<true, 128>(a, grid, p.MT, st, p.ve);
    else launch_attn_all<false, 128>(a, grid, p.MT, st);
  } else {
    if (bf) launch_attn_all<true, 64>(a, grid, p.MT, st, p.ve);
    else launch_attn_all<false, 64>(a, grid, p.MT, st);
  }
  return check_launch("sd_block_attn");
}

int sd_block_attn_append(const sd_attn_shape *sh, const void *q, const void *k_new, const void *v_new, void *k_cache,
                         void *v_cache, const int32_t *ctx_lens, const int32_t *block_lens, const int32_t *q_offsets,
                         int32_t mask_mode, void *out, void *workspace, size_t workspace_bytes, void *stream) {
  AttnPlan p;
  int rc = attn_plan(sh, &p);
  if (rc) return rc;
  if (sh->dtype != SD_BF16) return fail(SD_ERR_UNSUPPORTED, "sd_block_attn_append: bf16 only");
  if (sh->num_seqs == 0 || sh->total_q == 0) {
    if (mask_mode != SD_MASK_CAUSAL_IN_BLOCK && mask_mode != SD_MASK_BIDIR_IN_BLOCK)
      return fail(SD_ERR_INVALID_ARG, "unknown mask_mode %d", mask_mode);
    return ok();
  }
  if (!k_new || !v_new) return fail(SD_ERR_INVALID_ARG, "sd_block_attn_append: NULL pointer argument");
  if (!aligned16(k_new) || !aligned16(v_new)) return fail(SD_ERR_INVALID_ARG, "new rows must be 16-byte aligned");
  sdb::AttnArgs a;
  rc = attn_args(sh, p, q, k_cache, v_cache, ctx_lens, block_lens, q_offsets, mask_mode, out, workspace,
                 workspace_bytes, &a);
  if (rc) return rc;
  a.k_new = k_new;
  a.v_new = v_new;
  hipStream_t st = (hipStream_t)stream;
  if (p.bal) {
    if (sh->head_dim == 128) launch_attn_bal<128, false, true>(a, p.MT, st, p.ve);
    else launch_attn_bal<64, false, true>(a, p.MT, st, p.ve);
  } else if (sh->head_dim == 128) {
    launch_attn_all<true, 128, false, true>(a, p.grid, p.MT, st, p.ve);
  } else {
    launch_attn_all<true, 64, false, true>(a, p.grid, p.MT, st, p.ve);
  }
  return check_launch("sd_block_attn_append");
}

namespace {

int check_pages(const sd_attn_shape *sh, int32_t page_size, int32_t num_pages, int32_t max_pages, int *log2) {
  if (sh && sh->dtype != SD_BF16) return fail(SD_ERR_UNSUPPORTED, "paged caches are bf16 only");
  if (page_size < 16 || page_size > 4096 || (page_size & (page_size - 1)))
    return fail(SD_ERR_INVALID_ARG, "page_size must be a power of two in [16, 4096] (got %d)", page_size);
  if (num_pages < 1 || max_pages < 1) return fail(SD_ERR_INVALID_ARG, "num_pages and max_pages must be >= 1");
  if (sh && (long long)max_pages * page_size != sh->max_kv_len)
    return fail(SD_ERR_INVALID_ARG, "max_kv_len (%d) must equal max_pages * page_size (%d * %d)", sh->max_kv_len,
                max_pages, page_size);
  int l = 0;
  while ((1 << l) < page_size) ++l;
  *log2 = l;
  return ok();
}

}  // namespace

int sd_block_attn_paged(const sd_attn_shape *sh, int32_t page_size, int32_t num_pages, int32_t max_pages,
                        const int32_t *block_table, const void *q, const void *k_pages, const void *v_pages,
                        const int32_t *ctx_lens, const int32_t *block_lens, const int32_t *q_offsets,
                        int32_t mask_mode, void *out, void *workspace, size_t workspace_bytes, void *stream) {
  AttnPlan p;
  int rc = attn_plan(sh, &p);
  if (rc) return rc;
  int log2 = 0;
  rc = check_pages(sh, page_size, num_pages, max_pages, &log2);
  if (rc) return rc;
  if (sh->num_seqs == 0 || sh->total_q == 0) return ok();
  if (!block_table) return fail(SD_ERR_INVALID_ARG, "sd_block_attn_paged: block_table is NULL");
  sdb::AttnArgs a;
  rc = attn_args(sh, p, q, k_pages, v_pages, ctx_lens, block_lens, q_offsets, mask_mode, out, workspace,
                 workspace_bytes, &a);
  if (rc) return rc;
  a.block_table = block_table;
  a.page_log2 = log2;
  a.max_pages = max_pages;
  a.num_pages = num_pages;
  const int grid = p.grid;
  hipStream_t st = (hipStream_t)stream;
  if (p.bal) {
    if (sh->head_dim == 128) launch_attn_bal<128, true>(a, p.MT, st, p.ve);
    else launch_attn_bal<64, true>(a, p.MT, st, p.ve);
  } else if (sh->head_dim == 128) {
    launch_attn_all<true, 128, true>(a, grid, p.MT, st, p.ve);
  } else {
    launch_attn_all<true, 64, true>(a, grid, p.MT, st, p.ve);
  }
  return check_launch("sd_block_attn_paged");
}

int sd_kv_append_paged(const sd_attn_shape *sh, int32_t page_size, int32_t num_pages, int32_t max_pages,
                       const int32_t *block_table, const void *k_new, const void *v_new, void *k_pages, void *v_pages,
                       const int32_t *ctx_lens, const int32_t *q_offsets, void *stream) {
  int rc = check_cache_shape(sh, "sd_kv_append_paged");
  if (rc) return rc;
  int log2 = 0;
  rc = check_pages(nullptr, page_size, num_pages, max_pages, &log2);
  if (rc) return rc;
  if (sh->num_seqs == 0 || sh->total_q == 0) return ok();
  if (!k_new || !v_new || !k_pages || !v_pages || !ctx_lens || !q_offsets || !block_table)
    return fail(SD_ERR_INVALID_ARG, "sd_kv_append_paged: NULL pointer argument");
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pages) || !aligned16(v_pages))
    return fail(SD_ERR_INVALID_ARG, "new rows and page pools must be 16-byte aligned");
  sdb::AppendArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_cache = k_pages;
  a.v_cache = v_pages;
  a.ctx_lens = ctx_lens;
  a.q_offsets = q_offsets;
  a.S = sh->num_seqs;
  a.Hkv = sh->num_kv_heads;
  a.Lmax = max_pages * page_size;
  a.total_q = sh->total_q;
  a.row_vecs = sh->head_dim * (sh->dtype == SD_BF16 ? 2 : 4) / 16;
  a.block_table = block_table;
  a.page_log2 = log2;
  a.max_pages = max_pages;
  a.num_pages = num_pages;
  hipLaunchKernelGGL(sdb::kv_append_paged_kernel, dim3(sh->total_q, 2), dim3(256), 0, (hipStream_t)stream, a);
  return check_launch("sd_kv_append_paged");
}

int sd_accept_workspace_size(const sd_accept_shape *shape, float temperature, size_t *bytes) {
  if (!bytes) return fail(SD_ERR_INVALID_ARG, "bytes is NULL");
  AcceptPlan p;
  int rc = accept_plan(shape, temperature, &p);
  if (rc) return rc;
  *bytes = std::max(p.total, std::max(p.total_fused, p.total_draw));
  return ok();
}

namespace {

// Host-side checks of an sd_accept call (shape, pointers, alignment, workspace); nothing is
// enqueued.  Returns SD_OK with the plan filled in.
int check_accept_call(const sd_accept_shape *sh, const void *target_logits, const void *draft_logits,
                      const int32_t *draft_tokens, const float *uniforms, const int32_t *block_lens,
                      const int32_t *q_offsets, float temperature, const int32_t *accept_len,
                      const int32_t *next_token, const void *workspace, size_t workspace_bytes, AcceptPlan *p) {
  int rc = accept_plan(sh, temperature, p);
  if (rc) return rc;
  if (sh->num_seqs == 0) return ok();
  const bool sample = temperature > 0.f;
  if (!target_logits || !block_lens || !q_offsets || !accept_len || !next_token || !workspace)
    return fail(SD_ERR_INVALID_ARG, "sd_accept: NULL pointer argument");
  if (sh->total_q > sh->num_seqs && !draft_tokens) return fail(SD_ERR_INVALID_ARG, "draft_tokens is NULL");
  // draft rows exist only where some block holds a drafted token (total_q > S)
  const bool drafts = sh->total_q > sh->num_seqs;
  if (sample && ((drafts && !draft_logits) || !uniforms))
    return fail(SD_ERR_INVALID_ARG, "draft_logits (when total_q > num_seqs) and uniforms are required when temperature > 0");
  if (!aligned16(target_logits) || (sample && drafts && !aligned16(draft_logits)))
    return fail(SD_ERR_INVALID_ARG, "logits must be 16-byte aligned");
  if (((uintptr_t)workspace & 255u) != 0) return fail(SD_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (workspace_bytes < p->total)
    return fail(SD_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, p->total);
  return ok();
}

}  // namespace

namespace {

// Path selection for tests (sd_accept_set_path): 0 = single launch where possible, 1 = never;
// the poll limit of the single launch's waits (<= 0: the default).
std::atomic<int> g_accept_path{0};
std::atomic<int> g_accept_spin{0};
constexpr int kDefaultSpinLimit = 1 << 20;  // about a second of polling

// The tag of a single-launch call: a bijective 32-bit hash (MurmurHash3's finaliser) of a
// per-process call counter with a random start, so no two calls of a process within 2^32 share
// a tag and tags are spread over all 32-bit values, whatever data the workspace held before.
unsigned next_accept_tag() {
  static std::atomic<unsigned> ctr{0};
  static std::once_flag once;
  std::call_once(once, [] { ctr.store((unsigned)std::random_device{}()); });
  unsigned h = ctr.fetch_add(1, std::memory_order_relaxed);
  h ^= h >> 16;
  h *= 0x85ebca6bu;
  h ^= h >> 13;
  h *= 0xc2b2ae35u;
  h ^= h >> 16;
  return h;
}

constexpr int kMaxDevices = 64;  // devices whose per-device state the library keeps

// Workgroups of a single-launch acceptance kernel the current device holds at once (the least
// over the instantiations of accept_fused_kernel, kind 0, or accept_draw_kernel, kind 1), or 0
// if the runtime cannot tell; per device, computed on first use.
int resident_capacity(int kind) {
  static std::atomic<int> cap[2][kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return 0;
  }
  int c = cap[kind][dev].load(std::memory_order_relaxed);
  if (c > 0) return c;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) {
    (void)hipGetLastError();
    return 0;
  }
  const void *fused[] = {(const void *)sdb::accept_fused_kernel<true, true>, (const void *)sdb::accept_fused_kernel<true, false>,
                         (const void *)sdb::accept_fused_kernel<false, true>, (const void *)sdb::accept_fused_kernel<false, false>};
  const void *draw[] = {(const void *)sdb::accept_draw_kernel<true>, (const void *)sdb::accept_draw_kernel<false>};
  const void *const *ks = kind == 0 ? fused : draw;
  const int nk = kind == 0 ? 4 : 2;
  int per_cu = INT_MAX;
  for (int i = 0; i < nk; ++i) {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, ks[i], 256, 0) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    per_cu = std::min(per_cu, nb);
  }
  c = per_cu * cus;
  cap[kind][dev].store(c, std::memory_order_relaxed);
  return c;
}

// True when the single launch may run on this stream: it waits across workgroups on words
// tagged per call, so a graph that replays a captured launch (with its tag) must not hold it.
bool stream_allows_fused(hipStream_t st) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cs) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return cs == hipStreamCaptureStatusNone;
}

// Enqueue the acceptance kernels of a checked call; `workspace` holds workspace_bytes >=
// p.total bytes.
int accept_enqueue(const sd_accept_shape *sh, const AcceptPlan &p, const void *target_logits,
                   const void *draft_logits, const int32_t *draft_tokens, const float *uniforms,
                   const int32_t *block_lens, const int32_t *q_offsets, float temperature, int32_t *accept_len,
                   int32_t *next_token, void *workspace, size_t workspace_bytes, void *stream) {
  const bool sample = temperature > 0.f;

  sdb::AcceptArgs a{};
  a.target = target_logits;
  a.draft = draft_logits;
  a.draft_tokens = draft_tokens;
  a.uniforms = uniforms;
  a.block_lens = block_lens;
  a.q_offsets = q_offsets;
  a.accept_len = accept_len;
  a.next_token = next_token;
  char *ws = (char *)workspace;
  a.stats = (float4 *)(ws + p.off_stats);
  a.samp = (double2 *)(ws + p.off_samp);
  a.seqinfo = (float4 *)(ws + p.off_seq);
  a.S = sh->num_seqs;
  a.V = sh->vocab;
  a.total_q = sh->total_q;
  a.rows = p.rows;
  a.mb = sh->max_block;
  a.nch = p.nch;
  a.nch2 = p.nch2;
  a.c = sample ? (float)(1.4426950408889634 / (double)temperature) : 0.f;
  hipStream_t st = (hipStream_t)stream;
  const bool bf = sh->dtype == SD_BF16;
  const unsigned g1 = (unsigned)p.stats_grid;
  const unsigned S = (unsigned)sh->num_seqs;
  // every statistics chunk holds a whole 16-byte vector unless the vocabulary is tiny (then
  // there is one chunk and at most 2 VEC - 2 < 256 elements per row)
  const bool vecs = sh->vocab >= 2 * (bf ? 8 : 4) - 1;

  // Greedy acceptance in one launch when the shape, the workspace, the stream and the test
  // switch allow it (measured on the ragged Qwen3-4B batch: see accept_fused_kernel).  The
  // tail workgroups, which wait only for statistics workgroups (which never wait), must fit on
  // the device at once with a quarter of it to spare.
  if (p.fused_ok && workspace_bytes >= p.total_fused && g_accept_path.load(std::memory_order_relaxed) == 0 &&
      4LL * p.n_tail <= 3LL * resident_capacity(0) && stream_allows_fused(st)) {
    a.trec = (unsigned long long *)ws;
    a.tag = next_accept_tag();
    a.n_items = p.stats_grid;
    const int spin = g_accept_spin.load(std::memory_order_relaxed);
    a.spin_limit = spin > 0 ? spin : kDefaultSpinLimit;
    const unsigned grid = (unsigned)(p.stats_grid + p.n_tail);
    if (bf) {
      if (vecs) hipLaunchKernelGGL((sdb::accept_fused_kernel<true, true>), dim3(grid), dim3(256), 0, st, a);
      else hipLaunchKernelGGL((sdb::accept_fused_kernel<true, false>), dim3(grid), dim3(256), 0, st, a);
    } else {
      if (vecs) hipLaunchKernelGGL((sdb::accept_fused_kernel<false, true>), dim3(grid), dim3(256), 0, st, a);
      else hipLaunchKernelGGL((sdb::accept_fused_kernel<false, false>), dim3(grid), dim3(256), 0, st, a);
    }
    return check_launch("sd_accept");
  }
#define SDB_STATS(BF, SMP)                                                                                    \
  do {                                                                                                       \
    if (vecs) hipLaunchKernelGGL((sdb::accept_stats_kernel<BF, SMP, true>), dim3(g1), dim3(256), 0, st, a);  \
    else hipLaunchKernelGGL((sdb::accept_stats_kernel<BF, SMP, false>), dim3(g1), dim3(256), 0, st, a);      \
  } while (0)
#define SDB_TAIL(BF, NV)                                                                                      \
  do {                                                                                                       \
    hipLaunchKernelGGL((sdb::accept_mass_kernel<BF, NV>), dim3(S * p.nch2), dim3(256), 0, st, a);             \
    hipLaunchKernelGGL((sdb::accept_locate_kernel<BF, NV>), dim3(S), dim3(sdb::kLocThreads), 0, st, a);       \
  } while (0)
  // Sampling draw in one launch (mass and locate together) when the shape, the workspace, the
  // stream and the test switch allow it and the whole grid fits on the device at once with a
  // quarter to spare (every workgroup of accept_draw_kernel waits for its sequence's others).
  if (sample && p.draw_ok && workspace_bytes >= p.total_draw && g_accept_path.load(std::memory_order_relaxed) == 0 &&
      4LL * S * p.nch2 <= 3LL * resident_capacity(1) && stream_allows_fused(st)) {
    a.csum = (unsigned long long *)(ws + p.off_draw);
    a.tag = next_accept_tag();
    const int spin = g_accept_spin.load(std::memory_order_relaxed);
    a.spin_limit = spin > 0 ? spin : kDefaultSpinLimit;
    if (bf) {
      SDB_STATS(true, true);
      hipLaunchKernelGGL((sdb::accept_draw_kernel<true>), dim3(S * p.nch2), dim3(256), 0, st, a);
    } else {
      SDB_STATS(false, true);
      hipLaunchKernelGGL((sdb::accept_draw_kernel<false>), dim3(S * p.nch2), dim3(256), 0, st, a);
    }
  } else if (sample) {
    if (bf) {
      SDB_STATS(true, true);
      if (p.tail_wide) SDB_TAIL(true, sdb::kTailVecsWide);
      else SDB_TAIL(true, 1);
    } else {
      SDB_STATS(false, true);
      if (p.tail_wide) SDB_TAIL(false, sdb::kTailVecsWide);
      else SDB_TAIL(false, 1);
    }
  } else {
    if (bf) SDB_STATS(true, false);
    else SDB_STATS(false, false);
    hipLaunchKernelGGL(sdb::accept_greedy_kernel, dim3(S), dim3(64), 0, st, a);
  }
#undef SDB_STATS
#undef SDB_TAIL
  return check_launch("sd_accept");
}

// ---- the fixed scratch of sd_accept_noalloc ----
// Device memory for the acceptance workspace of callers that cannot allocate.  Each device
// the library runs on holds its own copy until the process ends.  Host code never uses the
// array's name as an address: the name is a host-side stand-in, so kernels get the device
// address that hipGetSymbolAddress returns, looked up once per device with that device current.
constexpr size_t kNoAllocScratchBytes = SD_ACCEPT_NOALLOC_SCRATCH_BYTES;
constexpr int kNoAllocMaxDevices = kMaxDevices;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];
std::atomic<void *> g_scratch_ptr[kNoAllocMaxDevices];
std::mutex g_scratch_mu;

int noalloc_scratch(void **ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SD_ERR_HIP, "sd_accept_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kNoAllocMaxDevices)
    return fail(SD_ERR_UNSUPPORTED, "sd_accept_noalloc: device %d beyond the %d devices served", dev,
                kNoAllocMaxDevices);
  void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail(SD_ERR_HIP, "sd_accept_noalloc: hipGetSymbolAddress(scratch) on device %d: %s", dev,
                    hipGetErrorString(e));
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return ok();
}

}  // namespace

int sd_accept(const sd_accept_shape *sh, const void *target_logits, const void *draft_logits,
              const int32_t *draft_tokens, const float *uniforms, const int32_t *block_lens,
              const int32_t *q_offsets, float temperature, int32_t *accept_len, int32_t *next_token,
              void *workspace, size_t workspace_bytes, void *stream) {
  AcceptPlan p;
  int rc = check_accept_call(sh, target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets,
                             temperature, accept_len, next_token, workspace, workspace_bytes, &p);
  if (rc) return rc;
  if (sh->num_seqs == 0) return ok();
  return accept_enqueue(sh, p, target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets,
                        temperature, accept_len, next_token, workspace, workspace_bytes, stream);
}

int sd_accept_noalloc(const sd_accept_shape *sh, const void *target_logits, const void *draft_logits,
                      const int32_t *draft_tokens, const float *uniforms, const int32_t *block_lens,
                      const int32_t *q_offsets, float temperature, int32_t *accept_len, int32_t *next_token,
                      void *stream) {
  AcceptPlan p;
  int rc = accept_plan(sh, temperature, &p);
  if (rc) return rc;
  if (p.total > kNoAllocScratchBytes)
    return fail(SD_ERR_WORKSPACE,
                "sd_accept_noalloc: this shape needs %zu bytes of scratch, the library holds %zu; "
                "call sd_accept with a workspace instead", p.total, kNoAllocScratchBytes);
  if (sh->num_seqs == 0) return ok();
  void *ws = nullptr;
  rc = noalloc_scratch(&ws);
  if (rc) return rc;
  rc = check_accept_call(sh, target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets,
                         temperature, accept_len, next_token, ws, kNoAllocScratchBytes, &p);
  if (rc) return rc;
  return accept_enqueue(sh, p, target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets,
                        temperature, accept_len, next_token, ws, kNoAllocScratchBytes, stream);
}

int sd_accept_set_path(int32_t mode, int32_t spin_limit) {
  if (mode != 0 && mode != 1) return fail(SD_ERR_INVALID_ARG, "sd_accept_set_path: mode must be 0 or 1 (got %d)", mode);
  g_accept_path.store(mode, std::memory_order_relaxed);
  g_accept_spin.store(spin_limit > 0 ? spin_limit : 0, std::memory_order_relaxed);
  return ok();
}

// ---------------------------------------------------------------------------
// the step around verification: append, commit, and the whole verify step
// ---------------------------------------------------------------------------
static_assert(SD_CHECK_CTX == sdb::kCheckCtx && SD_CHECK_BLOCK == sdb::kCheckBlock &&
                  SD_CHECK_OFFSETS == sdb::kCheckOffsets && SD_CHECK_TOKEN == sdb::kCheckToken &&
                  SD_CHECK_UNIFORM == sdb::kCheckUniform,
              "check bits of the header and the kernel agree");

int sd_check_attn_inputs(const sd_attn_shape *sh, const int32_t *ctx_lens, const int32_t *block_lens,
                         const int32_t *q_offsets, int32_t *status, void *stream) {
  if (!sh) return fail(SD_ERR_INVALID_ARG, "sd_check_attn_inputs: shape is NULL");
  if (sh->num_seqs < 0 || sh->total_q < 0 || sh->max_ctx < 0 || sh->max_block < 1 || sh->max_block > 64)
    return fail(SD_ERR_INVALID_ARG, "sd_check_attn_inputs: num_seqs, total_q, max_ctx or max_block out of range");
  if (!status || (sh->num_seqs > 0 && (!ctx_lens || !block_lens || !q_offsets)))
    return fail(SD_ERR_INVALID_ARG, "sd_check_attn_inputs: NULL pointer argument");
  sdb::CheckArgs a{};
  a.ctx_lens = ctx_lens;
  a.block_lens = block_lens;
  a.q_offsets = q_offsets;
  a.status = status;
  a.S = sh->num_seqs;
  a.total_q = sh->total_q;
  a.max_ctx = sh->max_ctx;
  a.min_block = 0;
  a.max_block = sh->max_block;
  hipLaunchKernelGGL(sdb::check_inputs_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, a);
  return check_launch("sd_check_attn_inputs");
}

int sd_check_accept_inputs(const sd_accept_shape *sh, const int32_t *draft_tokens, const float *uniforms,
                           const int32_t *block_lens, const int32_t *q_offsets, float temperature,
                           int32_t *status, void *stream) {
  if (!sh) return fail(SD_ERR_INVALID_ARG, "sd_check_accept_inputs: shape is NULL");
  if (sh->num_seqs < 0 || sh->total_q < 0 || sh->vocab < 1 || sh->max_block < 1 || sh->max_block > 64)
    return fail(SD_ERR_INVALID_ARG, "sd_check_accept_inputs: num_seqs, total_q, vocab or max_block out of range");
  if (!(temperature >= 0.f) || isinf(temperature))
    return fail(SD_ERR_INVALID_ARG, "temperature must be finite and >= 0");
  if (!status || (sh->num_seqs > 0 && (!draft_tokens || !block_lens || !q_offsets || (temperature > 0.f && !uniforms))))
    return fail(SD_ERR_INVALID_ARG, "sd_check_accept_inputs: NULL pointer argument");
  sdb::CheckArgs a{};
  a.block_lens = block_lens;
  a.q_offsets = q_offsets;
  a.draft_tokens = draft_tokens;
  a.uniforms = temperature > 0.f ? uniforms : nullptr;
  a.status = status;
  a.S = sh->num_seqs;
  a.total_q = sh->total_q;
  a.min_block = 1;
  a.max_block = sh->max_block;
  a.vocab = sh->vocab;
  hipLaunchKernelGGL(sdb::check_inputs_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, a);
  return check_launch("sd_check_accept_inputs");
}

int sd_kv_append(const sd_attn_shape *sh, const void *k_new, const void *v_new, void *k_cache, void *v_cache,
                 const int32_t *ctx_lens, const int32_t *q_offsets, void *stream) {
  int rc = check_cache_shape(sh, "sd_kv_append");
  if (rc) return rc;
  if (sh->num_seqs == 0 || sh->total_q == 0) return ok();
  if (!k_new || !v_new || !k_cache || !v_cache || !ctx_lens || !q_offsets)
    return fail(SD_ERR_INVALID_ARG, "sd_kv_append: NULL pointer argument");
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) || !aligned16(v_cache))
    return fail(SD_ERR_INVALID_ARG, "new rows and caches must be 16-byte aligned");
  sdb::AppendArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.ctx_lens = ctx_lens;
  a.q_offsets = q_offsets;
  a.S = sh->num_seqs;
  a.Hkv = sh->num_kv_heads;
  a.Lmax = sh->max_kv_len;
  a.total_q = sh->total_q;
  a.row_vecs = sh->head_dim * (sh->dtype == SD_BF16 ? 2 : 4) / 16;
  a.block_table = nullptr;
  a.page_log2 = a.max_pages = a.num_pages = 0;
  hipLaunchKernelGGL(sdb::kv_append_kernel, dim3(sh->total_q, 2), dim3(256), 0, (hipStream_t)stream, a);
  return check_launch("sd_kv_append");
}

int sd_commit(int32_t num_seqs, const int32_t *accept_len, int32_t *ctx_lens, void *stream) {
  if (num_seqs < 0) return fail(SD_ERR_INVALID_ARG, "num_seqs must be >= 0 (got %d)", num_seqs);
  if (num_seqs == 0) return ok();
  if (!accept_len || !ctx_lens) return fail(SD_ERR_INVALID_ARG, "sd_commit: NULL pointer argument");
  hipLaunchKernelGGL(sdb::commit_kernel, dim3((num_seqs + 255) / 256), dim3(256), 0, (hipStream_t)stream,
                     accept_len, ctx_lens, num_seqs);
  return check_launch("sd_commit");
}

int sd_verify_step_workspace_size(const sd_attn_shape *attn_shape, const sd_accept_shape *accept_shape,
                                  float temperature, size_t *bytes) {
  if (!bytes) return fail(SD_ERR_INVALID_ARG, "bytes is NULL");
  size_t wa = 0, wc = 0;
  int rc = sd_block_attn_workspace_size(attn_shape, &wa);
  if (rc) return rc;
  rc = sd_accept_workspace_size(accept_shape, temperature, &wc);
  if (rc) return rc;
  *bytes = wa > wc ? wa : wc;
  return ok();
}

int sd_verify_step(const sd_attn_shape *ash, int32_t num_layers, const sd_layer_buffers *layers,
                   int32_t *ctx_lens, const int32_t *block_lens, const int32_t *q_offsets, int32_t mask_mode,
                   const sd_accept_shape *csh, const void *target_logits, const void *draft_logits,
                   const int32_t *draft_tokens, const float *uniforms, float temperature, int32_t *accept_len,
                   int32_t *next_token, void *workspace, size_t workspace_bytes, void *stream) {
  if (num_layers < 1) return fail(SD_ERR_INVALID_ARG, "num_layers must be >= 1 (got %d)", num_layers);
  if (!layers) return fail(SD_ERR_INVALID_ARG, "sd_verify_step: layers is NULL");
  if (!ash || !csh) return fail(SD_ERR_INVALID_ARG, "sd_verify_step: shape is NULL");
  if (ash->num_seqs != csh->num_seqs || ash->total_q != csh->total_q || ash->max_block != csh->max_block)
    return fail(SD_ERR_INVALID_ARG, "attention and acceptance shapes disagree on num_seqs, total_q or max_block");
  for (int l = 0; l < num_layers; ++l) {  // every pointer is checked before any work is enqueued
    const sd_layer_buffers &L = layers[l];
    if (!L.q || !L.k_new || !L.v_new || !L.k_cache || !L.v_cache || !L.out)
      return fail(SD_ERR_INVALID_ARG, "sd_verify_step: NULL pointer in layer %d", l);
    if (!aligned16(L.q) || !aligned16(L.k_new) || !aligned16(L.v_new) || !aligned16(L.k_cache) ||
        !aligned16(L.v_cache) || !aligned16(L.out))
      return fail(SD_ERR_INVALID_ARG, "sd_verify_step: layer %d buffers must be 16-byte aligned", l);
  }
  size_t need = 0;
  int rc = sd_verify_step_workspace_size(ash, csh, temperature, &need);
  if (rc) return rc;
  if (workspace_bytes < need) return fail(SD_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  // the acceptance and commit arguments too, before the layers are enqueued
  AcceptPlan cp;
  rc = check_accept_call(csh, target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets, temperature,
                         accept_len, next_token, workspace, workspace_bytes, &cp);
  if (rc) return rc;
  if (!ctx_lens) return fail(SD_ERR_INVALID_ARG, "sd_verify_step: ctx_lens is NULL");
  for (int l = 0; l < num_layers; ++l) {
    const sd_layer_buffers &L = layers[l];
    if (ash->dtype == SD_BF16) {  // append fused into the attention launch
      rc = sd_block_attn_append(ash, L.q, L.k_new, L.v_new, L.k_cache, L.v_cache, ctx_lens, block_lens, q_offsets,
                                mask_mode, L.out, workspace, workspace_bytes, stream);
      if (rc) return rc;
    } else {
      rc = sd_kv_append(ash, L.k_new, L.v_new, L.k_cache, L.v_cache, ctx_lens, q_offsets, stream);
      if (rc) return rc;
      rc = sd_block_attn(ash, L.q, L.k_cache, L.v_cache, ctx_lens, block_lens, q_offsets, mask_mode, L.out, workspace,
                         workspace_bytes, stream);
      if (rc) return rc;
    }
  }
  rc = sd_accept(csh, target_logits, draft_logits, draft_tokens, uniforms, block_lens, q_offsets, temperature,
                 accept_len, next_token, workspace, workspace_bytes, stream);
  if (rc) return rc;
  return sd_commit(csh->num_seqs, accept_len, ctx_lens, stream);
}

// ---------------------------------------------------------------------------
// block-size policy (once per prompt)
// ---------------------------------------------------------------------------
int sd_policy_workspace_size(const sd_policy_shape *shape, size_t *bytes) {
  if (!bytes) return fail(SD_ERR_INVALID_ARG, "bytes is NULL");
  PolicyPlan p;
  int rc = policy_plan(shape, &p);
  if (rc) return rc;
  *bytes = p.total;
  return ok();
}

int sd_block_size_policy(const sd_policy_shape *sh, const void *last_logits, const void *w1, const float *b1,
                         const void *w2, const float *b2, const void *w3, const float *b3, float *scores,
                         int32_t *block_size, void *workspace, size_t workspace_bytes, void *stream) {
  PolicyPlan p;
  int rc = policy_plan(sh, &p);
  if (rc) return rc;
  if (sh->num_prompts == 0) return ok();
  if (!last_logits || !w1 || !b1 || !w2 || !b2 || !w3 || !b3 || !scores || !block_size || !workspace)
    return fail(SD_ERR_INVALID_ARG, "sd_block_size_policy: NULL pointer argument");
  if (!aligned16(w1) || !aligned16(w2) || !aligned16(w3) || !aligned16(last_logits))
    return fail(SD_ERR_INVALID_ARG, "logits and weights must be 16-byte aligned");
  if (((uintptr_t)workspace & 255u) != 0) return fail(SD_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (workspace_bytes < p.total)
    return fail(SD_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, p.total);
  hipStream_t st = (hipStream_t)stream;
  char *ws = (char *)workspace;
  const int P = sh->num_prompts, V = sh->vocab, H = sh->hidden, C = 2 * sh->radius + 1;
  sdb::PolicyArgs pa;
  pa.logits = last_logits;
  pa.stats = (float2 *)(ws + p.off_stats);
  pa.P = P;
  pa.V = V;
  pa.logits_bf16 = sh->logits_dtype == SD_BF16;
  const dim3 gsoft(P * sdb::kPolicyChunks);
  if (pa.logits_bf16) hipLaunchKernelGGL(sdb::policy_stats_kernel<true>, gsoft, dim3(256), 0, st, pa);
  else hipLaunchKernelGGL(sdb::policy_stats_kernel<false>, gsoft, dim3(256), 0, st, pa);
  float *h1 = (float *)(ws + p.off_h1), *h2 = (float *)(ws + p.off_h2);
  // dense layers in groups of kPolicyMaxPrompts prompts (each group reads the weights once);
  // the first takes the logits and makes p = softmax(z) from the chunk records on the fly
  const size_t zb = pa.logits_bf16 ? 2 : 4;
  for (int g0 = 0; g0 < P; g0 += sdb::kPolicyMaxPrompts) {
    const int np = std::min(sdb::kPolicyMaxPrompts, P - g0);
    sdb::DenseArgs d1{(const uint16_t *)w1, (const char *)last_logits + (size_t)g0 * V * zb, b1,
                      h1 + (size_t)g0 * H, H, V, np, pa.stats + (size_t)g0 * sdb::kPolicyChunks};
    if (pa.logits_bf16) launch_dense<true, 1>(d1, st);
    else launch_dense<true, 2>(d1, st);
    sdb::DenseArgs d2{(const uint16_t *)w2, h1 + (size_t)g0 * H, b2, h2 + (size_t)g0 * H, H, H, np, nullptr};
    launch_dense<true, 0>(d2, st);
  }
  sdb::HeadArgs ha{(const uint16_t *)w3, h2, b3, scores, block_size, C, H, sh->base_block, sh->radius};
  hipLaunchKernelGGL(sdb::policy_head_kernel, dim3(P), dim3(256), 0, st, ha);
  return check_launch("sd_block_size_policy");
}

}  // extern "C"

// ---------------------------------------------------------------------------
// prefix-survival model (App. A)
// ---------------------------------------------------------------------------
namespace {

int survival_check(const sd_survival_shape *sh, const float *gamma, sdb::SurvivalArgs *a) {
  if (!sh) return fail(SD_ERR_INVALID_ARG, "survival: shape is NULL");
  if (sh->num_samples < 0) return fail(SD_ERR_INVALID_ARG, "num_samples must be >= 0 (got %d)", sh->num_samples);
  if (sh->max_pos < 1 || sh->max_pos > sdb::kSurvMaxPos)
    return fail(SD_ERR_INVALID_ARG, "max_pos must be in [1, %d] (got %d)", sdb::kSurvMaxPos, sh->max_pos);
  if (sh->num_cands < 1 || sh->num_cands > sdb::kSurvMaxCands)
    return fail(SD_ERR_INVALID_ARG, "num_cands must be in [1, %d] (got %d)", sdb::kSurvMaxCands, sh->num_cands);
  for (int c = 0; c < sh->num_cands; ++c) {
    const int b = sh->cands[c];
    if (b < 1 || b > sh->max_pos) return fail(SD_ERR_INVALID_ARG, "candidate %d (%d) outside [1, max_pos]", c, b);
    if (c > 0 && b <= sh->cands[c - 1]) return fail(SD_ERR_INVALID_ARG, "candidates must be strictly ascending");
  }
  if (!(sh->alpha >= 0.0) || isinf(sh->alpha)) return fail(SD_ERR_INVALID_ARG, "alpha must be finite and >= 0");
  if ((long long)sh->num_samples * sh->max_pos > (1LL << 31) - 1)
    return fail(SD_ERR_INVALID_ARG, "num_samples * max_pos exceeds 2^31 - 1");
  if (sh->num_samples > 0 && !gamma) return fail(SD_ERR_INVALID_ARG, "gamma is NULL");
  if (gamma && !aligned16(gamma)) return fail(SD_ERR_INVALID_ARG, "gamma must be 16-byte aligned");
  memset(a, 0, sizeof *a);
  a->gamma = gamma;
  a->N = sh->num_samples;
  a->P = sh->max_pos;
  a->C = sh->num_cands;
  a->train_block = sh->train_block;
  a->alpha = sh->alpha;
  for (int c = 0; c < sh->num_cands; ++c) a->cands[c] = sh->cands[c];
  return ok();
}

}  // namespace

extern "C" {

int sd_survival_tau(const sd_survival_shape *sh, const float *gamma, const int32_t *b_hat, double *tau,
                    int32_t *b_star, double *regret, double *lipschitz, void *stream) {
  sdb::SurvivalArgs a;
  int rc = survival_check(sh, gamma, &a);
  if (rc) return rc;
  if (!b_hat != !regret) return fail(SD_ERR_INVALID_ARG, "b_hat and regret must both be given or both be NULL");
  if (a.N == 0) return ok();
  if (!tau || !b_star) return fail(SD_ERR_INVALID_ARG, "sd_survival_tau: NULL output");
  a.b_hat = b_hat;
  a.tau = tau;
  a.b_star = b_star;
  a.regret = regret;
  a.lipschitz = lipschitz;
  // samples per workgroup: the most of 256, 128, 64 whose staged rows fit the LDS budget
  const size_t row_bytes = (size_t)(a.P + 1) * sizeof(float), fixed = sdb::kSurvMaxCands * sizeof(double);
  int spw = 256;
  while (spw > 64 && fixed + spw * row_bytes > (size_t)sdb::kSurvLdsBytes) spw /= 2;
  const size_t lds = fixed + spw * row_bytes;
  const int grid = (a.N + spw - 1) / spw;
  hipLaunchKernelGGL(sdb::survival_tau_kernel, dim3(grid), dim3(spw), lds, (hipStream_t)stream, a);
  return check_launch("sd_survival_tau");
}

int sd_survival_sample(const sd_survival_shape *sh, const float *gamma, uint64_t seed, int32_t trials,
                       double *mean_len, int32_t *len_hist, void *stream) {
  sdb::SurvivalArgs a;
  int rc = survival_check(sh, gamma, &a);
  if (rc) return rc;
  if (trials < 1 || trials > (1 << 30)) return fail(SD_ERR_INVALID_ARG, "trials must be in [1, 2^30] (got %d)", trials);
  if (a.N == 0) return ok();
  if (!mean_len) return fail(SD_ERR_INVALID_ARG, "sd_survival_sample: mean_len is NULL");
  a.seed = seed;
  a.trials = trials;
  a.mean_len = mean_len;
  a.len_hist = len_hist;
  const long long pairs = (long long)a.N * a.C;
  const long long grid = (pairs + sdb::kSurvWavesPerWg - 1) / sdb::kSurvWavesPerWg;
  if (grid > 0x7fffffffLL) return fail(SD_ERR_INVALID_ARG, "num_samples * num_cands too large");
  const size_t lds = (size_t)sdb::kSurvWavesPerWg * (a.P + (a.P + 2) / 2) * sizeof(double);
  hipLaunchKernelGGL(sdb::survival_sample_kernel, dim3((unsigned)grid), dim3(64 * sdb::kSurvWavesPerWg), lds,
                     (hipStream_t)stream, a);
  return check_launch("sd_survival_sample");
}

}  // extern "C"
