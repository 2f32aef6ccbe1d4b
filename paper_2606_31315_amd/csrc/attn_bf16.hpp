// attn_bf16.hpp -- bf16 block attention kernel built around gfx950's asynchronous
// global-to-LDS loads.
//
// Same operation and work decomposition as block_attn_kernel (one workgroup per
// (sequence, kv head, KV split); all G*B_s query rows of the kv-head group packed into
// 16-row MFMA tiles), with the memory pipeline rebuilt for bandwidth:
//   * 8 wavefronts; wavefront w owns m-tiles w, w+8 (so up to 128 query rows per
//     m-tile slot).
//   * K and V tiles (64 keys each) are fetched with global_load_lds_dwordx4 straight
//     into an LDS ring of NS stages (3 by default, 96 KB at D = 128): NS-1 tiles stay in
//     flight while one is consumed, and no VGPRs hold data in transit.  One barrier per
//     tile.
//   * Rows in LDS are XOR-swizzled at 16-byte granularity (the swizzle is applied to
//     the global address each lane fetches, since a load-to-LDS instruction writes 1 KB
//     contiguously): K rows by (row mod 16) so the 16 rows an MFMA A-operand read
//     touches fall in distinct banks; V rows by 2*(row mod 8) for the transposed reads.
//   * The P.V contraction needs V^T operands (8 keys of one head dim per lane); they
//     come straight from the row-major V tile with ds_read_b64_tr_b16, which transposes
//     4x4 blocks of 16-bit elements across each 16-lane group.
//   * Tiles every row can see entirely skip the per-element mask; the O rescale is
//     skipped when no row's running maximum moved.
//   * K/V loads carry the non-temporal cache policy: each key row is read once per call
//     (ragged Qwen3-4B batch, 7 interleaved rounds: 36.6 -> 34.5 us per call).
#pragma once

#include <type_traits>

#include "attn.hpp"

namespace sdb {

#define SDB_LDS __attribute__((address_space(3)))

typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef float f32x2v __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  const f32x2v v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2v));
}

// ds_read_b64_tr_b16 issued as inline assembly: the intrinsic form makes the compiler
// assume it may alias the in-flight load-to-LDS writes and wait for all of them (the
// explicit vmcnt wait and barrier at the top of each tile already order these reads).
// The result is only valid after wait_lds_tr() below, which takes it as an operand.
template <int OFF>
__device__ __forceinline__ s16x4 ds_read_tr16(unsigned lds_addr) {
  s16x4 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(lds_addr), "n"(OFF) : "memory");
  return r;
}

// One K operand (16 bytes of a key row) by an explicit LDS read; valid after wait_k_step().
template <int OFF>
__device__ __forceinline__ bf16x8 ds_read_k(unsigned lds_addr) {
  bf16x8 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(lds_addr), "n"(OFF) : "memory");
  return r;
}

// Wait until at most N LDS reads are outstanding.  LDS reads complete in order, so with every
// K read of a tile issued step by step, the reads of step st are done once N = (steps after st)
// x (reads per step); the step's registers pass through the asm so no use of them is scheduled
// before it.
template <int N, int NSBW>
__device__ __forceinline__ void wait_k_step(bf16x8 (&v)[NSBW]) {
  static_assert(N <= 15, "lgkmcnt counts at most 15 outstanding reads");
  if constexpr (NSBW == 4)
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]) : "n"(N) : "memory");
  else if constexpr (NSBW == 2)
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(v[0]), "+v"(v[1]) : "n"(N) : "memory");
  else
    static_assert(NSBW == 4 || NSBW == 2, "whole or half tiles");
}

// Wait for outstanding LDS reads; the registers pass through the asm so no use of them
// can be scheduled before the wait.
template <int NDT>
__device__ __forceinline__ void wait_lds_tr(s16x4 (&v)[NDT][2]) {
  if constexpr (NDT == 8) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0][0]), "+v"(v[0][1]), "+v"(v[1][0]), "+v"(v[1][1]), "+v"(v[2][0]), "+v"(v[2][1]),
                   "+v"(v[3][0]), "+v"(v[3][1]), "+v"(v[4][0]), "+v"(v[4][1]), "+v"(v[5][0]), "+v"(v[5][1]),
                   "+v"(v[6][0]), "+v"(v[6][1]), "+v"(v[7][0]), "+v"(v[7][1])::"memory");
  } else {
    static_assert(NDT == 4, "head_dim 64 or 128");
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0][0]), "+v"(v[0][1]), "+v"(v[1][0]), "+v"(v[1][1]), "+v"(v[2][0]), "+v"(v[2][1]),
                   "+v"(v[3][0]), "+v"(v[3][1])::"memory");
  }
}

// 16-byte vector of new block rows (K or V) that a thread carries into the cache in an APPEND
// launch.  A vector type, not the u32x4 struct: a struct array held across the tile loop is
// copied through private memory.
typedef unsigned AppendVec __attribute__((ext_vector_type(4)));

template <int D, int KT_, int NS_>
struct Bf16Tile {
  static constexpr int KT = KT_;                // keys per tile
  static constexpr int ROWB = D * 2;            // bytes per key row
  static constexpr int CPR = ROWB / 16;         // 16-byte chunks per row
  static constexpr int TILEB = KT * ROWB;       // bytes of one K (or V) tile
  static constexpr int RPI = 1024 / ROWB;       // rows written by one 1 KB load instruction
  static constexpr int LPI = TILEB / 1024;      // load instructions per K (or V) tile
  static constexpr int NW = 8;                  // wavefronts per workgroup
  static constexpr int LPW = 2 * LPI / NW;      // load instructions per wavefront per tile
  static constexpr int NS = NS_;                // ring stages
  static constexpr int STAGEB = 2 * TILEB;      // K tile then V tile
  static_assert((2 * LPI) % NW == 0 && LPI % LPW == 0, "K and V loads split evenly over wavefronts");
  __device__ static int swz_k(int r) { return r % CPR; }
  __device__ static int swz_v(int r) { return (2 * r) % CPR; }
};

// Per-lane source offsets of this wavefront's share of one tile's loads (row*ROWB +
// swizzled chunk*16, relative to the tile's first key row).  Wavefronts 0-3 fetch K,
// 4-7 fetch V.
template <int D, int KT, int NS>
struct TileLoads {
  using T = Bf16Tile<D, KT, NS>;
  int row[T::LPW];
  unsigned src[T::LPW];
  unsigned cof[T::LPW];  // swizzled chunk offset within the row
  bool isv;
  __device__ void init(int wave, int lane) {
    isv = wave * T::LPW >= T::LPI;  // uniform per wavefront
#pragma unroll
    for (int q = 0; q < T::LPW; ++q) {
      const int li = wave * T::LPW + q - (isv ? T::LPI : 0);
      row[q] = li * T::RPI + lane / T::CPR;
      const int chunk = (lane % T::CPR) ^ (isv ? T::swz_v(row[q]) : T::swz_k(row[q]));
      src[q] = row[q] * T::ROWB + chunk * 16;
      cof[q] = chunk * 16;
    }
  }
  // The same tile from a page pool: key k of sequence s lives in pool page
  // table[k >> log2] at row k & (page_size - 1).  A wavefront's loads of one tile cover
  // 2 * KT / NW = 16 consecutive keys starting at a multiple of 16 (rows past key_last re-read
  // key_last, which lies in the same 16 keys), and pages hold a power of two >= 16 keys, so
  // they all read one page: one id per wavefront and tile, read with one scalar load (the
  // index is made wavefront-uniform with readfirstlane; a vector load would need a vmcnt wait
  // that drains the tile loads in flight).  The kernel reads the id one tile ahead, at the end
  // of a tile's arithmetic: scalar loads and LDS reads share one wait counter (lgkmcnt), so an
  // id load issued before the arithmetic would stall its first LDS read for a memory round
  // trip.  (An LDS lookup would make the compiler drain every in-flight load-to-LDS transfer
  // before it.)  Ids are clamped into the pool.
  static_assert(2 * KT / T::NW == 16 && T::LPW * T::RPI == 16, "16 keys per wavefront per tile");
  __device__ int fetch_page_raw(const int *table, int max_pages, int log2, int key0, int key_last, int wave) const {
    const int wrow = (wave % (T::NW / 2)) * 16;  // first key row of this wavefront's loads
    const int key = __builtin_amdgcn_readfirstlane(min(key0 + wrow, key_last));
    return ld_uniform(table, min(key >> log2, max_pages - 1));
  }
  __device__ static int clamp_page(int id, int num_pages) { return min(max(id, 0), num_pages - 1); }
  __device__ int fetch_page(const int *table, int max_pages, int num_pages, int log2, int key0, int key_last,
                            int wave) const {
    return clamp_page(fetch_page_raw(table, max_pages, log2, key0, key_last, wave), num_pages);
  }
  __device__ void issue_paged(char SDB_LDS *stage, const char *kpool, const char *vpool, int key0, int key_last,
                              int pg, int log2, int Hkv, int g, int wave) const {
    const char *pool = isv ? vpool : kpool;
    char SDB_LDS *dst = stage + (isv ? T::TILEB : 0) + (wave * T::LPW - (isv ? T::LPI : 0)) * 1024;
    const int mask = (1 << log2) - 1;
    const char *page = pool + ((((size_t)pg * Hkv + g) << log2) * T::ROWB);
#pragma unroll
    for (int q = 0; q < T::LPW; ++q) {
      const int key = min(key0 + row[q], key_last);
      __builtin_amdgcn_global_load_lds((const void *)(page + (unsigned)((key & mask) * T::ROWB) + cof[q]),
                                       (SDB_LDS void *)(dst + q * 1024), 16, 0, kLoadNT);
    }
  }
  // The tile starting at key0 when the block's own keys are not in the cache yet: key
  // k >= ctx is block row k - ctx, read from the new rows (nbase: the kv head's row of block
  // position 0; rows nstride bytes apart).  Rows past key_last re-read key_last.
  __device__ void issue_append(char SDB_LDS *stage, const char *kbase, const char *vbase, const char *knew,
                               const char *vnew, size_t nstride, int key0, int key_last, int ctx, int wave) const {
    const char *base = isv ? vbase : kbase;
    const char *nbase = isv ? vnew : knew;
    char SDB_LDS *dst = stage + (isv ? T::TILEB : 0) + (wave * T::LPW - (isv ? T::LPI : 0)) * 1024;
#pragma unroll
    for (int q = 0; q < T::LPW; ++q) {
      const int key = min(key0 + row[q], key_last);
      const char *src = key < ctx ? base + (size_t)key * T::ROWB + cof[q] : nbase + (size_t)(key - ctx) * nstride + cof[q];
      __builtin_amdgcn_global_load_lds((const void *)src, (SDB_LDS void *)(dst + q * 1024), 16, 0, kLoadNT);
    }
  }
  // Issue the loads of the tile starting at key0 into `stage`; rows past key_last
  // re-read key_last (only the split's last tile can need that).
  __device__ void issue(char SDB_LDS *stage, const char *kbase, const char *vbase, int key0, int key_last,
                        int wave) const {
    const char *base = (isv ? vbase : kbase) + (size_t)key0 * T::ROWB;
    char SDB_LDS *dst = stage + (isv ? T::TILEB : 0) + (wave * T::LPW - (isv ? T::LPI : 0)) * 1024;
    if (key0 + T::KT - 1 <= key_last) {
#pragma unroll
      for (int q = 0; q < T::LPW; ++q)
        __builtin_amdgcn_global_load_lds((const void *)(base + src[q]), (SDB_LDS void *)(dst + q * 1024), 16, 0, kLoadNT);
    } else {
#pragma unroll
      for (int q = 0; q < T::LPW; ++q) {
        const int shift = min(row[q], key_last - key0) - row[q];  // <= 0: back to the last valid key
        __builtin_amdgcn_global_load_lds((const void *)(base + src[q] + shift * T::ROWB), (SDB_LDS void *)(dst + q * 1024),
                                         16, 0, kLoadNT);
      }
    }
  }
};

// One 32-key step (keys KK*32 .. KK*32+31 of the tile) of O^T += V^T P^T.  P comes from
// the score registers (keys KK*32 + h*16 + kgrp*4 + r, h = 0,1); the matching V^T operand
// from two transposed LDS reads per head-dim tile.
template <int KK, int NDT, int NSB>
__device__ __forceinline__ void pv_step(const f32x4 (&p)[NSB], unsigned stage, const unsigned (&voff)[NDT],
                                        f32x4 (&oacc)[NDT]) {
  constexpr int ROWB = NDT * 32;  // bytes per key row (D * 2)
  const u32x4 praw{cvt_pk_bf16(p[2 * KK][0], p[2 * KK][1]), cvt_pk_bf16(p[2 * KK][2], p[2 * KK][3]),
                   cvt_pk_bf16(p[2 * KK + 1][0], p[2 * KK + 1][1]), cvt_pk_bf16(p[2 * KK + 1][2], p[2 * KK + 1][3])};
  const bf16x8 pb = __builtin_bit_cast(bf16x8, praw);
  s16x4 vv[NDT][2];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
    vv[dt][0] = ds_read_tr16<(KK * 32 + 0) * ROWB>(stage + voff[dt]);
    vv[dt][1] = ds_read_tr16<(KK * 32 + 16) * ROWB>(stage + voff[dt]);
  }
  wait_lds_tr<NDT>(vv);
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 v8 = {vv[dt][0][0], vv[dt][0][1], vv[dt][0][2], vv[dt][0][3],
                      vv[dt][1][0], vv[dt][1][1], vv[dt][1][2], vv[dt][1][3]};
    oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, v8), pb, oacc[dt], 0, 0, 0);
  }
}

// pv_step in two parts, so that the V^T operands can be read while the softmax runs: pv_issue
// starts the transposed LDS reads of the 32-key step KK; pv_mma waits for them (and every earlier
// LDS read) and multiplies.
template <int KK, int NDT>
__device__ __forceinline__ void pv_issue(unsigned stage, const unsigned (&voff)[NDT], s16x4 (&vv)[NDT][2]) {
  constexpr int ROWB = NDT * 32;  // bytes per key row (D * 2)
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
    vv[dt][0] = ds_read_tr16<(KK * 32 + 0) * ROWB>(stage + voff[dt]);
    vv[dt][1] = ds_read_tr16<(KK * 32 + 16) * ROWB>(stage + voff[dt]);
  }
}
template <int KK, int NDT, int NSB>
__device__ __forceinline__ void pv_mma(const f32x4 (&p)[NSB], s16x4 (&vv)[NDT][2], f32x4 (&oacc)[NDT]) {
  const u32x4 praw{cvt_pk_bf16(p[2 * KK][0], p[2 * KK][1]), cvt_pk_bf16(p[2 * KK][2], p[2 * KK][3]),
                   cvt_pk_bf16(p[2 * KK + 1][0], p[2 * KK + 1][1]), cvt_pk_bf16(p[2 * KK + 1][2], p[2 * KK + 1][3])};
  const bf16x8 pb = __builtin_bit_cast(bf16x8, praw);
  wait_lds_tr<NDT>(vv);
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 v8 = {vv[dt][0][0], vv[dt][0][1], vv[dt][0][2], vv[dt][0][3],
                      vv[dt][1][0], vv[dt][1][1], vv[dt][1][2], vv[dt][1][3]};
    oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, v8), pb, oacc[dt], 0, 0, 0);
  }
}

// The value of lane l combined with lane l ^ 16 (x16) or l ^ 32 (x32), by the gfx950 lane-swap
// instructions: v_permlane16_swap / v_permlane32_swap with both operands x return, in every lane,
// its own value and its partner's (one in each result), in VALU cycles instead of the LDS round
// trip of a ds_bpermute shuffle.
__device__ __forceinline__ float2 pair_x16(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return float2{__uint_as_float(p[0]), __uint_as_float(p[1])};
}
__device__ __forceinline__ float2 pair_x32(float x) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return float2{__uint_as_float(p[0]), __uint_as_float(p[1])};
}

// APPEND: the block's keys and values are read from a.k_new / a.v_new rather than the cache,
// and the split that covers them also writes them into the cache (sd_block_attn_append).
// BAL (the balanced plan): the workgroup streams its share of every pair's key tiles, one work
// item per pair its share touches (bal_item), the body below once per item; otherwise the body
// runs once, for the workgroup's one work item (attn_item).
// VE (one m-tile per wavefront, blocks of 7-8 m-tiles): each tile's V^T operands are read from
// LDS right after the QK^T products, so their latency runs under the softmax (8 sequences x 8
// kv heads, contexts 4096, 8 m-tiles: 42.1 -> 41.2 us per call; at 3-6 m-tiles no faster).
template <int D, int MT, int KT_, int NS_, bool PAGED, bool APPEND = false, bool BAL = false, bool VE = false>
__global__ __launch_bounds__(512) void block_attn_bf16_kernel(AttnArgs a) {
  using T = Bf16Tile<D, KT_, NS_>;
  constexpr int KT = T::KT, NS = T::NS, NDT = D / 16, NST = D / 32, NSB = KT / 16;
  static_assert(NS >= 2 && NS <= 5, "ring depth");
  static_assert(KT == 64 || KT == 128, "key tile of 64 or 128 keys");
  static_assert(!VE || MT == 1, "early V^T reads: registers for one m-tile per wavefront only");
  constexpr int EB = 2;
  __shared__ __attribute__((aligned(1024))) char ring_raw[NS * T::STAGEB];
  char SDB_LDS *ring = (char SDB_LDS *)(SDB_LDS void *)ring_raw;

  [[maybe_unused]] BalShare bsh;
  if constexpr (BAL) bsh = bal_share(a, blockIdx.x, KT);
  for (;;) {  // one pass per work item
    AttnItem it;
    if constexpr (BAL) {
      if (!bal_item(a, bsh, KT, it)) return;
    } else {
      if (!attn_item(a, blockIdx.x, it)) return;
    }
    const int s = it.s, g = it.g, k0 = it.k0, k1 = it.k1, nsplit = it.nsplit;
    const int ctx = it.ctx, B = it.B, qoff = it.qoff;
    const int M = a.G * B;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int l16 = lane & 15;
    const int kgrp = lane >> 4;
    const int nmt = (M + 15) >> 4;
    // Wavefront w runs on SIMD w % 4.  With 5 or 6 m-tiles, m-tiles 4 and 5 would put two whole
    // m-tiles of work on one SIMD while others idle, so wavefronts 4-7 instead take the two key
    // halves of m-tiles 4 and 5 (each keeps its own online-softmax state over its 32 keys of
    // every tile; the halves are merged once, after the last tile): at most 1.5 m-tiles of work
    // per SIMD instead of 2.
    const bool hsplit = MT == 1 && (nmt == 5 || nmt == 6);
    const int hlf = (hsplit && wave >= 4) ? ((wave - 4) & 1) : -1;  // key half, or -1: whole tiles
    auto mtile = [&](int j) { return (hlf >= 0) ? 4 + ((wave - 4) >> 1) : wave + T::NW * j; };

    const char *kbase = reinterpret_cast<const char *>(a.k);
    const char *vbase = reinterpret_cast<const char *>(a.v);
    if constexpr (!PAGED) {
      kbase += ((size_t)(s * a.Hkv + g) * a.Lmax) * D * EB;
      vbase += ((size_t)(s * a.Hkv + g) * a.Lmax) * D * EB;
    }

    // ---- query operands: element e of step st is dim st*32 + kgrp*8 + e of row m ----
    bf16x8 qop[MT][NST];
    f32x4 oacc[MT][NDT];
    float m_run[MT], l_run[MT];
    int row_i[MT];
    bool act[MT];
  #pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int mt = mtile(j);
      const int m = mt * 16 + l16;
      act[j] = mt < nmt;
      m_run[j] = -INFINITY;
      l_run[j] = 0.f;
  #pragma unroll
      for (int dt = 0; dt < NDT; ++dt) oacc[j][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
      const bool valid = act[j] && m < M;
      row_i[j] = valid ? m / a.G : 0;
      const char *qrow = reinterpret_cast<const char *>(a.q) +
                         ((size_t)(qoff + (valid ? m / a.G : 0)) * a.Hq + g * a.G + (valid ? m % a.G : 0)) * D * EB;
  #pragma unroll
      for (int st = 0; st < NST; ++st) {
        const u32x4 raw = valid ? *reinterpret_cast<const u32x4 *>(qrow + (st * 32 + kgrp * 8) * EB) : u32x4{0, 0, 0, 0};
        qop[j][st] = __builtin_bit_cast(bf16x8, raw);
      }
    }

    // ---- per-lane LDS offsets, fixed for the whole loop ----
    // K operand of sub-tile sb, step st: row sb*16 + l16, chunk (st*4 + kgrp) swizzled by the
    // row (the swizzle only depends on l16); sb*16 rows are an immediate offset.
    unsigned koff[NST];
  #pragma unroll
    for (int st = 0; st < NST; ++st) koff[st] = l16 * T::ROWB + (((st * 4 + kgrp) ^ T::swz_k(l16)) << 4);
    // V^T operand for head-dim tile dt: source row kgrp*4 + l16/4 (plus kk*32 + h*16 keys as
    // an immediate), head dims dt*16 + 4*(l16%4) .. +3 (swizzle depends only on the row mod 8).
    const int vrow = kgrp * 4 + (l16 >> 2);
    unsigned voff[NDT];
  #pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
      voff[dt] = T::TILEB + vrow * T::ROWB + (((2 * dt + ((l16 & 3) >> 1)) ^ T::swz_v(vrow)) << 4) + ((l16 & 1) << 3);

    TileLoads<D, KT, NS> ld;
    ld.init(wave, lane);
    // paged caches: this sequence's row of the block table
    [[maybe_unused]] const int *table = PAGED ? a.block_table + (size_t)s * a.max_pages : nullptr;
    [[maybe_unused]] int pgn = 0;  // paged caches: page id of this wavefront's share of the next tile
    // APPEND: the block rows of this kv head in the new-row arrays, and this split's share of
    // them ([ab0, k1) of the keys) copied into the cache through registers: loaded now, stored
    // after the last tile.  (Stores count in vmcnt: issued earlier, they would hold up the next
    // tile wait until they were acknowledged.)
    [[maybe_unused]] const size_t nstride = (size_t)a.Hkv * D * EB;
    [[maybe_unused]] const char *knew = nullptr, *vnew = nullptr;
    [[maybe_unused]] int ab0 = k1;
    constexpr int NAV = D / 32;  // 64 rows x 2 x D*2/16 vectors over 512 threads
    [[maybe_unused]] AppendVec cpv[NAV];
    if constexpr (APPEND) {
      knew = reinterpret_cast<const char *>(a.k_new) + ((size_t)qoff * a.Hkv + g) * D * EB;
      vnew = reinterpret_cast<const char *>(a.v_new) + ((size_t)qoff * a.Hkv + g) * D * EB;
      ab0 = max(k0, ctx);
      if (ab0 < k1) {  // uniform: this split covers block rows ab0 - ctx .. k1 - 1 - ctx
        constexpr int RV = D * EB / 16;  // 16-byte vectors per row
        const int half = (k1 - ab0) * RV;  // K vectors, then as many V vectors
  #pragma unroll
        for (int c = 0; c < NAV; ++c) {
          const int v = min(tid + 512 * c, 2 * half - 1);  // clamped: no per-load branch
          const int kv = v >= half, w = v - kv * half, r = w / RV, ch = w % RV;
          cpv[c] = *reinterpret_cast<const AppendVec *>((kv ? vnew : knew) + (size_t)(ab0 - ctx + r) * nstride + ch * 16);
        }
      }
    }
    auto issue = [&](char SDB_LDS *stage, int key0) {
      if constexpr (PAGED) {
        ld.issue_paged(stage, kbase, vbase, key0, k1 - 1, pgn, a.page_log2, a.Hkv, g, wave);
      } else if constexpr (APPEND) {
        if (key0 + KT > ctx) ld.issue_append(stage, kbase, vbase, knew, vnew, nstride, key0, k1 - 1, ctx, wave);
        else ld.issue(stage, kbase, vbase, key0, k1 - 1, wave);
      } else {
        ld.issue(stage, kbase, vbase, key0, k1 - 1, wave);
      }
    };

    // ---- pipeline prologue: tiles 0 .. NS-2 in flight ----
    const int ntiles = (k1 - k0 + KT - 1) / KT;
    if constexpr (PAGED) {
      // the page ids of the first NS tiles in one batch of scalar loads: one round trip rather
      // than one per tile (measured: 38.2 -> 35.6 us per call with shuffled 16-key pages,
      // together with one id per wavefront and tile)
      int pro[NS];
  #pragma unroll
      for (int t = 0; t < NS; ++t) pro[t] = ld.fetch_page_raw(table, a.max_pages, a.page_log2, k0 + t * KT, k1 - 1, wave);
      // one use of all the raw ids before any is clamped, so their loads go out together
      if constexpr (NS == 3) asm volatile("" : "+s"(pro[0]), "+s"(pro[1]), "+s"(pro[2]));
  #pragma unroll
      for (int t = 0; t < NS; ++t) pro[t] = TileLoads<D, KT, NS>::clamp_page(pro[t], a.num_pages);
  #pragma unroll
      for (int t = 0; t < NS - 1; ++t)
        if (t < ntiles) ld.issue_paged(ring + t * T::STAGEB, kbase, vbase, k0 + t * KT, k1 - 1, pro[t], a.page_log2, a.Hkv, g, wave);
      pgn = pro[NS - 1];
    } else {
  #pragma unroll
      for (int t = 0; t < NS - 1; ++t)
        if (t < ntiles) issue(ring + t * T::STAGEB, k0 + t * KT);
    }
    // keys every row can see: all of [k0, k1) when bidirectional, keys <= ctx when causal
    const int vis_all = a.causal ? min(k1, ctx + 1) : k1;
    const float sl2 = a.scale_log2;

    // One wavefront's work on one m-tile over NSBW 16-key sub-blocks of a tile, starting at key
    // kb (LDS rows from stg): scores, mask, online softmax, P.V.
    auto tile_work = [&](auto nsbw_c, int j, unsigned stg, int kb, bool full) {
      constexpr int NSBW = decltype(nsbw_c)::value;
      // S^T = K Q^T: sacc[sb][r] is key kb + sb*16 + kgrp*4 + r of row l16 (unscaled)
      f32x4 sacc[NSBW];
  #pragma unroll
      for (int sb = 0; sb < NSBW; ++sb) sacc[sb] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (MT == 1) {
        // Every K operand of the tile is read first, then each step's products follow a counted
        // wait for that step's reads only, so the LDS latency is exposed once per tile rather
        // than once per step (the compiler's own schedule waited for all reads in flight before
        // each group of products).  Ragged Qwen3-4B batch: 33.43 -> 33.21 us per call; not for
        // two m-tiles per wavefront, whose register budget would spill.
        bf16x8 kf[NST][NSBW];
  #pragma unroll
        for (int st = 0; st < NST; ++st) {
          const unsigned kp = stg + koff[st];
          kf[st][0] = ds_read_k<0 * 16 * T::ROWB>(kp);
          kf[st][1] = ds_read_k<1 * 16 * T::ROWB>(kp);
          if constexpr (NSBW == 4) {
            kf[st][NSBW == 4 ? 2 : 0] = ds_read_k<2 * 16 * T::ROWB>(kp);
            kf[st][NSBW == 4 ? 3 : 0] = ds_read_k<3 * 16 * T::ROWB>(kp);
          }
        }
        auto kstep = [&](auto st_c) {
          constexpr int st = decltype(st_c)::value;
          wait_k_step<(NST - 1 - st) * NSBW, NSBW>(kf[st]);
  #pragma unroll
          for (int sb = 0; sb < NSBW; ++sb)
            sacc[sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[st][sb], qop[j][st], sacc[sb], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);  // the next step's wait stays after these products
        };
        static_assert(NST == 2 || NST == 4, "head_dim 64 or 128");
        kstep(std::integral_constant<int, 0>{});
        kstep(std::integral_constant<int, 1>{});
        if constexpr (NST == 4) {
          kstep(std::integral_constant<int, (NST == 4 ? 2 : 0)>{});
          kstep(std::integral_constant<int, (NST == 4 ? 3 : 0)>{});
        }
      } else {
  #pragma unroll
        for (int st = 0; st < NST; ++st) {
          const char SDB_LDS *kp = (const char SDB_LDS *)(uintptr_t)(stg + koff[st]);
  #pragma unroll
          for (int sb = 0; sb < NSBW; ++sb) {
            const bf16x8 av = *(const bf16x8 SDB_LDS *)(kp + sb * 16 * T::ROWB);
            sacc[sb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, qop[j][st], sacc[sb], 0, 0, 0);
          }
        }
      }
      // VE: the V^T operands of this tile's 32-key steps, read now (after the K reads the products
      // above consumed), so that their LDS latency runs under the softmax below
      constexpr bool vearly = VE && NSBW <= 4;
      [[maybe_unused]] s16x4 vq[vearly ? NSBW / 2 : 1][NDT][2];
      if constexpr (vearly) {
        pv_issue<0, NDT>(stg, voff, vq[0]);
        if constexpr (NSBW > 2) pv_issue<1, NDT>(stg, voff, vq[NSBW > 2 ? 1 : 0]);
      }
      // online softmax in the log2 domain: max of the raw scores, then one FMA per score
      if (!full) {
        const int lim = a.causal ? min(k1, ctx + row_i[j] + 1) : k1;
  #pragma unroll
        for (int sb = 0; sb < NSBW; ++sb)
  #pragma unroll
          for (int r = 0; r < 4; ++r)
            if (kb + sb * 16 + kgrp * 4 + r >= lim) sacc[sb][r] = -INFINITY;
      }
      float tmax = -INFINITY;
  #pragma unroll
      for (int sb = 0; sb < NSBW; ++sb)
        tmax = fmaxf(tmax, fmaxf(fmaxf(sacc[sb][0], sacc[sb][1]), fmaxf(sacc[sb][2], sacc[sb][3])));
      {  // the row's maximum over the four key groups (lanes l, l ^ 16, l ^ 32, l ^ 48)
        const float2 p16 = pair_x16(tmax);
        const float2 p32 = pair_x32(fmaxf(p16.x, p16.y));
        tmax = fmaxf(p32.x, p32.y);
      }
      const float mnew = fmaxf(m_run[j], tmax * sl2);
      const float muse = (mnew == -INFINITY) ? 0.f : mnew;
      float psum = 0.f;
  #pragma unroll
      for (int sb = 0; sb < NSBW; ++sb)
  #pragma unroll
        for (int r = 0; r < 4; ++r) {
          sacc[sb][r] = fast_exp2(fmaf(sacc[sb][r], sl2, -muse));
          psum += sacc[sb][r];
        }
      if (__any(mnew != m_run[j])) {
        const float alpha = fast_exp2(m_run[j] - muse);
        l_run[j] *= alpha;
  #pragma unroll
        for (int dt = 0; dt < NDT; ++dt) oacc[j][dt] *= alpha;
      }
      m_run[j] = mnew;
      l_run[j] += psum;

      // O^T += V^T P^T over these keys in 32-key steps
      if constexpr (vearly) {
        pv_mma<0, NDT, NSBW>(sacc, vq[0], oacc[j]);
        if constexpr (NSBW > 2) pv_mma<1, NDT, NSBW>(sacc, vq[NSBW > 2 ? 1 : 0], oacc[j]);
      } else {
        pv_step<0, NDT, NSBW>(sacc, stg, voff, oacc[j]);
        if constexpr (NSBW > 2) pv_step<1, NDT, NSBW>(sacc, stg, voff, oacc[j]);
        if constexpr (NSBW > 4) {
          pv_step<2, NDT, NSBW>(sacc, stg, voff, oacc[j]);
          pv_step<3, NDT, NSBW>(sacc, stg, voff, oacc[j]);
        }
      }
    };

    for (int t = 0; t < ntiles; ++t) {
      const int kt = k0 + t * KT;
      const int ahead = min(ntiles - 1 - t, NS - 2);  // tiles issued after tile t
      if (NS > 4 && ahead >= 3) wait_vmcnt<3 * T::LPW>();
      else if (NS > 3 && ahead >= 2) wait_vmcnt<2 * T::LPW>();
      else if (NS > 2 && ahead >= 1) wait_vmcnt<T::LPW>();
      else wait_vmcnt<0>();
      __syncthreads();  // tile t landed for every wavefront; stage (t-1) % NS is free again
      if (t + NS - 1 < ntiles) issue(ring + ((t + NS - 1) % NS) * T::STAGEB, kt + (NS - 1) * KT);
      const unsigned stage = (unsigned)(uintptr_t)(ring + (t % NS) * T::STAGEB);
      const bool full = kt + KT <= vis_all;  // uniform: no key of this tile is masked for any row
  #pragma unroll
      for (int j = 0; j < MT; ++j) {
        if (!act[j]) continue;  // uniform per wavefront
        if (hlf < 0) tile_work(std::integral_constant<int, NSB>{}, j, stage, kt, full);
        else tile_work(std::integral_constant<int, NSB / 2>{}, j, stage + (unsigned)(hlf * (KT / 2) * T::ROWB),
                       kt + hlf * (KT / 2), full);
      }
      if constexpr (PAGED) {
        if (t + NS < ntiles) pgn = ld.fetch_page(table, a.max_pages, a.num_pages, a.page_log2, k0 + (t + NS) * KT, k1 - 1, wave);
      }
    }

    if constexpr (APPEND) {
      if (ab0 < k1) {  // the block rows this split covers, into the cache
        constexpr int RV = D * EB / 16;
        const int half = (k1 - ab0) * RV;
        char *kc = reinterpret_cast<char *>(const_cast<void *>(a.k)) + ((size_t)(s * a.Hkv + g) * a.Lmax) * D * EB;
        char *vc = reinterpret_cast<char *>(const_cast<void *>(a.v)) + ((size_t)(s * a.Hkv + g) * a.Lmax) * D * EB;
  #pragma unroll
        for (int c = 0; c < NAV; ++c) {
          const int v = tid + 512 * c;
          if (v < 2 * half) {
            const int kv = v >= half, w = v - kv * half, r = w / RV, ch = w % RV;
            *reinterpret_cast<AppendVec *>((kv ? vc : kc) + (size_t)(ab0 + r) * T::ROWB + ch * 16) = cpv[c];
          }
        }
      }
    }

    // ---- key halves of m-tiles 4 and 5: the second half's state joins the first's ----
    if (hsplit) {  // uniform
      constexpr int XS = NDT * 4 + 2;  // floats per lane: O, then m and l
      float SDB_LDS *xch = (float SDB_LDS *)(SDB_LDS void *)ring_raw;  // the ring is no longer read
      __syncthreads();
      if (hlf == 1 && act[0]) {
        float SDB_LDS *dst = xch + ((wave - 4) >> 1) * 64 * XS + lane;
  #pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
  #pragma unroll
          for (int r = 0; r < 4; ++r) dst[(dt * 4 + r) * 64] = oacc[0][dt][r];
        dst[(NDT * 4) * 64] = m_run[0];
        dst[(NDT * 4 + 1) * 64] = l_run[0];
      }
      __syncthreads();
      if (hlf == 0 && act[0]) {
        const float SDB_LDS *src = xch + ((wave - 4) >> 1) * 64 * XS + lane;
        const float mb = src[(NDT * 4) * 64], lb = src[(NDT * 4 + 1) * 64];
        const float mn = fmaxf(m_run[0], mb);
        const float mu = (mn == -INFINITY) ? 0.f : mn;
        const float sa = (m_run[0] == -INFINITY) ? 0.f : fast_exp2(m_run[0] - mu);
        const float sb = (mb == -INFINITY) ? 0.f : fast_exp2(mb - mu);
  #pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
  #pragma unroll
          for (int r = 0; r < 4; ++r) oacc[0][dt][r] = fmaf(oacc[0][dt][r], sa, src[(dt * 4 + r) * 64] * sb);
        l_run[0] = fmaf(l_run[0], sa, lb * sb);  // explicit: rounding independent of contraction choices
        m_run[0] = mn;
      }
      if (hlf == 1) act[0] = false;  // merged into the first half's wavefront
    }

    // ---- epilogue: row sums over the four key groups, then output or partials ----
  #pragma unroll
    for (int j = 0; j < MT; ++j) {
      const float2 p16 = pair_x16(l_run[j]);
      const float2 p32 = pair_x32(p16.x + p16.y);
      l_run[j] = p32.x + p32.y;
    }
    if (nsplit == 1) {
  #pragma unroll
      for (int j = 0; j < MT; ++j) {
        const int m = mtile(j) * 16 + l16;
        if (!act[j] || m >= M) continue;
        const float inv = 1.f / l_run[j];
        char *orow = reinterpret_cast<char *>(a.out) + ((size_t)(qoff + m / a.G) * a.Hq + g * a.G + m % a.G) * D * EB;
  #pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const f32x4 o = oacc[j][dt] * inv;
          *reinterpret_cast<uint2 *>(orow + (dt * 16 + kgrp * 4) * EB) = uint2{cvt_pk_bf16(o[0], o[1]), cvt_pk_bf16(o[2], o[3])};
        }
      }
      if constexpr (!BAL) return;
      __syncthreads();  // every wavefront is done with the ring before the next item's loads
      continue;
    }
    const size_t wrow = (size_t)it.slot * a.Mpad;
  #pragma unroll
    for (int j = 0; j < MT; ++j) {
      const int m = mtile(j) * 16 + l16;
      if (!act[j] || m >= M) continue;
      float *prow = a.part_o + (wrow + m) * D;
      // non-temporal: the partials are read once, by the merge kernel, so they go to memory now
      // instead of waiting dirty in L2 for the write-back at the kernel's end (ragged Qwen3-4B
      // batch, 7 interleaved rounds: 35.0 -> 34.0 us per call)
  #pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
        __builtin_nontemporal_store(oacc[j][dt], reinterpret_cast<f32x4 *>(prow + dt * 16 + kgrp * 4));
      if (kgrp == 0) {
        typedef float f2v __attribute__((ext_vector_type(2)));
        __builtin_nontemporal_store(f2v{m_run[j], l_run[j]}, reinterpret_cast<f2v *>(a.part_ml + wrow + m));
      }
    }
    if constexpr (!BAL) return;
    __syncthreads();  // every wavefront is done with the ring before the next item's loads
  }
}

}  // namespace sdb
