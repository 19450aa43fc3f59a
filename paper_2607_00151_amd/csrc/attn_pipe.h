// Software-pipelined form of the paged prefill attention (same work items,
// same LDS tiles and operand layouts as attn_kernel<P, 1, 4>).
//
// A CDNA4 SIMD overlaps matrix-core and VALU work only when both come from
// the same wave: an MFMA-only wave next to a VALU-only wave on one SIMD runs
// no faster than the two back to back, while a few VALU ops placed after each
// 32x32x16 MFMA of one wave cost little beyond the MFMA time (measured on
// MI355X).  So each wave splits key tile t into two interleaved phases,
//   phase 1:  S(t+1)^T = K(t+1) Q^T   16 MFMAs
//             P(t) = exp2(x(t)), keys 0-31     VALU (16 exp, 8 cvt, 16 add per
//                                               lane; the adds form l)
//   phase 2:  O^T += V(t)^T P(t)^T    16 MFMAs
//             P(t), keys 32-63        during the first 8 (the PV MFMAs of
//                                       keys 0-31), the same VALU work
//             row max of x(t+1)       during the last 8 (16 max3), then the
//                                       lazy rescale test
// with K one tile ahead of V.  The VALU work of each phase depends only on
// results of the previous phase or of earlier MFMAs, so it issues between the
// MFMAs; splitting the exponentials between the phases measured ~1% faster
// than making all of P(t) in phase 1.  Steps whose next tile needs the causal
// mask, and the last step, run the same sequence without the interleaving.
//
// Two ways to apply the softmax scale.  The default (kExact) keeps q as
// given, starts the S accumulations from zero and computes each exponent as
// fma(s, c, -m) in fp32 (c = softmax scale times log2 e, m the row's offset),
// with the offset moved whenever a row's max grows.  The fast mode folds the
// scale into the MFMA instead: the query rows are scaled by c once, when they
// are loaded, and every S accumulation starts from -m, which takes the 32 fma
// per lane and tile off the VALU; its offset moves only when the max grows by
// 2^kRescaleLog2.  Its price is one more bf16 rounding, of c q (each x moves
// by at most 2^-8 sum_d |c q_d k_d|, so the log-sum-exp by at most ln 2 times
// that), plus the rounding of a row's largest probability.
#pragma once

#include "attn_kernel.h"

namespace sa {


template <int N>
struct IntC {
  static constexpr int value = N;
};

// The phase-2 exponentials of the interleaved step go to PV slots
// ((e - 8 kG1) w2) / (32 - 8 kG1) - 1 and each pair is packed one slot after
// its second element; the PV MFMAs of 16-key group g are slots 4g .. 4g + 3.
// True if every group of phase 2 is packed before slot 4g - 1.
constexpr bool phase2_in_time(int kg1, int w2) {
  for (int g = kg1; g < 4; ++g) {
    const int e = 8 * g + 7;                                 // last element of the group
    const int pack = ((e - 8 * kg1) * w2) / (32 - 8 * kg1);
    if (pack >= 4 * g - 1) return false;
  }
  return true;
}

constexpr int kPipeWaves = 4;                              // waves per group, 32 rows each
constexpr int kPipeRows = 32 * kPipeWaves;                 // query rows per work item
constexpr int kTileBytes = kKT * kHD * 2;                  // one K or V tile, 16 KB

// LDS of one group: its double-buffered K and V tiles.  A second group also
// names the first group's partial-result area (four 16 KB arrays and a 2 KB
// array of row statistics), which the other group fills at the end.
struct PipeLds {
  lds_u8 *k0, *k1, *v0, *v1;
  lds_u8 *x0, *x1, *x2, *x3;
  __attribute__((address_space(3))) float* ml;
};

// Page slots of an item are checked once: true if every page its keys need is
// present and in range.  The first round of reads (four per thread, enough
// for an item of up to 4 x nthreads pages) is issued early and evaluated
// later, so its latency overlaps the first tile loads; every thread of the
// block takes part in the evaluation (one barrier).
struct TableCheck {
  int32_t v[4];
  int pg, pg_end;
  bool bad;
};

template <int P>
__device__ __forceinline__ TableCheck table_check_issue(const AttnArgs& a, const AttnItem& it, int32_t pt_base,
                                                        int32_t pt_count, int nthreads) {
  constexpr int kPagesPerTile = kKT / P;
  const int t0 = it.kv_begin / kKT;
  const int t1 = (it.kv_end + kKT - 1) / kKT;
  TableCheck c;
  c.bad = pt_count < (it.kv_end + P - 1) / P;
  c.pg = t0 * kPagesPerTile + (int)threadIdx.x;
  c.pg_end = min(t1 * kPagesPerTile, pt_count);
#pragma unroll
  for (int u = 0; u < 4; ++u) c.v[u] = c.pg + u * nthreads < c.pg_end ? a.indices[pt_base + c.pg + u * nthreads] : 0;
  return c;
}

__device__ __forceinline__ bool table_check_finish(const AttnArgs& a, TableCheck& c, int32_t pt_base, int nthreads) {
  bool bad = c.bad;
#pragma unroll
  for (int u = 0; u < 4; ++u) bad |= !(c.v[u] >= 0 && c.v[u] < a.num_slots);
  for (int pg = c.pg + 4 * nthreads; pg < c.pg_end; pg += nthreads) {
    const int32_t s = a.indices[pt_base + pg];
    bad |= !(s >= 0 && s < a.num_slots);
  }
  return !__syncthreads_or(bad);
}

// ---- the segment's rows, written by the launch that attends over them
//
// With kRead every block takes the segment's keys (positions kv_len - q_len
// on) from the token-major k_new / v_new and never from their pages, so no
// block depends on another block's writes.  The first key-range part of each
// row tile (kv_begin == 0) stores to the pages the rows of the tokens whose
// first query row lies in its tile: the row tiles partition the rows, so every
// token's row is written exactly once.  A row whose page is missing or lies
// outside the pool is not written and raises error flag 2, as the append
// kernel does.  Four chunks per thread are loaded before any is stored, so the
// block waits for one round trip per 1024 chunks (64 tokens).
template <int P>
__device__ __forceinline__ void write_own_rows(const AttnArgs& a, const AttnItem& it) {
  const int G = a.G;
  const int tb = (it.row0 + G - 1) / G;
  const int te = min((it.row0 + kPipeRows + G - 1) / G, it.q_len);
  const int n = (te - tb) * 16;                             // 16-byte chunks of K (and of V)
  const int pre = it.kv_len - it.q_len;
  const int32_t pt_base = ld_uniform(a.indptr + it.seq);
  const int32_t pt_count = ld_uniform(a.indptr + it.seq + 1) - pt_base;
  uint16_t* const kp = const_cast<uint16_t*>(a.k);
  uint16_t* const vp = const_cast<uint16_t*>(a.v);
  constexpr int kDepth = 4;
  for (int c0 = (int)threadIdx.x; c0 < n; c0 += kDepth * (int)blockDim.x) {
    int64_t dst[kDepth];
    u32x4 kx[kDepth], vx[kDepth];
#pragma unroll
    for (int u = 0; u < kDepth; ++u) {
      const int c = c0 + u * (int)blockDim.x;
      dst[u] = -1;
      if (c >= n) continue;
      const int tok = tb + (c >> 4), ch = c & 15;
      const int x = pre + tok;
      const int page = x / P, row = x - page * P;
      const int32_t slot = page < pt_count ? a.indices[pt_base + page] : -1;
      if (slot < 0 || slot >= a.num_slots) {
        atomicOr(a.err, 2);
        continue;
      }
      const int64_t src = ((int64_t)(it.q_start + tok) * a.Hkv + it.kvh) * kHD + ch * 8;
      kx[u] = ld_u32x4(a.k_new + src);
      vx[u] = ld_u32x4(a.v_new + src);
      dst[u] = (((int64_t)slot * a.Hkv + it.kvh) * P + row) * kHD + ch * 8;
    }
#pragma unroll
    for (int u = 0; u < kDepth; ++u)
      if (dst[u] >= 0) {
        st_u32x4(kp + dst[u], kx[u]);
        st_u32x4(vp + dst[u], vx[u]);
      }
  }
}

// One group of four waves runs the item's rows over the keys
// [g_lo, g_hi): the whole item when kGroups == 1; with two groups, group 0
// takes the first half of the item's key tiles and group 1 the rest, and the
// two meet at the end to merge their partial results.  With two groups every
// step holds two barriers (one before each phase) and group 1 runs one
// barrier behind group 0, so on each SIMD one group's phase 1 overlaps the
// other's phase 2.
//
// kPoolRsrc: a layer's K (and V) pool spans < 2^31 bytes, so one buffer
// resource per pool reaches every page through the 32-bit scalar offset;
// otherwise each page load builds a resource for its page.
//
// kRead: keys from kv_len - q_len on (the segment's) are loaded from k_new /
// v_new instead of from their pages (write_own_rows).  Within a tile the
// source is chosen per group of four keys; a group holding keys of both kinds
// (prefix lengths that are not a multiple of 4) takes the checked load, so the
// steps that load its tile are plain steps.
template <int P, bool kPoolRsrc, int kGroups, int GRP, bool kRead = false, bool kExact = false>
__device__ __attribute__((always_inline)) inline void pipe_group(const AttnArgs& a, const AttnItem& it,
                                                                 const SeqDesc& sd, const PipeLds& L) {
  static_assert(P == 16 || P == 32, "page size");
  static_assert(!kRead || (kPoolRsrc && kGroups == 1), "segment reads: one group, pool-wide resources");
  constexpr int WAVES = kPipeWaves;
  constexpr int kRows = kPipeRows;
  constexpr int kPagesPerTile = kKT / P;
  constexpr int kNJ = 16 / WAVES;                          // loads per wave per tile and operand
  constexpr int kAhead = 2;                                // operand reads issued this many steps ahead
  constexpr int kG1 = 2;                                   // 16-key groups of P(t) made in phase 1

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (WAVES - 1);
  const int hh = lane >> 5;
  const int G = a.G;
  const int rows_total = sd.q_len * G;
  const int pre = sd.kv_len - sd.q_len;

  const int r_row = it.row0 + wave * 32 + (lane & 31);
  const bool row_valid = r_row < rows_total;
  const int rr = row_valid ? r_row : rows_total - 1;
  const int tok = rr / G;
  const int head = it.kvh * G + (rr - tok * G);
  const int qpos = pre + tok;

  // this group's keys [g_lo, g_hi) and tiles [t0, t1)
  const int ti0 = it.kv_begin / kKT;
  const int ti1 = (it.kv_end + kKT - 1) / kKT;
  const int tmid = ti0 + (ti1 - ti0 + 1) / 2;
  const int g_lo = (kGroups == 2 && GRP == 1) ? tmid * kKT : it.kv_begin;
  const int g_hi = (kGroups == 2 && GRP == 0) ? min(it.kv_end, tmid * kKT) : it.kv_end;
  const int t0 = g_lo / kKT;
  const int t1 = g_lo < g_hi ? (g_hi + kKT - 1) / kKT : t0;

  const int wrow0 = it.row0 + wave * 32;
  const bool wave_active = wrow0 < rows_total;
  const int w_full = min(g_hi, pre + wrow0 / G + 1);         // keys below are visible to all rows

  // the query row; it is scaled by c (below) only once the first tiles and
  // the page-table check are under way, so its load latency overlaps theirs
  bf16x8 qop[8];             // c q, rounded to bf16
  {
    const uint16_t* qrow = a.q + ((int64_t)(sd.q_start + tok) * a.Hq + head) * kHD;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qop[ks] = ld_bf16x8(qrow + (2 * ks + hh) * 8);
  }

  const int32_t pt_base = ld_uniform(a.indptr + it.seq);
  const int32_t pt_count = ld_uniform(a.indptr + it.seq + 1) - pt_base;
  TableCheck tcheck = table_check_issue<P>(a, it, pt_base, pt_count, 64 * WAVES * kGroups);
  const int64_t slot_bytes = (int64_t)a.Hkv * P * kHD * 2;
  const char* kbase = (const char*)a.k;
  const char* vbase = (const char*)a.v;
  int koff[kNJ], voff[kNJ];
#pragma unroll
  for (int j = 0; j < kNJ; ++j) {
    const int key = 4 * (j * WAVES + wave) + (lane >> 4);
    const int row_bytes = (it.kvh * P + key % P) * (kHD * 2);
    koff[j] = row_bytes + (((lane & 15) ^ swz_k(key)) << 4);
    voff[j] = row_bytes + (((lane & 15) ^ swz_v(key)) << 4);
  }

  struct Slots {
    int32_t s[kPagesPerTile];
    int32_t ts;              // the tile's first key
  };
  auto fetch = [&](int t) __attribute__((always_inline)) {
    Slots S;
#pragma unroll
    for (int j = 0; j < kPagesPerTile; ++j) {
      const int pg = t * kPagesPerTile + j;
      S.s[j] = (pg >= 0 && pg < pt_count) ? ld_uniform(a.indices + pt_base + pg) : -1;
    }
    S.ts = t * kKT;
    return S;
  };
  auto slot_ok = [&](int32_t s) __attribute__((always_inline)) { return s >= 0 && s < a.num_slots; };

  // A block whose table is intact (table_ok) loads tiles without per-page
  // tests; otherwise every tile takes the checked path, which zero-fills
  // what it cannot load and raises the error flag.  The check itself runs
  // while the first tiles load, which take the checked path.
  bool table_ok = false;
  const uint32_t pool_bytes = kPoolRsrc ? (uint32_t)(a.num_slots * slot_bytes) : 0u;
  const __amdgpu_buffer_rsrc_t rsrc_k =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.k), (short)0, (int)pool_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsrc_v =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.v), (short)0, (int)pool_bytes, 0x00020000);

  // kRead: the segment's rows.  Key 4 gb + (lane >> 4) of the tile starting
  // at key ts is token q_start + ts + 4 gb + (lane >> 4) - pre of k_new; a
  // lane's offset within its group of four keys (the row within the group
  // and the swizzled chunk, which depends only on key % 16 for K and key % 4
  // for V, and key = 16 j + 4 wave + (lane >> 4)) is the same for every j,
  // and the group's start goes in the scalar offset.
  const __amdgpu_buffer_rsrc_t rsrc_nk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.k_new), (short)0, kRead ? (int)a.new_bytes : 0,
                                        0x00020000);
  const __amdgpu_buffer_rsrc_t rsrc_nv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.v_new), (short)0, kRead ? (int)a.new_bytes : 0,
                                        0x00020000);
  const int nk_off = (koff[0] & 255) + (lane >> 4) * a.Hkv * (kHD * 2);
  const int nv_off = (voff[0] & 255) + (lane >> 4) * a.Hkv * (kHD * 2);
  auto new_soff = [&](int ts, int gb) __attribute__((always_inline)) {
    return ((uint32_t)(sd.q_start + ts + 4 * gb - pre) * (uint32_t)a.Hkv + (uint32_t)it.kvh) * (uint32_t)(kHD * 2);
  };
  // the tile holding a group of four keys of both kinds, or -1
  const int t_mixed = (kRead && (pre & 3) != 0) ? pre / kKT : -1;

  // global -> LDS loads of one operand (K or V) of tile t into dst
  auto load_op = [&](int t, const Slots& S, const char* base, const __amdgpu_buffer_rsrc_t& rsrc, const int* off,
                     const __amdgpu_buffer_rsrc_t& nrsrc, int noff, lds_u8* dst) __attribute__((always_inline)) {
    const int ts = t * kKT;
    if (table_ok && ts + kKT <= g_hi && t != t_mixed) {
#pragma unroll
      for (int j = 0; j < kNJ; ++j) {
        const int gb = j * WAVES + wave;
        const int32_t slot = S.s[(4 * gb) / P];
        __attribute__((address_space(3))) void* d = (__attribute__((address_space(3))) void*)(dst + gb * 1024);
        if (kRead && ts + 4 * gb >= pre)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(nrsrc, d, 16, noff, new_soff(ts, gb), 0, 0);
        else if constexpr (kPoolRsrc)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, d, 16, off[j], (uint32_t)slot * (uint32_t)slot_bytes, 0, 0);
        else
          lds_dma16(base + (int64_t)slot * slot_bytes, (uint32_t)slot_bytes, off[j], d);
      }
    } else {
      bool bad = false;
#pragma unroll
      for (int j = 0; j < kNJ; ++j) {
        const int gb = j * WAVES + wave;
        const int32_t s = S.s[(4 * gb) / P];
        const int key = ts + 4 * gb + (lane >> 4);
        // the group's page is read when it holds keys of the item taken from pages
        const bool page_needed = ts + 4 * gb < g_hi && (!kRead || ts + 4 * gb < pre);
        bad |= page_needed && !slot_ok(s);
        const bool ld = page_needed && slot_ok(s) && key < g_hi && (!kRead || key < pre);
        const bool ldn = kRead && key < g_hi && key >= pre;
        __attribute__((address_space(3))) void* d = (__attribute__((address_space(3))) void*)(dst + gb * 1024);
        if (ld) lds_dma16(base + (int64_t)s * slot_bytes, (uint32_t)slot_bytes, off[j], d);
        if constexpr (kRead) {
          if (ldn)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                nrsrc, d, 16, (off[j] & 255) + ((sd.q_start + key - pre) * a.Hkv + it.kvh) * (kHD * 2), 0, 0, 0);
        }
        if (!ld && !ldn) {
          // absent keys: zero rows keep the masked products finite
          const u32x4 z = {0u, 0u, 0u, 0u};
          *(__attribute__((address_space(3))) u32x4*)(dst + gb * 1024 + lane * 16) = z;
        }
      }
      if (bad && lane == 0) atomicOr(a.err, 1);
    }
  };

  f32x16 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) oacc[dt] = f32x16{};
  float m_used = -INFINITY;  // exponent offset in use (log2 domain)
  float msub = 0.f;          // m_used, or 0 while it is -inf
  float m_seen = -INFINITY;  // (exact scale) c times the row's largest score so far
  float l = 0.f;             // this lane's share of the denominator
  float corr = 0.f;          // (exact scale) bf16 roundings of its rows' largest probabilities
  f32x16 negm = f32x16{};    // -msub in every element: where each S accumulation starts
  f32x16 sc[2][2];           // [buffer][32-key block] scores of tiles t and t + 1
  bf16x8 pop[4];             // [16-key group] probabilities of tile t

  const int krow = lane & 31;
  const int tr_g = lane >> 4, tr_s = lane & 15;
  const int tr_key = 4 * (tr_g >> 1) + (tr_s >> 2);
  const int tr_d = 16 * (tr_g & 1) + 4 * (tr_s & 3);

  // MFMA operands from LDS.  S step i: 32-key block i & 1, d-chunk pair
  // i >> 1 (the two accumulation chains alternate).  PV step i: 16-key group
  // i >> 2, 32-wide d block i & 3.
  auto read_k = [&](const lds_u8* kb, int i) __attribute__((always_inline)) {
    const int key = 32 * (i & 1) + krow;
    return *(const __attribute__((address_space(3))) bf16x8*)(
        kb + key * 256 + (((2 * (i >> 1) + hh) ^ swz_k(key)) << 4));
  };
  auto read_v = [&](const lds_u8* vb, int i) __attribute__((always_inline)) {
    bf16x8 vop;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int vkey = 16 * (i >> 2) + 8 * r + tr_key;
      const int d = 32 * (i & 3) + tr_d;
      const bf16x4 x = lds_read_tr(vb + vkey * 256 + ((((d >> 3) ^ swz_v(vkey)) << 4) | ((d & 7) << 1)));
#pragma unroll
      for (int e = 0; e < 4; ++e) vop[4 * r + e] = x[e];
    }
    return vop;
  };
  auto s_step = [&](f32x16* S, bf16x8 kop, int i) __attribute__((always_inline)) {
    S[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[i >> 1], i < 2 ? negm : S[i & 1], 0, 0, 0);
  };
  auto pv_step = [&](bf16x8 vop, int i) __attribute__((always_inline)) {
    oacc[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pop[i >> 2], oacc[i & 3], 0, 0, 0);
  };
  // probabilities of pair j (elements 2j, 2j + 1 of the tile, in P^T slot
  // order: group j >> 2, slots 2 (j & 3) and 2 (j & 3) + 1)
  auto xpair = [&](const f32x16* X, int j, int h) __attribute__((always_inline)) {
    const int g = j >> 2;
    return X[g >> 1][8 * (g & 1) + 2 * (j & 3) + h];
  };
  // probability of one score: the accumulator holds x - m already, or (exact
  // scale) the raw q.k, which is scaled and offset here in fp32
  auto xexp = [&](float v) __attribute__((always_inline)) {
    if constexpr (kExact) return exp2f_fast(__builtin_fmaf(v, a.c, -msub));
    else return exp2f_fast(v);
  };
  auto exp_pair = [&](const f32x16* X, int j) __attribute__((always_inline)) {
    const int g = j >> 2, e = 2 * (j & 3);
    const float p0 = xexp(xpair(X, j, 0));
    const float p1 = xexp(xpair(X, j, 1));
    pop[g][e] = (__bf16)p0;
    pop[g][e + 1] = (__bf16)p1;
    return p0 + p1;
  };
  auto mask_tile = [&](int t, f32x16* S) __attribute__((always_inline)) {
    const int ts = t * kKT;
    const int lim = min(qpos, g_hi - 1);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = ts + 32 * kt + 8 * (e >> 2) + 4 * hh + (e & 3);
        if (key > lim) S[kt][e] = -INFINITY;
      }
  };
  // rescale test, given this lane's max mx of a tile's x values (raw scores
  // with exact scale): move the offset when c (row max) outgrows it by
  // 2^kRescaleLog2, rescale O and l, and shift the tile's x values to the new
  // offset.
  // With exact scale the offset lags the row's max, so the largest
  // probability of a row is 2^x for some x in [0, kRescaleLog2], which the
  // bf16 packing of P rounds; the numerator then carries that rounding and
  // the fp32 denominator would not.  Whenever a row's max grows, the lane
  // holding the new largest score therefore adds its key's rounding,
  // bf16(p) - p, to corr (rescaled with l): p is formed exactly as the tile's
  // exponentials will form it (same fma, same offset), so the output, divided
  // by l + corr, carries in numerator and denominator the same value for
  // every key that was its row's largest when it arrived, as when the offset
  // tracks every growth of the max (largest probability exactly 1), without
  // the rescale of O that this would take at each growth.  The log-sum-exp
  // takes l alone, the fp32 sum.
  auto rescale_test = [&](float mx, f32x16* X) __attribute__((always_inline)) {
    const float mine = mx;
    mx = pair_max(mx);
    const float cand = kExact ? mx * a.c : mx + msub;       // c * row max
    bool grew = false;
    if constexpr (kExact) grew = __ballot(cand > m_seen) != 0;
    if ((!kExact || grew) && __ballot(cand > m_used + kRescaleLog2)) {
      const float m_new = fmaxf(m_used, cand);
      const float alpha = (m_new == -INFINITY) ? 1.f : exp2f_fast(m_used - m_new);
      m_used = m_new;
      const float msub_new = (m_used == -INFINITY) ? 0.f : m_used;
      const float shift = msub_new - msub;
      msub = msub_new;
      // the accumulators start from the new offset (x values only; exact-scale
      // scores carry no offset)
      if constexpr (!kExact) {
#pragma unroll
        for (int e = 0; e < 16; ++e) negm[e] = -msub;
      }
      l *= alpha;
      if constexpr (kExact) corr *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[dt][e] *= alpha;
      if constexpr (!kExact) {
        // and the tile's x values move to it
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) X[kt][e] -= shift;
      } else {
        (void)shift;
        (void)X;
      }
    }
    if constexpr (kExact) {
      if (grew) {
        const float p = exp2f_fast(__builtin_fmaf(mx, a.c, -msub));
        const float d = (float)(__bf16)p - p;
        corr += (cand > m_seen && mine == mx) ? d : 0.f;
        m_seen = fmaxf(m_seen, cand);
      }
    }
  };
  auto row_max = [&](const f32x16* S) __attribute__((always_inline)) {
    float mx = S[0][0];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = vmax(mx, S[kt][e]);
    return mx;
  };

  // plain step, S(t) in sc[0]: S(t+1) into sc[1] if there is a next tile;
  // P(t); O += V(t) P(t); sum; mask and rescale test of tile t+1, which then
  // moves to sc[0]
  auto plain_step = [&](int t, const lds_u8* kb, const lds_u8* vb) __attribute__((always_inline)) {
    const bool has_next = t + 1 < t1;
    float ls = 0.f;
    if (wave_active) {
      if (has_next) {
        // operand reads two MFMAs ahead, P(t) between the MFMAs
        bf16x8 kop[16];
#pragma unroll
        for (int i = 0; i < 2; ++i) kop[i] = read_k(kb, i);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          if (i + 2 < 16) kop[i + 2] = read_k(kb, i + 2);
          s_step(sc[1], kop[i], i);
          ls += exp_pair(sc[0], i);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) ls += exp_pair(sc[0], j);
      }
    }
    if constexpr (kGroups == 2) lds_barrier();
    if (wave_active) {
      bf16x8 vop[16];
#pragma unroll
      for (int i = 0; i < 2; ++i) vop[i] = read_v(vb, i);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (i + 2 < 16) vop[i + 2] = read_v(vb, i + 2);
        pv_step(vop[i], i);
      }
      l += ls;
      if (has_next) {
        if ((t + 2) * kKT > w_full) mask_tile(t + 1, sc[1]);
        rescale_test(row_max(sc[1]), sc[1]);
        sc[0][0] = sc[1][0];
        sc[0][1] = sc[1][1];
      }
    }
  };

  // interleaved step (next tile exists and needs no mask)
  Slots s_a, s_b;          // pages of tiles t + 1 and t + 2 in step t

  // one 16-byte-per-lane load of a full tile with an intact table: from the
  // group's page, or (kRead) from the segment's rows, chosen without a branch
  auto tile_load = [&](const Slots& S, const char* base, const __amdgpu_buffer_rsrc_t& rsrc, const int* off,
                       const __amdgpu_buffer_rsrc_t& nrsrc, int noff, lds_u8* dst, int j) __attribute__((always_inline)) {
    const int gb = j * WAVES + wave;
    const int32_t slot = S.s[(4 * gb) / P];
    __attribute__((address_space(3))) void* d = (__attribute__((address_space(3))) void*)(dst + gb * 1024);
    if constexpr (kRead) {
      const bool seg = S.ts + 4 * gb >= pre;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(seg ? nrsrc : rsrc, d, 16, seg ? noff : off[j],
                                               seg ? new_soff(S.ts, gb) : (uint32_t)slot * (uint32_t)slot_bytes, 0, 0);
    } else if constexpr (kPoolRsrc) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, d, 16, off[j], (uint32_t)slot * (uint32_t)slot_bytes, 0, 0);
    } else {
      lds_dma16(base + (int64_t)slot * slot_bytes, (uint32_t)slot_bytes, off[j], d);
    }
  };

  // interleaved step; also issues this step's loads, K(t+2) into kn and
  // V(t+1) into vn (full tiles, intact table), one per MFMA of phase 1.
  // The exponentials of P(t) are split between the phases: the first
  // 4 kG1 pairs (16-key groups 0 .. kG1 - 1) between the S(t+1) MFMAs of
  // phase 1, the rest between the PV MFMAs of phase 2, each group finished
  // at least one MFMA before the PV MFMA that reads it.  Every VALU op waits on one
  // issued a step earlier, never on its neighbour, so the next MFMA issues on
  // time.
  auto fast_step = [&](auto bc, const lds_u8* kb, const lds_u8* vb, lds_u8* kn, lds_u8* vn) __attribute__((always_inline)) {
    constexpr int B = decltype(bc)::value, N = 1 - B;
    constexpr int E1 = 8 * kG1;              // exponentials in phase 1 (of 32)
    constexpr int E2 = 32 - E1;              // in phase 2
    // phase-2 steps that take them: spread up to the step before the PV MFMA
    // of the last group (slot 4 kG1 + 4 ... 12 with two groups per phase) needs
    // it, rather than packed into the first 4 kG1 slots (measured ~1% faster at
    // c2 with kG1 = 2)
    constexpr int W2 = kG1 == 2 ? 11 : (kG1 < 4 ? 4 * kG1 : 1);
    // step of element e (pair e / 2, half e % 2); -1: before the first MFMA
    auto p1_step = [](int e) constexpr { return (e * 16) / E1 - 1; };
    auto p2_step = [](int e) constexpr { return ((e - E1) * W2) / (E2 > 0 ? E2 : 1) - 1; };
    // a pair is packed and summed one step after its second element
    auto p1_pack = [&](int j) constexpr { return p1_step(2 * j + 1) + 1; };
    auto p2_pack = [&](int j) constexpr { return p2_step(2 * j + 1) + 1; };
    // row max of x(t+1), 16 three-way maxes: in the phase-2 steps past the exponentials
    auto mx_step = [](int k) constexpr { return kG1 <= 2 ? 8 + k / 2 : k; };
    static_assert(phase2_in_time(kG1, W2), "a 16-key group of P packed after the PV MFMA that reads it");
    bf16x8 kop[16], vop[16];
    float ex[16][2];
    // two accumulation chains for the denominator; -0 + y is y, so the first
    // add of each chain folds away
    float ls[2] = {-0.f, -0.f};
    // (exact scale) exponents c s - m, each made one MFMA slot before its
    // exponential, so the exponential never waits on the fma beside it
    float xv[32];
    auto do_x = [&](int e) __attribute__((always_inline)) {
      if constexpr (kExact) xv[e] = __builtin_fmaf(xpair(sc[B], e >> 1, e & 1), a.c, -msub);
    };
    auto do_exp = [&](int e) __attribute__((always_inline)) {
      if constexpr (kExact) ex[e >> 1][e & 1] = exp2f_fast(xv[e]);
      else ex[e >> 1][e & 1] = exp2f_fast(xpair(sc[B], e >> 1, e & 1));
    };
    auto do_pack = [&](int j) __attribute__((always_inline)) {
      ls[j & 1] += ex[j][0] + ex[j][1];
      pop[j >> 2][2 * (j & 3)] = (__bf16)ex[j][0];
      pop[j >> 2][2 * (j & 3) + 1] = (__bf16)ex[j][1];
    };
    // phase 1: S(t+1) MFMAs
#pragma unroll
    for (int i = 0; i < kAhead; ++i) kop[i] = read_k(kb, i);
#pragma unroll
    for (int e = 0; e < E1; ++e)
      if (p1_step(e) <= 0) do_x(e);
#pragma unroll
    for (int e = 0; e < E1; ++e)
      if (p1_step(e) < 0) do_exp(e);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i + kAhead < 16) kop[i + kAhead] = read_k(kb, i + kAhead);
      if (i < kNJ) tile_load(s_b, kbase, rsrc_k, koff, rsrc_nk, nk_off, kn, i);
      else if (i < 2 * kNJ) tile_load(s_a, vbase, rsrc_v, voff, rsrc_nv, nv_off, vn, i - kNJ);
      s_step(sc[N], kop[i], i);
      int nv = 0;
#pragma unroll
      for (int e = 0; e < E1; ++e)
        if (p1_step(e) == i) { do_exp(e); ++nv; }
      if constexpr (kExact) {
#pragma unroll
        for (int e = 0; e < E1; ++e)
          if (p1_step(e) == i + 1) { do_x(e); ++nv; }
        // the exponents of the first elements of phase 2
#pragma unroll
        for (int e = E1; e < 32; ++e)
          if (i == 15 && p2_step(e) < 0) { do_x(e); ++nv; }
      }
#pragma unroll
      for (int j = 0; j < E1 / 2; ++j)
        if (p1_pack(j) == i) { do_pack(j); nv += 3; }
      // pin each step's operand read, tile load, MFMA and VALU work to this step
      if (i + kAhead < 16) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (i < 2 * kNJ) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (nv > 0) __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // the pairs of phase 1 packed after its last MFMA
#pragma unroll
    for (int j = 0; j < E1 / 2; ++j)
      if (p1_pack(j) >= 16) do_pack(j);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (kGroups == 2) lds_barrier();
    // phase 2: PV MFMAs; the rest of P(t) and the row max of x(t+1) between them
#pragma unroll
    for (int i = 0; i < kAhead; ++i) vop[i] = read_v(vb, i);
#pragma unroll
    for (int e = E1; e < 32; ++e)
      if (p2_step(e) < 0) do_exp(e);
#pragma unroll
    for (int e = E1; e < 32; ++e)
      if (p2_step(e) == 0) do_x(e);
    float mx[2] = {-INFINITY, -INFINITY};   // two accumulation chains
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i + kAhead < 16) vop[i + kAhead] = read_v(vb, i + kAhead);
      pv_step(vop[i], i);
      int nv = 0;
#pragma unroll
      for (int e = E1; e < 32; ++e)
        if (p2_step(e) == i) { do_exp(e); ++nv; }
      if constexpr (kExact) {
#pragma unroll
        for (int e = E1; e < 32; ++e)
          if (p2_step(e) == i + 1) { do_x(e); ++nv; }
      }
#pragma unroll
      for (int j = E1 / 2; j < 16; ++j)
        if (p2_pack(j) == i) { do_pack(j); nv += 3; }
#pragma unroll
      for (int k = 0; k < 16; ++k)
        if (mx_step(k) == i) {
          mx[k & 1] = vmax(vmax(mx[k & 1], sc[N][k & 1][2 * (k >> 1)]), sc[N][k & 1][2 * (k >> 1) + 1]);
          ++nv;
        }
      if (i + kAhead < 16) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (nv > 0) __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_sched_barrier(0);
    l += ls[0] + ls[1];
    rescale_test(vmax(mx[0], mx[1]), sc[N]);
  };

  lds_u8* const K0 = L.k0;
  lds_u8* const K1 = L.k1;
  lds_u8* const V0 = L.v0;
  lds_u8* const V1 = L.v1;

  // ---- prologue: K(t0), V(t0), K(t0 + 1); S(t0) and its rescale test
  if (t0 < t1) {
    const Slots s0 = fetch(t0);
    load_op(t0, s0, kbase, rsrc_k, koff, rsrc_nk, nk_off, K0);
    load_op(t0, s0, vbase, rsrc_v, voff, rsrc_nv, nv_off, V0);
  }
  s_b = fetch(t0 + 1);
  if (t0 + 1 < t1) load_op(t0 + 1, s_b, kbase, rsrc_k, koff, rsrc_nk, nk_off, K1);
  // Interleaved steps take the page slots of their loads from a vector load
  // issued a step ahead: it is counted with the tile loads and has a whole
  // step to land, where a scalar load would be waited for at the next barrier.
  const __amdgpu_buffer_rsrc_t rsrc_pt = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t*>(a.indices + pt_base), (short)0, pt_count * 4, 0x00020000);
  typedef uint32_t slot_vec __attribute__((ext_vector_type(kPagesPerTile)));
  auto fetch_vec = [&](int t) __attribute__((always_inline)) {
    if constexpr (kPagesPerTile == 4)
      return __builtin_bit_cast(slot_vec, __builtin_amdgcn_raw_buffer_load_b128(rsrc_pt, t * 16, 0, 0));
    else
      return __builtin_bit_cast(slot_vec, __builtin_amdgcn_raw_buffer_load_b64(rsrc_pt, t * 8, 0, 0));
  };
  slot_vec v_next = fetch_vec(t0 + 2);                      // pages of tile t + 2, in flight
  table_ok = table_check_finish(a, tcheck, pt_base, 64 * WAVES * kGroups);
#pragma unroll
  for (int ks = 0; ks < 8; ++ks)
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if constexpr (!kExact) qop[ks][e] = (__bf16)((float)qop[ks][e] * a.c);
  __builtin_amdgcn_s_waitcnt(0x0070);
  lds_barrier();
  if (kGroups == 2 && GRP == 1) lds_barrier();             // group 1 runs a barrier behind
  if (wave_active && t0 < t1) {
#pragma unroll
    for (int i = 0; i < 16; ++i) s_step(sc[0], read_k(K0, i), i);
    if ((t0 + 1) * kKT > w_full) mask_tile(t0, sc[0]);
    rescale_test(row_max(sc[0]), sc[0]);
  }

  // ---- step t reads K(t+1) and V(t) and loads K(t+2), V(t+1).  K(t) and
  // V(t) sit in buffer (t - t0) & 1.
  auto wait_tiles = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0x0070);                     // my loads of K(t+1), V(t) landed
    lds_barrier();                                          // everyone's; the next buffers are free
  };
  // the item's first `boost` steps run at raised wave priority
  const int t_boost = t0 + (kGroups == 1 ? it.boost : 0);
  auto priority = [&](int t) __attribute__((always_inline)) {
    if (t == t_boost) __builtin_amdgcn_s_setprio(0);
  };
  if (t_boost > t0) __builtin_amdgcn_s_setprio(1);
  auto top = [&](int t, lds_u8* kn, lds_u8* vn) __attribute__((always_inline)) {
    wait_tiles();
    if (t + 2 < t1) load_op(t + 2, s_b, kbase, rsrc_k, koff, rsrc_nk, nk_off, kn);
    if (t + 1 < t1) load_op(t + 1, s_a, vbase, rsrc_v, voff, rsrc_nv, nv_off, vn);
  };
  auto advance = [&](int t) __attribute__((always_inline)) {
    s_a = s_b;
    s_b = fetch(t + 3);
  };
  // start of interleaved step t: s_a <- pages of t + 1, s_b <- pages of t + 2
  // (landed with the last tile loads), pages of t + 3 requested
  auto advance_fast = [&](int t) __attribute__((always_inline)) {
    s_a = s_b;
#pragma unroll
    for (int j = 0; j < kPagesPerTile; ++j) s_b.s[j] = (int32_t)__builtin_amdgcn_readfirstlane(v_next[j]);
    s_b.ts = (t + 2) * kKT;
    v_next = fetch_vec(t + 3);
  };
  // Steps t < t_fast interleave: their next tile needs no mask, V(t+1) is a
  // full tile and K(t+2) a tile of the item (the last one may be partial: its
  // rows past the end are whatever the page holds, and the step that scores
  // them masks them), all covered by an intact table.  Waves run different
  // numbers of each kind of step but the same number of steps, each with one
  // barrier and its share of the tile loads.
  int t_fast = (wave_active && table_ok) ? max(t0, min(w_full / kKT - 1, t1 - 2)) : t0;
  // (kRead) no interleaved step loads the tile with a mixed group of keys
  if (t_mixed >= 0) t_fast = max(t0, min(t_fast, t_mixed - 2));
  int t = t0;
  for (; t + 1 < t_fast; t += 2) {
    priority(t);
    wait_tiles();
    advance_fast(t);
    fast_step(IntC<0>{}, K1, V0, K0, V1);
    priority(t + 1);
    wait_tiles();
    advance_fast(t + 1);
    fast_step(IntC<1>{}, K0, V1, K1, V0);
  }
  if (t < t_fast) {
    priority(t);
    wait_tiles();
    advance_fast(t);
    fast_step(IntC<0>{}, K1, V0, K0, V1);
    ++t;
  }
  // plain steps: scalar page reads (-1 for pages the table lacks)
  s_a = fetch(t + 1);
  s_b = fetch(t + 2);
  if ((t - t0) & 1) {                                       // S(t) is in sc[1]
    sc[0][0] = sc[1][0];
    sc[0][1] = sc[1][1];
  }
  for (; t < t1; ++t) {
    const bool odd = (t - t0) & 1;
    priority(t);
    top(t, odd ? K1 : K0, odd ? V0 : V1);
    plain_step(t, odd ? K0 : K1, odd ? V1 : V0);
    advance(t);
  }

  // (two groups) the partial results merge through l alone
  if constexpr (kExact && kGroups == 2) {
    l += corr;
    corr = 0.f;
  }
  if constexpr (kGroups == 2) {
    // Both groups pass the same number of barriers: group g has passed
    // 1 + g + 2 (its steps) so far; pad to the larger count, then one more
    // barrier frees the tile buffers for group 1's partial results and
    // another publishes them.
    const int n0 = tmid - ti0, n1 = ti1 - tmid;              // steps of each group
    const int passed = 1 + GRP + 2 * (GRP == 0 ? n0 : n1);
    const int total = max(1 + 2 * n0, 2 + 2 * n1);
    for (int k = passed; k < total; ++k) lds_barrier();
    __builtin_amdgcn_s_waitcnt(0x0070);                     // no tile load of mine in flight
    lds_barrier();
    auto slot = [&](int k) __attribute__((always_inline)) {
      lds_u8* const x[4] = {L.x0, L.x1, L.x2, L.x3};
      return (__attribute__((address_space(3))) f32x4*)(x[k >> 2] + ((k & 3) * WAVES + wave) * 1024 + lane * 16);
    };
    if (GRP == 1) {
      if (wave_active) {
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const int dt = k >> 2, i = k & 3;
          *slot(k) = f32x4{oacc[dt][4 * i], oacc[dt][4 * i + 1], oacc[dt][4 * i + 2], oacc[dt][4 * i + 3]};
        }
        L.ml[wave * 64 + lane] = m_used;
        L.ml[kRows * 2 + wave * 64 + lane] = l;
      }
      lds_barrier();
      return;
    }
    lds_barrier();
    if (!wave_active) return;
    // merge: both partials are sums against their own exponent offsets
    const float m_b = L.ml[wave * 64 + lane];
    const float l_b = L.ml[kRows * 2 + wave * 64 + lane];
    const float m_new = fmaxf(m_used, m_b);
    const float alpha = (m_used == -INFINITY) ? 0.f : exp2f_fast(m_used - m_new);
    const float beta = (m_b == -INFINITY) ? 0.f : exp2f_fast(m_b - m_new);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int dt = k >> 2, i = k & 3;
      const f32x4 ob = *slot(k);
#pragma unroll
      for (int e = 0; e < 4; ++e) oacc[dt][4 * i + e] = oacc[dt][4 * i + e] * alpha + ob[e] * beta;
    }
    l = l * alpha + l_b * beta;
    m_used = m_new;
  }

  if (!wave_active) return;
  const float l_tot = pair_sum(l);
  const float l_out = kExact ? pair_sum(l + corr) : l_tot;
  const float inv = l_out > 0.f ? 1.f / l_out : 0.f;
  const float lse2 = l_tot > 0.f ? m_used + __builtin_amdgcn_logf(l_tot) : -INFINITY;
  // The output row is worked out again from the lane index here rather than
  // kept from the start: values live across the loops beyond its registers
  // are spilled to scratch memory.
  const int lane_o = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int hh_o = lane_o >> 5;
  const int o_row = it.row0 + wave * 32 + (lane_o & 31);
  const int o_tok = o_row / G;
  const int o_head = it.kvh * G + (o_row - o_tok * G);
  if (it.part < 0) {
    if (o_row < rows_total) {
      uint16_t* orow = a.o + ((int64_t)(sd.q_start + o_tok) * a.Hq + o_head) * kHD;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d = 32 * dt + 8 * i + 4 * hh_o;
          st_bf16x4(orow + d, oacc[dt][4 * i] * inv, oacc[dt][4 * i + 1] * inv,
                    oacc[dt][4 * i + 2] * inv, oacc[dt][4 * i + 3] * inv);
        }
      if (a.lse != nullptr && hh_o == 0)
        a.lse[(int64_t)(sd.q_start + o_tok) * a.Hq + o_head] = lse2 * 0.69314718055994531f;
    }
  } else {
    const int lrow = wave * 32 + (lane_o & 31);
    float* po = a.part_o + ((int64_t)it.part * kRows + lrow) * kHD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = 32 * dt + 8 * i + 4 * hh_o;
        f32x4 w = {oacc[dt][4 * i] * inv, oacc[dt][4 * i + 1] * inv, oacc[dt][4 * i + 2] * inv,
                   oacc[dt][4 * i + 3] * inv};
        *(f32x4*)(po + d) = w;
      }
    if (hh_o == 0) a.part_lse[(int64_t)it.part * kRows + lrow] = lse2;
  }
}

// ---- work items of at most 32 packed rows (decode requests)
//
// A decode request has one query token, so its item holds the G query heads
// of one KV head -- a single 32-row MFMA block -- over the whole cached
// context.  Run like a prefill item, one wave would carry every matrix
// instruction of the item on one SIMD while the other three only load tiles,
// and a prefill block sharing the CU, whose waves wait on each other at every
// barrier, would run at the pace of its wave on that SIMD.  Here the four
// waves split the item's keys instead: wave w takes the 32-key tiles
// u0 + w, u0 + w + 4, ..., keeps its own online-softmax state over the same
// rows, and needs no barrier.  Its K tiles go straight into registers (they
// are the A operand of S^T = K Q^T, so no LDS round trip is needed) and its V
// tiles into two 8 KB LDS slices of its own (the PV product reads them
// transposed); K is requested one tile ahead and V two, so a wave keeps up to
// 24 KB in flight.  The four partial results are merged through LDS at
// the end.  The item stays bound by HBM, and its matrix work falls evenly on
// the CU's four SIMDs.
constexpr int kDecRows = kDecodeRows;        // rows of an item this path takes
constexpr int kDecKeys = 32;                 // keys per tile of one wave

template <int P, bool kExact>
__device__ __attribute__((always_inline)) inline void decode_group(const AttnArgs& a, const AttnItem& it,
                                                                   const SeqDesc& sd, const PipeLds& L) {
  static_assert(P == 16 || P == 32, "page size");
  constexpr int kWaves = 4;
  constexpr int kPagesPerTile = kDecKeys / P;                // 2 or 1
  constexpr int kSliceBytes = kDecKeys * kHD * 2;            // 8 KB: one V tile of one wave
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (kWaves - 1);
  const int hh = lane >> 5;
  const int G = a.G;
  const int rows_total = sd.q_len * G;
  const int pre = sd.kv_len - sd.q_len;

  // every wave holds the same rows: row r of the block is lane r % 32
  const int r_row = it.row0 + (lane & 31);
  const int rr = r_row < rows_total ? r_row : rows_total - 1;
  const int tok = rr / G;
  const int head = it.kvh * G + (rr - tok * G);
  const int qpos = pre + tok;
  const int g_lo = it.kv_begin, g_hi = it.kv_end;
  const int w_full = min(g_hi, pre + it.row0 / G + 1);      // keys below are visible to all rows

  bf16x8 qop[8];
  {
    const uint16_t* qrow = a.q + ((int64_t)(sd.q_start + tok) * a.Hq + head) * kHD;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qop[ks] = ld_bf16x8(qrow + (2 * ks + hh) * 8);
  }
  const int32_t pt_base = ld_uniform(a.indptr + it.seq);
  const int32_t pt_count = ld_uniform(a.indptr + it.seq + 1) - pt_base;
  TableCheck tcheck = table_check_issue<P>(a, it, pt_base, pt_count, 64 * kWaves);
  if constexpr (!kExact) {
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) qop[ks][e] = (__bf16)((float)qop[ks][e] * a.c);
  }
  const bool table_ok = table_check_finish(a, tcheck, pt_base, 64 * kWaves);

  lds_u8* const vslice[2] = {(wave & 2 ? L.k1 : L.k0) + (wave & 1) * kSliceBytes,
                             (wave & 2 ? L.v1 : L.v0) + (wave & 1) * kSliceBytes};
  const int64_t slot_bytes = (int64_t)a.Hkv * P * kHD * 2;
  const uint32_t pool_bytes = (uint32_t)(a.num_slots * slot_bytes);      // < 2^31 (caller's condition)
  const __amdgpu_buffer_rsrc_t rsrc_k =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.k), (short)0, (int)pool_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsrc_v =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.v), (short)0, (int)pool_bytes, 0x00020000);
  const int krow = lane & 31;
  const int krow_off = (it.kvh * P + krow % P) * (kHD * 2) + hh * 16;   // this lane's K row, d-chunk parity
  bool bad = false;

  // Slot of page pg of the sequence, or -1 when the table lacks it or it lies
  // outside the pool (then the page is not read and the error flag is raised).
  auto slot_of = [&](int pg) __attribute__((always_inline)) {
    const int32_t s = pg < pt_count ? ld_uniform(a.indices + pt_base + pg) : -1;
    return (s >= 0 && s < a.num_slots) ? s : -1;
  };
  // Every tile issues exactly 8 K loads and 8 V loads, so that "the next
  // tile's 16 loads may still be outstanding" is an exact wait: a row that must
  // not be read gets an offset past the pool's buffer resource (the pool spans
  // < 2^31 bytes), which returns zeros -- into registers or into LDS alike.
  constexpr uint32_t kOutside = 0x80000000u;
  // K of tile u into registers: lane l holds key l % 32, d-chunks 2 i + l / 32
  // (the MFMA's A operand).  Keys past the item's end and absent pages are zeros
  // (the former are masked; the latter behave as zero rows, and raise the flag).
  auto load_k = [&](int u, bf16x8* kr) __attribute__((always_inline)) {
    int32_t sl[kPagesPerTile];
#pragma unroll
    for (int p = 0; p < kPagesPerTile; ++p) {
      sl[p] = slot_of(u * kPagesPerTile + p);
      bad |= sl[p] < 0 && u * kDecKeys + p * P < g_hi;
    }
    const int32_t s = (kPagesPerTile == 2 && krow >= P) ? sl[kPagesPerTile - 1] : sl[0];
    const bool ok = s >= 0 && u * kDecKeys + krow < g_hi;
    const uint32_t base = ok ? (uint32_t)s * (uint32_t)slot_bytes + (uint32_t)krow_off : kOutside;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      kr[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rsrc_k, base + i * 32, 0, 0));
  };
  // V of tile u into an LDS slice: load j fills rows 4j .. 4j + 3, lane i one
  // 16-byte chunk of row 4j + i / 16 (XOR-swizzled as the prefill path's).
  // Keys past the item's end and absent pages are zero rows, which keep the
  // masked products finite.
  auto load_v = [&](int u, lds_u8* dst) __attribute__((always_inline)) {
    const int ts = u * kDecKeys;
    int32_t sl[kPagesPerTile];
#pragma unroll
    for (int p = 0; p < kPagesPerTile; ++p) sl[p] = slot_of(u * kPagesPerTile + p);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int key = 4 * j + (lane >> 4);
      const int s = sl[(4 * j) / P];
      const uint32_t off = (uint32_t)((it.kvh * P + key % P) * (kHD * 2) + (((lane & 15) ^ swz_v(key)) << 4));
      const bool ok = s >= 0 && ts + key < g_hi;
      __attribute__((address_space(3))) void* d = (__attribute__((address_space(3))) void*)(dst + j * 1024);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc_v, d, 16, ok ? off : kOutside,
                                               s >= 0 ? (uint32_t)s * (uint32_t)slot_bytes : 0u, 0, 0);
    }
  };

  const int tr_g = lane >> 4, tr_s = lane & 15;
  const int tr_key = 4 * (tr_g >> 1) + (tr_s >> 2);
  const int tr_d = 16 * (tr_g & 1) + 4 * (tr_s & 3);
  f32x16 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) oacc[dt] = f32x16{};
  float m_used = -INFINITY, msub = 0.f, l = 0.f;
  bf16x8 kr[8];

  // Issue order: K(u), V(u), V(u + 4); then in the step of tile u, K(u + 4)
  // once S(u) has read K(u) out of the registers, and V(u + 8) once the PV
  // product has read V(u) out of its slice.  At the top of the step of tile
  // u, K(u) and V(u) have landed once at most V(u + 4)'s 8 loads are
  // outstanding (K(u + 4) is issued later, within the step).
  const int u0 = g_lo / kDecKeys;
  const int u1 = (g_hi + kDecKeys - 1) / kDecKeys;
  int u = u0 + wave;
  if (u < u1) {
    load_k(u, kr);
    load_v(u, vslice[0]);
  }
  if (u + kWaves < u1) load_v(u + kWaves, vslice[1]);
  auto step = [&](auto bc) __attribute__((always_inline)) {
    constexpr int b = decltype(bc)::value;
    if (u + kWaves < u1) __builtin_amdgcn_s_waitcnt(0x0078);             // vmcnt(8), lgkmcnt(0)
    else __builtin_amdgcn_s_waitcnt(0x0070);                             // vmcnt(0), lgkmcnt(0)
    asm volatile("" ::: "memory");
    // S^T = K Q^T over the tile's 32 keys (one 32 x 32 block, 8 MFMAs over d)
    f32x16 S = f32x16{};
    if constexpr (!kExact) {
#pragma unroll
      for (int e = 0; e < 16; ++e) S[e] = -msub;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kr[i], qop[i], S, 0, 0, 0);
    if (u + kWaves < u1) load_k(u + kWaves, kr);
    // mask keys past the row's own position or the item's end
    const int ts = u * kDecKeys;
    if (ts + kDecKeys > w_full) {
      const int lim = min(qpos, g_hi - 1);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = ts + 8 * (e >> 2) + 4 * hh + (e & 3);
        if (key > lim) S[e] = -INFINITY;
      }
    }
    // offset test (exact scale: whenever the row max grows; folded: past 2^kRescaleLog2)
    float mx = S[0];
#pragma unroll
    for (int e = 1; e < 16; ++e) mx = vmax(mx, S[e]);
    mx = pair_max(mx);
    const float cand = kExact ? mx * a.c : mx + msub;
    if (__ballot(cand > m_used + (kExact ? kRescaleLog2Exact : kRescaleLog2))) {
      const float m_new = fmaxf(m_used, cand);
      const float alpha = (m_new == -INFINITY) ? 1.f : exp2f_fast(m_used - m_new);
      m_used = m_new;
      const float msub_new = (m_used == -INFINITY) ? 0.f : m_used;
      const float shift = msub_new - msub;
      msub = msub_new;
      l *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[dt][e] *= alpha;
      if constexpr (!kExact) {
#pragma unroll
        for (int e = 0; e < 16; ++e) S[e] -= shift;
      } else {
        (void)shift;
      }
    }
    // P = exp2(x), packed to bf16 in the P^T operand order (16-key group g,
    // slots 2 (j & 3) and 2 (j & 3) + 1 from accumulator 8 g + 2 (j & 3) + h)
    bf16x8 pop[2];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int g = j >> 2, e = 2 * (j & 3);
      const float x0 = S[8 * g + e], x1 = S[8 * g + e + 1];
      const float p0 = kExact ? exp2f_fast(__builtin_fmaf(x0, a.c, -msub)) : exp2f_fast(x0);
      const float p1 = kExact ? exp2f_fast(__builtin_fmaf(x1, a.c, -msub)) : exp2f_fast(x1);
      pop[g][e] = (__bf16)p0;
      pop[g][e + 1] = (__bf16)p1;
      l += p0 + p1;
    }
    // O^T += V^T P^T: 2 groups of 16 keys x 4 blocks of 32 d
    const lds_u8* const vb = vslice[b];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      bf16x8 vop;
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int vkey = 16 * (i >> 2) + 8 * r + tr_key;
        const int d = 32 * (i & 3) + tr_d;
        const bf16x4 x = lds_read_tr(vb + vkey * 256 + ((((d >> 3) ^ swz_v(vkey)) << 4) | ((d & 7) << 1)));
#pragma unroll
        for (int e = 0; e < 4; ++e) vop[4 * r + e] = x[e];
      }
      oacc[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pop[i >> 2], oacc[i & 3], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);                    // lgkmcnt(0): V operands read out of LDS
    asm volatile("" ::: "memory");
    if (u + 2 * kWaves < u1) load_v(u + 2 * kWaves, vslice[b]);
    u += kWaves;
  };
  while (u < u1) {
    step(IntC<0>{});
    if (u >= u1) break;
    step(IntC<1>{});
  }
  if (bad && lane == 0) atomicOr(a.err, 1);

  // ---- merge the four waves' partial results through LDS (the tile slices are free)
  __builtin_amdgcn_s_waitcnt(0x0070);
  __syncthreads();
  // wave w > 0 leaves its O^T in one 16 KB array (k0, k1, v0), m and l in v1
  auto xo = [&](int w) __attribute__((always_inline)) {
    lds_u8* const x[3] = {L.k0, L.k1, L.v0};
    return (__attribute__((address_space(3))) float*)x[w];
  };
  __attribute__((address_space(3))) float* const xml = (__attribute__((address_space(3))) float*)L.v1;
  if (wave > 0) {
    __attribute__((address_space(3))) float* const dst = xo(wave - 1);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int dt = k >> 2, i = k & 3;
      *(__attribute__((address_space(3))) f32x4*)(dst + (k * 64 + lane) * 4) =
          f32x4{oacc[dt][4 * i], oacc[dt][4 * i + 1], oacc[dt][4 * i + 2], oacc[dt][4 * i + 3]};
    }
    xml[((wave - 1) * 2) * 64 + lane] = m_used;
    xml[((wave - 1) * 2 + 1) * 64 + lane] = l;
  }
  __syncthreads();
  if (wave > 0) return;
#pragma unroll
  for (int w = 0; w < kWaves - 1; ++w) {
    const float m_b = xml[(w * 2) * 64 + lane];
    const float l_b = xml[(w * 2 + 1) * 64 + lane];
    const float m_new = fmaxf(m_used, m_b);
    const float alpha = (m_used == -INFINITY) ? 0.f : exp2f_fast(m_used - m_new);
    const float beta = (m_b == -INFINITY) ? 0.f : exp2f_fast(m_b - m_new);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int dt = k >> 2, i = k & 3;
      const f32x4 ob = *(const __attribute__((address_space(3))) f32x4*)(xo(w) + (k * 64 + lane) * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) oacc[dt][4 * i + e] = oacc[dt][4 * i + e] * alpha + ob[e] * beta;
    }
    l = l * alpha + l_b * beta;
    m_used = m_new;
  }
  const float l_tot = pair_sum(l);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse2 = l_tot > 0.f ? m_used + __builtin_amdgcn_logf(l_tot) : -INFINITY;
  if (it.part < 0) {
    if (r_row < rows_total) {
      uint16_t* orow = a.o + ((int64_t)(sd.q_start + tok) * a.Hq + head) * kHD;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d = 32 * dt + 8 * i + 4 * hh;
          st_bf16x4(orow + d, oacc[dt][4 * i] * inv, oacc[dt][4 * i + 1] * inv, oacc[dt][4 * i + 2] * inv,
                    oacc[dt][4 * i + 3] * inv);
        }
      if (a.lse != nullptr && hh == 0)
        a.lse[(int64_t)(sd.q_start + tok) * a.Hq + head] = lse2 * 0.69314718055994531f;
    }
  } else {
    // partial of a key-range part: rows 0 .. 31 of the part's slot
    float* po = a.part_o + ((int64_t)it.part * kPipeRows + (lane & 31)) * kHD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = 32 * dt + 8 * i + 4 * hh;
        *(f32x4*)(po + d) = f32x4{oacc[dt][4 * i] * inv, oacc[dt][4 * i + 1] * inv, oacc[dt][4 * i + 2] * inv,
                                  oacc[dt][4 * i + 3] * inv};
      }
    if (hh == 0) a.part_lse[(int64_t)it.part * kPipeRows + (lane & 31)] = lse2;
  }
}

// One group of four waves per block, two blocks per CU.
// kRead: the launch also writes the segment's new K/V rows (write_own_rows)
// and reads the segment's keys from them, not from their pages.  A decode item
// reads its keys through the pages: it is then the only reader of its rows, so
// it writes them itself first and reads them back after a barrier; a later
// key-range part of a split decode item that holds segment keys takes the
// general path, which reads them from k_new / v_new.
// kExact: the softmax scale is applied in fp32 to each score instead of to
// the query rows in bf16 (one fma per score; no rounding of c q).
template <int P, bool kPoolRsrc, bool kRead, bool kExact = false>
__global__ __launch_bounds__(256, 2) void attn_pipe_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds0[kTileBytes], k_lds1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds0[kTileBytes], v_lds1[kTileBytes];
  const AttnItem it = ld_uniform(a.items + blockIdx.x);
  if (a.blk_clock != nullptr && threadIdx.x == 0) {
    uint64_t* r = a.blk_clock + 4 * (int64_t)blockIdx.x;
    r[0] = __builtin_amdgcn_s_memrealtime();
    // {sequence, KV head, first key tile mod 2^16}, {q_len, first row}
    r[2] = (uint64_t)(uint32_t)it.seq | ((uint64_t)(uint16_t)it.kvh << 32) |
           ((uint64_t)(uint16_t)(it.kv_begin / kKT) << 48);
    r[3] = (uint64_t)(uint32_t)it.q_len | ((uint64_t)(uint32_t)it.row0 << 32);
  }
  if (it.kv_begin < it.kv_end) {                            // else a padding item
    const SeqDesc sd{it.q_start, it.q_len, it.kv_len, 0};
    const PipeLds L{(lds_u8*)k_lds0, (lds_u8*)k_lds1, (lds_u8*)v_lds0, (lds_u8*)v_lds1,
                    nullptr, nullptr, nullptr, nullptr, nullptr};
    const bool decode = kPoolRsrc && it.q_len * a.G <= kDecRows &&
                        (!kRead || it.kv_begin == 0 || it.kv_end <= it.kv_len - it.q_len);
    if constexpr (kRead) {
      if (it.kv_begin == 0) {
        write_own_rows<P>(a, it);
        if (decode) __syncthreads();                         // its own rows, read back below
      }
    }
    if (decode)
      decode_group<P, kExact>(a, it, sd, L);
    else
      pipe_group<P, kPoolRsrc, 1, 0, kRead, kExact>(a, it, sd, L);
  }
  if (a.blk_clock != nullptr) {
    // every wave's stores are done once the barrier is passed
    __syncthreads();
    if (threadIdx.x == 0) a.blk_clock[4 * (int64_t)blockIdx.x + 1] = __builtin_amdgcn_s_memrealtime();
  }
}

// Two groups of four waves per block on the same rows, each over half of the
// item's key tiles, one block per CU; the halves merge in LDS.
template <int P, bool kPoolRsrc>
__global__ __launch_bounds__(512, 1) void attn_pp_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t k_a0[kTileBytes], k_a1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_a0[kTileBytes], v_a1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t k_b0[kTileBytes], k_b1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_b0[kTileBytes], v_b1[kTileBytes];
  __shared__ float ml[4 * kPipeRows];
  const AttnItem it = ld_uniform(a.items + blockIdx.x);
  if (it.kv_begin >= it.kv_end) return;                     // padding item
  const SeqDesc sd{it.q_start, it.q_len, it.kv_len, 0};
  lds_u8* const xb0 = (lds_u8*)k_b0;
  lds_u8* const xb1 = (lds_u8*)k_b1;
  lds_u8* const xb2 = (lds_u8*)v_b0;
  lds_u8* const xb3 = (lds_u8*)v_b1;
  __attribute__((address_space(3))) float* const mlp = (__attribute__((address_space(3))) float*)ml;
  if (__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) < kPipeWaves) {
    const PipeLds L{(lds_u8*)k_a0, (lds_u8*)k_a1, (lds_u8*)v_a0, (lds_u8*)v_a1, xb0, xb1, xb2, xb3, mlp};
    pipe_group<P, kPoolRsrc, 2, 0>(a, it, sd, L);
  } else {
    const PipeLds L{xb0, xb1, xb2, xb3, xb0, xb1, xb2, xb3, mlp};
    pipe_group<P, kPoolRsrc, 2, 1>(a, it, sd, L);
  }
}

}  // namespace sa
