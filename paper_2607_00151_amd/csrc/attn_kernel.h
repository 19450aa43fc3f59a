// Paged causal grouped-query prefill attention for gfx950 (CDNA4).
//
// One work item = one (sequence, KV head, tile of query rows, key range).
// Query rows of a KV head are its G query heads packed per token:
// row r <-> (segment token r / G, query head kvh*G + r % G), so every K/V tile
// staged in LDS serves all G heads of the group.  Each wave owns 32*QT rows;
// keys advance in tiles of 64.
//
// Per tile and wave:
//   S^T[64 keys x 32 rows] = K_tile . Q^T      8 v_mfma_f32_32x32x16_bf16 per
//                                              (32-key block, 32-row block)
//   online softmax in the exp2 domain          lane l owns row l % 32 of each
//                                              row block; its scores sit in its
//                                              own registers and in lane l ^ 32
//   O^T[128 d x 32 rows] += V^T . P^T          16 MFMAs per row block
// The transposed products keep one row's statistics on one lane pair: the row
// max needs one v_permlane32_swap, the O^T rescale is a per-lane multiply, and
// the P^T operand of the PV product comes straight from the S^T accumulators.
//
// A 32x32 accumulator puts, for lane l (h = l / 32), keys 8i + 4h + j of the
// 32-key block in register 4i + j, so the k-slots of lane half h carry keys
// {4h..4h+3, 8+4h..8+4h+3} of each 16-key group.  The V^T operand is read
// with ds_read_b64_tr_b16, which hands each lane of a 16-lane group one
// column of a 4-row x 16-column block; two such reads give a lane exactly the
// 8 keys its P^T slots hold, at its own d.
//
// K and V tiles move global -> LDS with global_load_lds_dwordx4 (no register
// staging), double buffered: the loads of tile t+1 are in flight while tile t
// is computed.  Rows of both tiles are 256 bytes; 16-byte chunks are XOR
// swizzled (K by key & 15, V by 4 * (key & 3)) so the MFMA operand reads of a
// wave spread over the LDS banks.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"
#include "plan.h"

namespace sa {

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;        // pools offset to the layer
  const uint16_t* v;
  uint16_t* o;
  float* lse;               // nullable
  float* part_o;            // [parts][rows_per_item][kHD] normalised partial outputs
  float* part_lse;          // [parts][rows_per_item] log2-domain LSE of each partial
  const AttnItem* items;
  const SeqDesc* seqs;
  const int32_t* indptr;
  const int32_t* indices;
  int32_t* err;
  int32_t num_slots;
  int32_t n_items;
  int32_t Hq, Hkv, G;
  float c;                  // softmax_scale * log2(e)
  // The segment's own K/V rows (attn_pipe_kernel with kRead only): blocks
  // read the segment's keys from here instead of from their pages, and the
  // first key-range part of each row tile writes its tokens' rows to the pages.
  const uint16_t* k_new;    // [sum q_len][Hkv][kHD], token-major like q
  const uint16_t* v_new;
  uint32_t new_bytes;       // bytes of each of k_new, v_new (< 2^31)
  // nullable (attn_pipe_kernel only): per block {start, end} of the device's
  // constant-rate clock and the item's {sequence, q_len}, four words per block
  uint64_t* blk_clock;
};

// Lazy rescaling (folded-scale mode only): the exponent offset only moves
// when a row's running max grows by more than this many powers of two, so P
// stays below 2^kRescaleLog2 (bf16 and fp32 hold that easily) and the O
// rescale is rare.  Its price is accuracy: a row's largest probability is
// then 2^x for some x in (0, kRescaleLog2], which bf16 rounds by up to 2^-9
// of itself, an error that reaches the output undiluted when one key
// dominates the row.
constexpr float kRescaleLog2 = 8.0f;
// The exact-scale kernels move the offset whenever a row's max grows
// (threshold 0): the largest probability of every row is then exactly 1 in
// bf16, and the only roundings left on the dominant term are the output's.
constexpr float kRescaleLog2Exact = 0.0f;

__device__ __forceinline__ int swz_k(int key) { return key & 15; }
__device__ __forceinline__ int swz_v(int key) { return (key & 3) << 2; }

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) uint8_t lds_u8;

__device__ __forceinline__ bf16x4 lds_read_tr(const lds_u8* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
}

__device__ __forceinline__ float pair_max(float x) {
  // lanes l and l ^ 32 exchange; both halves see the same pair
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int P, int QT, int WAVES>
__global__ __launch_bounds__(64 * WAVES, (QT == 1 ? 2 : 1)) void attn_kernel(AttnArgs a) {
  static_assert(P == 16 || P == 32, "page size");
  static_assert(16 % WAVES == 0 && (WAVES & (WAVES - 1)) == 0, "waves: a power of two dividing 16");
  constexpr int kRowsW = 32 * QT;                          // rows per wave
  constexpr int kRows = kRowsW * WAVES;                    // rows per item
  constexpr int kTileBytes = kKT * kHD * 2;                // 16 KB
  constexpr int kPagesPerTile = kKT / P;
  constexpr int kNJ = 16 / WAVES;                          // loads per wave per tile and operand
  // one array per buffer: distinct objects let the compiler see that the DMA
  // writes into one buffer never alias the operand reads of the other
  __shared__ __attribute__((aligned(1024))) uint8_t k_lds0[kTileBytes], k_lds1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v_lds0[kTileBytes], v_lds1[kTileBytes];

  const AttnItem it = ld_uniform(a.items + blockIdx.x);
  if (it.kv_begin >= it.kv_end) return;                     // padding item
  const SeqDesc sd = ld_uniform(a.seqs + it.seq);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // the mask tells the compiler wave < WAVES, so per-load page indices fold to constants
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (WAVES - 1);
  const int hh = lane >> 5;                                 // lane half
  const int G = a.G;
  const int rows_total = sd.q_len * G;
  const int pre = sd.kv_len - sd.q_len;

  // ---- this lane's query rows (one per 32-row block)
  int tok[QT], head[QT], qpos[QT];
  bool row_valid[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int r = it.row0 + wave * kRowsW + 32 * qt + (lane & 31);
    row_valid[qt] = r < rows_total;
    const int rr = row_valid[qt] ? r : rows_total - 1;
    tok[qt] = rr / G;
    head[qt] = it.kvh * G + (rr - tok[qt] * G);
    qpos[qt] = pre + tok[qt];
  }

  // ---- wave-uniform bounds
  const int wrow0 = it.row0 + wave * kRowsW;
  const bool wave_active = wrow0 < rows_total;
  const int wlast = min(wrow0 + kRowsW - 1, rows_total - 1);
  const int w_kv_end = min(it.kv_end, pre + wlast / G + 1);  // keys any row of the wave needs
  const int w_full = min(it.kv_end, pre + wrow0 / G + 1);    // keys below are visible to all rows

  // ---- Q operand (B of S^T = K Q^T): lane holds d-chunks 2ks + hh
  bf16x8 qop[QT][8];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const uint16_t* qrow = a.q + ((int64_t)(sd.q_start + tok[qt]) * a.Hq + head[qt]) * kHD;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qop[qt][ks] = ld_bf16x8(qrow + (2 * ks + hh) * 8);
  }

  // ---- page table of this sequence (scalar reads)
  const int32_t pt_base = ld_uniform(a.indptr + it.seq);
  const int32_t pt_count = ld_uniform(a.indptr + it.seq + 1) - pt_base;
  const int64_t slot_bytes = (int64_t)a.Hkv * P * kHD * 2;
  const char* kbase = (const char*)a.k;
  const char* vbase = (const char*)a.v;

  // load j of this wave fills LDS rows 4*gb .. 4*gb + 3 (gb = j*WAVES + wave);
  // lane i writes 16 bytes at row 4*gb + i/16, swizzled chunk i & 15
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
  };
  auto fetch = [&](int t) {
    Slots S;
#pragma unroll
    for (int j = 0; j < kPagesPerTile; ++j) {
      const int pg = t * kPagesPerTile + j;
      if (pg < pt_count) S.s[j] = ld_uniform(a.indices + pt_base + pg);
      else S.s[j] = -1;
    }
    return S;
  };
  auto slot_ok = [&](int32_t s) { return s >= 0 && s < a.num_slots; };

  // issue the global -> LDS loads of tile t into the buffers kb, vb
  auto load_tile = [&](int t, const Slots& S, lds_u8* kb, lds_u8* vb) {
    const int ts = t * kKT;
    bool fast = ts + kKT <= it.kv_end;
#pragma unroll
    for (int j = 0; j < kPagesPerTile; ++j) fast = fast && slot_ok(S.s[j]);
    if (fast) {
#pragma unroll
      for (int j = 0; j < kNJ; ++j) {
        const int gb = j * WAVES + wave;
        const int64_t sb = (int64_t)S.s[(4 * gb) / P] * slot_bytes;
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(kbase + sb + koff[j]),
                                         (__attribute__((address_space(3))) void*)(kb + gb * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(vbase + sb + voff[j]),
                                         (__attribute__((address_space(3))) void*)(vb + gb * 1024), 16, 0, 0);
      }
    } else {
      bool bad = false;
#pragma unroll
      for (int j = 0; j < kNJ; ++j) {
        const int gb = j * WAVES + wave;
        const int32_t s = S.s[(4 * gb) / P];
        const bool page_needed = ts + 4 * gb < it.kv_end;
        bad |= page_needed && !slot_ok(s);
        const bool ld = page_needed && slot_ok(s) && ts + 4 * gb + (lane >> 4) < it.kv_end;
        if (ld) {
          const int64_t sb = (int64_t)s * slot_bytes;
          __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(kbase + sb + koff[j]),
                                           (__attribute__((address_space(3))) void*)(kb + gb * 1024), 16, 0, 0);
          __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(vbase + sb + voff[j]),
                                           (__attribute__((address_space(3))) void*)(vb + gb * 1024), 16, 0, 0);
        } else {
          // absent keys: zero K and V so masked products stay finite
          const u32x4 z = {0u, 0u, 0u, 0u};
          *(__attribute__((address_space(3))) u32x4*)(kb + gb * 1024 + lane * 16) = z;
          *(__attribute__((address_space(3))) u32x4*)(vb + gb * 1024 + lane * 16) = z;
        }
      }
      if (bad && lane == 0) atomicOr(a.err, 1);
    }
  };

  f32x16 oacc[4][QT];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) oacc[dt][qt] = f32x16{};
  float m_used[QT], l[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_used[qt] = -INFINITY;  // exponent offset in use (log2 domain)
    l[qt] = 0.f;             // this lane's share of the denominator
  }

  // per-lane LDS offsets of the MFMA operand reads
  const int krow = lane & 31;                               // key within a 32-key block
  const int tr_g = lane >> 4, tr_s = lane & 15;             // 16-lane group, lane in group
  const int tr_key = 4 * (tr_g >> 1) + (tr_s >> 2);         // + 16 kb + 8 r
  const int tr_d = 16 * (tr_g & 1) + 4 * (tr_s & 3);        // + 32 dt

  const int t0 = it.kv_begin / kKT;
  const int t1 = (it.kv_end + kKT - 1) / kKT;
  lds_u8* const K0 = (lds_u8*)k_lds0;
  lds_u8* const K1 = (lds_u8*)k_lds1;
  lds_u8* const V0 = (lds_u8*)v_lds0;
  lds_u8* const V1 = (lds_u8*)v_lds1;
  load_tile(t0, fetch(t0), K0, V0);
  Slots nxt = fetch(t0 + 1 < t1 ? t0 + 1 : t0);

  // one key tile: wait for its loads, start the next tile's, compute
  auto step = [&](int t, const lds_u8* kb, const lds_u8* vb, lds_u8* kn, lds_u8* vn) {
    __builtin_amdgcn_s_waitcnt(0x0070);                     // vmcnt(0) lgkmcnt(0): my loads landed
    __syncthreads();                                        // everyone's landed; kn, vn are free
    if (t + 1 < t1) {
      load_tile(t + 1, nxt, kn, vn);
      if (t + 2 < t1) nxt = fetch(t + 2);
    }
    const int ts = t * kKT;
    if (!(wave_active && ts < w_kv_end)) return;
      f32x16 s[2][QT];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int key = 32 * kt + krow;
        const lds_u8* kr = kb + key * 256;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const bf16x8 kop = *(const __attribute__((address_space(3))) bf16x8*)(kr + (((2 * ks + hh) ^ swz_k(key)) << 4));
#pragma unroll
          for (int qt = 0; qt < QT; ++qt)
            s[kt][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[qt][ks], ks == 0 ? f32x16{} : s[kt][qt], 0, 0, 0);
        }
      }
      const bool need_mask = ts + kKT > w_full;
      bf16x8 pop[QT][4];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        if (need_mask) {
          const int lim = min(qpos[qt], it.kv_end - 1);
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int key = ts + 32 * kt + 8 * (e >> 2) + 4 * hh + (e & 3);
              if (key > lim) s[kt][qt][e] = -INFINITY;
            }
        }
        float mx = s[0][qt][0];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) mx = vmax(mx, s[kt][qt][e]);
        mx = pair_max(mx);
        const float cand = mx * a.c;
        if (__ballot(cand > m_used[qt] + kRescaleLog2Exact)) {
          const float m_new = fmaxf(m_used[qt], cand);
          const float alpha = (m_new == -INFINITY) ? 1.f : exp2f_fast(m_used[qt] - m_new);
          m_used[qt] = m_new;
          l[qt] *= alpha;
#pragma unroll
          for (int dt = 0; dt < 4; ++dt)
#pragma unroll
            for (int e = 0; e < 16; ++e) oacc[dt][qt][e] *= alpha;
        }
        const float msub = (m_used[qt] == -INFINITY) ? 0.f : m_used[qt];
        float lsum = 0.f;
#pragma unroll
        for (int kb2 = 0; kb2 < 4; ++kb2) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float p = exp2f_fast(__builtin_fmaf(s[kb2 >> 1][qt][8 * (kb2 & 1) + e], a.c, -msub));
            lsum += p;
            pop[qt][kb2][e] = (__bf16)p;
          }
        }
        l[qt] += lsum;
      }
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int kb2 = 0; kb2 < 4; ++kb2) {
          bf16x8 vop;
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            const int key = 16 * kb2 + 8 * r + tr_key;
            const int d = 32 * dt + tr_d;
            const bf16x4 x = lds_read_tr(vb + key * 256 + ((((d >> 3) ^ swz_v(key)) << 4) | ((d & 7) << 1)));
#pragma unroll
            for (int e = 0; e < 4; ++e) vop[4 * r + e] = x[e];
          }
#pragma unroll
          for (int qt = 0; qt < QT; ++qt)
            oacc[dt][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pop[qt][kb2], oacc[dt][qt], 0, 0, 0);
        }
      }
  };
  for (int t = t0; t < t1; t += 2) {
    step(t, K0, V0, K1, V1);
    if (t + 1 < t1) step(t + 1, K1, V1, K0, V0);
  }

  if (!wave_active) return;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float l_tot = pair_sum(l[qt]);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse2 = l_tot > 0.f ? m_used[qt] + __builtin_amdgcn_logf(l_tot) : -INFINITY;
    if (it.part < 0) {
      if (row_valid[qt]) {
        uint16_t* orow = a.o + ((int64_t)(sd.q_start + tok[qt]) * a.Hq + head[qt]) * kHD;
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int d = 32 * dt + 8 * i + 4 * hh;
            st_bf16x4(orow + d, oacc[dt][qt][4 * i] * inv, oacc[dt][qt][4 * i + 1] * inv,
                      oacc[dt][qt][4 * i + 2] * inv, oacc[dt][qt][4 * i + 3] * inv);
          }
        if (a.lse != nullptr && hh == 0)
          a.lse[(int64_t)(sd.q_start + tok[qt]) * a.Hq + head[qt]] = lse2 * 0.69314718055994531f;
      }
    } else {
      const int lrow = wave * kRowsW + 32 * qt + (lane & 31);
      float* po = a.part_o + ((int64_t)it.part * kRows + lrow) * kHD;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d = 32 * dt + 8 * i + 4 * hh;
          f32x4 w = {oacc[dt][qt][4 * i] * inv, oacc[dt][qt][4 * i + 1] * inv,
                     oacc[dt][qt][4 * i + 2] * inv, oacc[dt][qt][4 * i + 3] * inv};
          *(f32x4*)(po + d) = w;
        }
      if (hh == 0) a.part_lse[(int64_t)it.part * kRows + lrow] = lse2;
    }
  }
}

// Combine the key-range partials of split work items by their log-sum-exp.
struct MergeArgs {
  const float* part_o;
  const float* part_lse;
  const MergeGroup* groups;
  const SeqDesc* seqs;
  uint16_t* o;
  float* lse;
  int32_t Hq, G;
  int32_t rows;              // rows per work item
};

// grid: x = merge group, y = 32-row slice of the group's rows.  Thread
// (row, c) of a block merges 16 consecutive d of one row: every partial's
// 64-byte piece of that row is read with four 16-byte loads, the LSE of the
// row once per partial.
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
  const MergeGroup g = a.groups[blockIdx.x];
  const SeqDesc sd = a.seqs[g.seq];
  const int rows_total = sd.q_len * a.G;
  const int lrow = blockIdx.y * 32 + (threadIdx.x >> 3);
  const int d0 = (threadIdx.x & 7) * 16;
  const int r = g.row0 + lrow;
  if (lrow >= a.rows || r >= rows_total) return;
  float mx = -INFINITY;
  for (int s = 0; s < g.nsplit; ++s) mx = fmaxf(mx, a.part_lse[(int64_t)(g.part0 + s) * a.rows + lrow]);
  f32x4 num[4] = {};
  float den = 0.f;
  if (mx != -INFINITY) {
#pragma unroll 2
    for (int s = 0; s < g.nsplit; ++s) {
      const int64_t p = (int64_t)(g.part0 + s) * a.rows + lrow;
      const float w = exp2f_fast(a.part_lse[p] - mx);
      const f32x4* src = (const f32x4*)(a.part_o + p * kHD + d0);
      den += w;
#pragma unroll
      for (int c = 0; c < 4; ++c) num[c] += w * src[c];
    }
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
  const int tok = r / a.G;
  const int head = g.kvh * a.G + (r - tok * a.G);
  const int64_t orow = (int64_t)(sd.q_start + tok) * a.Hq + head;
#pragma unroll
  for (int c = 0; c < 4; ++c)
    st_bf16x4(a.o + orow * kHD + d0 + 4 * c, num[c][0] * inv, num[c][1] * inv, num[c][2] * inv, num[c][3] * inv);
  if (a.lse != nullptr && d0 == 0)
    a.lse[orow] = den > 0.f ? (mx + __builtin_amdgcn_logf(den)) * 0.69314718055994531f : -INFINITY;
}

}  // namespace sa
