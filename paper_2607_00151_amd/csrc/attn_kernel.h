// Paged causal grouped-query prefill attention for gfx950 (CDNA4).
//
// One work item = one (sequence, KV head, tile of 128 query rows, key range).
// Query rows of a KV head are its G query heads packed per token:
// row r <-> (segment token r / G, query head kvh*G + r % G), so every K/V tile
// staged in LDS serves all G heads of the group.  Each of the 4 waves owns 32
// rows.  Keys advance in tiles of 64.
//
// Per tile and wave (all in registers except the K/V tile):
//   S^T[64 keys x 32 rows] = K_tile . Q^T      2 x 8 v_mfma_f32_32x32x16_bf16
//   online softmax in the exp2 domain          lane l owns row l % 32: its
//                                              32 scores per tile sit in its own
//                                              registers plus lane l ^ 32
//   O^T[128 d x 32 rows] += V^T . P^T          4 x 4 v_mfma_f32_32x32x16_bf16
// Computing the transposed products keeps one row's statistics on one lane
// pair, so the row max needs a single cross-half exchange and the rescale of
// O^T is a per-lane scalar multiply.
//
// The accumulator layout of a 32x32 MFMA puts, for lane l (h = l / 32), the
// keys 8i + 4h + j (i, j in 0..3) of the 32-key block into accumulator 4i + j.
// The P^T operand of the PV product is fed straight from those registers: the
// k-slots of lane half h carry keys {4h..4h+3, 8+4h..8+4h+3} of each 16-key
// group.  The V^T operand must use the same key order, which the LDS layout of
// V provides: V is stored transposed ([d][key]) with the middle two 4-key
// quads of every 16-key group swapped, so each lane's 8 keys are one 16-byte
// LDS read.  Both K and V^T rows are XOR-swizzled in 16-byte units to spread a
// wave's reads over all LDS banks.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace sa {

constexpr int kHD = 128;          // head dim
constexpr int kKT = 64;           // keys per tile
constexpr int kWaves = 4;
constexpr int kRows = 32 * kWaves;  // query rows per work item
constexpr int kThreads = 64 * kWaves;

struct AttnItem {
  int32_t seq;
  int32_t kvh;
  int32_t row0;      // first packed row
  int32_t kv_begin;  // first key, multiple of kKT
  int32_t kv_end;    // one past the last key this item reads (<= kv_len)
  int32_t part;      // -1: final output; else index of this item's partial slot
};

struct SeqDesc {
  int32_t q_start;   // first token of the sequence in Q / O
  int32_t q_len;
  int32_t kv_len;
  int32_t pad;
};

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;        // pools offset to the layer
  const uint16_t* v;
  uint16_t* o;
  float* lse;               // nullable
  float* part_o;            // [parts][kRows][kHD] normalised partial outputs
  float* part_lse;          // [parts][kRows] log2-domain LSE of each partial
  const AttnItem* items;
  const SeqDesc* seqs;
  const int32_t* indptr;
  const int32_t* indices;
  int32_t* err;
  int64_t num_slots;
  int32_t n_items;
  int32_t Hq, Hkv, G;
  float c;                  // softmax_scale * log2(e)
};

__device__ __forceinline__ int swap_mid_quads(int x) { return ((x & 1) << 1) | (x >> 1); }

template <int P>
__global__ __launch_bounds__(kThreads, 2) void attn_kernel(AttnArgs a) {
  static_assert(P == 16 || P == 32, "page size");
  constexpr int kTileBytes = kKT * kHD * 2;                 // 16 KB
  __shared__ __attribute__((aligned(16))) uint8_t smem[4 * kTileBytes];  // 2 x (K, V^T)

  const AttnItem it = a.items[blockIdx.x];
  if (it.kv_begin >= it.kv_end) return;                     // padding item
  const SeqDesc sd = a.seqs[it.seq];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5;                                 // lane half
  const int G = a.G;
  const int rows_total = sd.q_len * G;
  const int pre = sd.kv_len - sd.q_len;

  // ---- this lane's query row
  const int r = it.row0 + wave * 32 + (lane & 31);
  const bool row_valid = r < rows_total;
  const int rr = row_valid ? r : rows_total - 1;
  const int tok = rr / G;
  const int head = it.kvh * G + (rr - tok * G);
  const int qpos = pre + tok;                               // last visible key

  // ---- wave-uniform bounds
  const int wrow0 = it.row0 + wave * 32;
  const bool wave_active = wrow0 < rows_total;
  const int wlast = min(wrow0 + 31, rows_total - 1);
  const int w_kv_end = min(it.kv_end, pre + wlast / G + 1);  // keys any row of the wave needs
  const int w_full = min(it.kv_end, pre + wrow0 / G + 1);    // keys below are visible to all rows

  // ---- Q operand (B of S^T = K Q^T): lane holds d-chunks 2ks + hh
  bf16x8 qop[8];
  {
    const uint16_t* qrow = a.q + ((int64_t)(sd.q_start + tok) * a.Hq + head) * kHD;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qop[ks] = ld_bf16x8(qrow + (2 * ks + hh) * 8);
  }

  // ---- page table of this sequence
  const int32_t pt_base = a.indptr[it.seq];
  const int32_t pt_count = a.indptr[it.seq + 1] - pt_base;
  const int64_t slot_stride = (int64_t)a.Hkv * P * kHD;     // elements per slot
  const int64_t head_off = (int64_t)it.kvh * P * kHD;

  // loader roles: K chunks (key (tid>>4) + 16i, chunk tid&15); V quads (keys 4(tid>>4)+i, chunk tid&15)
  const int ld_chunk = tid & 15;
  const int ld_key = tid >> 4;

  u32x4 kreg[4], vreg[4];

  auto slot_of = [&](int page) -> int64_t {
    // uniform page index; returns -1 for a page outside the table or a bad slot
    if (page >= pt_count) return -1;
    const int32_t s = a.indices[pt_base + page];
    if (s < 0 || (int64_t)s >= a.num_slots) return -1;
    return s;
  };

  auto load_tile = [&](int t) {
    const int ts = t * kKT;
    // K: load i covers keys ts + 16i .. ts + 16i + 15
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = ts + ld_key + 16 * i;
      const int page = (ts + 16 * i) / P;                   // uniform
      const int row = (ld_key + 16 * i) % P;
      u32x4 x = {0u, 0u, 0u, 0u};
      if (ts + 16 * i < it.kv_end) {
        const int64_t s = slot_of(page);
        if (s < 0) {
          if (lane == 0) atomicOr(a.err, 1);
        } else if (key < it.kv_end) {
          x = ld_u32x4(a.k + s * slot_stride + head_off + row * kHD + ld_chunk * 8);
        }
      }
      kreg[i] = x;
    }
    // V: this wave's quads hold keys ts + 16*wave .. ts + 16*wave + 15
    {
      const int page = (ts + 16 * wave) / P;               // uniform
      u32x4 z = {0u, 0u, 0u, 0u};
      int64_t s = -1;
      if (ts + 16 * wave < it.kv_end) {
        s = slot_of(page);
        if (s < 0 && lane == 0) atomicOr(a.err, 1);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = ts + 4 * ld_key + i;
        const int row = (4 * ld_key + i) % P;
        vreg[i] = (s >= 0 && key < it.kv_end)
                      ? ld_u32x4(a.v + s * slot_stride + head_off + row * kHD + ld_chunk * 8)
                      : z;
      }
    }
  };

  auto store_tile = [&](int buf) {
    uint8_t* kb = smem + buf * 2 * kTileBytes;
    uint8_t* vb = kb + kTileBytes;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = ld_key + 16 * i;
      *(u32x4*)(kb + key * 256 + ((ld_chunk ^ (key & 7)) << 4)) = kreg[i];
    }
    // transpose 4 keys x 8 d into 8 rows of 4 keys
    const int qa = ld_key;                                  // key quad 0..15
    const int pos = 16 * (qa >> 2) + 4 * swap_mid_quads(qa & 3);
    const int cidx = pos >> 3, half = (pos >> 2) & 1;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int d = ld_chunk * 8 + e;
      const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
      const uint32_t lo = __builtin_amdgcn_perm(vreg[1][e >> 1], vreg[0][e >> 1], sel);
      const uint32_t hi = __builtin_amdgcn_perm(vreg[3][e >> 1], vreg[2][e >> 1], sel);
      u32x2 w = {lo, hi};
      *(u32x2*)(vb + d * 128 + ((cidx ^ (d & 7)) << 4) + half * 8) = w;
    }
  };

  f32x16 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) oacc[dt] = f32x16{};
  float m = -INFINITY;    // running max, log2 domain
  float l = 0.f;          // this lane's share of the denominator

  const int t0 = it.kv_begin / kKT;
  const int t1 = (it.kv_end + kKT - 1) / kKT;
  load_tile(t0);
  for (int t = t0; t < t1; ++t) {
    const int buf = (t - t0) & 1;
    store_tile(buf);
    __syncthreads();
    if (t + 1 < t1) load_tile(t + 1);
    const int ts = t * kKT;
    if (wave_active && ts < w_kv_end) {
      const uint8_t* kb = smem + buf * 2 * kTileBytes;
      const uint8_t* vb = kb + kTileBytes;
      f32x16 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        s[kt] = f32x16{};
        const int key = 32 * kt + (lane & 31);
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const bf16x8 kop = *(const bf16x8*)(kb + key * 256 + (((2 * ks + hh) ^ (key & 7)) << 4));
          s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[ks], s[kt], 0, 0, 0);
        }
      }
      // mask keys past this row's position or past the item's range
      if (ts + kKT > w_full) {
        const int lim = min(qpos, it.kv_end - 1);
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = ts + 32 * kt + 8 * (e >> 2) + 4 * hh + (e & 3);
            if (key > lim) s[kt][e] = -INFINITY;
          }
      }
      float mx = s[0][0];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m, mx * a.c);
      const float alpha = (m_new == -INFINITY) ? 1.f : exp2f_fast(m - m_new);
      const float msub = (m_new == -INFINITY) ? 0.f : m_new;
      m = m_new;
      if (__ballot(alpha != 1.f)) {
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int e = 0; e < 16; ++e) oacc[dt][e] *= alpha;
      }
      float lsum = 0.f;
      bf16x8 pop[4];
#pragma unroll
      for (int kb2 = 0; kb2 < 4; ++kb2) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float p = exp2f_fast(__builtin_fmaf(s[kb2 >> 1][8 * (kb2 & 1) + e], a.c, -msub));
          lsum += p;
          pop[kb2][e] = (__bf16)p;
        }
      }
      l = l * alpha + lsum;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int d = 32 * dt + (lane & 31);
#pragma unroll
        for (int kb2 = 0; kb2 < 4; ++kb2) {
          const bf16x8 vop = *(const bf16x8*)(vb + d * 128 + (((2 * kb2 + hh) ^ (d & 7)) << 4));
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pop[kb2], oacc[dt], 0, 0, 0);
        }
      }
    }
  }

  if (!wave_active) return;
  const float l_tot = l + __shfl_xor(l, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse2 = l_tot > 0.f ? m + __builtin_amdgcn_logf(l_tot) : -INFINITY;
  if (it.part < 0) {
    if (row_valid) {
      uint16_t* orow = a.o + ((int64_t)(sd.q_start + tok) * a.Hq + head) * kHD;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d = 32 * dt + 8 * i + 4 * hh;
          st_bf16x4(orow + d, oacc[dt][4 * i] * inv, oacc[dt][4 * i + 1] * inv,
                    oacc[dt][4 * i + 2] * inv, oacc[dt][4 * i + 3] * inv);
        }
      if (a.lse != nullptr && hh == 0)
        a.lse[(int64_t)(sd.q_start + tok) * a.Hq + head] = lse2 * 0.69314718055994531f;
    }
  } else {
    const int lrow = wave * 32 + (lane & 31);
    float* po = a.part_o + ((int64_t)it.part * kRows + lrow) * kHD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = 32 * dt + 8 * i + 4 * hh;
        f32x4 w = {oacc[dt][4 * i] * inv, oacc[dt][4 * i + 1] * inv, oacc[dt][4 * i + 2] * inv,
                   oacc[dt][4 * i + 3] * inv};
        *(f32x4*)(po + d) = w;
      }
    if (hh == 0) a.part_lse[(int64_t)it.part * kRows + lrow] = lse2;
  }
}

// Combine the key-range partials of split work items by their log-sum-exp.
struct MergeGroup {
  int32_t seq, kvh, row0, nsplit, part0, pad;
};

struct MergeArgs {
  const float* part_o;
  const float* part_lse;
  const MergeGroup* groups;
  const SeqDesc* seqs;
  uint16_t* o;
  float* lse;
  int32_t Hq, G;
};

__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
  const MergeGroup g = a.groups[blockIdx.x];
  const SeqDesc sd = a.seqs[g.seq];
  const int rows_total = sd.q_len * a.G;
  for (int idx = threadIdx.x; idx < kRows * kHD; idx += 256) {
    const int lrow = idx / kHD, d = idx % kHD;
    const int r = g.row0 + lrow;
    if (r >= rows_total) continue;
    float mx = -INFINITY;
    for (int s = 0; s < g.nsplit; ++s) mx = fmaxf(mx, a.part_lse[(int64_t)(g.part0 + s) * kRows + lrow]);
    float num = 0.f, den = 0.f;
    if (mx != -INFINITY) {
      for (int s = 0; s < g.nsplit; ++s) {
        const int64_t p = (int64_t)(g.part0 + s) * kRows + lrow;
        const float w = exp2f_fast(a.part_lse[p] - mx);
        den += w;
        num += w * a.part_o[p * kHD + d];
      }
    }
    const int tok = r / a.G;
    const int head = g.kvh * a.G + (r - tok * a.G);
    const int64_t orow = (int64_t)(sd.q_start + tok) * a.Hq + head;
    a.o[orow * kHD + d] = f32_to_bf16_rne(den > 0.f ? num / den : 0.f);
    if (a.lse != nullptr && d == 0)
      a.lse[orow] = den > 0.f ? (mx + __builtin_amdgcn_logf(den)) * 0.69314718055994531f : -INFINITY;
  }
}

}  // namespace sa
