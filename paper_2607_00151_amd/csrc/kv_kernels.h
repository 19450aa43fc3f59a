// Bandwidth-bound page kernels: segment append (scatter) and commit-splice
// assembly (whole-page gather into fresh slots).  Both move 16-byte chunks
// with every lane of a wave on consecutive addresses, and range-check every
// page id before touching memory.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"
#include "plan.h"

namespace sa {

// ---------------------------------------------------------------- append

struct AppendArgs {
  uint16_t* k_pool;          // offset to the layer
  uint16_t* v_pool;
  const uint16_t* k_new;     // [sum new][Hkv][128]
  const uint16_t* v_new;
  const int32_t* tok_begin;  // [B + 1] first new token of each sequence
  const int32_t* start;      // [B] logical position of each sequence's first new token
  const int32_t* indptr;
  const int32_t* indices;
  int32_t* err;
  int64_t num_slots;
  int64_t total_chunks;      // sum new * Hkv * 16
  int32_t B, Hkv, P;
};

// Largest b with tok_begin[b] <= t (tok_begin is non-decreasing).
__device__ __forceinline__ int find_seq(const int32_t* tok_begin, int B, int t) {
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (tok_begin[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

constexpr int kAppendChunksPerThread = 4;

// Batches of kSeqLdsMin to kSeqLds sequences: a block first copies the
// per-sequence records its threads look up (token offsets, positions,
// page-table offsets) into LDS with one coalesced read, so finding a token's
// sequence is a search in LDS rather than a chain of dependent global loads
// (seven for a batch of 68 sequences: 1.4x the append rate measured there).
// Smaller batches search the global arrays directly, where the search is
// short and the barrier would cost more than it saves (a single sequence:
// ~2% slower staged); larger ones too.
constexpr int kSeqLdsMin = 8;
constexpr int kSeqLds = 1024;
__device__ __forceinline__ bool stage_seqs(int B) { return B >= kSeqLdsMin && B <= kSeqLds; }

// Each thread resolves the slots of its chunks first, then issues every load,
// then every store: the stores may alias the new rows as far as the compiler
// knows, so a load placed after a store would wait for it.  tb, st, ip: the
// token offsets, start positions and page-table offsets, in LDS or global.
__device__ __forceinline__ void append_rows(const AppendArgs& a, const int32_t* tb, const int32_t* st,
                                            const int32_t* ip) {
  const int per_tok = a.Hkv * 16;
  int64_t dst[kAppendChunksPerThread];
#pragma unroll
  for (int u = 0; u < kAppendChunksPerThread; ++u) {
    const int64_t c = ((int64_t)blockIdx.x * kAppendChunksPerThread + u) * 256 + threadIdx.x;
    dst[u] = -1;
    if (c >= a.total_chunks) continue;
    const int t = (int)(c / per_tok);
    const int rem = (int)(c - (int64_t)t * per_tok);
    const int g = rem >> 4, ch = rem & 15;
    const int b = find_seq(tb, a.B, t);
    const int x = st[b] + (t - tb[b]);
    const int page = x / a.P, row = x - page * a.P;
    const int32_t base = ip[b];
    if (page >= ip[b + 1] - base) { atomicOr(a.err, 2); continue; }
    const int32_t slot = a.indices[base + page];
    if (slot < 0 || (int64_t)slot >= a.num_slots) { atomicOr(a.err, 2); continue; }
    dst[u] = (((int64_t)slot * a.Hkv + g) * a.P + row) * 128 + ch * 8;
  }
  u32x4 kx[kAppendChunksPerThread], vx[kAppendChunksPerThread];
#pragma unroll
  for (int u = 0; u < kAppendChunksPerThread; ++u)
    if (dst[u] >= 0) {
      const int64_t c = ((int64_t)blockIdx.x * kAppendChunksPerThread + u) * 256 + threadIdx.x;
      kx[u] = ld_u32x4(a.k_new + c * 8);
      vx[u] = ld_u32x4(a.v_new + c * 8);
    }
#pragma unroll
  for (int u = 0; u < kAppendChunksPerThread; ++u)
    if (dst[u] >= 0) {
      st_u32x4(a.k_pool + dst[u], kx[u]);
      st_u32x4(a.v_pool + dst[u], vx[u]);
    }
}

__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
  __shared__ int32_t s_tb[kSeqLds + 1], s_st[kSeqLds], s_ip[kSeqLds + 1];
  if (stage_seqs(a.B)) {
    for (int i = (int)threadIdx.x; i <= a.B; i += 256) {
      s_tb[i] = a.tok_begin[i];
      s_ip[i] = a.indptr[i];
      if (i < a.B) s_st[i] = a.start[i];
    }
    __syncthreads();
    append_rows(a, s_tb, s_st, s_ip);
  } else {
    append_rows(a, a.tok_begin, a.start, a.indptr);
  }
}

// ---------------------------------------------------------------- assemble

// One copied page: which sequence, its logical source page, and its position
// in the destination table (also its index into the fresh-slot list).
struct AsmArgs {
  const uint16_t* k_src;
  const uint16_t* v_src;
  uint16_t* k_dst;
  uint16_t* v_dst;
  const AsmUnit* units;        // [n_units]
  const int32_t* dst_indptr;   // [B + 1] plan copy of the destination table offsets
  const int32_t* src_indptr;
  const int32_t* src_indices;
  const int32_t* fresh;
  int32_t* out_indptr;         // [B + 1]
  int32_t* out_indices;        // [n_dst]
  int32_t* err;
  int64_t num_slots;
  int64_t slot_elems;          // Hkv * P * 128
  int64_t layer_elems;         // num_slots * slot_elems
  int32_t n_units, n_dst, B;
  // append of a segment in the same launch (app_layer < 0: none).  Blocks
  // 0 .. app_blocks - 1 of that layer write the new rows that land on fresh
  // pages (they go first: their address chains are the longest); blocks
  // app_blocks .. app_blocks + n_units - 1 copy pages.  Tokens are listed per
  // sequence like the append plan:
  const uint16_t* k_new;       // [sum new][Hkv][128]
  const uint16_t* v_new;
  const int32_t* app_tok_begin;  // [B + 1] first listed token of each sequence
  const int32_t* app_start;      // [B] its logical position in the replacement cache
  const int32_t* app_knew;       // [B] its row in k_new / v_new
  int64_t app_chunks;            // listed tokens * Hkv * 16
  int32_t app_layer, app_blocks, Hkv, P;
};

constexpr int kAsmThreads = 512;
constexpr int kAsmDepth = 4;   // 16-byte chunks of K (and of V) in flight per thread

// Page copies stream through with non-temporal loads and stores (measured the
// faster pairing for this scattered whole-page copy on MI355X).
__device__ __forceinline__ u32x4 ld_stream(const uint16_t* p) {
  return __builtin_nontemporal_load((const u32x4*)p);
}
__device__ __forceinline__ void st_stream(uint16_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, (u32x4*)p);
}

// One page pair, kAsmDepth chunks of K and of V in flight per thread.  kMix:
// the partial last surviving page of an append, whose rows
// [app_row0, app_row0 + app_rows) are taken from the new rows instead.
template <bool kMix>
__device__ __forceinline__ void copy_page(const AsmArgs& a, const AsmUnit& un, const uint16_t* ks,
                                          const uint16_t* vs, uint16_t* kd, uint16_t* vd, int tid) {
  const int n_chunks = (int)(a.slot_elems / 8);
  for (int base = 0; base < n_chunks; base += kAsmThreads * kAsmDepth) {
    u32x4 kx[kAsmDepth], vx[kAsmDepth];
#pragma unroll
    for (int j = 0; j < kAsmDepth; ++j) {
      const int c = base + j * kAsmThreads + tid;
      if (c < n_chunks) {
        const uint16_t* kp = ks + c * 8;
        const uint16_t* vp = vs + c * 8;
        if (kMix) {
          const int g = c / (a.P * 16), r = (c >> 4) % a.P - un.app_row0;
          if (r >= 0 && r < un.app_rows) {
            const int64_t src = ((int64_t)(un.app_tok + r) * a.Hkv + g) * 128 + (c & 15) * 8;
            kp = a.k_new + src;
            vp = a.v_new + src;
          }
        }
        kx[j] = ld_stream(kp);
        vx[j] = ld_stream(vp);
      }
    }
#pragma unroll
    for (int j = 0; j < kAsmDepth; ++j) {
      const int c = base + j * kAsmThreads + tid;
      if (c < n_chunks) {
        st_stream(kd + c * 8, kx[j]);
        st_stream(vd + c * 8, vx[j]);
      }
    }
  }
}

// The append part of a splice + append launch, block u of the append layer:
// new rows onto fresh pages (the destination table is the free list in order,
// so the slot comes from it, not from the table being written).  All
// addresses are resolved first, then every load is issued, then every store,
// so no chunk waits behind another chunk's store.  tb, st, kn, ip: the listed
// token offsets, logical positions, rows in k_new / v_new and destination
// table offsets of the sequences, in LDS or global.
__device__ __forceinline__ void assemble_append_rows(const AsmArgs& a, int u, int layer, const int32_t* tb,
                                                     const int32_t* st, const int32_t* kn, const int32_t* ip) {
  const int tid = threadIdx.x;
  const int per_tok = a.Hkv * 16;
  const int64_t lo = (int64_t)layer * a.layer_elems;
  int64_t src[kAsmDepth], dst[kAsmDepth];
#pragma unroll
  for (int j = 0; j < kAsmDepth; ++j) {
    const int64_t c = ((int64_t)u * kAsmDepth + j) * kAsmThreads + tid;
    src[j] = -1;
    if (c >= a.app_chunks) continue;
    const int t = (int)(c / per_tok);
    const int rem = (int)(c - (int64_t)t * per_tok);
    const int g = rem >> 4, ch = rem & 15;
    const int b = find_seq(tb, a.B, t);
    const int x = st[b] + (t - tb[b]);
    const int page = x / a.P, row = x - page * a.P;
    if (page >= ip[b + 1] - ip[b]) { atomicOr(a.err, 2); continue; }
    const int32_t slot = a.fresh[ip[b] + page];
    if (slot < 0 || (int64_t)slot >= a.num_slots) { atomicOr(a.err, 2); continue; }
    src[j] = ((int64_t)(kn[b] + (t - tb[b])) * a.Hkv + g) * 128 + ch * 8;
    dst[j] = lo + (((int64_t)slot * a.Hkv + g) * a.P + row) * 128 + ch * 8;
  }
  u32x4 kx[kAsmDepth], vx[kAsmDepth];
#pragma unroll
  for (int j = 0; j < kAsmDepth; ++j)
    if (src[j] >= 0) {
      kx[j] = ld_stream(a.k_new + src[j]);
      vx[j] = ld_stream(a.v_new + src[j]);
    }
#pragma unroll
  for (int j = 0; j < kAsmDepth; ++j)
    if (src[j] >= 0) {
      st_stream(a.k_dst + dst[j], kx[j]);
      st_stream(a.v_dst + dst[j], vx[j]);
    }
}

// grid: x = max(app_blocks + units, table blocks), y = layer.  One block of 512 threads
// copies one page of one layer, slot_elems * 2 bytes of K and as many of V,
// with every chunk of a 32 KiB page pair in flight at once (512 threads were
// measured ~4% faster than 256 for this copy on MI355X).  A unit's slots take
// two dependent reads: its source page-table offset, then the slot.
__global__ __launch_bounds__(kAsmThreads) void assemble_kernel(AsmArgs a) {
  __shared__ int32_t s_tb[kSeqLds + 1], s_st[kSeqLds], s_kn[kSeqLds], s_ip[kSeqLds + 1];
  int u = blockIdx.x;
  const int layer = blockIdx.y;
  const int tid = threadIdx.x;

  // the destination table (layer 0 blocks write disjoint slices of it)
  if (layer == 0) {
    const int idx = u * kAsmThreads + tid;
    if (idx < a.n_dst) a.out_indices[idx] = a.fresh[idx];
    if (idx <= a.B) a.out_indptr[idx] = a.dst_indptr[idx];
  }
  if (u < a.app_blocks) {
    if (layer != a.app_layer) return;
    if (stage_seqs(a.B)) {
      for (int i = tid; i <= a.B; i += kAsmThreads) {
        s_tb[i] = a.app_tok_begin[i];
        s_ip[i] = a.dst_indptr[i];
        if (i < a.B) {
          s_st[i] = a.app_start[i];
          s_kn[i] = a.app_knew[i];
        }
      }
      __syncthreads();
      assemble_append_rows(a, u, layer, s_tb, s_st, s_kn, s_ip);
    } else {
      assemble_append_rows(a, u, layer, a.app_tok_begin, a.app_start, a.app_knew, a.dst_indptr);
    }
    return;
  }
  u -= a.app_blocks;
  if (u >= a.n_units) return;

  const AsmUnit un = a.units[u];
  const int32_t sbase = a.src_indptr[un.seq];
  const int32_t scount = a.src_indptr[un.seq + 1] - sbase;
  const int32_t d_slot = a.fresh[un.dst_index];
  if (un.src_page >= scount) { if (tid == 0) atomicOr(a.err, 4); return; }
  const int32_t s_slot = a.src_indices[sbase + un.src_page];
  if (s_slot < 0 || (int64_t)s_slot >= a.num_slots || d_slot < 0 || (int64_t)d_slot >= a.num_slots) {
    if (tid == 0) atomicOr(a.err, 4);
    return;
  }
  const int64_t lo_off = (int64_t)layer * a.layer_elems;
  const uint16_t* ks = a.k_src + lo_off + (int64_t)s_slot * a.slot_elems;
  const uint16_t* vs = a.v_src + lo_off + (int64_t)s_slot * a.slot_elems;
  uint16_t* kd = a.k_dst + lo_off + (int64_t)d_slot * a.slot_elems;
  uint16_t* vd = a.v_dst + lo_off + (int64_t)d_slot * a.slot_elems;
  if (layer == a.app_layer && un.app_rows > 0)
    copy_page<true>(a, un, ks, vs, kd, vd, tid);
  else
    copy_page<false>(a, un, ks, vs, kd, vd, tid);
}

// ---------------------------------------------------------------- zero-copy splice

struct AliasArgs {
  const AsmUnit* units;        // surviving pages (sequence, source page)
  const int32_t* entry;        // [n_dst] unit index, or -(fresh position + 1) for a reserved page
  const int32_t* dst_indptr;   // [B + 1] plan copy of the destination table offsets
  const int32_t* src_indptr;
  const int32_t* src_indices;
  const int32_t* fresh;
  int32_t* out_indptr;
  int32_t* out_indices;
  int32_t* err;
  int64_t num_slots;
  int32_t n_dst, B;
};

// One thread per destination table entry: a surviving page's entry is its
// source slot, a reserved page's entry the next fresh slot.  Nothing is copied.
// A missing source page or a slot outside [0, num_slots) raises the error
// flag (the entry is written as -1 for a missing page, as found otherwise).
__global__ __launch_bounds__(256) void splice_alias_kernel(AliasArgs a) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e <= a.B) a.out_indptr[e] = a.dst_indptr[e];
  if (e >= a.n_dst) return;
  const int32_t code = a.entry[e];
  int32_t slot;
  if (code >= 0) {
    const AsmUnit un = a.units[code];
    const int32_t sbase = a.src_indptr[un.seq];
    const int32_t scount = a.src_indptr[un.seq + 1] - sbase;
    slot = un.src_page < scount ? a.src_indices[sbase + un.src_page] : -1;
  } else {
    slot = a.fresh[-code - 1];
  }
  if (slot < 0 || (int64_t)slot >= a.num_slots) atomicOr(a.err, 4);
  a.out_indices[e] = slot;
}

}  // namespace sa
