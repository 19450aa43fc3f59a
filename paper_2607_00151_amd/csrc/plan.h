// Host-side planning behind the C ABI: argument validation, the commit
// splice's page plan and the attention launch's work list.  Plain C++17 with
// no HIP dependency: the library includes it, and the host tests build it on
// its own under AddressSanitizer and UndefinedBehaviorSanitizer to check the
// plans' invariants on many shapes without a GPU.
//
// The records defined here are also the device-side plan formats (uploaded
// as bytes and read by the kernels), so they are plain int32 structs.
#pragma once

#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <map>
#include <string>
#include <vector>

#include "sa.h"

namespace sa {

constexpr int kHD = 128;          // head dim
constexpr int kKT = 64;           // keys per attention tile
constexpr int kMaxRows = 256;     // largest query-row tile of a work item
constexpr int kNumXcd = 8;        // MI355X: 8 accelerator complex dies, 32 CUs each
// Items of at most this many packed query rows (decode requests: one token,
// G query heads) take the kernel's decode path, which spreads the item's keys
// over the block's four waves instead of its rows.
constexpr int kDecodeRows = 32;

// One attention work item: a tile of packed query rows of one (sequence, KV
// head) over a key range.
struct AttnItem {
  int32_t seq;
  int32_t kvh;
  int32_t row0;      // first packed row
  int32_t kv_begin;  // first key, multiple of kKT
  int32_t kv_end;    // one past the last key this item reads (<= kv_len)
  int32_t part;      // -1: final output; else index of this item's partial slot
  int32_t boost;     // steps at the start that run at raised wave priority (0: none)
  int32_t q_start;   // the sequence's SeqDesc fields, repeated so that one read
  int32_t q_len;     // of the item gives a workgroup all it needs to start
  int32_t kv_len;
};

struct SeqDesc {
  int32_t q_start;   // first token of the sequence in Q / O
  int32_t q_len;
  int32_t kv_len;
  int32_t pad;
};

// The key-range parts of one split work item, merged by log-sum-exp.
struct MergeGroup {
  int32_t seq, kvh, row0, nsplit, part0, pad;
};

// One surviving page of a commit splice.
struct AsmUnit {
  int32_t seq;
  int32_t src_page;
  int32_t dst_index;
  // with an append in the same launch: rows app_row0 .. app_row0 + app_rows - 1
  // of this page (the last surviving one, when partial) come from new-row
  // token app_tok onwards instead of from the source page
  int32_t app_row0, app_rows, app_tok;
};

inline sa_status plan_fail(std::string& err, sa_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  err = buf;
  return s;
}

inline int64_t slot_elems(const sa_layout* L) { return (int64_t)L->num_kv_heads * L->page_size * kHD; }
inline int64_t layer_elems(const sa_layout* L) { return L->num_slots * slot_elems(L); }

inline sa_status check_layout(const sa_layout* L, std::string& err) {
  if (!L) return plan_fail(err, SA_ERR_NULL, "layout is NULL");
  if (L->num_q_heads <= 0 || L->num_kv_heads <= 0 || L->num_layers <= 0 || L->num_slots <= 0)
    return plan_fail(err, SA_ERR_SHAPE, "layout: heads, layers and slots must be positive");
  if (L->num_q_heads % L->num_kv_heads != 0)
    return plan_fail(err, SA_ERR_SHAPE, "layout: num_q_heads %d is not a multiple of num_kv_heads %d",
                     L->num_q_heads, L->num_kv_heads);
  if (L->head_dim != kHD) return plan_fail(err, SA_ERR_UNSUPPORTED, "head_dim %d (only 128)", L->head_dim);
  if (L->page_size != 16 && L->page_size != 32)
    return plan_fail(err, SA_ERR_UNSUPPORTED, "page_size %d (only 16 or 32)", L->page_size);
  if (L->num_slots > INT32_MAX || L->num_slots > (INT64_MAX / 4) / slot_elems(L) / L->num_layers)
    return plan_fail(err, SA_ERR_SHAPE, "layout: pool too large");
  return SA_OK;
}

// ------------------------------------------------------------ commit splice

// Host plan of a commit splice: validated spans, one record per surviving
// page, and the destination table's offsets.  With `alias`, surviving pages
// keep their source slots and only the reserved pages take fresh slots.
struct SplicePlan {
  std::vector<AsmUnit> units;          // surviving pages, in destination order
  std::vector<int32_t> dst_indptr, dst_len;
  std::vector<int32_t> entry;          // alias: per destination entry, unit index or -(fresh position + 1)
  int64_t n_dst = 0, fresh_used = 0;
};

inline sa_status plan_splice(const sa_layout* layout, int32_t batch, const int32_t* h_src_len,
                             const int32_t* h_keep_indptr, const int32_t* h_keep_spans, const int32_t* h_reserve,
                             bool alias, int32_t num_fresh, int32_t dst_capacity, SplicePlan& out,
                             std::string& err) {
  sa_status s = check_layout(layout, err);
  if (s != SA_OK) return s;
  if (batch < 1) return plan_fail(err, SA_ERR_SHAPE, "batch %d < 1", batch);
  if (!h_src_len || !h_keep_indptr || !h_reserve) return plan_fail(err, SA_ERR_NULL, "a host length array is NULL");
  if (h_keep_indptr[0] != 0) return plan_fail(err, SA_ERR_SHAPE, "keep_indptr[0] must be 0");
  for (int b = 0; b < batch; ++b)
    if (h_keep_indptr[b + 1] < h_keep_indptr[b])
      return plan_fail(err, SA_ERR_SHAPE, "keep_indptr decreases at %d", b);
  if (h_keep_indptr[batch] > 0 && !h_keep_spans) return plan_fail(err, SA_ERR_NULL, "h_keep_spans is NULL");
  if (num_fresh < 0 || dst_capacity < 0) return plan_fail(err, SA_ERR_SHAPE, "negative capacity");
  const int P = layout->page_size;
  out = SplicePlan{};
  out.dst_indptr.assign(batch + 1, 0);
  out.dst_len.assign(batch, 0);
  int64_t n_dst = 0, fresh_used = 0;
  for (int b = 0; b < batch; ++b) {
    if (h_src_len[b] < 0 || h_reserve[b] < 0)
      return plan_fail(err, SA_ERR_SHAPE, "sequence %d: src_len %d, reserve %d", b, h_src_len[b], h_reserve[b]);
    const int n_src_pages = (int)(((int64_t)h_src_len[b] + P - 1) / P);
    int prev_end = 0;
    int64_t kept_pages = 0, kept = 0;
    for (int k = h_keep_indptr[b]; k < h_keep_indptr[b + 1]; ++k) {
      const int beg = h_keep_spans[2 * k], end = h_keep_spans[2 * k + 1];
      if (beg < prev_end || beg >= end || end > n_src_pages)
        return plan_fail(err, SA_ERR_RANGE, "sequence %d: keep span [%d, %d) invalid (previous end %d, %d pages)",
                         b, beg, end, prev_end, n_src_pages);
      for (int p = beg; p < end; ++p) {
        if (alias) out.entry.push_back((int32_t)out.units.size());
        out.units.push_back({b, p, (int32_t)(n_dst + kept_pages + (p - beg)), 0, 0, 0});
        kept += std::min<int64_t>(P, (int64_t)h_src_len[b] - (int64_t)p * P);
      }
      kept_pages += end - beg;
      prev_end = end;
    }
    const int64_t pages_b = std::max<int64_t>(kept_pages, (kept + h_reserve[b] + P - 1) / P);
    const int64_t fresh_b = alias ? pages_b - kept_pages : pages_b;
    if (alias)
      for (int64_t j = 0; j < fresh_b; ++j) out.entry.push_back((int32_t)(-(fresh_used + j) - 1));
    out.dst_len[b] = (int32_t)kept;
    n_dst += pages_b;
    fresh_used += fresh_b;
    if (n_dst > INT32_MAX || fresh_used > INT32_MAX) return plan_fail(err, SA_ERR_SHAPE, "destination table too large");
    out.dst_indptr[b + 1] = (int32_t)n_dst;
  }
  if (fresh_used > num_fresh)
    return plan_fail(err, SA_ERR_NO_PAGES, "need %lld fresh slots, %d given", (long long)fresh_used, num_fresh);
  if (n_dst > dst_capacity)
    return plan_fail(err, SA_ERR_NO_PAGES, "destination table needs %lld entries, capacity %d", (long long)n_dst,
                     dst_capacity);
  out.n_dst = n_dst;
  out.fresh_used = fresh_used;
  return SA_OK;
}

// The append that rides with a copy splice: new rows that land on a partial
// last surviving page go with that page's copy (recorded in its unit); the
// rest are listed per sequence for the append blocks.
struct SpliceAppendPlan {
  std::vector<int32_t> tok_begin;      // [B + 1] first new token (of those the append blocks write) per sequence
  std::vector<int32_t> start;          // [B] logical position of that token
  std::vector<int32_t> knew;           // [B] its index among all new tokens
  int64_t total = 0;                   // tokens the append blocks write
  int64_t all_new = 0;                 // every new token
};

inline sa_status plan_splice_append(const sa_layout* layout, int32_t batch, const int32_t* h_new_len, int32_t layer,
                                    SplicePlan& sp, SpliceAppendPlan& out, std::string& err) {
  if (layer < 0 || layer >= layout->num_layers)
    return plan_fail(err, SA_ERR_SHAPE, "layer %d outside [0, %d)", layer, layout->num_layers);
  const int P = layout->page_size;
  out = SpliceAppendPlan{};
  out.tok_begin.assign(batch + 1, 0);
  out.start.assign(batch, 0);
  out.knew.assign(batch, 0);
  int64_t knew = 0, total = 0;
  size_t unit_end = 0;
  for (int b = 0; b < batch; ++b) {
    const int n = h_new_len[b];
    const int64_t pages_b = sp.dst_indptr[b + 1] - sp.dst_indptr[b];
    if (n < 0 || sp.dst_len[b] + (int64_t)n > pages_b * P)
      return plan_fail(err, SA_ERR_SHAPE, "sequence %d: %d new tokens after %d kept do not fit its %lld pages", b, n,
                       sp.dst_len[b], (long long)pages_b);
    while (unit_end < sp.units.size() && sp.units[unit_end].seq == b) ++unit_end;
    int first = 0;                                      // new tokens on the last surviving page
    if (n > 0 && sp.dst_len[b] % P != 0 && unit_end > 0 && sp.units[unit_end - 1].seq == b) {
      AsmUnit& last = sp.units[unit_end - 1];
      last.app_row0 = sp.dst_len[b] % P;
      last.app_rows = std::min(P - last.app_row0, n);
      last.app_tok = (int32_t)knew;
      first = last.app_rows;
    }
    out.tok_begin[b] = (int32_t)total;
    out.start[b] = sp.dst_len[b] + first;
    out.knew[b] = (int32_t)(knew + first);
    total += n - first;
    knew += n;
    if (knew > INT32_MAX / 2) return plan_fail(err, SA_ERR_SHAPE, "too many new tokens");
  }
  out.tok_begin[batch] = (int32_t)total;
  out.total = total;
  out.all_new = knew;
  return SA_OK;
}

// ---------------------------------------------------------------- attention

// Shape checks of an attention call and its sequence records.
inline sa_status plan_attn_check(const sa_layout* layout, int32_t layer, int32_t batch, const int32_t* h_q_len,
                                 const int32_t* h_kv_len, float softmax_scale, std::vector<SeqDesc>& seqs,
                                 int64_t& total_q, std::string& err) {
  sa_status s = check_layout(layout, err);
  if (s != SA_OK) return s;
  if (layer < 0 || layer >= layout->num_layers)
    return plan_fail(err, SA_ERR_SHAPE, "layer %d outside [0, %d)", layer, layout->num_layers);
  if (batch < 1) return plan_fail(err, SA_ERR_SHAPE, "batch %d < 1", batch);
  if (!h_q_len || !h_kv_len) return plan_fail(err, SA_ERR_NULL, "h_q_len / h_kv_len is NULL");
  if (!std::isfinite(softmax_scale) || softmax_scale <= 0.f)
    return plan_fail(err, SA_ERR_SHAPE, "softmax_scale must be finite and positive");
  const int G = layout->num_q_heads / layout->num_kv_heads;
  seqs.assign(batch, SeqDesc{0, 0, 0, 0});
  total_q = 0;
  for (int b = 0; b < batch; ++b) {
    if (h_q_len[b] < 0 || h_q_len[b] > h_kv_len[b])
      return plan_fail(err, SA_ERR_SHAPE, "sequence %d: need 0 <= q_len (%d) <= kv_len (%d)", b, h_q_len[b],
                       h_kv_len[b]);
    if ((int64_t)h_q_len[b] * G > INT32_MAX - kMaxRows)
      return plan_fail(err, SA_ERR_SHAPE, "sequence %d: q_len * G too large", b);
    seqs[b] = {(int32_t)total_q, h_q_len[b], h_kv_len[b], 0};
    total_q += h_q_len[b];
    if (total_q > INT32_MAX) return plan_fail(err, SA_ERR_SHAPE, "too many query tokens");
  }
  return SA_OK;
}

struct AttnShape {
  int rows_item = 128;       // packed query rows per work item
  int num_cu = 256;
  bool pair_rounds = true;   // two blocks share a CU (the dispatcher pairs block i with i + num_cu)
  int64_t max_parts = -1;    // cap on key-range parts of split items (-1: none)
};

// The relative XCD speeds of sa_set_xcd_weights and the last weighting's
// input and result: a launch repeating the same work reuses it.
struct XcdState {
  bool weighted = false;
  float speed[kNumXcd] = {1, 1, 1, 1, 1, 1, 1, 1};
  std::vector<std::vector<AttnItem>> in, out;
};

struct AttnPlan {
  std::vector<AttnItem> items;         // one per workgroup, in launch order (kv_begin >= kv_end: padding)
  std::vector<MergeGroup> groups;      // split items to merge
  int32_t n_parts = 0;
};

inline int64_t item_tiles(const AttnItem& it) { return (it.kv_end - it.kv_begin + kKT - 1) / kKT; }

// Longest first within each XCD's queue.
inline void sort_longest_first(std::vector<AttnItem>& q) {
  std::stable_sort(q.begin(), q.end(),
                   [](const AttnItem& x, const AttnItem& y) { return item_tiles(x) > item_tiles(y); });
}

// Key tiles of the most loaded CU of an XCD whose queue q is sorted longest
// first and runs in at most two rounds of `round` blocks, the second reversed
// (block k and block round + k share a CU): q[k] + q[n - 1 - k].
inline int64_t busiest_cu(const std::vector<AttnItem>& q, size_t round) {
  const size_t n = q.size();
  int64_t m = 0;
  for (size_t k = 0; k < std::min(n, round); ++k)
    m = std::max<int64_t>(m, item_tiles(q[k]) + (k + round < n ? item_tiles(q[n - 1 - k]) : 0));
  return m;
}

// The XCDs of one chip do not run equally fast under this load (measured:
// the slowest one's workgroups take ~5-7% longer than the fastest one's on
// the same work, whichever KV head it serves), and the launch ends with the
// slowest.  Given relative speeds, the XCDs are paired by speed -- the
// slowest with the fastest, the second slowest with the second fastest, and
// so on -- and within each pair work moves from the one whose busiest CU has
// the more key tiles per unit of speed to the other, by swapping the longest
// item of the first for the shortest of the second while neither ends above
// the first's present cost.  Every XCD keeps its number of items, so the
// launch keeps its rounds.  An item that moves reads another KV head's K/V
// than its XCD's others, through that XCD's L2: keeping the exchanges inside
// fixed pairs bounds those foreign KV heads at one per XCD (measured at c2:
// a search over all XCDs reached 20-28 foreign (KV head, XCD) pairs and 2.6x
// the HBM reads of the unweighted launch for ~0.5% more balance).
// Queues of at most two rounds come back sorted longest first.
inline void weigh_xcds(std::vector<std::vector<AttnItem>>& queue, size_t round, const float* speed) {
  // More than two rounds: each XCD's CUs take its items as they free; moving
  // the last items of the most loaded XCD to the least loaded one was tried
  // and measured -1.5% to +1.4% on 16 ragged contexts and on a 64K-key
  // context, so those launches are left as placed.
  for (const auto& q : queue)
    if (q.size() > 2 * round) return;
  for (auto& q : queue) sort_longest_first(q);
  int order[kNumXcd];
  for (int x = 0; x < kNumXcd; ++x) order[x] = x;
  std::stable_sort(order, order + kNumXcd, [&](int a, int b) { return speed[a] < speed[b]; });
  for (int k = 0; k < kNumXcd / 2; ++k) {
    const int x0 = order[k], x1 = order[kNumXcd - 1 - k];
    double c0 = busiest_cu(queue[x0], round) / speed[x0], c1 = busiest_cu(queue[x1], round) / speed[x1];
    for (int iter = 0; iter < 4096 && c0 != c1; ++iter) {
      const bool first = c0 > c1;               // the more loaded of the pair gives
      const int s = first ? x0 : x1, f = first ? x1 : x0;
      const double cs = first ? c0 : c1;
      auto& qs = queue[s];
      auto& qf = queue[f];
      if (qs.empty() || qf.empty() || item_tiles(qs.front()) <= item_tiles(qf.back())) break;
      std::vector<AttnItem> ns = qs, nf = qf;
      std::swap(ns.front(), nf.back());
      sort_longest_first(ns);
      sort_longest_first(nf);
      // a swap may leave s's busiest CU where it was (another CU of s carries as
      // much): it is taken as long as neither XCD ends above s's present cost,
      // since it lowers s's total and the next swaps then lower that CU
      const double ns_c = busiest_cu(ns, round) / speed[s], nf_c = busiest_cu(nf, round) / speed[f];
      if (ns_c > cs || nf_c >= cs) break;
      qs.swap(ns);
      qf.swap(nf);
      (first ? c0 : c1) = ns_c;
      (first ? c1 : c0) = nf_c;
    }
  }
}

// The attention launch's work items: (sequence, KV head, row tile) items,
// split by key range when too few to fill the chip, ordered and placed over
// the XCDs.  `seqs` comes from plan_attn_check.
inline void plan_attn_items(const sa_layout* layout, const std::vector<SeqDesc>& seqs, const AttnShape& shape,
                            XcdState* xcd, AttnPlan& out) {
  const int Hq = layout->num_q_heads, Hkv = layout->num_kv_heads, G = Hq / Hkv;
  const int rows_item = shape.rows_item;
  const int num_cu = shape.num_cu;
  const int batch = (int)seqs.size();
  out = AttnPlan{};

  // ---- work items: (sequence, kv head, row tile)
  struct Work {
    AttnItem it;
    int64_t tiles;
    bool decode;
    int xcd;
    int64_t group = 0;         // items that stay together in the launch order
    int64_t group_tiles = 0;   // the longest item of that group
  };
  std::vector<Work> work;
  int64_t total_tiles = 0;
  for (int b = 0; b < batch; ++b) {
    const int ql = seqs[b].q_len;
    if (ql == 0) continue;
    const int rows = ql * G, pre = seqs[b].kv_len - ql;
    for (int g = 0; g < Hkv; ++g)
      for (int r0 = 0; r0 < rows; r0 += rows_item) {
        const int last = std::min(r0 + rows_item - 1, rows - 1);
        const int kv_end = pre + last / G + 1;
        const int64_t tiles = (kv_end + kKT - 1) / kKT;
        work.push_back({{b, g, r0, 0, kv_end, -1, 0, 0, 0, 0}, tiles, rows <= kDecodeRows, (b * Hkv + g) % kNumXcd});
        total_tiles += tiles;
      }
  }
  // Split long items by key range when there are too few to fill the chip:
  // always below one item per CU; below two per CU (both workgroup slots of
  // a CU) only when items average >= 128 key tiles, where the pairing gains
  // more than the partial-merge launch costs (measured: a CU's two blocks
  // together run ~1.3x one alone; the merge adds ~10-15 us).  A cap on the
  // parts (a caller's fixed scratch) coarsens the split until it fits.
  const int64_t n_work = (int64_t)work.size();
  if (shape.max_parts != 0 &&
      (n_work < num_cu || (n_work < 2 * num_cu && total_tiles >= 128 * n_work))) {
    int64_t chunk = std::max<int64_t>(16, (total_tiles + 2 * num_cu - 1) / (2 * num_cu));
    auto parts_for = [&](int64_t c) {
      int64_t n = 0;
      for (const Work& w : work)
        if (w.tiles > c) n += (w.tiles + c - 1) / c;
      return n;
    };
    if (shape.max_parts > 0)
      while (parts_for(chunk) > shape.max_parts) chunk *= 2;
    std::vector<Work> split;
    for (const Work& w : work) {
      if (w.tiles <= chunk) {
        split.push_back(w);
        continue;
      }
      const int64_t n = (w.tiles + chunk - 1) / chunk;
      out.groups.push_back({w.it.seq, w.it.kvh, w.it.row0, (int32_t)n, out.n_parts, 0});
      for (int64_t k = 0; k < n; ++k) {
        Work p = w;
        p.it.kv_begin = (int32_t)(k * chunk * kKT);
        p.it.kv_end = (int32_t)std::min<int64_t>((k + 1) * chunk * kKT, w.it.kv_end);
        p.it.part = out.n_parts++;
        p.tiles = (p.it.kv_end - p.it.kv_begin + kKT - 1) / kKT;
        split.push_back(p);
      }
    }
    work.swap(split);
  }
  // Order: decode work first, then longest first, except that the row tiles of
  // one (sequence, KV head) prefill stay next to each other (ranked by the
  // group's longest tile): they read the same K/V range, so run together on
  // their XCD they stream it through its L2 once.  Decode items and the
  // key-range parts of split items share no K/V with their neighbours and
  // keep the plain longest-first order.
  {
    std::map<int64_t, int64_t> group_len;                       // (seq, kvh) -> longest row tile
    auto grouped = [](const Work& w) { return !w.decode && w.it.part < 0; };
    for (const Work& w : work)
      if (grouped(w)) {
        int64_t& g = group_len[(int64_t)w.it.seq * Hkv + w.it.kvh];
        g = std::max(g, w.tiles);
      }
    for (size_t i = 0; i < work.size(); ++i) {
      Work& w = work[i];
      if (grouped(w)) {
        w.group = (int64_t)w.it.seq * Hkv + w.it.kvh;
        w.group_tiles = group_len[w.group];
      } else {
        w.group = (int64_t)i - (int64_t)work.size();              // a group of its own, in list order
        w.group_tiles = w.tiles;
      }
    }
  }
  std::stable_sort(work.begin(), work.end(), [](const Work& x, const Work& y) {
    if (x.decode != y.decode) return x.decode;
    if (x.group_tiles != y.group_tiles) return x.group_tiles > y.group_tiles;
    if (x.group != y.group) return x.group < y.group;
    return x.tiles > y.tiles;
  });
  // XCD-aware placement: block i runs on XCD i % 8, so all items of one
  // (sequence, kv head) go to one XCD and share its L2 -- if that balances.
  int64_t load[kNumXcd] = {0};
  for (const Work& w : work) load[w.xcd] += w.tiles;
  const int64_t mx = *std::max_element(load, load + kNumXcd);
  const int64_t mn = *std::min_element(load, load + kNumXcd);
  // Two blocks share a CU, and with a grid of at most two rounds the
  // dispatcher pairs block i with block i + (number of CUs) (measured): the
  // second round is reversed so the longest items share CUs with the
  // shortest and every CU gets about the same work.  A kernel with one block
  // per CU keeps the longest-first order: each later block goes to the CU
  // that frees first.
  //
  // Mixed launches (decode requests beside prefill chunks) are placed so that
  // every CU holds a decode item and a prefill item from the start: decode
  // items are bound by HBM and prefill items by the matrix cores, so the two
  // overlap.  In each queue the first round is decode items, the second
  // prefill items (their partners), then the remaining decode items -- the
  // dispatcher gives later blocks the slots that free first, and the decode
  // items free theirs first -- then the remaining prefill items.
  bool any_decode = false, any_prefill = false;
  for (const Work& w : work) (w.decode ? any_decode : any_prefill) = true;
  const bool mixed = any_decode && any_prefill;
  auto mix_rounds = [&](std::vector<AttnItem>& q, size_t round) {
    std::vector<AttnItem> d, p;
    for (const AttnItem& x : q) ((int64_t)seqs[x.seq].q_len * G <= kDecodeRows ? d : p).push_back(x);
    if (d.empty() || p.empty()) return;
    const size_t nd = std::min(d.size(), round), np = std::min(p.size(), round);
    q.clear();
    q.insert(q.end(), d.begin(), d.begin() + nd);
    q.insert(q.end(), p.begin(), p.begin() + np);
    q.insert(q.end(), d.begin() + nd, d.end());
    q.insert(q.end(), p.begin() + np, p.end());
  };
  const bool pair = shape.pair_rounds && !mixed;
  auto pair_rounds = [&](std::vector<AttnItem>& q, size_t first_round) {
    if (mixed) {
      mix_rounds(q, first_round);
      return;
    }
    if (!pair) return;
    if (q.size() > first_round && q.size() <= 2 * first_round) std::reverse(q.begin() + first_round, q.end());
  };
  std::vector<AttnItem>& items = out.items;
  const size_t xcd_round = (size_t)std::max(1, num_cu / kNumXcd);
  if (mx > 0 && (double)(mx - mn) <= 0.1 * (double)mx) {
    std::vector<std::vector<AttnItem>> queue(kNumXcd);
    for (const Work& w : work) queue[w.xcd].push_back(w.it);
    if (xcd != nullptr && xcd->weighted && !mixed) {
      bool same = xcd->in.size() == queue.size();
      for (size_t x = 0; same && x < queue.size(); ++x)
        same = xcd->in[x].size() == queue[x].size() &&
               (queue[x].empty() ||
                memcmp(xcd->in[x].data(), queue[x].data(), queue[x].size() * sizeof(AttnItem)) == 0);
      if (same) {
        queue = xcd->out;
      } else {
        xcd->in = queue;
        weigh_xcds(queue, xcd_round, xcd->speed);
        xcd->out = queue;
      }
    }
    for (auto& qd : queue) pair_rounds(qd, xcd_round);
    size_t depth = 0;
    for (auto& qd : queue) depth = std::max(depth, qd.size());
    items.assign(depth * kNumXcd, AttnItem{0, 0, 0, 0, 0, -1, 0, 0, 0, 0});
    for (int x = 0; x < kNumXcd; ++x)
      for (size_t i = 0; i < queue[x].size(); ++i) items[i * kNumXcd + x] = queue[x][i];
  } else {
    for (const Work& w : work) items.push_back(w.it);
    pair_rounds(items, (size_t)num_cu);
  }
  for (AttnItem& x : items) {
    if (x.kv_end <= x.kv_begin) continue;              // padding
    x.q_start = seqs[x.seq].q_start;
    x.q_len = seqs[x.seq].q_len;
    x.kv_len = seqs[x.seq].kv_len;
  }
  // Finishing a CU's two blocks together.  Of two co-resident blocks the
  // older (first-round) one wins the SIMD's issue arbitration: measured at
  // c2, the favoured block advances at about 1.4 times the other's rate
  // (kSlowShare = 0.715 of it), and a block left alone on the CU uses it
  // less well than the pair.  The later block of a pair therefore runs its
  // first `boost` steps at raised priority, chosen so that under those rates
  // both blocks end at the same time: with S = L_old + L_new tiles and
  // D = L_old - L_new, boost = (S / (1 + r) - D / (1 - r)) / 2.
  if (pair && items.size() > (size_t)num_cu && items.size() <= 2 * (size_t)num_cu) {
    constexpr double kSlowShare = 0.715;
    auto tiles_of = [](const AttnItem& x) {
      return x.kv_end > x.kv_begin ? (x.kv_end + kKT - 1) / kKT - x.kv_begin / kKT : 0;
    };
    for (size_t b = num_cu; b < items.size(); ++b) {
      const double l_new = tiles_of(items[b]), l_old = tiles_of(items[b - num_cu]);
      const double x = 0.5 * ((l_old + l_new) / (1.0 + kSlowShare) - (l_old - l_new) / (1.0 - kSlowShare));
      items[b].boost = (int32_t)std::lround(std::min(std::max(x, 0.0), l_new));
    }
  }
}

// Shape of a planned attention launch, for latency models: its workgroups,
// the key-range parts of split items (a partial-merge launch follows when
// there are any), its 64-key tiles, and its makespan in tiles when the items
// are taken in launch order by the first of 2 x num_cu workgroup slots to
// free (a decode item counts a quarter of its tiles: its four waves split
// them).
struct AttnPlanStats {
  int64_t items = 0, parts = 0, tiles = 0, makespan_tiles = 0;
};

inline AttnPlanStats attn_plan_stats(const AttnPlan& plan, const std::vector<SeqDesc>& seqs, int G, int num_cu) {
  AttnPlanStats st;
  st.items = (int64_t)plan.items.size();
  st.parts = plan.n_parts;
  const size_t slots = (size_t)std::max(1, 2 * num_cu);
  std::vector<int64_t> free_at(slots, 0);          // a min-heap of slot finish times (in tiles x 4)
  for (const AttnItem& it : plan.items) {
    if (it.kv_end <= it.kv_begin) continue;
    const int64_t t = item_tiles(it);
    st.tiles += t;
    const int64_t cost = (int64_t)seqs[it.seq].q_len * G <= kDecodeRows ? t : 4 * t;
    std::pop_heap(free_at.begin(), free_at.end(), std::greater<int64_t>());
    free_at.back() += cost;
    std::push_heap(free_at.begin(), free_at.end(), std::greater<int64_t>());
  }
  st.makespan_tiles = (*std::max_element(free_at.begin(), free_at.end()) + 3) / 4;
  return st;
}

// ------------------------------------------------ debug checks of slot lists
//
// Page ids inside device tables are not checked on the hot path beyond the
// kernels' range tests.  With SA_DEBUG=1 the library copies the tables a call
// will use back to the host and runs these checks before launching; they
// return SA_ERR_RANGE for an id outside [0, num_slots) or a page a sequence
// lacks, SA_ERR_OVERLAP for slots that repeat where they must not.

// Commit splice.  surv[u]: the source slot of surviving page u (sp.units
// order); fresh[0 .. sp.fresh_used): the free-list slots the plan consumes.
// Every destination slot must be distinct -- the fresh slots among
// themselves, and with `alias` also the surviving slots, which the
// destination table then lists beside them -- and no fresh slot may be a
// surviving source slot: the copy reads those while it writes the fresh
// ones (a read-after-write race), and an aliased table would name one slot
// for two pages.
inline sa_status debug_check_splice(const SplicePlan& sp, const int32_t* surv, const int32_t* fresh,
                                    int64_t num_slots, bool alias, std::string& err) {
  std::vector<std::pair<int32_t, int>> seen;     // (slot, 0 surviving / 1 fresh)
  seen.reserve(sp.units.size() + (size_t)sp.fresh_used);
  for (size_t u = 0; u < sp.units.size(); ++u) {
    if (surv[u] < 0 || surv[u] >= num_slots)
      return plan_fail(err, SA_ERR_RANGE, "sequence %d: surviving page %d has slot %d outside [0, %lld)",
                       sp.units[u].seq, sp.units[u].src_page, surv[u], (long long)num_slots);
    seen.push_back({surv[u], 0});
  }
  for (int64_t f = 0; f < sp.fresh_used; ++f) {
    if (fresh[f] < 0 || fresh[f] >= num_slots)
      return plan_fail(err, SA_ERR_RANGE, "free-list entry %lld is slot %d, outside [0, %lld)", (long long)f,
                       fresh[f], (long long)num_slots);
    seen.push_back({fresh[f], 1});
  }
  std::sort(seen.begin(), seen.end());
  for (size_t i = 1; i < seen.size(); ++i) {
    if (seen[i].first != seen[i - 1].first) continue;
    const int a = seen[i - 1].second, b = seen[i].second;
    if (a == 1 && b == 1)
      return plan_fail(err, SA_ERR_OVERLAP, "slot %d appears twice in the free list", seen[i].first);
    if (a != b)
      return plan_fail(err, SA_ERR_OVERLAP, "fresh slot %d is also a surviving source slot", seen[i].first);
    if (alias)
      return plan_fail(err, SA_ERR_OVERLAP, "surviving slot %d is listed for two pages", seen[i].first);
  }
  return SA_OK;
}

// Append.  indptr [B + 1] and indices (the whole table) are host copies of
// the device page table.  Every written position must have its page, every
// page's slot must be in range, and no two sequences may write the same row
// of the same slot.
inline sa_status debug_check_append(int32_t batch, const int32_t* start, const int32_t* new_len,
                                    const int32_t* indptr, const int32_t* indices, int P, int64_t num_slots,
                                    std::string& err) {
  struct Span {
    int32_t slot, lo, hi, seq;   // rows [lo, hi) of slot, written by seq
  };
  std::vector<Span> spans;
  for (int b = 0; b < batch; ++b) {
    if (new_len[b] == 0) continue;
    const int64_t x0 = start[b], x1 = (int64_t)start[b] + new_len[b];     // positions [x0, x1)
    const int64_t n_pages = (int64_t)indptr[b + 1] - indptr[b];
    for (int64_t pg = x0 / P; pg <= (x1 - 1) / P; ++pg) {
      if (pg >= n_pages)
        return plan_fail(err, SA_ERR_RANGE, "sequence %d: position %lld needs page %lld, the table has %lld", b,
                         (long long)std::max(x0, pg * P), (long long)pg, (long long)n_pages);
      const int32_t slot = indices[indptr[b] + pg];
      if (slot < 0 || slot >= num_slots)
        return plan_fail(err, SA_ERR_RANGE, "sequence %d: page %lld has slot %d outside [0, %lld)", b,
                         (long long)pg, slot, (long long)num_slots);
      const int32_t lo = (int32_t)(std::max(x0, pg * P) - pg * P);
      const int32_t hi = (int32_t)(std::min(x1, (pg + 1) * P) - pg * P);
      spans.push_back({slot, lo, hi, b});
    }
  }
  std::sort(spans.begin(), spans.end(),
            [](const Span& x, const Span& y) { return x.slot != y.slot ? x.slot < y.slot : x.lo < y.lo; });
  for (size_t i = 1; i < spans.size(); ++i)
    if (spans[i].slot == spans[i - 1].slot && spans[i].lo < spans[i - 1].hi)
      return plan_fail(err, SA_ERR_OVERLAP, "sequences %d and %d both write rows of slot %d", spans[i - 1].seq,
                       spans[i].seq, spans[i].slot);
  return SA_OK;
}

}  // namespace sa
