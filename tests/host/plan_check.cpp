// Host-only checks of the library's planner (paper_2607_00151_amd/csrc/plan.h),
// built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_sanitizers.py and run without a GPU.
//
// Over thousands of seeded random shapes (empty sequences first, in the
// middle and last; prefixes of zero; decode rows; G from 1 to 16; both page
// sizes; few and many compute units; with and without XCD speeds; with and
// without a cap on split parts) it checks that
//   * the attention work list covers every (sequence, KV head, row tile)
//     exactly once, as one whole item or as key-range parts that tile
//     [0, kv_end) in order, with the causal key bound of the tile's last row;
//   * split parts are numbered once each and their merge groups agree;
//   * the XCD weighting moves items, never changes them, and a repeated
//     launch reuses the same placement;
//   * the splice plan matches a direct page-by-page count (kept tokens,
//     destination offsets, fresh slots, alias entries) and the splice's
//     append records fit each sequence's pages;
//   * the debug slot checks accept valid lists and refuse repeats, overlaps
//     and out-of-range slots;
//   * malformed arguments are refused with the documented status codes.
// Prints "ALL OK" and exits 0 on success; any failure prints and exits 1.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <tuple>
#include <vector>

#include "plan.h"

static int g_fail = 0;
#define CHECK(cond, ...)                                                        \
  do {                                                                          \
    if (!(cond)) {                                                              \
      std::fprintf(stderr, "FAIL %s:%d: %s: ", __FILE__, __LINE__, #cond);      \
      std::fprintf(stderr, __VA_ARGS__);                                        \
      std::fprintf(stderr, "\n");                                               \
      if (++g_fail > 20) std::exit(1);                                          \
    }                                                                           \
  } while (0)

static sa_layout layout(int Hq, int Hkv, int P, int64_t slots = 1 << 20, int layers = 1) {
  sa_layout L;
  L.num_q_heads = Hq;
  L.num_kv_heads = Hkv;
  L.head_dim = 128;
  L.page_size = P;
  L.num_layers = layers;
  L.num_slots = slots;
  return L;
}

// ------------------------------------------------------------- attention

static void check_attention_case(std::mt19937_64& r, int case_id) {
  const int Hkv = 1 << (r() % 4);                // 1..8
  const int G = std::vector<int>{1, 2, 3, 4, 8, 16}[r() % 6];
  const int P = (r() & 1) ? 16 : 32;
  const sa_layout L = layout(Hkv * G, Hkv, P);
  const int B = 1 + (int)(r() % 7);
  std::vector<int32_t> ql(B), kl(B);
  for (int b = 0; b < B; ++b) {
    const int kind = (int)(r() % 5);
    const int pre = (r() % 4 == 0) ? 0 : (int)(r() % 9000);
    int q = kind == 0 ? 0 : kind == 1 ? 1 : (int)(1 + r() % 2500);
    ql[b] = q;
    kl[b] = pre + q;
  }
  if (case_id % 7 == 0) ql[0] = 0, kl[0] = (int)(r() % 100);          // empty first
  if (case_id % 11 == 0) ql[B - 1] = 0;                               // empty last
  if (case_id % 13 == 0 && B > 2) ql[B / 2] = 0, kl[B / 2] = 0;       // empty middle, nothing cached

  std::string err;
  std::vector<sa::SeqDesc> seqs;
  int64_t total_q = 0;
  sa_status s = sa::plan_attn_check(&L, 0, B, ql.data(), kl.data(), 0.0884f, seqs, total_q, err);
  CHECK(s == SA_OK, "case %d: %s", case_id, err.c_str());
  if (s != SA_OK) return;
  int64_t t = 0;
  for (int b = 0; b < B; ++b) {
    CHECK(seqs[b].q_start == t && seqs[b].q_len == ql[b] && seqs[b].kv_len == kl[b], "seq desc %d", b);
    t += ql[b];
  }
  CHECK(t == total_q, "total_q");

  sa::AttnShape shape;
  shape.rows_item = 128;
  shape.num_cu = std::vector<int>{256, 256, 64, 8}[r() % 4];
  shape.pair_rounds = (r() % 4) != 0;
  shape.max_parts = (r() % 3 == 0) ? (int64_t)(r() % 40) : -1;
  sa::XcdState xcd;
  const bool weighted = (r() % 2) == 0;
  if (weighted) {
    xcd.weighted = true;
    for (int x = 0; x < sa::kNumXcd; ++x) xcd.speed[x] = 0.8f + 0.05f * (float)(r() % 9);
  }
  sa::AttnPlan plan;
  sa::plan_attn_items(&L, seqs, shape, &xcd, plan);

  // expected row tiles: (seq, kvh, row0) -> causal key bound of its last row
  std::map<std::tuple<int, int, int>, int> want;
  for (int b = 0; b < B; ++b) {
    const int rows = ql[b] * G, pre = kl[b] - ql[b];
    for (int g = 0; g < Hkv; ++g)
      for (int r0 = 0; r0 < rows; r0 += shape.rows_item) {
        const int last = std::min(r0 + shape.rows_item - 1, rows - 1);
        want[{b, g, r0}] = pre + last / G + 1;
      }
  }
  // whole items and parts found
  std::map<std::tuple<int, int, int>, std::vector<sa::AttnItem>> got;
  std::set<int> part_ids;
  size_t real = 0;
  for (const sa::AttnItem& it : plan.items) {
    if (it.kv_end <= it.kv_begin) continue;             // padding
    ++real;
    CHECK(it.seq >= 0 && it.seq < B && ql[it.seq] > 0, "item of an empty or unknown sequence %d", it.seq);
    if (!(it.seq >= 0 && it.seq < B)) continue;
    CHECK(it.q_start == seqs[it.seq].q_start && it.q_len == ql[it.seq] && it.kv_len == kl[it.seq],
          "item copies of the sequence fields");
    CHECK(it.kv_begin % sa::kKT == 0, "kv_begin %d not tile aligned", it.kv_begin);
    CHECK(it.boost >= 0 && it.boost <= sa::item_tiles(it), "boost %d of %lld tiles", it.boost,
          (long long)sa::item_tiles(it));
    if (it.part >= 0) {
      CHECK(part_ids.insert(it.part).second, "part %d listed twice", it.part);
      CHECK(it.part < plan.n_parts, "part %d of %d", it.part, plan.n_parts);
    }
    got[{it.seq, it.kvh, it.row0}].push_back(it);
  }
  CHECK((int)part_ids.size() == plan.n_parts, "%zu parts listed, n_parts %d", part_ids.size(), plan.n_parts);
  if (shape.max_parts >= 0) CHECK(plan.n_parts <= shape.max_parts, "%d parts over the cap", plan.n_parts);
  CHECK(got.size() == want.size(), "case %d: %zu row tiles planned, %zu expected", case_id, got.size(), want.size());
  std::map<std::tuple<int, int, int>, const sa::MergeGroup*> groups;
  for (const sa::MergeGroup& g : plan.groups) {
    CHECK(groups.insert({{g.seq, g.kvh, g.row0}, &g}).second, "merge group listed twice");
    CHECK(g.nsplit >= 2 && g.part0 >= 0 && g.part0 + g.nsplit <= plan.n_parts, "merge group range");
  }
  for (auto& kv : want) {
    auto it = got.find(kv.first);
    CHECK(it != got.end(), "row tile (%d, %d, %d) missing", std::get<0>(kv.first), std::get<1>(kv.first),
          std::get<2>(kv.first));
    if (it == got.end()) continue;
    auto& v = it->second;
    std::sort(v.begin(), v.end(), [](const sa::AttnItem& a, const sa::AttnItem& b) { return a.kv_begin < b.kv_begin; });
    if (v.size() == 1) {
      CHECK(v[0].part < 0 && v[0].kv_begin == 0 && v[0].kv_end == kv.second, "whole item keys [%d, %d), want [0, %d)",
            v[0].kv_begin, v[0].kv_end, kv.second);
      CHECK(groups.find(kv.first) == groups.end(), "whole item with a merge group");
    } else {
      auto g = groups.find(kv.first);
      CHECK(g != groups.end() && g->second->nsplit == (int)v.size(), "split item without its merge group");
      int next = 0;
      for (size_t k = 0; k < v.size(); ++k) {
        CHECK(v[k].part >= 0 && v[k].kv_begin == next, "parts do not tile the keys");
        if (g != groups.end())
          CHECK(v[k].part == g->second->part0 + (int)k, "part numbering within a group");
        next = v[k].kv_end;
      }
      CHECK(next == kv.second, "parts end at %d, want %d", next, kv.second);
    }
  }
  (void)real;

  // the weighting moves items, never changes them; a repeat reuses the placement
  if (weighted) {
    sa::AttnPlan plain, again;
    sa::plan_attn_items(&L, seqs, shape, nullptr, plain);
    sa::plan_attn_items(&L, seqs, shape, &xcd, again);
    auto key = [](const sa::AttnItem& x) {
      return std::make_tuple(x.seq, x.kvh, x.row0, x.kv_begin, x.kv_end, x.part);
    };
    std::multiset<std::tuple<int, int, int, int, int, int>> a, b;
    for (const auto& x : plain.items)
      if (x.kv_end > x.kv_begin) a.insert(key(x));
    for (const auto& x : plan.items)
      if (x.kv_end > x.kv_begin) b.insert(key(x));
    CHECK(a == b, "case %d: the weighted plan holds other items than the plain one", case_id);
    CHECK(again.items.size() == plan.items.size() &&
              (plan.items.empty() ||
               std::memcmp(again.items.data(), plan.items.data(), plan.items.size() * sizeof(sa::AttnItem)) == 0),
          "a repeated launch changed its placement");
  }
}

static void check_attention_errors() {
  std::string err;
  std::vector<sa::SeqDesc> seqs;
  int64_t tq = 0;
  const sa_layout L = layout(32, 8, 16);
  int32_t ql[2] = {4, 9}, kl[2] = {8, 8};
  CHECK(sa::plan_attn_check(&L, 0, 2, ql, kl, 0.1f, seqs, tq, err) == SA_ERR_SHAPE, "q_len > kv_len");
  ql[1] = -1;
  CHECK(sa::plan_attn_check(&L, 0, 2, ql, kl, 0.1f, seqs, tq, err) == SA_ERR_SHAPE, "negative q_len");
  ql[1] = 2;
  CHECK(sa::plan_attn_check(&L, 1, 2, ql, kl, 0.1f, seqs, tq, err) == SA_ERR_SHAPE, "layer");
  CHECK(sa::plan_attn_check(&L, 0, 0, ql, kl, 0.1f, seqs, tq, err) == SA_ERR_SHAPE, "batch 0");
  CHECK(sa::plan_attn_check(&L, 0, 2, nullptr, kl, 0.1f, seqs, tq, err) == SA_ERR_NULL, "NULL q_len");
  CHECK(sa::plan_attn_check(&L, 0, 2, ql, kl, -1.f, seqs, tq, err) == SA_ERR_SHAPE, "negative scale");
  CHECK(sa::plan_attn_check(&L, 0, 2, ql, kl, NAN, seqs, tq, err) == SA_ERR_SHAPE, "NaN scale");
  sa_layout bad = L;
  bad.head_dim = 64;
  CHECK(sa::check_layout(&bad, err) == SA_ERR_UNSUPPORTED, "head_dim");
  bad = L;
  bad.page_size = 8;
  CHECK(sa::check_layout(&bad, err) == SA_ERR_UNSUPPORTED, "page size");
  bad = L;
  bad.num_q_heads = 12;
  CHECK(sa::check_layout(&bad, err) == SA_ERR_SHAPE, "GQA ratio");
  bad = L;
  bad.num_slots = (int64_t)1 << 40;
  CHECK(sa::check_layout(&bad, err) == SA_ERR_SHAPE, "pool too large");
  CHECK(sa::check_layout(nullptr, err) == SA_ERR_NULL, "NULL layout");
}

// ------------------------------------------------------------------ splice

static void check_splice_case(std::mt19937_64& r, int case_id) {
  const int P = (r() & 1) ? 16 : 32;
  const sa_layout L = layout(8, 2, P, 1 << 16);
  const int B = 1 + (int)(r() % 5);
  std::vector<int32_t> src_len(B), reserve(B), keep_indptr(B + 1, 0), spans, new_len(B);
  for (int b = 0; b < B; ++b) {
    src_len[b] = (r() % 5 == 0) ? 0 : (int)(r() % 3000);
    reserve[b] = (int)(r() % 700);
    const int n_pages = (src_len[b] + P - 1) / P;
    int p = 0;
    while (p < n_pages) {
      const int gap = (int)(r() % 4), len = 1 + (int)(r() % 40);
      const int beg = p + gap;
      if (beg >= n_pages) break;
      const int end = std::min(n_pages, beg + len);
      if (r() % 3) {
        spans.push_back(beg);
        spans.push_back(end);
      }
      p = end;
    }
    keep_indptr[b + 1] = (int32_t)(spans.size() / 2);
  }
  for (int alias = 0; alias < 2; ++alias) {
    // direct count
    int64_t n_dst = 0, fresh = 0;
    std::vector<int32_t> want_len(B), want_ip(B + 1, 0);
    int64_t units = 0;
    for (int b = 0; b < B; ++b) {
      int64_t kept = 0, kp = 0;
      for (int k = keep_indptr[b]; k < keep_indptr[b + 1]; ++k)
        for (int p = spans[2 * k]; p < spans[2 * k + 1]; ++p) {
          kept += std::min(P, src_len[b] - p * P);
          ++kp;
        }
      const int64_t pages = std::max<int64_t>(kp, (kept + reserve[b] + P - 1) / P);
      want_len[b] = (int32_t)kept;
      n_dst += pages;
      fresh += alias ? pages - kp : pages;
      units += kp;
      want_ip[b + 1] = (int32_t)n_dst;
    }
    std::string err;
    sa::SplicePlan sp;
    const sa_status s = sa::plan_splice(&L, B, src_len.data(), keep_indptr.data(), spans.empty() ? nullptr : spans.data(),
                                        reserve.data(), alias != 0, (int32_t)fresh, (int32_t)n_dst, sp, err);
    CHECK(s == SA_OK, "case %d: %s", case_id, err.c_str());
    if (s != SA_OK) continue;
    CHECK(sp.n_dst == n_dst && sp.fresh_used == fresh && (int64_t)sp.units.size() == units, "splice counts");
    CHECK(sp.dst_len == want_len && sp.dst_indptr == want_ip, "splice lengths / offsets");
    // units: per sequence, in span order, destination indexes from the sequence's offset up
    size_t u = 0;
    for (int b = 0; b < B; ++b) {
      int32_t d = want_ip[b];
      for (int k = keep_indptr[b]; k < keep_indptr[b + 1]; ++k)
        for (int p = spans[2 * k]; p < spans[2 * k + 1]; ++p, ++u, ++d)
          CHECK(u < sp.units.size() && sp.units[u].seq == b && sp.units[u].src_page == p && sp.units[u].dst_index == d,
                "unit %zu", u);
    }
    if (alias) {
      CHECK((int64_t)sp.entry.size() == n_dst, "alias entries");
      int64_t next_fresh = 0;
      size_t next_unit = 0;
      for (int64_t e = 0; e < (int64_t)sp.entry.size(); ++e) {
        if (sp.entry[e] >= 0) CHECK(sp.entry[e] == (int32_t)next_unit++, "alias unit entry order");
        else CHECK(sp.entry[e] == -(int32_t)next_fresh++ - 1, "alias fresh entry order");
      }
      CHECK(next_fresh == fresh && next_unit == sp.units.size(), "alias entries consume everything");
    } else {
      // the append riding with the splice: up to the room left in each sequence's pages
      for (int b = 0; b < B; ++b) {
        const int64_t room = (int64_t)(want_ip[b + 1] - want_ip[b]) * P - want_len[b];
        new_len[b] = (int32_t)(room > 0 ? (int64_t)(r() % (room + 1)) : 0);
      }
      sa::SpliceAppendPlan ap;
      const sa_status s2 = sa::plan_splice_append(&L, B, new_len.data(), 0, sp, ap, err);
      CHECK(s2 == SA_OK, "splice append: %s", err.c_str());
      if (s2 == SA_OK) {
        int64_t listed = 0, on_units = 0, all = 0;
        for (int b = 0; b < B; ++b) {
          all += new_len[b];
          listed += ap.tok_begin[b + 1] - ap.tok_begin[b];
        }
        for (const auto& x : sp.units) {
          on_units += x.app_rows;
          CHECK(x.app_rows == 0 || (x.app_row0 > 0 && x.app_row0 + x.app_rows <= P), "unit append rows");
        }
        CHECK(ap.all_new == all && listed + on_units == all && ap.total == listed, "every new token placed once");
      }
      // one token too many for the first sequence is refused
      std::vector<int32_t> over = new_len;
      over[0] = (int32_t)((int64_t)(want_ip[1] - want_ip[0]) * P - want_len[0] + 1);
      sa::SplicePlan sp2;
      sa::plan_splice(&L, B, src_len.data(), keep_indptr.data(), spans.empty() ? nullptr : spans.data(),
                      reserve.data(), false, (int32_t)fresh, (int32_t)n_dst, sp2, err);
      CHECK(sa::plan_splice_append(&L, B, over.data(), 0, sp2, ap, err) == SA_ERR_SHAPE, "overfull append");
    }
    // too few fresh slots / too small a table
    if (fresh > 0)
      CHECK(sa::plan_splice(&L, B, src_len.data(), keep_indptr.data(), spans.empty() ? nullptr : spans.data(),
                            reserve.data(), alias != 0, (int32_t)fresh - 1, (int32_t)n_dst, sp, err) == SA_ERR_NO_PAGES,
            "free list short by one");
    if (n_dst > 0)
      CHECK(sa::plan_splice(&L, B, src_len.data(), keep_indptr.data(), spans.empty() ? nullptr : spans.data(),
                            reserve.data(), alias != 0, (int32_t)fresh, (int32_t)n_dst - 1, sp, err) == SA_ERR_NO_PAGES,
            "destination table short by one");
  }
}

static void check_splice_errors() {
  const sa_layout L = layout(8, 2, 16, 1 << 16);
  std::string err;
  sa::SplicePlan sp;
  int32_t src_len[1] = {100}, reserve[1] = {10};
  int32_t ki[2] = {0, 2}, ov[4] = {0, 2, 1, 7};
  CHECK(sa::plan_splice(&L, 1, src_len, ki, ov, reserve, false, 100, 100, sp, err) == SA_ERR_RANGE, "overlap");
  int32_t past[2] = {0, 8};
  int32_t k1[2] = {0, 1};
  CHECK(sa::plan_splice(&L, 1, src_len, k1, past, reserve, false, 100, 100, sp, err) == SA_ERR_RANGE, "past end");
  int32_t empty[2] = {3, 3};
  CHECK(sa::plan_splice(&L, 1, src_len, k1, empty, reserve, false, 100, 100, sp, err) == SA_ERR_RANGE, "empty span");
  int32_t k_bad[2] = {1, 1};
  CHECK(sa::plan_splice(&L, 1, src_len, k_bad, past, reserve, false, 100, 100, sp, err) == SA_ERR_SHAPE, "indptr[0]");
  int32_t k_dec[3] = {0, 1, 0};
  int32_t two_len[2] = {100, 100}, two_res[2] = {0, 0};
  CHECK(sa::plan_splice(&L, 2, two_len, k_dec, past, two_res, false, 100, 100, sp, err) == SA_ERR_SHAPE,
        "decreasing indptr");
  CHECK(sa::plan_splice(&L, 1, src_len, k1, nullptr, reserve, false, 100, 100, sp, err) == SA_ERR_NULL, "NULL spans");
  int32_t neg[1] = {-1};
  CHECK(sa::plan_splice(&L, 1, neg, ki, ov, reserve, false, 100, 100, sp, err) == SA_ERR_SHAPE, "negative length");
}

// ------------------------------------------------------------ debug checks

static void check_debug_checks() {
  std::string err;
  const sa_layout L = layout(8, 2, 16, 64);
  // two sequences, 40 and 20 tokens, keep everything: 3 + 2 surviving pages
  int32_t src_len[2] = {40, 20}, reserve[2] = {30, 0}, ki[3] = {0, 1, 2}, spans[4] = {0, 3, 0, 2};
  sa::SplicePlan sp;
  CHECK(sa::plan_splice(&L, 2, src_len, ki, spans, reserve, false, 100, 100, sp, err) == SA_OK, "%s", err.c_str());
  std::vector<int32_t> surv = {1, 2, 3, 4, 5};
  std::vector<int32_t> fresh;
  for (int i = 0; i < (int)sp.fresh_used; ++i) fresh.push_back(10 + i);
  CHECK(sa::debug_check_splice(sp, surv.data(), fresh.data(), 64, false, err) == SA_OK, "valid lists: %s", err.c_str());
  auto f2 = fresh;
  f2[2] = f2[0];
  CHECK(sa::debug_check_splice(sp, surv.data(), f2.data(), 64, false, err) == SA_ERR_OVERLAP, "repeated fresh slot");
  f2 = fresh;
  f2[1] = 3;
  CHECK(sa::debug_check_splice(sp, surv.data(), f2.data(), 64, false, err) == SA_ERR_OVERLAP, "fresh = surviving");
  f2 = fresh;
  f2[0] = 64;
  CHECK(sa::debug_check_splice(sp, surv.data(), f2.data(), 64, false, err) == SA_ERR_RANGE, "fresh out of range");
  auto s2 = surv;
  s2[4] = -1;
  CHECK(sa::debug_check_splice(sp, s2.data(), fresh.data(), 64, false, err) == SA_ERR_RANGE, "surviving out of range");
  s2 = surv;
  s2[4] = s2[0];
  CHECK(sa::debug_check_splice(sp, s2.data(), fresh.data(), 64, false, err) == SA_OK, "copy may read one slot twice");
  // alias: the surviving slots become destination slots, so they must not repeat
  sa::SplicePlan spa;
  CHECK(sa::plan_splice(&L, 2, src_len, ki, spans, reserve, true, 100, 100, spa, err) == SA_OK, "%s", err.c_str());
  std::vector<int32_t> fa;
  for (int i = 0; i < (int)spa.fresh_used; ++i) fa.push_back(20 + i);
  CHECK(sa::debug_check_splice(spa, surv.data(), fa.data(), 64, true, err) == SA_OK, "alias valid");
  CHECK(sa::debug_check_splice(spa, s2.data(), fa.data(), 64, true, err) == SA_ERR_OVERLAP, "alias repeat");

  // append: sequence 0 writes positions 10..39 over pages {3, 7}, sequence 1 0..9 of page {9}
  int32_t indptr[3] = {0, 3, 4}, indices[4] = {3, 7, 8, 9};
  int32_t start[2] = {10, 0}, len[2] = {30, 10};
  CHECK(sa::debug_check_append(2, start, len, indptr, indices, 16, 64, err) == SA_OK, "append valid: %s", err.c_str());
  int32_t shared[4] = {3, 7, 8, 3};       // sequence 1 writes rows 0..9 of slot 3, sequence 0 rows 10..15
  CHECK(sa::debug_check_append(2, start, len, indptr, shared, 16, 64, err) == SA_OK, "disjoint rows of one slot");
  int32_t clash[4] = {3, 7, 8, 7};        // both write rows 0..9 of slot 7
  CHECK(sa::debug_check_append(2, start, len, indptr, clash, 16, 64, err) == SA_ERR_OVERLAP, "same rows twice");
  int32_t len_far[2] = {60, 10};          // position 69 needs page 4 of 3
  CHECK(sa::debug_check_append(2, start, len_far, indptr, indices, 16, 64, err) == SA_ERR_RANGE, "missing page");
  int32_t oob[4] = {3, 70, 8, 9};
  CHECK(sa::debug_check_append(2, start, len, indptr, oob, 16, 64, err) == SA_ERR_RANGE, "slot out of range");
  int32_t none[2] = {0, 0};
  CHECK(sa::debug_check_append(2, start, none, indptr, oob, 16, 64, err) == SA_OK, "nothing written");
}

int main() {
  std::mt19937_64 r(20260);
  for (int c = 0; c < 3000; ++c) check_attention_case(r, c);
  check_attention_errors();
  for (int c = 0; c < 3000; ++c) check_splice_case(r, c);
  check_splice_errors();
  check_debug_checks();
  if (g_fail) {
    std::fprintf(stderr, "%d failures\n", g_fail);
    return 1;
  }
  std::printf("ALL OK\n");
  return 0;
}
