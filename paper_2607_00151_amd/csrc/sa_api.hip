// Host side of the C ABI declared in include/sa.h: argument validation, work
// planning, plan upload and kernel launches.  Every entry point validates on
// the host before its first HIP call.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <map>
#include <vector>

#include "sa.h"
#include "attn_kernel.h"
#include "attn_pipe.h"
#include "kv_kernels.h"

namespace {

thread_local std::string g_err;

sa_status fail(sa_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define SA_HIP(call)                                                                 \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess)                                                            \
      return fail(SA_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e_));        \
  } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int kNumXcd = 8;         // MI355X: 8 accelerator complex dies, 32 CUs each
constexpr int kRing = 8;           // pinned staging buffers in flight

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Byte image of a plan: sub-arrays at 256-byte aligned offsets.
struct PlanImage {
  std::vector<uint8_t> bytes;
  template <class T>
  size_t add(const T* data, size_t n) {
    size_t off = align_up(bytes.size(), 256);
    bytes.resize(off + sizeof(T) * n);
    if (n) memcpy(bytes.data() + off, data, sizeof(T) * n);
    return off;
  }
};

enum PlanKind { kPlanAppend = 0, kPlanAssemble = 1, kPlanAttn = 2, kPlanAlias = 3, kPlanKinds = 4 };

}  // namespace

struct sa_ctx {
  int device = 0;
  int num_cu = 256;
  int32_t* d_err = nullptr;
  struct DevPlan {
    uint8_t* dev = nullptr;
    size_t cap = 0;
    std::vector<uint8_t> shadow;   // what the device buffer holds
    void* stream = nullptr;        // stream that last wrote it
    bool valid = false;
  } plans[kPlanKinds];
  struct Stage {
    void* host = nullptr;
    size_t cap = 0;
    hipEvent_t ev = nullptr;
    bool pending = false;
  } ring[kRing];
  int ring_next = 0;
  float* part = nullptr;           // split-KV partials
  size_t part_cap = 0;             // bytes
  uint32_t* d_sync = nullptr;      // counters of an attention launch that appends (zero between launches)
  bool exact_scale = true;         // sa_set_exact_scale (0: scale folded into q)
  hipEvent_t kernel_ev[2][2] = {};   // sa_set_kernel_events: [SA_TIMED_ATTN | SA_TIMED_PAGES][start, stop]
  uint64_t* blk_clock = nullptr;     // sa_set_block_clock: device buffer, 4 words per block
  float xcd_weight[8] = {1, 1, 1, 1, 1, 1, 1, 1};   // sa_set_xcd_weights: relative XCD speeds
  bool xcd_weighted = false;
  // the last weighting's input queues and result: a launch repeating the same
  // work reuses it instead of searching again
  std::vector<std::vector<sa::AttnItem>> wq_in, wq_out;
  int64_t blk_clock_cap = 0;         // blocks it holds
};

namespace {

// Make the device copy of a plan current; returns its device address.
sa_status upload_plan(sa_ctx* ctx, PlanKind kind, const PlanImage& img, hipStream_t stream,
                      uint8_t** dev) {
  sa_ctx::DevPlan& dp = ctx->plans[kind];
  const size_t n = img.bytes.size();
  if (dp.valid && dp.stream == (void*)stream && dp.shadow.size() == n &&
      memcmp(dp.shadow.data(), img.bytes.data(), n) == 0) {
    *dev = dp.dev;
    return SA_OK;
  }
  if (n > dp.cap) {
    if (dp.dev) {
      SA_HIP(hipDeviceSynchronize());   // an in-flight kernel may still read the old plan
      SA_HIP(hipFree(dp.dev));
      dp.dev = nullptr;
    }
    size_t cap = std::max<size_t>(align_up(n * 2, 4096), 65536);
    SA_HIP(hipMalloc(&dp.dev, cap));
    dp.cap = cap;
  }
  sa_ctx::Stage& st = ctx->ring[ctx->ring_next];
  ctx->ring_next = (ctx->ring_next + 1) % kRing;
  if (st.pending) {
    SA_HIP(hipEventSynchronize(st.ev));
    st.pending = false;
  }
  if (n > st.cap) {
    if (st.host) SA_HIP(hipHostFree(st.host));
    st.host = nullptr;
    size_t cap = std::max<size_t>(align_up(n * 2, 4096), 65536);
    SA_HIP(hipHostMalloc(&st.host, cap, hipHostMallocDefault));
    st.cap = cap;
  }
  if (n) {
    memcpy(st.host, img.bytes.data(), n);
    SA_HIP(hipMemcpyAsync(dp.dev, st.host, n, hipMemcpyHostToDevice, stream));
    SA_HIP(hipEventRecord(st.ev, stream));
    st.pending = true;
  }
  dp.shadow = img.bytes;
  dp.stream = (void*)stream;
  dp.valid = true;
  *dev = dp.dev;
  return SA_OK;
}

sa_status check_layout(const sa_layout* L) {
  if (!L) return fail(SA_ERR_NULL, "layout is NULL");
  if (L->num_q_heads <= 0 || L->num_kv_heads <= 0 || L->num_layers <= 0 || L->num_slots <= 0)
    return fail(SA_ERR_SHAPE, "layout: heads, layers and slots must be positive");
  if (L->num_q_heads % L->num_kv_heads != 0)
    return fail(SA_ERR_SHAPE, "layout: num_q_heads %d is not a multiple of num_kv_heads %d",
                L->num_q_heads, L->num_kv_heads);
  if (L->head_dim != 128) return fail(SA_ERR_UNSUPPORTED, "head_dim %d (only 128)", L->head_dim);
  if (L->page_size != 16 && L->page_size != 32)
    return fail(SA_ERR_UNSUPPORTED, "page_size %d (only 16 or 32)", L->page_size);
  const int64_t slot_elems = (int64_t)L->num_kv_heads * L->page_size * 128;
  if (L->num_slots > INT32_MAX || L->num_slots > (INT64_MAX / 4) / slot_elems / L->num_layers)
    return fail(SA_ERR_SHAPE, "layout: pool too large");
  return SA_OK;
}

int64_t slot_elems(const sa_layout* L) { return (int64_t)L->num_kv_heads * L->page_size * 128; }
int64_t layer_elems(const sa_layout* L) { return L->num_slots * slot_elems(L); }

sa_status check_ctx(sa_ctx* ctx) {
  if (!ctx) return fail(SA_ERR_NULL, "context is NULL");
  SA_HIP(hipSetDevice(ctx->device));
  return SA_OK;
}

// Attention kernel variants: 0 = the software-pipelined kernel (default),
// 1 = the phase-separated kernel (32 rows per wave, 4 waves), 2 = the
// pipelined kernel with two groups of four waves per block splitting each
// item's keys.  The SA_ATTN_VARIANT environment variable selects one
// (comparison and tuning).
struct AttnVariant {
  int qt, waves, pipe;
};
constexpr AttnVariant kVariants[] = {{1, 4, 1}, {1, 4, 0}, {1, 4, 2}};
constexpr int kDefaultVariant = 0;

AttnVariant attn_variant() {
  static int v = [] {
    const char* e = getenv("SA_ATTN_VARIANT");
    int x = e ? atoi(e) : kDefaultVariant;
    return (x >= 0 && x < (int)(sizeof(kVariants) / sizeof(kVariants[0]))) ? x : kDefaultVariant;
  }();
  return kVariants[v];
}

// sa_segment_prefill_attn_append writes the segment's rows with the append
// kernel and then runs the attention (two launches) unless
// SA_APPEND_IN_ATTN=1, which has the default attention kernel write them
// itself in the same launch (measured slower at the c2 workload: the
// cross-block publication of the rows costs more than the launch it saves).
bool append_in_attention() {
  static bool v = [] {
    const char* e = getenv("SA_APPEND_IN_ATTN");
    return e != nullptr && atoi(e) == 1;
  }();
  return v;
}

// A kernel launch; with timing events set (sa_set_kernel_events) it goes
// through hipExtLaunchKernelGGL, which binds both events to the kernel itself,
// so their elapsed time is the kernel's execution on the device.
template <typename K, typename A>
void launch_timed(K kernel, dim3 grid, dim3 block, hipStream_t st, const hipEvent_t* ev, const A& a) {
  if (ev[0] != nullptr)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, ev[0], ev[1], 0, a);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, st, a);
}

template <int P>
void launch_attn_p(AttnVariant v, bool pool_rsrc, bool exact, dim3 grid, hipStream_t st, const hipEvent_t* ev,
                   const sa::AttnArgs& a) {
  if (v.pipe == 1 && exact && pool_rsrc)
    launch_timed(sa::attn_pipe_kernel<P, true, false, true>, grid, dim3(256), st, ev, a);
  else if (v.pipe == 1 && exact)
    launch_timed(sa::attn_pipe_kernel<P, false, false, true>, grid, dim3(256), st, ev, a);
  else if (v.pipe == 2 && pool_rsrc)
    launch_timed(sa::attn_pp_kernel<P, true>, grid, dim3(512), st, ev, a);
  else if (v.pipe == 2)
    launch_timed(sa::attn_pp_kernel<P, false>, grid, dim3(512), st, ev, a);
  else if (v.pipe && a.app_tickets > 0 && pool_rsrc)
    launch_timed(sa::attn_pipe_kernel<P, true, true>, grid, dim3(256), st, ev, a);
  else if (v.pipe && a.app_tickets > 0)
    launch_timed(sa::attn_pipe_kernel<P, false, true>, grid, dim3(256), st, ev, a);
  else if (v.pipe && pool_rsrc)
    launch_timed(sa::attn_pipe_kernel<P, true, false>, grid, dim3(256), st, ev, a);
  else if (v.pipe)
    launch_timed(sa::attn_pipe_kernel<P, false, false>, grid, dim3(256), st, ev, a);
  else
    launch_timed(sa::attn_kernel<P, 1, 4>, grid, dim3(256), st, ev, a);
}

// pool_rsrc: a layer's K (and V) pool spans < 2^31 bytes, so one buffer
// resource per pool addresses every page with a 32-bit offset
void launch_attn(int page_size, AttnVariant v, bool pool_rsrc, bool exact, dim3 grid, hipStream_t st,
                 const hipEvent_t* ev, const sa::AttnArgs& a) {
  if (page_size == 16) launch_attn_p<16>(v, pool_rsrc, exact, grid, st, ev, a);
  else launch_attn_p<32>(v, pool_rsrc, exact, grid, st, ev, a);
}

}  // namespace

extern "C" {

const char* sa_status_string(sa_status s) {
  switch (s) {
    case SA_OK: return "ok";
    case SA_ERR_NULL: return "null pointer";
    case SA_ERR_SHAPE: return "inconsistent shape or length";
    case SA_ERR_UNSUPPORTED: return "unsupported configuration";
    case SA_ERR_ALIGN: return "pointer not 16-byte aligned";
    case SA_ERR_RANGE: return "value out of range";
    case SA_ERR_NO_PAGES: return "not enough pages";
    case SA_ERR_HIP: return "HIP runtime error";
    case SA_ERR_DEVICE: return "no usable gfx950 device";
  }
  return "unknown status";
}

const char* sa_last_error(void) { return g_err.c_str(); }

sa_status sa_create(int device, sa_ctx** out) {
  if (!out) return fail(SA_ERR_NULL, "out is NULL");
  *out = nullptr;
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n)
    return fail(SA_ERR_DEVICE, "HIP device %d not present (%d visible)", device, n);
  hipDeviceProp_t prop;
  SA_HIP(hipGetDeviceProperties(&prop, device));
  if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(SA_ERR_DEVICE, "device %d is %s, not gfx950", device, prop.gcnArchName);
  SA_HIP(hipSetDevice(device));
  sa_ctx* c = new sa_ctx();
  c->device = device;
  c->num_cu = prop.multiProcessorCount;
  hipError_t e = hipMalloc(&c->d_err, sizeof(int32_t));
  if (e == hipSuccess) e = hipMemset(c->d_err, 0, sizeof(int32_t));
  const size_t sync_bytes = 3 * sa::kSyncStride * sizeof(uint32_t);
  if (e == hipSuccess) e = hipMalloc(&c->d_sync, sync_bytes);
  if (e == hipSuccess) e = hipMemset(c->d_sync, 0, sync_bytes);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  for (int i = 0; e == hipSuccess && i < kRing; ++i)
    e = hipEventCreateWithFlags(&c->ring[i].ev, hipEventDisableTiming);
  if (e != hipSuccess) {
    sa_destroy(c);
    return fail(SA_ERR_HIP, "context setup failed: %s", hipGetErrorString(e));
  }
  *out = c;
  return SA_OK;
}

void sa_destroy(sa_ctx* ctx) {
  if (!ctx) return;
  (void)hipSetDevice(ctx->device);
  (void)hipDeviceSynchronize();
  for (auto& p : ctx->plans)
    if (p.dev) (void)hipFree(p.dev);
  for (auto& s : ctx->ring) {
    if (s.host) (void)hipHostFree(s.host);
    if (s.ev) (void)hipEventDestroy(s.ev);
  }
  if (ctx->part) (void)hipFree(ctx->part);
  if (ctx->d_sync) (void)hipFree(ctx->d_sync);
  if (ctx->d_err) (void)hipFree(ctx->d_err);
  delete ctx;
}

sa_status sa_sync_check(sa_ctx* ctx, void* stream) {
  sa_status s = check_ctx(ctx);
  if (s != SA_OK) return s;
  SA_HIP(hipStreamSynchronize((hipStream_t)stream));
  int32_t flag = 0;
  SA_HIP(hipMemcpy(&flag, ctx->d_err, sizeof flag, hipMemcpyDeviceToHost));
  if (flag) {
    SA_HIP(hipMemset(ctx->d_err, 0, sizeof(int32_t)));
    return fail(SA_ERR_RANGE, "a kernel met an out-of-range page id or slot (flags 0x%x)", flag);
  }
  return SA_OK;
}

// ------------------------------------------------------------------- append

sa_status sa_kv_append(sa_ctx* ctx, const sa_layout* layout, int32_t layer, void* k_pool,
                       void* v_pool, const void* k_new, const void* v_new, int32_t batch,
                       const int32_t* h_start, const int32_t* h_new_len, sa_pages pages,
                       void* stream) {
  sa_status s = check_layout(layout);
  if (s != SA_OK) return s;
  if (layer < 0 || layer >= layout->num_layers)
    return fail(SA_ERR_SHAPE, "layer %d outside [0, %d)", layer, layout->num_layers);
  if (batch < 1) return fail(SA_ERR_SHAPE, "batch %d < 1", batch);
  if (!h_start || !h_new_len) return fail(SA_ERR_NULL, "h_start / h_new_len is NULL");
  std::vector<int32_t> tok_begin(batch + 1);
  int64_t total = 0;
  for (int b = 0; b < batch; ++b) {
    if (h_start[b] < 0 || h_new_len[b] < 0 || (int64_t)h_start[b] + h_new_len[b] > INT32_MAX)
      return fail(SA_ERR_SHAPE, "sequence %d: start %d, new_len %d", b, h_start[b], h_new_len[b]);
    tok_begin[b] = (int32_t)total;
    total += h_new_len[b];
    if (total > INT32_MAX / 2) return fail(SA_ERR_SHAPE, "too many new tokens");
  }
  tok_begin[batch] = (int32_t)total;
  if (!k_pool || !v_pool || !pages.indptr || !pages.indices)
    return fail(SA_ERR_NULL, "pool or page table pointer is NULL");
  if (total > 0 && (!k_new || !v_new)) return fail(SA_ERR_NULL, "k_new / v_new is NULL");
  if (!aligned16(k_pool) || !aligned16(v_pool) || !aligned16(k_new) || !aligned16(v_new))
    return fail(SA_ERR_ALIGN, "pool or new-row pointer not 16-byte aligned");
  s = check_ctx(ctx);
  if (s != SA_OK) return s;
  if (total == 0) return SA_OK;

  PlanImage img;
  const size_t o_tok = img.add(tok_begin.data(), tok_begin.size());
  const size_t o_start = img.add(h_start, (size_t)batch);
  uint8_t* dev = nullptr;
  s = upload_plan(ctx, kPlanAppend, img, (hipStream_t)stream, &dev);
  if (s != SA_OK) return s;

  sa::AppendArgs a{};
  const int64_t lo = (int64_t)layer * layer_elems(layout);
  a.k_pool = (uint16_t*)k_pool + lo;
  a.v_pool = (uint16_t*)v_pool + lo;
  a.k_new = (const uint16_t*)k_new;
  a.v_new = (const uint16_t*)v_new;
  a.tok_begin = (const int32_t*)(dev + o_tok);
  a.start = (const int32_t*)(dev + o_start);
  a.indptr = pages.indptr;
  a.indices = pages.indices;
  a.err = ctx->d_err;
  a.num_slots = layout->num_slots;
  a.total_chunks = total * layout->num_kv_heads * 16;
  a.B = batch;
  a.Hkv = layout->num_kv_heads;
  a.P = layout->page_size;
  const int64_t per_block = 256 * sa::kAppendChunksPerThread;
  const int64_t blocks = (a.total_chunks + per_block - 1) / per_block;
  launch_timed(sa::append_kernel, dim3((unsigned)blocks), dim3(256), (hipStream_t)stream,
               ctx->kernel_ev[SA_TIMED_PAGES], a);
  SA_HIP(hipGetLastError());
  return SA_OK;
}

// ----------------------------------------------------------------- assemble

}  // extern "C"

namespace {

// Host plan of a commit splice: validated spans, one record per surviving
// page, and the destination table's offsets.  With `alias`, surviving pages
// keep their source slots and only the reserved pages take fresh slots.
struct SplicePlan {
  std::vector<sa::AsmUnit> units;      // surviving pages, in destination order
  std::vector<int32_t> dst_indptr, dst_len;
  std::vector<int32_t> entry;          // alias: per destination entry, unit index or -(fresh position + 1)
  int64_t n_dst = 0, fresh_used = 0;
};

sa_status plan_splice(const sa_layout* layout, int32_t batch, const int32_t* h_src_len,
                      const int32_t* h_keep_indptr, const int32_t* h_keep_spans, const int32_t* h_reserve,
                      bool alias, int32_t num_fresh, int32_t dst_capacity, int32_t* h_dst_len,
                      SplicePlan& out) {
  sa_status s = check_layout(layout);
  if (s != SA_OK) return s;
  if (batch < 1) return fail(SA_ERR_SHAPE, "batch %d < 1", batch);
  if (!h_src_len || !h_keep_indptr || !h_reserve || !h_dst_len)
    return fail(SA_ERR_NULL, "a host length array is NULL");
  if (h_keep_indptr[0] != 0) return fail(SA_ERR_SHAPE, "keep_indptr[0] must be 0");
  if (h_keep_indptr[batch] > 0 && !h_keep_spans) return fail(SA_ERR_NULL, "h_keep_spans is NULL");
  if (num_fresh < 0 || dst_capacity < 0) return fail(SA_ERR_SHAPE, "negative capacity");
  const int P = layout->page_size;
  out.dst_indptr.assign(batch + 1, 0);
  out.dst_len.assign(batch, 0);
  int64_t n_dst = 0, fresh_used = 0;
  for (int b = 0; b < batch; ++b) {
    if (h_src_len[b] < 0 || h_reserve[b] < 0)
      return fail(SA_ERR_SHAPE, "sequence %d: src_len %d, reserve %d", b, h_src_len[b], h_reserve[b]);
    if (h_keep_indptr[b + 1] < h_keep_indptr[b])
      return fail(SA_ERR_SHAPE, "keep_indptr decreases at %d", b);
    const int n_src_pages = (h_src_len[b] + P - 1) / P;
    int prev_end = 0, kept_pages = 0;
    int64_t kept = 0;
    for (int k = h_keep_indptr[b]; k < h_keep_indptr[b + 1]; ++k) {
      const int beg = h_keep_spans[2 * k], end = h_keep_spans[2 * k + 1];
      if (beg < prev_end || beg >= end || end > n_src_pages)
        return fail(SA_ERR_RANGE, "sequence %d: keep span [%d, %d) invalid (previous end %d, %d pages)",
                    b, beg, end, prev_end, n_src_pages);
      for (int p = beg; p < end; ++p) {
        if (alias) out.entry.push_back((int32_t)out.units.size());
        out.units.push_back({b, p, (int32_t)(n_dst + kept_pages + (p - beg))});
        kept += std::min(P, h_src_len[b] - p * P);
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
    if (n_dst > INT32_MAX) return fail(SA_ERR_SHAPE, "destination table too large");
    out.dst_indptr[b + 1] = (int32_t)n_dst;
  }
  if (fresh_used > num_fresh)
    return fail(SA_ERR_NO_PAGES, "need %lld fresh slots, %d given", (long long)fresh_used, num_fresh);
  if (n_dst > dst_capacity)
    return fail(SA_ERR_NO_PAGES, "destination table needs %lld entries, capacity %d",
                (long long)n_dst, dst_capacity);
  out.n_dst = n_dst;
  out.fresh_used = fresh_used;
  return SA_OK;
}

}  // namespace

extern "C" {


}  // extern "C"

namespace {

// The copy splice, and with new_len non-NULL an append of new rows of layer
// `layer` behind each sequence's kept tokens in the same launch.
sa_status splice_launch(sa_ctx* ctx, const sa_layout* layout, const void* k_src, const void* v_src,
                        void* k_dst, void* v_dst, int32_t batch, const int32_t* h_src_len,
                        const int32_t* h_keep_indptr, const int32_t* h_keep_spans, const int32_t* h_reserve,
                        sa_pages src, const int32_t* d_fresh, int32_t num_fresh, int32_t* d_dst_indptr,
                        int32_t* d_dst_indices, int32_t dst_capacity, int32_t* h_dst_len, int32_t layer,
                        const void* k_new, const void* v_new, const int32_t* h_new_len, void* stream) {
  SplicePlan sp;
  sa_status s = plan_splice(layout, batch, h_src_len, h_keep_indptr, h_keep_spans, h_reserve, false,
                            num_fresh, dst_capacity, h_dst_len, sp);
  if (s != SA_OK) return s;
  std::vector<sa::AsmUnit>& unit_list = sp.units;
  std::vector<int32_t>& dst_indptr = sp.dst_indptr;
  std::vector<int32_t>& dst_len = sp.dst_len;
  const int64_t units = (int64_t)unit_list.size(), n_dst = sp.n_dst;
  const int P = layout->page_size;
  // append plan: the new rows landing on a partial last surviving page go with
  // that page's copy; the rest are listed per sequence for the append blocks
  const bool app = h_new_len != nullptr;
  std::vector<int32_t> app_tok_begin(batch + 1, 0), app_start(batch, 0), app_knew(batch, 0);
  int64_t app_total = 0;
  if (app) {
    if (layer < 0 || layer >= layout->num_layers)
      return fail(SA_ERR_SHAPE, "layer %d outside [0, %d)", layer, layout->num_layers);
    int64_t knew = 0;
    size_t unit_end = 0;
    for (int b = 0; b < batch; ++b) {
      const int n = h_new_len[b];
      const int64_t pages_b = dst_indptr[b + 1] - dst_indptr[b];
      if (n < 0 || dst_len[b] + (int64_t)n > pages_b * P)
        return fail(SA_ERR_SHAPE, "sequence %d: %d new tokens after %d kept do not fit its %lld pages", b, n,
                    dst_len[b], (long long)pages_b);
      while (unit_end < unit_list.size() && unit_list[unit_end].seq == b) ++unit_end;
      int first = 0;                                      // new tokens on the last surviving page
      if (n > 0 && dst_len[b] % P != 0 && unit_end > 0 && unit_list[unit_end - 1].seq == b) {
        sa::AsmUnit& last = unit_list[unit_end - 1];
        last.app_row0 = dst_len[b] % P;
        last.app_rows = std::min(P - last.app_row0, n);
        last.app_tok = (int32_t)knew;
        first = last.app_rows;
      }
      app_tok_begin[b] = (int32_t)app_total;
      app_start[b] = dst_len[b] + first;
      app_knew[b] = (int32_t)(knew + first);
      app_total += n - first;
      knew += n;
      if (knew > INT32_MAX / 2) return fail(SA_ERR_SHAPE, "too many new tokens");
    }
    app_tok_begin[batch] = (int32_t)app_total;
    if (knew > 0 && (!k_new || !v_new)) return fail(SA_ERR_NULL, "k_new / v_new is NULL");
    if (!aligned16(k_new) || !aligned16(v_new)) return fail(SA_ERR_ALIGN, "new-row pointer not 16-byte aligned");
  }
  // the source slots are read only for surviving pages, the free list and the
  // destination slots only for destination pages
  if (!k_src || !v_src || !k_dst || !v_dst || !src.indptr || !d_dst_indptr ||
      (units > 0 && !src.indices) || (n_dst > 0 && (!d_fresh || !d_dst_indices)))
    return fail(SA_ERR_NULL, "a device pointer is NULL");
  if (!aligned16(k_src) || !aligned16(v_src) || !aligned16(k_dst) || !aligned16(v_dst))
    return fail(SA_ERR_ALIGN, "pool pointer not 16-byte aligned");
  s = check_ctx(ctx);
  if (s != SA_OK) return s;
  memcpy(h_dst_len, dst_len.data(), sizeof(int32_t) * batch);

  PlanImage img;
  const size_t o_un = img.add(unit_list.data(), unit_list.size());
  const size_t o_ip = img.add(dst_indptr.data(), dst_indptr.size());
  const size_t o_at = img.add(app_tok_begin.data(), app ? app_tok_begin.size() : 0);
  const size_t o_as = img.add(app_start.data(), app ? app_start.size() : 0);
  const size_t o_ak = img.add(app_knew.data(), app ? app_knew.size() : 0);
  uint8_t* dev = nullptr;
  s = upload_plan(ctx, kPlanAssemble, img, (hipStream_t)stream, &dev);
  if (s != SA_OK) return s;

  sa::AsmArgs a{};
  a.k_src = (const uint16_t*)k_src;
  a.v_src = (const uint16_t*)v_src;
  a.k_dst = (uint16_t*)k_dst;
  a.v_dst = (uint16_t*)v_dst;
  a.units = (const sa::AsmUnit*)(dev + o_un);
  a.dst_indptr = (const int32_t*)(dev + o_ip);
  a.src_indptr = src.indptr;
  a.src_indices = src.indices;
  a.fresh = d_fresh;
  a.out_indptr = d_dst_indptr;
  a.out_indices = d_dst_indices;
  a.err = ctx->d_err;
  a.num_slots = layout->num_slots;
  a.slot_elems = slot_elems(layout);
  a.layer_elems = layer_elems(layout);
  a.n_units = (int32_t)units;
  a.n_dst = (int32_t)n_dst;
  a.B = batch;
  a.app_layer = app ? layer : -1;
  a.Hkv = layout->num_kv_heads;
  a.P = P;
  if (app) {
    a.k_new = (const uint16_t*)k_new;
    a.v_new = (const uint16_t*)v_new;
    a.app_tok_begin = (const int32_t*)(dev + o_at);
    a.app_start = (const int32_t*)(dev + o_as);
    a.app_knew = (const int32_t*)(dev + o_ak);
    a.app_chunks = app_total * layout->num_kv_heads * 16;
    a.app_blocks = (int32_t)((a.app_chunks + sa::kAsmThreads * sa::kAsmDepth - 1) / (sa::kAsmThreads * sa::kAsmDepth));
  }
  const int64_t table_blocks = (std::max<int64_t>(n_dst, batch + 1) + sa::kAsmThreads - 1) / sa::kAsmThreads;
  const int64_t gx = std::max<int64_t>(units + a.app_blocks, table_blocks);
  if (gx > 0)
    launch_timed(sa::assemble_kernel, dim3((unsigned)gx, (unsigned)layout->num_layers),
                 dim3(sa::kAsmThreads), (hipStream_t)stream, ctx->kernel_ev[SA_TIMED_PAGES], a);
  SA_HIP(hipGetLastError());
  return SA_OK;
}

}  // namespace

extern "C" {

sa_status sa_kv_assemble(sa_ctx* ctx, const sa_layout* layout, const void* k_src,
                         const void* v_src, void* k_dst, void* v_dst, int32_t batch,
                         const int32_t* h_src_len, const int32_t* h_keep_indptr,
                         const int32_t* h_keep_spans, const int32_t* h_reserve, sa_pages src,
                         const int32_t* d_fresh, int32_t num_fresh, int32_t* d_dst_indptr,
                         int32_t* d_dst_indices, int32_t dst_capacity, int32_t* h_dst_len,
                         void* stream) {
  return splice_launch(ctx, layout, k_src, v_src, k_dst, v_dst, batch, h_src_len, h_keep_indptr,
                       h_keep_spans, h_reserve, src, d_fresh, num_fresh, d_dst_indptr, d_dst_indices,
                       dst_capacity, h_dst_len, 0, nullptr, nullptr, nullptr, stream);
}

sa_status sa_kv_assemble_append(sa_ctx* ctx, const sa_layout* layout, const void* k_src,
                                const void* v_src, void* k_dst, void* v_dst, int32_t batch,
                                const int32_t* h_src_len, const int32_t* h_keep_indptr,
                                const int32_t* h_keep_spans, const int32_t* h_reserve, sa_pages src,
                                const int32_t* d_fresh, int32_t num_fresh, int32_t* d_dst_indptr,
                                int32_t* d_dst_indices, int32_t dst_capacity, int32_t* h_dst_len,
                                int32_t layer, const void* k_new, const void* v_new,
                                const int32_t* h_new_len, void* stream) {
  if (!h_new_len) return fail(SA_ERR_NULL, "h_new_len is NULL");
  return splice_launch(ctx, layout, k_src, v_src, k_dst, v_dst, batch, h_src_len, h_keep_indptr,
                       h_keep_spans, h_reserve, src, d_fresh, num_fresh, d_dst_indptr, d_dst_indices,
                       dst_capacity, h_dst_len, layer, k_new, v_new, h_new_len, stream);
}

sa_status sa_kv_splice_alias(sa_ctx* ctx, const sa_layout* layout, int32_t batch,
                             const int32_t* h_src_len, const int32_t* h_keep_indptr,
                             const int32_t* h_keep_spans, const int32_t* h_reserve, sa_pages src,
                             const int32_t* d_fresh, int32_t num_fresh, int32_t* d_dst_indptr,
                             int32_t* d_dst_indices, int32_t dst_capacity, int32_t* h_dst_len,
                             void* stream) {
  SplicePlan sp;
  sa_status s = plan_splice(layout, batch, h_src_len, h_keep_indptr, h_keep_spans, h_reserve, true,
                            num_fresh, dst_capacity, h_dst_len, sp);
  if (s != SA_OK) return s;
  if (!src.indptr || !d_dst_indptr || (!sp.units.empty() && !src.indices) || (sp.n_dst > 0 && !d_dst_indices) ||
      (sp.fresh_used > 0 && !d_fresh))
    return fail(SA_ERR_NULL, "a device pointer is NULL");
  s = check_ctx(ctx);
  if (s != SA_OK) return s;
  memcpy(h_dst_len, sp.dst_len.data(), sizeof(int32_t) * batch);

  PlanImage img;
  const size_t o_un = img.add(sp.units.data(), sp.units.size());
  const size_t o_ip = img.add(sp.dst_indptr.data(), sp.dst_indptr.size());
  const size_t o_en = img.add(sp.entry.data(), sp.entry.size());
  uint8_t* dev = nullptr;
  s = upload_plan(ctx, kPlanAlias, img, (hipStream_t)stream, &dev);
  if (s != SA_OK) return s;

  sa::AliasArgs a{};
  a.units = (const sa::AsmUnit*)(dev + o_un);
  a.entry = (const int32_t*)(dev + o_en);
  a.dst_indptr = (const int32_t*)(dev + o_ip);
  a.src_indptr = src.indptr;
  a.src_indices = src.indices;
  a.fresh = d_fresh;
  a.out_indptr = d_dst_indptr;
  a.out_indices = d_dst_indices;
  a.err = ctx->d_err;
  a.num_slots = layout->num_slots;
  a.n_dst = (int32_t)sp.n_dst;
  a.B = batch;
  const int64_t blocks = (std::max<int64_t>(sp.n_dst, batch + 1) + 255) / 256;
  launch_timed(sa::splice_alias_kernel, dim3((unsigned)blocks), dim3(256), (hipStream_t)stream,
               ctx->kernel_ev[SA_TIMED_PAGES], a);
  SA_HIP(hipGetLastError());
  return SA_OK;
}

// ---------------------------------------------------------------- attention

}  // extern "C"

namespace {

// The attention launch; with `append` it first writes each sequence's q_len
// new K/V rows (k_new, v_new) to its positions kv_len - q_len .. kv_len - 1:
// as an append launch before the attention, or inside the attention launch
// (append_in_attention()).
int64_t item_tiles(const sa::AttnItem& it) { return (it.kv_end - it.kv_begin + sa::kKT - 1) / sa::kKT; }

// Longest first within each XCD's queue.
void sort_longest_first(std::vector<sa::AttnItem>& q) {
  std::stable_sort(q.begin(), q.end(),
                   [](const sa::AttnItem& x, const sa::AttnItem& y) { return item_tiles(x) > item_tiles(y); });
}

// Key tiles of the most loaded CU of an XCD whose queue q is sorted longest
// first and runs in at most two rounds of `round` blocks, the second reversed
// (block k and block round + k share a CU): q[k] + q[n - 1 - k].
int64_t busiest_cu(const std::vector<sa::AttnItem>& q, size_t round) {
  const size_t n = q.size();
  int64_t m = 0;
  for (size_t k = 0; k < std::min(n, round); ++k)
    m = std::max<int64_t>(m, item_tiles(q[k]) + (k + round < n ? item_tiles(q[n - 1 - k]) : 0));
  return m;
}

// The XCDs of one chip do not run equally fast under this load (measured:
// the slowest one's workgroups take ~5-7% longer than the fastest one's on
// the same work, whichever KV head it serves), and the launch ends with the
// slowest.  Given relative speeds, move work from the XCD whose busiest CU
// has the most key tiles per unit of speed to the one with the fewest, by
// swapping the longest item of the first for the shortest of the second
// while neither ends above the first's present cost: every XCD keeps its number of
// items, so the launch keeps its rounds; the items that move read another
// KV head's K/V than their XCD's others, which the balance pays for.
// Queues of at most two rounds come back sorted longest first.
void weigh_xcds(std::vector<std::vector<sa::AttnItem>>& queue, size_t round, const float* speed) {
  // More than two rounds: each XCD's CUs take its items as they free; moving
  // the last items of the most loaded XCD to the least loaded one was tried
  // and measured -1.5% to +1.4% on 16 ragged contexts and on a 64K-key
  // context, so those launches are left as placed.
  for (const auto& q : queue)
    if (q.size() > 2 * round) return;
  for (auto& q : queue) sort_longest_first(q);
  double cost[kNumXcd];
  for (int x = 0; x < kNumXcd; ++x) cost[x] = busiest_cu(queue[x], round) / speed[x];
  for (int iter = 0; iter < 4096; ++iter) {
    int s = 0, f = 0;
    for (int x = 1; x < kNumXcd; ++x) {
      if (cost[x] > cost[s]) s = x;
      if (cost[x] < cost[f]) f = x;
    }
    if (s == f || queue[s].empty() || queue[f].empty()) return;
    auto& qs = queue[s];
    auto& qf = queue[f];
    if (item_tiles(qs.front()) <= item_tiles(qf.back())) return;
    std::vector<sa::AttnItem> ns = qs, nf = qf;
    std::swap(ns.front(), nf.back());
    sort_longest_first(ns);
    sort_longest_first(nf);
    // a swap may leave s's busiest CU where it was (another CU of s carries as
    // much): it is taken as long as neither XCD ends above s's present cost,
    // since it lowers s's total and the next swaps then lower that CU
    const double cs = busiest_cu(ns, round) / speed[s], cf = busiest_cu(nf, round) / speed[f];
    if (cs > cost[s] || cf >= cost[s]) return;
    qs.swap(ns);
    qf.swap(nf);
    cost[s] = cs;
    cost[f] = cf;
  }
}

sa_status attn_launch(sa_ctx* ctx, const sa_layout* layout, int32_t layer, const void* q,
                      const void* k_pool, const void* v_pool, bool append, const void* k_new,
                      const void* v_new, int32_t batch, const int32_t* h_q_len, const int32_t* h_kv_len,
                      sa_pages pages, float softmax_scale, void* o, float* lse, void* stream) {
  sa_status s = check_layout(layout);
  if (s != SA_OK) return s;
  if (layer < 0 || layer >= layout->num_layers)
    return fail(SA_ERR_SHAPE, "layer %d outside [0, %d)", layer, layout->num_layers);
  if (batch < 1) return fail(SA_ERR_SHAPE, "batch %d < 1", batch);
  if (!h_q_len || !h_kv_len) return fail(SA_ERR_NULL, "h_q_len / h_kv_len is NULL");
  if (!std::isfinite(softmax_scale) || softmax_scale <= 0.f)
    return fail(SA_ERR_SHAPE, "softmax_scale must be finite and positive");
  const int Hq = layout->num_q_heads, Hkv = layout->num_kv_heads, G = Hq / Hkv;
  std::vector<sa::SeqDesc> seqs(batch);
  int64_t total_q = 0;
  for (int b = 0; b < batch; ++b) {
    if (h_q_len[b] < 0 || h_q_len[b] > h_kv_len[b])
      return fail(SA_ERR_SHAPE, "sequence %d: need 0 <= q_len (%d) <= kv_len (%d)", b, h_q_len[b],
                  h_kv_len[b]);
    if ((int64_t)h_q_len[b] * G > INT32_MAX - sa::kMaxRows)
      return fail(SA_ERR_SHAPE, "sequence %d: q_len * G too large", b);
    seqs[b] = {(int32_t)total_q, h_q_len[b], h_kv_len[b], 0};
    total_q += h_q_len[b];
    if (total_q > INT32_MAX) return fail(SA_ERR_SHAPE, "too many query tokens");
  }
  if (total_q > 0 && (!q || !o)) return fail(SA_ERR_NULL, "q / o is NULL");
  if (!k_pool || !v_pool || !pages.indptr || !pages.indices)
    return fail(SA_ERR_NULL, "pool or page table pointer is NULL");
  if (!aligned16(q) || !aligned16(o) || !aligned16(k_pool) || !aligned16(v_pool) ||
      (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(SA_ERR_ALIGN, "q, o, pools must be 16-byte aligned (lse 4-byte)");
  if (append && total_q > 0 && (!k_new || !v_new)) return fail(SA_ERR_NULL, "k_new / v_new is NULL");
  if (append && (!aligned16(k_new) || !aligned16(v_new)))
    return fail(SA_ERR_ALIGN, "new-row pointer not 16-byte aligned");
  s = check_ctx(ctx);
  if (s != SA_OK) return s;
  if (total_q == 0) return SA_OK;

  // ---- kernel variant: query rows per wave (32 * qt) and waves per work item
  const AttnVariant var = attn_variant();
  // the exact-scale form of the pipelined kernel has no in-launch append
  const bool exact = ctx->exact_scale && var.pipe == 1;
  const bool fused = append && var.pipe == 1 && !exact && append_in_attention();
  if (append && !fused) {
    // the new rows go in with an append launch of their own
    std::vector<int32_t> start(batch);
    for (int b = 0; b < batch; ++b) start[b] = h_kv_len[b] - h_q_len[b];
    s = sa_kv_append(ctx, layout, layer, const_cast<void*>(k_pool), const_cast<void*>(v_pool), k_new, v_new,
                     batch, start.data(), h_q_len, pages, stream);
    if (s != SA_OK) return s;
  }
  const int rows_item = 32 * var.qt * var.waves;

  // ---- work items: (sequence, kv head, row tile), longest first
  struct Work {
    sa::AttnItem it;
    int64_t tiles;
    bool decode;
    int xcd;
    int64_t group = 0;         // items that stay together in the launch order
    int64_t group_tiles = 0;   // the longest item of that group
  };
  std::vector<Work> work;
  int64_t total_tiles = 0;
  for (int b = 0; b < batch; ++b) {
    const int ql = h_q_len[b];
    if (ql == 0) continue;
    const int rows = ql * G, pre = h_kv_len[b] - ql;
    for (int g = 0; g < Hkv; ++g)
      for (int r0 = 0; r0 < rows; r0 += rows_item) {
        const int last = std::min(r0 + rows_item - 1, rows - 1);
        const int kv_end = pre + last / G + 1;
        const int64_t tiles = (kv_end + sa::kKT - 1) / sa::kKT;
        work.push_back({{b, g, r0, 0, kv_end, -1}, tiles, rows <= 32, (b * Hkv + g) % kNumXcd});
        total_tiles += tiles;
      }
  }
  // Split long items by key range when there are too few to fill the chip:
  // always below one item per CU; below two per CU (both workgroup slots of
  // a CU) only when items average >= 128 key tiles, where the pairing gains
  // more than the partial-merge launch costs (measured: a CU's two blocks
  // together run ~1.3x one alone; the merge adds ~10-15 us).
  std::vector<sa::MergeGroup> groups;
  int32_t n_parts = 0;
  const int64_t n_work = (int64_t)work.size();
  if (n_work < ctx->num_cu || (n_work < 2 * ctx->num_cu && total_tiles >= 128 * n_work)) {
    const int64_t chunk = std::max<int64_t>(16, (total_tiles + 2 * ctx->num_cu - 1) / (2 * ctx->num_cu));
    std::vector<Work> split;
    for (const Work& w : work) {
      if (w.tiles <= chunk) {
        split.push_back(w);
        continue;
      }
      const int64_t n = (w.tiles + chunk - 1) / chunk;
      groups.push_back({w.it.seq, w.it.kvh, w.it.row0, (int32_t)n, n_parts, 0});
      for (int64_t k = 0; k < n; ++k) {
        Work p = w;
        p.it.kv_begin = (int32_t)(k * chunk * sa::kKT);
        p.it.kv_end = (int32_t)std::min<int64_t>((k + 1) * chunk * sa::kKT, w.it.kv_end);
        p.it.part = n_parts++;
        p.tiles = (p.it.kv_end - p.it.kv_begin + sa::kKT - 1) / sa::kKT;
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
  const bool one_block_per_cu = var.pipe == 2;
  auto pair_rounds = [one_block_per_cu](std::vector<sa::AttnItem>& q, size_t first_round) {
    if (one_block_per_cu) return;
    if (q.size() > first_round && q.size() <= 2 * first_round) std::reverse(q.begin() + first_round, q.end());
  };
  std::vector<sa::AttnItem> items;
  if (mx > 0 && (double)(mx - mn) <= 0.1 * (double)mx) {
    std::vector<std::vector<sa::AttnItem>> queue(kNumXcd);
    for (const Work& w : work) queue[w.xcd].push_back(w.it);
    if (ctx->xcd_weighted) {
      bool same = ctx->wq_in.size() == queue.size();
      for (size_t x = 0; same && x < queue.size(); ++x)
        same = ctx->wq_in[x].size() == queue[x].size() &&
               memcmp(ctx->wq_in[x].data(), queue[x].data(), queue[x].size() * sizeof(sa::AttnItem)) == 0;
      if (same) {
        queue = ctx->wq_out;
      } else {
        ctx->wq_in = queue;
        weigh_xcds(queue, (size_t)std::max(1, ctx->num_cu / kNumXcd), ctx->xcd_weight);
        ctx->wq_out = queue;
      }
    }
    for (auto& qd : queue) pair_rounds(qd, (size_t)std::max(1, ctx->num_cu / kNumXcd));
    size_t depth = 0;
    for (auto& qd : queue) depth = std::max(depth, qd.size());
    items.assign(depth * kNumXcd, sa::AttnItem{0, 0, 0, 0, 0, -1});
    for (int x = 0; x < kNumXcd; ++x)
      for (size_t i = 0; i < queue[x].size(); ++i) items[i * kNumXcd + x] = queue[x][i];
  } else {
    for (const Work& w : work) items.push_back(w.it);
    pair_rounds(items, (size_t)ctx->num_cu);
  }
  for (sa::AttnItem& x : items) {
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
  if (!one_block_per_cu && items.size() > (size_t)ctx->num_cu && items.size() <= 2 * (size_t)ctx->num_cu) {
    constexpr double kSlowShare = 0.715;
    auto tiles_of = [](const sa::AttnItem& x) {
      return x.kv_end > x.kv_begin ? (x.kv_end + sa::kKT - 1) / sa::kKT - x.kv_begin / sa::kKT : 0;
    };
    for (size_t b = ctx->num_cu; b < items.size(); ++b) {
      const double l_new = tiles_of(items[b]), l_old = tiles_of(items[b - ctx->num_cu]);
      const double x = 0.5 * ((l_old + l_new) / (1.0 + kSlowShare) - (l_old - l_new) / (1.0 - kSlowShare));
      items[b].boost = (int32_t)std::lround(std::min(std::max(x, 0.0), l_new));
    }
  }

  if (n_parts > 0) {
    const size_t need = (size_t)n_parts * rows_item * (sa::kHD + 1) * sizeof(float);
    if (need > ctx->part_cap) {
      if (ctx->part) {
        SA_HIP(hipDeviceSynchronize());
        SA_HIP(hipFree(ctx->part));
        ctx->part = nullptr;
      }
      SA_HIP(hipMalloc(&ctx->part, need));
      ctx->part_cap = need;
    }
  }

  PlanImage img;
  const size_t o_seq = img.add(seqs.data(), seqs.size());
  const size_t o_it = img.add(items.data(), items.size());
  const size_t o_gr = img.add(groups.data(), groups.size());
  uint8_t* dev = nullptr;
  s = upload_plan(ctx, kPlanAttn, img, (hipStream_t)stream, &dev);
  if (s != SA_OK) return s;

  sa::AttnArgs a{};
  const int64_t lo = (int64_t)layer * layer_elems(layout);
  a.q = (const uint16_t*)q;
  a.k = (const uint16_t*)k_pool + lo;
  a.v = (const uint16_t*)v_pool + lo;
  a.o = (uint16_t*)o;
  a.lse = lse;
  a.part_o = ctx->part;
  a.part_lse = ctx->part ? ctx->part + (size_t)n_parts * rows_item * sa::kHD : nullptr;
  a.items = (const sa::AttnItem*)(dev + o_it);
  a.seqs = (const sa::SeqDesc*)(dev + o_seq);
  a.indptr = pages.indptr;
  a.indices = pages.indices;
  a.err = ctx->d_err;
  a.num_slots = (int32_t)layout->num_slots;
  a.n_items = (int32_t)items.size();
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.G = G;
  a.c = softmax_scale * 1.4426950408889634f;
  a.B = batch;
  if (fused) {
    a.k_new = (const uint16_t*)k_new;
    a.v_new = (const uint16_t*)v_new;
    a.sync = ctx->d_sync;
    a.app_chunks = total_q * Hkv * 16;
    // whole groups of 64 tickets (one wave's draw) cover the chunks
    const int64_t tickets = (a.app_chunks + 64 * sa::kAppTicket - 1) / (64 * sa::kAppTicket) * 64;
    if (tickets > INT32_MAX / 2) return fail(SA_ERR_SHAPE, "too many new rows for one launch");
    a.app_tickets = (int32_t)tickets;
  }
  if (ctx->blk_clock != nullptr && var.pipe == 1) {
    if ((int64_t)items.size() > ctx->blk_clock_cap)
      return fail(SA_ERR_SHAPE, "block clock buffer holds %lld blocks, the launch has %zu",
                  (long long)ctx->blk_clock_cap, items.size());
    a.blk_clock = ctx->blk_clock;
  }
  const bool pool_rsrc = layer_elems(layout) * 2 < ((int64_t)1 << 31);
  launch_attn(layout->page_size, var, pool_rsrc, exact, dim3((unsigned)items.size()), (hipStream_t)stream,
              ctx->kernel_ev[SA_TIMED_ATTN], a);
  SA_HIP(hipGetLastError());
  if (!groups.empty()) {
    sa::MergeArgs m{};
    m.part_o = a.part_o;
    m.part_lse = a.part_lse;
    m.groups = (const sa::MergeGroup*)(dev + o_gr);
    m.seqs = a.seqs;
    m.o = a.o;
    m.lse = lse;
    m.Hq = Hq;
    m.G = G;
    m.rows = rows_item;
    hipLaunchKernelGGL(sa::merge_kernel, dim3((unsigned)groups.size(), (unsigned)((rows_item + 31) / 32)), dim3(256), 0,
                       (hipStream_t)stream, m);
    SA_HIP(hipGetLastError());
  }
  return SA_OK;
}

}  // namespace

extern "C" {

sa_status sa_segment_prefill_attn(sa_ctx* ctx, const sa_layout* layout, int32_t layer,
                                  const void* q, const void* k_pool, const void* v_pool,
                                  int32_t batch, const int32_t* h_q_len, const int32_t* h_kv_len,
                                  sa_pages pages, float softmax_scale, void* o, float* lse,
                                  void* stream) {
  return attn_launch(ctx, layout, layer, q, k_pool, v_pool, false, nullptr, nullptr, batch, h_q_len,
                     h_kv_len, pages, softmax_scale, o, lse, stream);
}

sa_status sa_set_exact_scale(sa_ctx* ctx, int32_t enable) {
  sa_status s = check_ctx(ctx);
  if (s != SA_OK) return s;
  ctx->exact_scale = enable != 0;
  return SA_OK;
}

sa_status sa_set_kernel_events(sa_ctx* ctx, int32_t which, void* start_event, void* stop_event) {
  sa_status s = check_ctx(ctx);
  if (s != SA_OK) return s;
  if (which != SA_TIMED_ATTN && which != SA_TIMED_PAGES)
    return fail(SA_ERR_SHAPE, "sa_set_kernel_events: which = %d (SA_TIMED_ATTN or SA_TIMED_PAGES)", which);
  if ((start_event == nullptr) != (stop_event == nullptr))
    return fail(SA_ERR_NULL, "sa_set_kernel_events: give both events or neither");
  ctx->kernel_ev[which][0] = (hipEvent_t)start_event;
  ctx->kernel_ev[which][1] = (hipEvent_t)stop_event;
  return SA_OK;
}

sa_status sa_set_xcd_weights(sa_ctx* ctx, const float* h_speed) {
  sa_status s = check_ctx(ctx);
  if (s != SA_OK) return s;
  if (h_speed == nullptr) {
    ctx->xcd_weighted = false;
    for (float& w : ctx->xcd_weight) w = 1.f;
    return SA_OK;
  }
  for (int x = 0; x < kNumXcd; ++x)
    if (!(h_speed[x] > 0.f) || !std::isfinite(h_speed[x]))
      return fail(SA_ERR_SHAPE, "sa_set_xcd_weights: speed[%d] = %g (must be finite and > 0)", x, h_speed[x]);
  for (int x = 0; x < kNumXcd; ++x) ctx->xcd_weight[x] = h_speed[x];
  ctx->xcd_weighted = true;
  ctx->wq_in.clear();                                      // new speeds: search again
  ctx->wq_out.clear();
  return SA_OK;
}

sa_status sa_set_block_clock(sa_ctx* ctx, void* d_buf, int64_t max_blocks, int64_t* clock_khz) {
  sa_status s = check_ctx(ctx);
  if (s != SA_OK) return s;
  if ((d_buf == nullptr) != (max_blocks == 0) || max_blocks < 0)
    return fail(SA_ERR_SHAPE, "sa_set_block_clock: a buffer needs max_blocks > 0, none needs 0");
  if (d_buf != nullptr && (reinterpret_cast<uintptr_t>(d_buf) & 7u) != 0)
    return fail(SA_ERR_ALIGN, "sa_set_block_clock: buffer not 8-byte aligned");
  if (clock_khz != nullptr) {
    int khz = 0;
    SA_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, ctx->device));
    *clock_khz = khz;
  }
  ctx->blk_clock = (uint64_t*)d_buf;
  ctx->blk_clock_cap = max_blocks;
  return SA_OK;
}

sa_status sa_segment_prefill_attn_append(sa_ctx* ctx, const sa_layout* layout, int32_t layer,
                                         const void* q, void* k_pool, void* v_pool, const void* k_new,
                                         const void* v_new, int32_t batch, const int32_t* h_q_len,
                                         const int32_t* h_kv_len, sa_pages pages, float softmax_scale,
                                         void* o, float* lse, void* stream) {
  return attn_launch(ctx, layout, layer, q, k_pool, v_pool, true, k_new, v_new, batch, h_q_len,
                     h_kv_len, pages, softmax_scale, o, lse, stream);
}

}  // extern "C"
