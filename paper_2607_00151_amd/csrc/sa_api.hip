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
#include <mutex>
#include <vector>

#include "sa.h"
#include "plan.h"
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

// Fixed device scratch of sa_segment_prefill_attn_noalloc: the launch's plan
// (sequence records, work items, merge groups) in its first kNoAllocPlanBytes,
// the key-range partials of split items after it.  Every device the library
// runs on holds one copy for the life of the process, shared by all contexts
// on that device.
constexpr size_t kNoAllocBytes = size_t(32) << 20;
constexpr size_t kNoAllocPlanBytes = size_t(2) << 20;
constexpr int kMaxDevices = 64;

}  // namespace

static __device__ __align__(256) uint8_t scratch[kNoAllocBytes];

namespace {

// Device address of `scratch` on each device: the array's name is only a
// host-side stand-in, so host code uses this address (looked up once per
// device, with that device current) wherever it needs the array's memory.
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

hipError_t scratch_address(int device, void** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  if (g_scratch_ptr[device] == nullptr) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[device] = ptr;
  }
  *out = g_scratch_ptr[device];
  return hipSuccess;
}

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
  bool exact_scale = true;         // sa_set_exact_scale (0: scale folded into q)
  bool fused_append = false;       // sa_set_fused_append (0, the default: append launch, then attention)
  hipEvent_t kernel_ev[2][2] = {};   // sa_set_kernel_events: [SA_TIMED_ATTN | SA_TIMED_PAGES][start, stop]
  uint64_t* blk_clock = nullptr;     // sa_set_block_clock: device buffer, 4 words per block
  int64_t blk_clock_cap = 0;         // blocks it holds
  sa::XcdState xcd;                  // sa_set_xcd_weights and the last weighting
  // buffers outgrown by a larger plan: kernels already enqueued may still read
  // them, so they are freed with the context rather than behind a device sync
  std::vector<void*> retired_dev, retired_host;
  // sa_segment_prefill_attn_noalloc: this device's `scratch` array, and pinned
  // staging for the plans copied into it
  uint8_t* scratch = nullptr;
  void* na_host = nullptr;
  hipEvent_t na_ev = nullptr;
  bool na_pending = false;
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
    if (dp.dev) ctx->retired_dev.push_back(dp.dev);   // an enqueued kernel may still read it
    dp.dev = nullptr;
    dp.cap = 0;
    dp.valid = false;
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
    if (st.host) ctx->retired_host.push_back(st.host);   // its last copy has completed
    st.host = nullptr;
    st.cap = 0;
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

sa_status check_layout(const sa_layout* L) { return sa::check_layout(L, g_err); }
using sa::layer_elems;
using sa::slot_elems;

// SA_DEBUG=1 (read once per process): the page-table and free-list checks of
// plan.h run before each splice and append (they copy the tables back to the
// host, so they are for debugging only).
bool debug_checks() {
  static bool v = [] {
    const char* e = getenv("SA_DEBUG");
    return e != nullptr && atoi(e) == 1;
  }();
  return v;
}

// Host copy of a device page table: indptr [batch + 1] and all its entries.
sa_status fetch_table(const int32_t* d_indptr, const int32_t* d_indices, int32_t batch, hipStream_t stream,
                      std::vector<int32_t>& indptr, std::vector<int32_t>& indices) {
  SA_HIP(hipStreamSynchronize(stream));
  indptr.assign(batch + 1, 0);
  SA_HIP(hipMemcpy(indptr.data(), d_indptr, sizeof(int32_t) * (batch + 1), hipMemcpyDeviceToHost));
  if (indptr[0] < 0 || indptr[batch] < indptr[0])
    return fail(SA_ERR_RANGE, "page table indptr runs from %d to %d", indptr[0], indptr[batch]);
  for (int b = 0; b < batch; ++b)
    if (indptr[b + 1] < indptr[b]) return fail(SA_ERR_RANGE, "page table indptr decreases at %d", b);
  indices.assign(indptr[batch], 0);
  if (indptr[batch] > 0 && d_indices == nullptr) return fail(SA_ERR_NULL, "page table indices are NULL");
  if (indptr[batch] > 0)
    SA_HIP(hipMemcpy(indices.data(), d_indices, sizeof(int32_t) * indptr[batch], hipMemcpyDeviceToHost));
  return SA_OK;
}

// SA_DEBUG check of a splice plan against the device's source table and free list.
sa_status debug_splice(const sa::SplicePlan& sp, sa_pages src, const int32_t* d_fresh, int32_t batch,
                       int64_t num_slots, bool alias, hipStream_t stream) {
  std::vector<int32_t> ip, ix;
  sa_status s = fetch_table(src.indptr, src.indices, batch, stream, ip, ix);
  if (s != SA_OK) return s;
  std::vector<int32_t> surv(sp.units.size()), fresh(sp.fresh_used);
  for (size_t u = 0; u < sp.units.size(); ++u) {
    const sa::AsmUnit& x = sp.units[u];
    if (x.src_page >= ip[x.seq + 1] - ip[x.seq])
      return fail(SA_ERR_RANGE, "sequence %d: surviving page %d is not in its source table (%d pages)", x.seq,
                  x.src_page, ip[x.seq + 1] - ip[x.seq]);
    surv[u] = ix[ip[x.seq] + x.src_page];
  }
  if (sp.fresh_used > 0)
    SA_HIP(hipMemcpy(fresh.data(), d_fresh, sizeof(int32_t) * sp.fresh_used, hipMemcpyDeviceToHost));
  return sa::debug_check_splice(sp, surv.data(), fresh.data(), num_slots, alias, g_err);
}

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

// read: the pipelined kernel that also writes the segment's rows and reads
// the segment's keys from them (pool_rsrc only)
template <int P>
void launch_attn_p(AttnVariant v, bool pool_rsrc, bool exact, bool read, dim3 grid, hipStream_t st,
                   const hipEvent_t* ev, const sa::AttnArgs& a) {
  if (v.pipe == 1 && read && exact)
    launch_timed(sa::attn_pipe_kernel<P, true, true, true>, grid, dim3(256), st, ev, a);
  else if (v.pipe == 1 && read)
    launch_timed(sa::attn_pipe_kernel<P, true, true, false>, grid, dim3(256), st, ev, a);
  else if (v.pipe == 1 && exact && pool_rsrc)
    launch_timed(sa::attn_pipe_kernel<P, true, false, true>, grid, dim3(256), st, ev, a);
  else if (v.pipe == 1 && exact)
    launch_timed(sa::attn_pipe_kernel<P, false, false, true>, grid, dim3(256), st, ev, a);
  else if (v.pipe == 2 && pool_rsrc)
    launch_timed(sa::attn_pp_kernel<P, true>, grid, dim3(512), st, ev, a);
  else if (v.pipe == 2)
    launch_timed(sa::attn_pp_kernel<P, false>, grid, dim3(512), st, ev, a);
  else if (v.pipe && pool_rsrc)
    launch_timed(sa::attn_pipe_kernel<P, true, false>, grid, dim3(256), st, ev, a);
  else if (v.pipe)
    launch_timed(sa::attn_pipe_kernel<P, false, false>, grid, dim3(256), st, ev, a);
  else
    launch_timed(sa::attn_kernel<P, 1, 4>, grid, dim3(256), st, ev, a);
}

// pool_rsrc: a layer's K (and V) pool spans < 2^31 bytes, so one buffer
// resource per pool addresses every page with a 32-bit offset
void launch_attn(int page_size, AttnVariant v, bool pool_rsrc, bool exact, bool read, dim3 grid, hipStream_t st,
                 const hipEvent_t* ev, const sa::AttnArgs& a) {
  if (page_size == 16) launch_attn_p<16>(v, pool_rsrc, exact, read, grid, st, ev, a);
  else launch_attn_p<32>(v, pool_rsrc, exact, read, grid, st, ev, a);
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
    case SA_ERR_OVERLAP: return "slot lists overlap or repeat";
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
  if (e == hipSuccess) e = hipDeviceSynchronize();
  for (int i = 0; e == hipSuccess && i < kRing; ++i)
    e = hipEventCreateWithFlags(&c->ring[i].ev, hipEventDisableTiming);
  if (e == hipSuccess) e = scratch_address(device, (void**)&c->scratch);
  if (e == hipSuccess) e = hipHostMalloc(&c->na_host, kNoAllocPlanBytes, hipHostMallocDefault);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->na_ev, hipEventDisableTiming);
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
  for (void* p : ctx->retired_dev) (void)hipFree(p);
  for (void* p : ctx->retired_host) (void)hipHostFree(p);
  if (ctx->d_err) (void)hipFree(ctx->d_err);
  if (ctx->na_host) (void)hipHostFree(ctx->na_host);
  if (ctx->na_ev) (void)hipEventDestroy(ctx->na_ev);
  delete ctx;
}

sa_status sa_reserve(sa_ctx* ctx, int64_t plan_bytes, int64_t split_bytes) {
  sa_status s = check_ctx(ctx);
  if (s != SA_OK) return s;
  if (plan_bytes < 0 || split_bytes < 0) return fail(SA_ERR_SHAPE, "sa_reserve: negative size");
  const size_t pb = align_up((size_t)plan_bytes, 4096);
  for (auto& dp : ctx->plans)
    if (dp.cap < pb) {
      if (dp.dev) ctx->retired_dev.push_back(dp.dev);
      dp.dev = nullptr;
      dp.cap = 0;
      dp.valid = false;
      SA_HIP(hipMalloc(&dp.dev, pb));
      dp.cap = pb;
    }
  for (auto& st : ctx->ring)
    if (st.cap < pb) {
      if (st.pending) {
        SA_HIP(hipEventSynchronize(st.ev));
        st.pending = false;
      }
      if (st.host) ctx->retired_host.push_back(st.host);
      st.host = nullptr;
      st.cap = 0;
      SA_HIP(hipHostMalloc(&st.host, pb, hipHostMallocDefault));
      st.cap = pb;
    }
  if (ctx->part_cap < (size_t)split_bytes) {
    if (ctx->part) ctx->retired_dev.push_back(ctx->part);
    ctx->part = nullptr;
    ctx->part_cap = 0;
    SA_HIP(hipMalloc(&ctx->part, (size_t)split_bytes));
    ctx->part_cap = (size_t)split_bytes;
  }
  return SA_OK;
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
  if (debug_checks()) {
    std::vector<int32_t> ip, ix;
    s = fetch_table(pages.indptr, pages.indices, batch, (hipStream_t)stream, ip, ix);
    if (s != SA_OK) return s;
    s = sa::debug_check_append(batch, h_start, h_new_len, ip.data(), ix.data(), layout->page_size,
                               layout->num_slots, g_err);
    if (s != SA_OK) return s;
  }

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


// The copy splice, and with new_len non-NULL an append of new rows of layer
// `layer` behind each sequence's kept tokens in the same launch.
sa_status splice_launch(sa_ctx* ctx, const sa_layout* layout, const void* k_src, const void* v_src,
                        void* k_dst, void* v_dst, int32_t batch, const int32_t* h_src_len,
                        const int32_t* h_keep_indptr, const int32_t* h_keep_spans, const int32_t* h_reserve,
                        sa_pages src, const int32_t* d_fresh, int32_t num_fresh, int32_t* d_dst_indptr,
                        int32_t* d_dst_indices, int32_t dst_capacity, int32_t* h_dst_len, int32_t layer,
                        const void* k_new, const void* v_new, const int32_t* h_new_len, void* stream) {
  sa::SplicePlan sp;
  sa_status s = sa::plan_splice(layout, batch, h_src_len, h_keep_indptr, h_keep_spans, h_reserve, false, num_fresh,
                                dst_capacity, sp, g_err);
  if (s != SA_OK) return s;
  if (!h_dst_len) return fail(SA_ERR_NULL, "h_dst_len is NULL");
  const int64_t units = (int64_t)sp.units.size(), n_dst = sp.n_dst;
  const int P = layout->page_size;
  const bool app = h_new_len != nullptr;
  sa::SpliceAppendPlan ap;
  if (app) {
    s = sa::plan_splice_append(layout, batch, h_new_len, layer, sp, ap, g_err);
    if (s != SA_OK) return s;
    if (ap.all_new > 0 && (!k_new || !v_new)) return fail(SA_ERR_NULL, "k_new / v_new is NULL");
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
  if (debug_checks()) {
    s = debug_splice(sp, src, d_fresh, batch, layout->num_slots, false, (hipStream_t)stream);
    if (s != SA_OK) return s;
  }
  memcpy(h_dst_len, sp.dst_len.data(), sizeof(int32_t) * batch);

  PlanImage img;
  const size_t o_un = img.add(sp.units.data(), sp.units.size());
  const size_t o_ip = img.add(sp.dst_indptr.data(), sp.dst_indptr.size());
  const size_t o_at = img.add(ap.tok_begin.data(), app ? ap.tok_begin.size() : 0);
  const size_t o_as = img.add(ap.start.data(), app ? ap.start.size() : 0);
  const size_t o_ak = img.add(ap.knew.data(), app ? ap.knew.size() : 0);
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
    a.app_chunks = ap.total * layout->num_kv_heads * 16;
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
  sa::SplicePlan sp;
  sa_status s = sa::plan_splice(layout, batch, h_src_len, h_keep_indptr, h_keep_spans, h_reserve, true, num_fresh,
                                dst_capacity, sp, g_err);
  if (s != SA_OK) return s;
  if (!h_dst_len) return fail(SA_ERR_NULL, "h_dst_len is NULL");
  if (!src.indptr || !d_dst_indptr || (!sp.units.empty() && !src.indices) || (sp.n_dst > 0 && !d_dst_indices) ||
      (sp.fresh_used > 0 && !d_fresh))
    return fail(SA_ERR_NULL, "a device pointer is NULL");
  s = check_ctx(ctx);
  if (s != SA_OK) return s;
  if (debug_checks()) {
    s = debug_splice(sp, src, d_fresh, batch, layout->num_slots, true, (hipStream_t)stream);
    if (s != SA_OK) return s;
  }
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

// The attention launch; with `append` each sequence's q_len new K/V rows
// (k_new, v_new) also go to its positions kv_len - q_len .. kv_len - 1: by the
// attention launch itself, which then reads the segment's keys from k_new /
// v_new (ctx->fused_append, the pipelined kernel, a pool and new rows that a
// buffer resource spans), else by an append launch before the attention.
//
// With `noalloc` the plan and the split partials go to this device's fixed
// `scratch` array (no append then): the plan must fit kNoAllocPlanBytes, and
// split items are coarsened until their partials fit the rest.
sa_status attn_launch(sa_ctx* ctx, const sa_layout* layout, int32_t layer, const void* q,
                      const void* k_pool, const void* v_pool, bool append, const void* k_new,
                      const void* v_new, int32_t batch, const int32_t* h_q_len, const int32_t* h_kv_len,
                      sa_pages pages, float softmax_scale, void* o, float* lse, void* stream,
                      bool noalloc = false) {
  std::vector<sa::SeqDesc> seqs;
  int64_t total_q = 0;
  sa_status s = sa::plan_attn_check(layout, layer, batch, h_q_len, h_kv_len, softmax_scale, seqs, total_q, g_err);
  if (s != SA_OK) return s;
  const int Hq = layout->num_q_heads, Hkv = layout->num_kv_heads, G = Hq / Hkv;
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
  const bool exact = ctx->exact_scale && var.pipe == 1;
  const bool pool_rsrc = layer_elems(layout) * 2 < ((int64_t)1 << 31);
  const int64_t new_bytes = total_q * Hkv * sa::kHD * 2;
  const bool fused = append && ctx->fused_append && var.pipe == 1 && pool_rsrc && new_bytes < ((int64_t)1 << 31);
  if (fused && debug_checks()) {
    // the rows the launch writes (sa_kv_append checks its own): no two
    // sequences write one slot row
    std::vector<int32_t> ip, ix, start(batch);
    s = fetch_table(pages.indptr, pages.indices, batch, (hipStream_t)stream, ip, ix);
    if (s != SA_OK) return s;
    for (int b = 0; b < batch; ++b) start[b] = h_kv_len[b] - h_q_len[b];
    s = sa::debug_check_append(batch, start.data(), h_q_len, ip.data(), ix.data(), layout->page_size,
                               layout->num_slots, g_err);
    if (s != SA_OK) return s;
  }
  if (append && !fused) {
    // the new rows go in with an append launch of their own
    std::vector<int32_t> start(batch);
    for (int b = 0; b < batch; ++b) start[b] = h_kv_len[b] - h_q_len[b];
    s = sa_kv_append(ctx, layout, layer, const_cast<void*>(k_pool), const_cast<void*>(v_pool), k_new, v_new,
                     batch, start.data(), h_q_len, pages, stream);
    if (s != SA_OK) return s;
  }
  const int rows_item = 32 * var.qt * var.waves;

  sa::AttnShape shape;
  shape.rows_item = rows_item;
  shape.num_cu = ctx->num_cu;
  shape.pair_rounds = var.pipe != 2;      // the two-group kernel runs one block per CU
  const size_t part_bytes = (size_t)rows_item * (sa::kHD + 1) * sizeof(float);   // one key-range part
  if (noalloc) shape.max_parts = (int64_t)((kNoAllocBytes - kNoAllocPlanBytes) / part_bytes);
  sa::AttnPlan plan;
  sa::plan_attn_items(layout, seqs, shape, &ctx->xcd, plan);
  std::vector<sa::AttnItem>& items = plan.items;
  std::vector<sa::MergeGroup>& groups = plan.groups;
  const int32_t n_parts = plan.n_parts;

  if (n_parts > 0 && !noalloc) {
    const size_t need = (size_t)n_parts * rows_item * (sa::kHD + 1) * sizeof(float);
    if (need > ctx->part_cap) {
      if (ctx->part) ctx->retired_dev.push_back(ctx->part);    // an enqueued merge may still read it
      ctx->part = nullptr;
      ctx->part_cap = 0;
      SA_HIP(hipMalloc(&ctx->part, need));
      ctx->part_cap = need;
    }
  }

  PlanImage img;
  const size_t o_seq = img.add(seqs.data(), seqs.size());
  const size_t o_it = img.add(items.data(), items.size());
  const size_t o_gr = img.add(groups.data(), groups.size());
  uint8_t* dev = nullptr;
  float* part = ctx->part;
  if (noalloc) {
    // the plan goes to the front of the fixed scratch, through pinned staging
    // whose previous copy must have been read first; the partials follow it
    const size_t n = img.bytes.size();
    if (n > kNoAllocPlanBytes)
      return fail(SA_ERR_SHAPE, "the launch's plan needs %zu bytes; the fixed scratch of the allocation-free "
                  "entry point holds %zu (about %zu work items)", n, kNoAllocPlanBytes,
                  kNoAllocPlanBytes / sizeof(sa::AttnItem));
    if (ctx->na_pending) {
      SA_HIP(hipEventSynchronize(ctx->na_ev));
      ctx->na_pending = false;
    }
    memcpy(ctx->na_host, img.bytes.data(), n);
    SA_HIP(hipMemcpyAsync(ctx->scratch, ctx->na_host, n, hipMemcpyHostToDevice, (hipStream_t)stream));
    SA_HIP(hipEventRecord(ctx->na_ev, (hipStream_t)stream));
    ctx->na_pending = true;
    dev = ctx->scratch;
    part = (float*)(ctx->scratch + kNoAllocPlanBytes);
  } else {
    s = upload_plan(ctx, kPlanAttn, img, (hipStream_t)stream, &dev);
    if (s != SA_OK) return s;
  }

  sa::AttnArgs a{};
  const int64_t lo = (int64_t)layer * layer_elems(layout);
  a.q = (const uint16_t*)q;
  a.k = (const uint16_t*)k_pool + lo;
  a.v = (const uint16_t*)v_pool + lo;
  a.o = (uint16_t*)o;
  a.lse = lse;
  a.part_o = n_parts > 0 ? part : nullptr;
  a.part_lse = n_parts > 0 ? part + (size_t)n_parts * rows_item * sa::kHD : nullptr;
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
  if (fused) {
    a.k_new = (const uint16_t*)k_new;
    a.v_new = (const uint16_t*)v_new;
    a.new_bytes = (uint32_t)new_bytes;
  }
  if (ctx->blk_clock != nullptr && var.pipe == 1) {
    if ((int64_t)items.size() > ctx->blk_clock_cap)
      return fail(SA_ERR_SHAPE, "block clock buffer holds %lld blocks, the launch has %zu",
                  (long long)ctx->blk_clock_cap, items.size());
    a.blk_clock = ctx->blk_clock;
  }
  launch_attn(layout->page_size, var, pool_rsrc, exact, fused, dim3((unsigned)items.size()), (hipStream_t)stream,
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

sa_status sa_attn_plan_stats(const sa_layout* layout, int32_t batch, const int32_t* h_q_len,
                             const int32_t* h_kv_len, int32_t num_cu, int64_t* out) {
  std::vector<sa::SeqDesc> seqs;
  int64_t total_q = 0;
  sa_status s = sa::plan_attn_check(layout, 0, batch, h_q_len, h_kv_len, 1.f, seqs, total_q, g_err);
  if (s != SA_OK) return s;
  if (!out) return fail(SA_ERR_NULL, "out is NULL");
  if (num_cu < 1) return fail(SA_ERR_SHAPE, "num_cu %d < 1", num_cu);
  const AttnVariant var = attn_variant();
  sa::AttnShape shape;
  shape.rows_item = 32 * var.qt * var.waves;
  shape.num_cu = num_cu;
  shape.pair_rounds = var.pipe != 2;
  sa::AttnPlan plan;
  sa::plan_attn_items(layout, seqs, shape, nullptr, plan);
  const sa::AttnPlanStats st = sa::attn_plan_stats(plan, seqs, layout->num_q_heads / layout->num_kv_heads, num_cu);
  out[0] = st.items;
  out[1] = st.parts;
  out[2] = st.tiles;
  out[3] = st.makespan_tiles;
  return SA_OK;
}

sa_status sa_segment_prefill_attn_noalloc(sa_ctx* ctx, const sa_layout* layout, int32_t layer,
                                          const void* q, const void* k_pool, const void* v_pool,
                                          int32_t batch, const int32_t* h_q_len, const int32_t* h_kv_len,
                                          sa_pages pages, float softmax_scale, void* o, float* lse,
                                          void* stream) {
  return attn_launch(ctx, layout, layer, q, k_pool, v_pool, false, nullptr, nullptr, batch, h_q_len, h_kv_len,
                     pages, softmax_scale, o, lse, stream, true);
}

sa_status sa_set_exact_scale(sa_ctx* ctx, int32_t enable) {
  sa_status s = check_ctx(ctx);
  if (s != SA_OK) return s;
  ctx->exact_scale = enable != 0;
  return SA_OK;
}

sa_status sa_set_fused_append(sa_ctx* ctx, int32_t enable) {
  sa_status s = check_ctx(ctx);
  if (s != SA_OK) return s;
  ctx->fused_append = enable != 0;
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
    ctx->xcd = sa::XcdState{};
    return SA_OK;
  }
  for (int x = 0; x < sa::kNumXcd; ++x)
    if (!(h_speed[x] > 0.f) || !std::isfinite(h_speed[x]))
      return fail(SA_ERR_SHAPE, "sa_set_xcd_weights: speed[%d] = %g (must be finite and > 0)", x, h_speed[x]);
  for (int x = 0; x < sa::kNumXcd; ++x) ctx->xcd.speed[x] = h_speed[x];
  ctx->xcd.weighted = true;
  ctx->xcd.in.clear();                                      // new speeds: search again
  ctx->xcd.out.clear();
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
