// C ABI of the memory-slice hot path (declared in include/ema_slice.h).
//
// One handle = host bookkeeping (SliceBook) + two separately allocated device
// pools + library scratch, all allocated at create: a kernel error counter, an
// upload area for the plans and copy lists that reclaim and run prefetches
// build on the host (with its pinned host staging, sized for the largest
// plan), and the stream-K attention workspace (partials and combine records
// for the largest batch the stream-K form takes). Only the grid form of
// attention (batches above the stream-K limit, or EMA_CREATE_ATTN_GRID) grows
// a workspace on first use; growing synchronizes the device.
#include "ema_slice.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <exception>
#include <memory>
#include <new>
#include <string>
#include <vector>

#include "kernels.h"
#include "slice_book.h"

struct ema_slice {
  ema_kv_shape shape{};
  int64_t bb = 0;
  bool host_only = false;
  bool checked = false;
  int device = -1;
  ema::SliceBook book;
  char* local = nullptr;
  char* slice = nullptr;
  int32_t* d_err = nullptr;
  int32_t* d_work = nullptr;
  size_t work_cap = 0;          // ints
  int32_t* h_work = nullptr;    // pinned
  size_t h_work_cap = 0;        // ints
  hipEvent_t h_work_ev = nullptr;   // after the last upload from h_work
  bool h_work_pending = false;
  hipEvent_t d_work_ev = nullptr;   // after the last kernel that read d_work
  bool d_work_pending = false;
  float* d_part = nullptr;          // stream-K partial slots (fixed size)
  size_t part_cap = 0;              // floats
  int32_t* d_info = nullptr;        // stream-K: per (sequence, KV head) partial ranges
  size_t info_cap = 0;              // ints
  float* d_gpart = nullptr;         // grid form: split-K partials (grows)
  size_t gpart_cap = 0;             // floats
  bool attn_grid = false;           // EMA_CREATE_ATTN_GRID: always the grid form
  void* noalloc_ws = nullptr;       // this device's fixed workspace (not owned)
  // slab mode: every layer group's swap sources (staging order), on the device
  int32_t* d_slab = nullptr;
  int32_t* h_slab = nullptr;        // pinned
  size_t slab_cap = 0;              // ints
  int64_t slab_built = -1;          // slab version the device lists were built for
  int32_t slab_m = 0;               // borrowed slabs when they were built
  hipEvent_t slab_up_ev = nullptr;  // after the last upload of the lists
  hipEvent_t slab_use_ev = nullptr; // after the last kernel that read them
  bool slab_up_pending = false, slab_use_pending = false;
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

}  // namespace

namespace ema {
// Records the message behind an error code for ema_last_error (used by the
// scheduler's entry points too).
int set_error(int code, const std::string& msg) { return fail(code, msg); }

// Called from the catch handler of every entry point: no C++ exception
// crosses the C ABI; host allocation failures become EMA_ERR_NOMEM.
int internal_error() {
  try {
    throw;
  } catch (const std::bad_alloc&) {
    return fail(EMA_ERR_NOMEM, "out of host memory");
  } catch (const std::exception& e) {
    return fail(EMA_ERR_INVAL, std::string("internal error: ") + e.what());
  } catch (...) {
    return fail(EMA_ERR_INVAL, "internal error");
  }
}
}  // namespace ema

using ema::internal_error;

namespace {

int hip_fail(hipError_t e, const char* what) {
  return fail(EMA_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(call, what)                    \
  do {                                         \
    hipError_t e_ = (call);                    \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

bool supported_block_size(int bs) {
  return bs == 16 || bs == 32 || bs == 64 || bs == 128 || bs == 256;
}

ema::PoolView pool_view(const ema_slice* h) {
  ema::PoolView pv;
  pv.local = h->local;
  pv.slice = h->slice;
  pv.block_bytes = h->bb;
  pv.n_local = h->book.n_local();
  pv.n_slice = h->book.n_slice();
  pv.kv_heads = h->shape.num_kv_heads;
  pv.block_size = h->shape.block_size;
  pv.slice_layout = h->shape.slice_layout;
  return pv;
}

// Makes the handle's device current for the rest of an entry point and puts
// the caller's device back when the entry point returns.
class DeviceScope {
 public:
  DeviceScope() = default;
  DeviceScope(const DeviceScope&) = delete;
  DeviceScope& operator=(const DeviceScope&) = delete;
  ~DeviceScope() {
    if (prev_ >= 0) (void)hipSetDevice(prev_);
  }
  int enter(const ema_slice* h) {
    int cur = -1;
    HIP_TRY(hipGetDevice(&cur), "hipGetDevice");
    if (cur != h->device) {
      HIP_TRY(hipSetDevice(h->device), "hipSetDevice");
      prev_ = cur;
    }
    return EMA_OK;
  }

 private:
  int prev_ = -1;
};

// Reads n ints of a device array to the host (checked mode).
int fetch_ints(const int32_t* dev, int64_t n, hipStream_t st, std::vector<int32_t>* out) {
  out->resize(size_t(n));
  if (n == 0) return EMA_OK;
  HIP_TRY(hipMemcpyAsync(out->data(), dev, size_t(n) * 4, hipMemcpyDeviceToHost, st),
          "hipMemcpyAsync(check)");
  HIP_TRY(hipStreamSynchronize(st), "hipStreamSynchronize(check)");
  return EMA_OK;
}

int grow_device(void** p, size_t* cap, size_t need, size_t elem, hipStream_t st) {
  if (need <= *cap) return EMA_OK;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  HIP_TRY(hipStreamIsCapturing(st, &cs), "hipStreamIsCapturing");
  if (cs != hipStreamCaptureStatusNone)
    return fail(EMA_ERR_INVAL, "attention: the grid-form workspace would grow during stream "
                               "capture; run a call of this size once before capturing");
  HIP_TRY(hipDeviceSynchronize(), "hipDeviceSynchronize(grow)");
  if (*p) HIP_TRY(hipFree(*p), "hipFree(grow)");
  *p = nullptr;
  *cap = 0;
  size_t n = need + need / 4;
  HIP_TRY(hipMalloc(p, n * elem), "hipMalloc(scratch)");
  *cap = n;
  return EMA_OK;
}

void release(ema_slice* h) {
  if (!h->host_only) {
    (void)hipDeviceSynchronize();
    if (h->local) (void)hipFree(h->local);
    if (h->slice) (void)hipFree(h->slice);
    if (h->d_err) (void)hipFree(h->d_err);
    if (h->d_work) (void)hipFree(h->d_work);
    if (h->d_part) (void)hipFree(h->d_part);
    if (h->d_info) (void)hipFree(h->d_info);
    if (h->d_gpart) (void)hipFree(h->d_gpart);
    if (h->h_work) (void)hipHostFree(h->h_work);
    if (h->h_work_ev) (void)hipEventDestroy(h->h_work_ev);
    if (h->d_work_ev) (void)hipEventDestroy(h->d_work_ev);
    if (h->d_slab) (void)hipFree(h->d_slab);
    if (h->h_slab) (void)hipHostFree(h->h_slab);
    if (h->slab_up_ev) (void)hipEventDestroy(h->slab_up_ev);
    if (h->slab_use_ev) (void)hipEventDestroy(h->slab_use_ev);
  }
  delete h;
}

// Contiguous runs of a copy list (src[i + 1] == src[i] + 1 and likewise dst),
// or false when there are more than max_runs of them.
bool list_runs(const std::vector<int32_t>& src, const std::vector<int32_t>& dst, int max_runs,
               std::vector<int32_t>* rs, std::vector<int32_t>* rd, std::vector<int32_t>* rn) {
  rs->clear();
  rd->clear();
  rn->clear();
  for (size_t i = 0; i < src.size(); ++i) {
    if (!rn->empty() && rs->back() + rn->back() == src[i] && rd->back() + rn->back() == dst[i]) {
      ++rn->back();
      continue;
    }
    if (int(rn->size()) == max_runs) return false;
    rs->push_back(src[i]);
    rd->push_back(dst[i]);
    rn->push_back(1);
  }
  return true;
}

// A set of block ids as a bitmap over [base, base + n): bit i of word i / 32
// stands for id base + i.
struct Bits {
  int32_t base = 0;
  int32_t n = 0;
  size_t words = 0;
};
Bits bit_span(const std::vector<int32_t>& ids) {
  Bits b;
  if (ids.empty()) return b;
  const auto mm = std::minmax_element(ids.begin(), ids.end());
  b.base = *mm.first;
  b.n = *mm.second - *mm.first + 1;
  b.words = (size_t(b.n) + 31) / 32;
  return b;
}
void put_bits(const std::vector<int32_t>& ids, const Bits& b, uint32_t* w) {
  std::fill(w, w + b.words, 0u);
  for (int32_t u : ids) {
    const uint32_t i = uint32_t(u - b.base);
    w[i >> 5] |= 1u << (i & 31);
  }
}

// The plan upload area (h_work -> d_work) is shared by reclaim and run
// prefetches, which may be issued on different streams. begin_upload waits on
// the host until the previous upload has left h_work, and makes `st` wait on
// the device until the previous kernels that read d_work have finished;
// end_upload marks the point after this call's kernels.
int begin_upload(ema_slice* h, hipStream_t st) {
  if (h->h_work_pending) {
    HIP_TRY(hipEventSynchronize(h->h_work_ev), "hipEventSynchronize(upload)");
    h->h_work_pending = false;
  }
  if (h->d_work_pending) HIP_TRY(hipStreamWaitEvent(st, h->d_work_ev, 0), "hipStreamWaitEvent");
  return EMA_OK;
}

int upload(ema_slice* h, size_t n_ints, hipStream_t st) {
  HIP_TRY(hipMemcpyAsync(h->d_work, h->h_work, n_ints * 4, hipMemcpyHostToDevice, st),
          "hipMemcpyAsync(upload)");
  HIP_TRY(hipEventRecord(h->h_work_ev, st), "hipEventRecord(upload)");
  h->h_work_pending = true;
  return EMA_OK;
}

int end_upload(ema_slice* h, hipStream_t st) {
  HIP_TRY(hipEventRecord(h->d_work_ev, st), "hipEventRecord(kernels)");
  h->d_work_pending = true;
  return EMA_OK;
}

}  // namespace

extern "C" {

const char* ema_last_error(void) { return g_err.c_str(); }

int ema_slice_create(const ema_kv_shape* shape, size_t local_bytes, size_t lent_bytes,
                     uint32_t flags, ema_slice_t* out) try {
  if (!shape || !out) return fail(EMA_ERR_INVAL, "create: NULL argument");
  *out = nullptr;
  if (shape->num_kv_heads < 1 || shape->num_kv_heads > 64 || shape->head_dim != 128 ||
      !supported_block_size(shape->block_size) ||
      (shape->dtype != EMA_F16 && shape->dtype != EMA_BF16) ||
      (shape->slice_layout != EMA_LAYOUT_ATTN && shape->slice_layout != EMA_LAYOUT_NHD))
    return fail(EMA_ERR_INVAL, "create: unsupported shape");
  if (flags & ~(EMA_CREATE_HOST_ONLY | EMA_CREATE_CHECKED | EMA_CREATE_ATTN_GRID))
    return fail(EMA_ERR_INVAL, "create: unknown flags");
  const int64_t bb = 2LL * shape->block_size * shape->num_kv_heads * shape->head_dim * 2;
  const uint64_t nl = local_bytes / uint64_t(bb), ns = lent_bytes / uint64_t(bb);
  if (nl + ns >= (1ull << 31)) return fail(EMA_ERR_INVAL, "create: more than 2^31 blocks");

  // Owned here until the handle is complete: an exception on the way (host
  // memory) releases it.
  std::unique_ptr<ema_slice, void (*)(ema_slice*)> guard(new ema_slice, release);
  ema_slice* h = guard.get();
  h->shape = *shape;
  h->bb = bb;
  h->host_only = (flags & EMA_CREATE_HOST_ONLY) != 0;
  h->checked = (flags & EMA_CREATE_CHECKED) != 0;
  h->attn_grid = (flags & EMA_CREATE_ATTN_GRID) != 0;
  h->book.init(int32_t(nl), int32_t(ns));
  if (h->host_only) {
    *out = guard.release();
    return EMA_OK;
  }
  hipError_t e = hipGetDevice(&h->device);
  const int32_t n_total = int32_t(nl + ns);
  if (e == hipSuccess && nl) e = hipMalloc(&h->local, nl * bb);
  if (e == hipSuccess && ns) e = hipMalloc(&h->slice, ns * bb);
  if (e == hipSuccess) e = hipMalloc(&h->d_err, 4);
  if (e == hipSuccess) e = hipMemset(h->d_err, 0, 4);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&h->h_work_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&h->d_work_ev, hipEventDisableTiming);
  // Reclaim's plan upload (movers' sources and destinations, the returned
  // range's remap, the released blocks outside it: at most 4 ints per block)
  // and run prefetches' block lists (2 per block), so neither ever allocates.
  const size_t work = size_t(4) * size_t(n_total > 0 ? n_total : 1) + 16;
  if (e == hipSuccess) e = hipHostMalloc(&h->h_work, work * 4, hipHostMallocDefault);
  if (e == hipSuccess) h->h_work_cap = work;
  if (e == hipSuccess) e = hipMalloc(&h->d_work, work * 4);
  if (e == hipSuccess) h->work_cap = work;
  // Stream-K attention workspace for every head count and the largest batch.
  const size_t part = size_t(2) * ema::attn_streamk_grid() * ema::kMaxGroup * (ema::kHeadDim + 2);
  const size_t info = size_t(ema::streamk_max_batch(1)) * shape->num_kv_heads * 3;
  if (e == hipSuccess) e = hipMalloc(&h->d_part, part * 4);
  if (e == hipSuccess) h->part_cap = part;
  if (e == hipSuccess) e = hipMalloc(&h->d_info, info * 4);
  if (e == hipSuccess) h->info_cap = info;
  // the no-allocation attention call's workspace on this device
  if (e == hipSuccess) e = ema::noalloc_workspace(&h->noalloc_ws);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "create");   // the guard releases h
  *out = guard.release();
  return EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slice_destroy(ema_slice_t h) try {
  if (!h) return fail(EMA_ERR_INVAL, "destroy: NULL handle");
  if (!h->host_only) {
    DeviceScope ds;
    int rc = ds.enter(h);
    if (rc) return rc;
  }
  release(h);
  return EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slice_get_info(ema_slice_t h, ema_slice_info* out) try {
  if (!h || !out) return fail(EMA_ERR_INVAL, "info: NULL argument");
  out->block_bytes = h->bb;
  out->n_local = h->book.n_local();
  out->n_slice = h->book.n_slice();
  out->lim = h->book.lim();
  out->free_local = h->book.free_local();
  out->free_slice = h->book.free_slice();
  out->device = h->device;
  out->local_base = h->local;
  out->slice_base = h->slice;
  return EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slice_owners(ema_slice_t h, int32_t* own_local, int32_t* own_slice) try {
  if (!h) return fail(EMA_ERR_INVAL, "owners: NULL handle");
  if (own_local && h->book.n_local())
    std::memcpy(own_local, h->book.own_local().data(), size_t(h->book.n_local()) * 4);
  if (own_slice && h->book.n_slice())
    std::memcpy(own_slice, h->book.own_slice().data(), size_t(h->book.n_slice()) * 4);
  return EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slice_alloc_blocks(ema_slice_t h, int32_t pool, int32_t n, const int32_t* owners,
                           int32_t* out_ids) try {
  if (!h) return fail(EMA_ERR_INVAL, "alloc: NULL handle");
  std::string err;
  const int rc = h->book.alloc(pool, n, owners, out_ids, &err);
  return rc ? fail(rc, err) : EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slice_free_blocks(ema_slice_t h, const int32_t* ids, int32_t n) try {
  if (!h) return fail(EMA_ERR_INVAL, "free: NULL handle");
  std::string err;
  const int rc = h->book.free_blocks(ids, n, &err);
  return rc ? fail(rc, err) : EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slice_lend(ema_slice_t h, int32_t n_blocks, int32_t* added) try {
  if (!h) return fail(EMA_ERR_INVAL, "lend: NULL handle");
  std::string err;
  const int rc = h->book.lend(n_blocks, added, &err);
  return rc ? fail(rc, err) : EMA_OK;
} catch (...) {
  return internal_error();
}

enum class CopyKind { kPrefetch, kMigrate, kWriteback };

static int check_copy(const ema_slice* h, CopyKind kind, const int32_t* src, const int32_t* dst,
                      int32_t n, std::string* err) {
  switch (kind) {
    case CopyKind::kPrefetch: return h->book.check_prefetch(src, dst, n, err);
    case CopyKind::kMigrate: return h->book.check_migrate(src, dst, n, err);
    default: return h->book.check_writeback(src, dst, n, err);
  }
}

static int copy_entry(ema_slice_t h, const int32_t* src, const int32_t* dst, int32_t n,
                      void* stream, CopyKind kind) {
  const char* what = kind == CopyKind::kPrefetch ? "prefetch"
                     : kind == CopyKind::kMigrate ? "migrate"
                                                  : "writeback";
  if (!h) return fail(EMA_ERR_INVAL, std::string(what) + ": NULL handle");
  if (n < 0 || (n > 0 && (!src || !dst)))
    return fail(EMA_ERR_INVAL, std::string(what) + ": n < 0 or NULL array");
  std::string err;
  if (h->host_only) {
    const int rc = check_copy(h, kind, src, dst, n, &err);
    return rc ? fail(rc, err) : EMA_OK;
  }
  if (n == 0) return EMA_OK;
  DeviceScope ds;
  int rc = ds.enter(h);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (h->checked) {
    std::vector<int32_t> hs, hd;
    if ((rc = fetch_ints(src, n, st, &hs)) || (rc = fetch_ints(dst, n, st, &hd))) return rc;
    rc = check_copy(h, kind, hs.data(), hd.data(), n, &err);
    if (rc) return fail(rc, err);
  }
  HIP_TRY(ema::launch_block_copy(pool_view(h), src, dst, n, h->d_err, st), what);
  return EMA_OK;
}

int ema_slice_prefetch(ema_slice_t h, const int32_t* block_ids, const int32_t* dst_block_table,
                       int32_t n, void* stream) try {
  return copy_entry(h, block_ids, dst_block_table, n, stream, CopyKind::kPrefetch);
} catch (...) {
  return internal_error();
}

int ema_slice_migrate(ema_slice_t h, const int32_t* src_ids, const int32_t* dst_ids, int32_t n,
                      void* stream) try {
  return copy_entry(h, src_ids, dst_ids, n, stream, CopyKind::kMigrate);
} catch (...) {
  return internal_error();
}

int ema_slice_prefetch_runs(ema_slice_t h, const int32_t* src_first, const int32_t* dst_first,
                            const int32_t* run_blocks, int32_t n_runs, int32_t engine,
                            void* stream) try {
  if (!h) return fail(EMA_ERR_INVAL, "prefetch_runs: NULL handle");
  if (n_runs < 0 || (n_runs > 0 && (!src_first || !dst_first || !run_blocks)))
    return fail(EMA_ERR_INVAL, "prefetch_runs: n_runs < 0 or NULL array");
  if (engine != EMA_ENGINE_KERNEL && engine != EMA_ENGINE_DMA)
    return fail(EMA_ERR_INVAL, "prefetch_runs: unknown engine");
  if (engine == EMA_ENGINE_DMA && h->shape.slice_layout != EMA_LAYOUT_ATTN)
    return fail(EMA_ERR_INVAL, "prefetch_runs: the copy engines need the slice in the local layout");
  const int64_t n_total = int64_t(h->book.n_local()) + h->book.n_slice();
  int64_t blocks = 0;
  for (int32_t r = 0; r < n_runs; ++r) {
    const int64_t a = src_first[r], b = dst_first[r], k = run_blocks[r];
    if (k < 0 || a < 0 || b < 0 || a + k > n_total || b + k > n_total || blocks + k > n_total)
      return fail(EMA_ERR_INVAL, "prefetch_runs: run out of range");
    blocks += k;
  }
  std::vector<int32_t> src, dst;
  src.reserve(size_t(blocks));
  dst.reserve(size_t(blocks));
  for (int32_t r = 0; r < n_runs; ++r) {
    const int64_t a = src_first[r], b = dst_first[r], k = run_blocks[r];
    for (int64_t i = 0; i < k; ++i) {
      src.push_back(int32_t(a + i));
      dst.push_back(int32_t(b + i));
    }
  }
  const int32_t n = int32_t(src.size());
  std::string err;
  int rc = h->book.check_prefetch(src.data(), dst.data(), n, &err);
  if (rc) return fail(rc, err);
  if (h->host_only || n == 0) return EMA_OK;
  DeviceScope ds;
  if ((rc = ds.enter(h))) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (engine == EMA_ENGINE_DMA) {
    const ema::PoolView pv = pool_view(h);
    for (int32_t r = 0; r < n_runs; ++r) {
      if (run_blocks[r] == 0) continue;
      char* d = pv.local + int64_t(dst_first[r]) * h->bb;
      const char* sp = pv.slice + (int64_t(src_first[r]) - pv.n_local) * h->bb;
      HIP_TRY(hipMemcpyAsync(d, sp, size_t(run_blocks[r]) * h->bb, hipMemcpyDeviceToDeviceNoCU, st),
              "prefetch_runs copy");
    }
    return EMA_OK;
  }
  if (n_runs <= ema::kArgRuns) {      // the runs travel in the launch arguments
    HIP_TRY(ema::launch_block_copy_runs(pool_view(h), src_first, dst_first, run_blocks, n_runs,
                                        h->d_err, st),
            "prefetch_runs launch");
    return EMA_OK;
  }
  if (size_t(2) * n > h->h_work_cap || size_t(2) * n > h->work_cap)
    return fail(EMA_ERR_INVAL, "prefetch_runs: more blocks than the plan buffer holds");
  if ((rc = begin_upload(h, st))) return rc;
  std::copy(src.begin(), src.end(), h->h_work);
  std::copy(dst.begin(), dst.end(), h->h_work + n);
  if ((rc = upload(h, size_t(2) * n, st))) return rc;
  HIP_TRY(ema::launch_block_copy(pool_view(h), h->d_work, h->d_work + n, n, h->d_err, st, true),
          "prefetch_runs launch");
  return end_upload(h, st);
} catch (...) {
  return internal_error();
}

int ema_slice_writeback(ema_slice_t h, const int32_t* staging_ids, const int32_t* slice_ids,
                        int32_t n, void* stream) try {
  return copy_entry(h, staging_ids, slice_ids, n, stream, CopyKind::kWriteback);
} catch (...) {
  return internal_error();
}

int ema_kv_append(ema_slice_t h, const void* k_new, const void* v_new, const int32_t* block_table,
                  const int32_t* seq_lens, int32_t batch, int32_t max_blocks, void* stream) try {
  if (!h) return fail(EMA_ERR_INVAL, "append: NULL handle");
  if (batch < 0 || max_blocks < 0) return fail(EMA_ERR_INVAL, "append: bad batch or max_blocks");
  if (batch > 0 && (!k_new || !v_new || !block_table || !seq_lens))
    return fail(EMA_ERR_INVAL, "append: NULL array");
  if (batch > 65535) return fail(EMA_ERR_INVAL, "append: batch too large");
  const int32_t bs = h->shape.block_size;
  auto check = [&](const int32_t* lens, const int32_t* tab) -> int {
    for (int32_t b = 0; b < batch; ++b) {
      if (lens[b] <= 0) continue;
      const int32_t j = (lens[b] - 1) / bs;
      if (j >= max_blocks) return fail(EMA_ERR_INVAL, "append: position past the block table");
      const int32_t id = tab[size_t(b) * max_blocks + j];
      if (id < 0 || id >= h->book.n_local())
        return fail(EMA_ERR_INVAL, "append: target is not a local block");
    }
    return EMA_OK;
  };
  if (h->host_only) return batch ? check(seq_lens, block_table) : EMA_OK;
  if (batch == 0) return EMA_OK;
  DeviceScope ds;
  int rc = ds.enter(h);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (h->checked) {
    std::vector<int32_t> lens, tab;
    if ((rc = fetch_ints(seq_lens, batch, st, &lens)) ||
        (rc = fetch_ints(block_table, int64_t(batch) * max_blocks, st, &tab)))
      return rc;
    if ((rc = check(lens.data(), tab.data()))) return rc;
  }
  HIP_TRY(ema::launch_kv_append(pool_view(h), k_new, v_new, block_table, seq_lens, batch,
                                max_blocks, h->d_err, st),
          "append launch");
  return EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slice_reclaim(ema_slice_t h, int32_t n_blocks, int32_t* canon_tables, int64_t n_entries,
                      void* stream, ema_reclaim_result* result, int32_t* victims,
                      int32_t victims_cap, int32_t* moves_src, int32_t* moves_dst,
                      int32_t moves_cap) try {
  if (!h || !result) return fail(EMA_ERR_INVAL, "reclaim: NULL handle or result");
  if (n_blocks < 0 || n_entries < 0 || (n_entries > 0 && !canon_tables))
    return fail(EMA_ERR_INVAL, "reclaim: bad count or table pointer");
  if (h->host_only && (canon_tables || n_entries))
    return fail(EMA_ERR_INVAL, "reclaim: host-only slices take no device tables");
  int rc;
  DeviceScope ds;
  if (!h->host_only && (rc = ds.enter(h))) return rc;

  ema::ReclaimPlan plan;
  std::string err;
  rc = h->book.reclaim(n_blocks, &plan, &err);
  if (rc) return fail(rc, err);

  const int32_t m = int32_t(plan.move_src.size());
  const int32_t nv = int32_t(plan.victim_blocks.size());
  result->reclaimed = plan.reclaimed;
  result->moved = m;
  result->written_back = plan.written_back;
  result->n_victims = int32_t(plan.victims.size());
  result->lim = h->book.lim();
  if (victims)
    for (int32_t i = 0; i < result->n_victims && i < victims_cap; ++i) victims[i] = plan.victims[i];
  if (moves_src && moves_dst)
    for (int32_t i = 0; i < m && i < moves_cap; ++i) {
      moves_src[i] = plan.move_src[i];
      moves_dst[i] = plan.move_dst[i];
    }
  if (h->host_only) return EMA_OK;
  const bool rewrite = n_entries > 0 && (m > 0 || nv > 0);
  if (m == 0 && !rewrite) return EMA_OK;

  hipStream_t st = static_cast<hipStream_t>(stream);
  // Few runs and no preemption (the usual reclaim of a contiguous range): the
  // runs travel in the launch arguments and the rewrite maps the range through
  // them, with no upload at all.
  std::vector<int32_t> rs, rd, rn;
  if (nv == 0 && list_runs(plan.move_src, plan.move_dst, ema::kArgRuns, &rs, &rd, &rn)) {
    ema::TableRewrite rw;
    if (rewrite) {
      rw.tables = canon_tables;
      rw.n_entries = n_entries;
      rw.base = h->book.n_local() + plan.cut;
      rw.n_range = plan.reclaimed;
    }
    HIP_TRY(ema::launch_block_copy_runs(pool_view(h), rs.data(), rd.data(), rn.data(),
                                        int32_t(rn.size()), h->d_err, st, &rw),
            "reclaim launch");
    return EMA_OK;
  }
  // Upload: move sources [m] | destinations [m] | remap of the returned range
  // [n'] | bitmap of the released blocks outside the range. One launch then
  // copies the movers and (its first workgroups) rewrites the tables.
  const int32_t n_range = plan.reclaimed;
  const int32_t base = h->book.n_local() + plan.cut;
  std::vector<int32_t> vout;
  for (int32_t u : plan.victim_blocks)
    if (u < base || u >= base + n_range) vout.push_back(u);
  const Bits bits = bit_span(vout);
  const size_t need = size_t(2) * m + (rewrite ? size_t(n_range) + bits.words : 0);
  // movers, the range and released blocks are within n_total, so the buffers
  // sized at create always hold the plan
  if (need > h->h_work_cap || need > h->work_cap)
    return fail(EMA_ERR_INVAL, "reclaim: plan larger than the work buffers");
  if ((rc = begin_upload(h, st))) return rc;
  int32_t* w = h->h_work;
  std::copy(plan.move_src.begin(), plan.move_src.end(), w);
  std::copy(plan.move_dst.begin(), plan.move_dst.end(), w + m);
  if (rewrite) {
    int32_t* rmap = w + 2 * size_t(m);
    for (int32_t i = 0; i < n_range; ++i) rmap[i] = base + i;
    for (int32_t i = 0; i < m; ++i) rmap[plan.move_src[i] - base] = plan.move_dst[i];
    for (int32_t u : plan.victim_blocks)
      if (u >= base && u < base + n_range) rmap[u - base] = -1;
    put_bits(vout, bits, reinterpret_cast<uint32_t*>(rmap + n_range));
  }
  if ((rc = upload(h, need, st))) return rc;
  ema::TableRewrite rw;
  if (rewrite) {
    rw.tables = canon_tables;
    rw.n_entries = n_entries;
    rw.range_map = h->d_work + 2 * size_t(m);
    rw.released_bits = reinterpret_cast<const uint32_t*>(h->d_work + 2 * size_t(m) + n_range);
    rw.base = base;
    rw.n_range = n_range;
    rw.bits_base = bits.base;
    rw.n_bits = bits.n;
  }
  HIP_TRY(ema::launch_block_copy(pool_view(h), h->d_work, h->d_work + m, m, h->d_err, st, true,
                                 &rw),
          "reclaim launch");
  return end_upload(h, st);
} catch (...) {
  return internal_error();
}

}  // extern "C"

namespace {

// Both attention entry points. `noalloc`: stream-K only, in the fixed
// per-device workspace, no host validation (checked mode reads arrays back)
// and nothing that allocates.
int attention_call(ema_slice_t h, const void* q, const int32_t* block_table,
                   const int32_t* seq_lens, int32_t batch, int32_t num_q_heads,
                   int32_t max_blocks, float scale, void* out, int32_t out_dtype, void* stream,
                   bool noalloc) {
  if (!h) return fail(EMA_ERR_INVAL, "attention: NULL handle");
  const int32_t hkv = h->shape.num_kv_heads;
  if (batch < 0 || max_blocks < 0 || num_q_heads < hkv || num_q_heads % hkv != 0)
    return fail(EMA_ERR_INVAL, "attention: bad batch, max_blocks or head counts");
  const int32_t G = num_q_heads / hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8 && G != 16)
    return fail(EMA_ERR_INVAL, "attention: query heads per kv head must be 1, 2, 4, 8 or 16");
  if (out_dtype != EMA_F32 && out_dtype != EMA_F16 && out_dtype != EMA_BF16)
    return fail(EMA_ERR_INVAL, "attention: out_dtype must be EMA_F32, EMA_F16 or EMA_BF16");
  if (batch > 65535 || hkv > 65535) return fail(EMA_ERR_INVAL, "attention: grid too large");
  if (batch > 0 && (!q || !block_table || !seq_lens || !out))
    return fail(EMA_ERR_INVAL, "attention: NULL array");
  const int64_t max_tokens = int64_t(max_blocks) * h->shape.block_size;
  if (max_tokens > (1LL << 30)) return fail(EMA_ERR_INVAL, "attention: max_blocks too large");
  if (h->host_only || batch == 0) return EMA_OK;
  if (h->book.n_local() == 0) return fail(EMA_ERR_INVAL, "attention: the local pool is empty");
  DeviceScope ds;
  int rc = ds.enter(h);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (h->checked && !noalloc) {
    std::vector<int32_t> lens, tab;
    if ((rc = fetch_ints(seq_lens, batch, st, &lens)) ||
        (rc = fetch_ints(block_table, int64_t(batch) * max_blocks, st, &tab)))
      return rc;
    for (int32_t b = 0; b < batch; ++b) {
      if (lens[b] < 0 || lens[b] > max_tokens)
        return fail(EMA_ERR_INVAL, "attention: seq_len out of range");
      const int32_t nb = (lens[b] + h->shape.block_size - 1) / h->shape.block_size;
      for (int32_t j = 0; j < nb; ++j) {
        const int32_t id = tab[size_t(b) * max_blocks + j];
        if (id < 0 || id >= h->book.n_local())
          return fail(EMA_ERR_INVAL, "attention: block table entry is not a local block");
      }
    }
  }
  // Scheduling: stream-K (equal tile ranges, one workgroup per CU, at most two
  // partials each; workspace allocated at create) when the batch fits its LDS
  // work list, else a grid of 1024-token chunks with one partial per
  // (sequence, head, chunk) in a workspace that grows on first use.
  const int64_t tiles = int64_t(batch) * hkv * ((max_tokens + 31) / 32);
  const bool fits_streamk = batch <= ema::streamk_max_batch(G) && tiles < (int64_t(1) << 30);
  if (noalloc) {
    if (!fits_streamk)
      return fail(EMA_ERR_INVAL, "attention_noalloc: batch above the stream-K limit (4096, or "
                                 "2048 at 16 query heads per KV head) or max_blocks too large");
    if (int64_t(batch) * hkv > ema::kNoAllocPairs)
      return fail(EMA_ERR_INVAL, "attention_noalloc: batch * num_kv_heads above 32768");
    if (ema::attn_streamk_grid() > ema::kNoAllocGrid)
      return fail(EMA_ERR_INVAL, "attention_noalloc: more compute units than the fixed "
                                 "workspace holds (512)");
    if (!h->noalloc_ws) return fail(EMA_ERR_INVAL, "attention_noalloc: no fixed workspace");
  }
  const bool stream_k = noalloc || (!h->attn_grid && fits_streamk);
  const int32_t chunk = ema::kMfmaGridChunk;
  const int32_t n_split = int32_t(std::max<int64_t>(1, (max_tokens + chunk - 1) / chunk));
  if (!stream_k && n_split > 65535) return fail(EMA_ERR_INVAL, "attention: max_blocks too large");
  ema::AttnArgs a;
  float* part = nullptr;
  size_t part_rows = 0;
  if (noalloc) {
    part_rows = size_t(2) * ema::attn_streamk_grid() * G;
    part = static_cast<float*>(h->noalloc_ws);
    a.info = reinterpret_cast<int32_t*>(static_cast<char*>(h->noalloc_ws) +
                                        ema::kNoAllocPartFloats * 4);
  } else if (stream_k) {
    part_rows = size_t(2) * ema::attn_streamk_grid() * G;
    part = h->d_part;
    a.info = h->d_info;
  } else {
    if (n_split > 1) {
      part_rows = size_t(batch) * num_q_heads * n_split;
      if ((rc = grow_device(reinterpret_cast<void**>(&h->d_gpart), &h->gpart_cap,
                            part_rows * (ema::kHeadDim + 2), 4, st)))
        return rc;
    }
    part = h->d_gpart;
    a.info = nullptr;
  }
  a.q = q;
  a.table = block_table;
  a.seq_lens = seq_lens;
  a.out = out;
  a.out_dtype = out_dtype;
  a.part_o = part;
  a.part_ml = part ? part + part_rows * ema::kHeadDim : nullptr;
  a.stream_k = stream_k ? 1 : 0;
  a.err_count = h->d_err;
  a.local = h->local;
  a.block_bytes = h->bb;
  a.n_local = h->book.n_local();
  a.batch = batch;
  a.q_heads = num_q_heads;
  a.kv_heads = hkv;
  a.block_size = h->shape.block_size;
  a.max_blocks = max_blocks;
  a.n_split = n_split;
  a.dtype = h->shape.dtype;
  a.chunk = chunk;
  const float sc = scale > 0.0f ? scale : 1.0f / std::sqrt(float(h->shape.head_dim));
  a.scale_log2 = sc * 1.4426950408889634f;
  HIP_TRY(ema::launch_paged_attention_mfma(a, st), "attention launch");
  return EMA_OK;
}

}  // namespace

extern "C" {

int ema_paged_decode_attention(ema_slice_t h, const void* q, const int32_t* block_table,
                               const int32_t* seq_lens, int32_t batch, int32_t num_q_heads,
                               int32_t max_blocks, float scale, void* out, int32_t out_dtype,
                               void* stream) try {
  return attention_call(h, q, block_table, seq_lens, batch, num_q_heads, max_blocks, scale, out,
                        out_dtype, stream, false);
} catch (...) {
  return internal_error();
}

int ema_paged_decode_attention_noalloc(ema_slice_t h, const void* q, const int32_t* block_table,
                                       const int32_t* seq_lens, int32_t batch,
                                       int32_t num_q_heads, int32_t max_blocks, float scale,
                                       void* out, int32_t out_dtype, void* stream) try {
  return attention_call(h, q, block_table, seq_lens, batch, num_q_heads, max_blocks, scale, out,
                        out_dtype, stream, true);
} catch (...) {
  return internal_error();
}

// ---- slab mode ---------------------------------------------------------------

int ema_slab_init(ema_slice_t h, const ema_slab_cfg* cfg) try {
  if (!h || !cfg) return fail(EMA_ERR_INVAL, "slab_init: NULL argument");
  ema::SlabCfg c;
  c.layers = cfg->layers;
  c.slab_blocks = cfg->slab_blocks;
  c.group = cfg->group;
  c.layout = cfg->layout;
  if (h->host_only) {
    std::string err;
    const int rc = h->book.slab_init(c, &err);
    return rc ? fail(rc, err) : EMA_OK;
  }
  DeviceScope ds;
  int rc = ds.enter(h);
  if (rc) return rc;
  // device lists of every group's swap sources: at most every slabbed slot once
  const size_t cap = size_t(h->book.n_slice()) + 1;
  hipError_t e = hipSuccess;
  if (!h->d_slab) {
    e = hipMalloc(&h->d_slab, cap * 4);
    if (e == hipSuccess) e = hipHostMalloc(&h->h_slab, cap * 4, hipHostMallocDefault);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->slab_up_ev, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->slab_use_ev, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "slab_init");
    h->slab_cap = cap;
  }
  std::string err;
  rc = h->book.slab_init(c, &err);
  return rc ? fail(rc, err) : EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slab_get_info(ema_slice_t h, ema_slab_info* out, int32_t* slab_tag, int32_t* pos_owner) try {
  if (!h || !out) return fail(EMA_ERR_INVAL, "slab_info: NULL argument");
  if (!h->book.slab_mode()) return fail(EMA_ERR_INVAL, "slab_info: the slice is not in slabs");
  const ema::SlabCfg& c = h->book.slab_cfg();
  out->n_slabs = h->book.n_slabs();
  out->layers = c.layers;
  out->slab_blocks = c.slab_blocks;
  out->group = c.group;
  out->layout = c.layout;
  out->borrowed = int32_t(h->book.borrowed_slabs().size());
  if (slab_tag) std::copy(h->book.slab_tag().begin(), h->book.slab_tag().end(), slab_tag);
  if (pos_owner) std::copy(h->book.pos_owner().begin(), h->book.pos_owner().end(), pos_owner);
  return EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slab_alloc(ema_slice_t h, int32_t n, const int32_t* owners, int32_t* out_pos) try {
  if (!h) return fail(EMA_ERR_INVAL, "slab_alloc: NULL handle");
  std::string err;
  const int rc = h->book.slab_alloc(n, owners, out_pos, &err);
  return rc ? fail(rc, err) : EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slab_free(ema_slice_t h, const int32_t* pos, int32_t n) try {
  if (!h) return fail(EMA_ERR_INVAL, "slab_free: NULL handle");
  std::string err;
  const int rc = h->book.slab_free(pos, n, &err);
  return rc ? fail(rc, err) : EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slab_block_ids(ema_slice_t h, const int32_t* pos, int32_t n, int32_t layer,
                       int32_t staging_first, int32_t* out_ids) try {
  if (!h) return fail(EMA_ERR_INVAL, "slab_block_ids: NULL handle");
  if (!h->book.slab_mode()) return fail(EMA_ERR_INVAL, "slab_block_ids: the slice is not in slabs");
  if (n < 0 || (n > 0 && (!pos || !out_ids)))
    return fail(EMA_ERR_INVAL, "slab_block_ids: n < 0 or NULL array");
  const ema::SlabCfg& c = h->book.slab_cfg();
  if (layer < 0 || layer >= c.layers) return fail(EMA_ERR_INVAL, "slab_block_ids: bad layer");
  const int32_t S = c.slab_blocks;
  const int64_t n_pos = int64_t(h->book.n_slabs()) * S;
  std::vector<int32_t> rank;
  int32_t m = 0;
  if (staging_first >= 0) {
    rank.assign(size_t(h->book.n_slabs()), -1);
    for (int32_t i : h->book.borrowed_slabs()) rank[i] = m++;
  }
  for (int32_t k = 0; k < n; ++k) {
    if (pos[k] < 0 || pos[k] >= n_pos)
      return fail(EMA_ERR_INVAL, "slab_block_ids: position out of range");
    const int32_t i = pos[k] / S, p = pos[k] % S;
    if (staging_first < 0) {
      out_ids[k] = int32_t(h->book.n_local() + h->book.slab_slot(i, layer, p));
    } else {
      if (rank[i] < 0) return fail(EMA_ERR_INVAL, "slab_block_ids: position of a slab not borrowed");
      const int64_t id = staging_first + h->book.stage_index(rank[i], m, layer % c.group, p);
      if (id >= h->book.n_local())
        return fail(EMA_ERR_INVAL, "slab_block_ids: staging image past the local pool");
      out_ids[k] = int32_t(id);
    }
  }
  return EMA_OK;
} catch (...) {
  return internal_error();
}

// Runs of group g's swap into the staging image at staging_first: maximal
// ranges contiguous on both sides, in staging order.
static void slab_runs(const ema_slice* h, int32_t g, int32_t staging_first,
                      std::vector<int32_t>* rs, std::vector<int32_t>* rd, std::vector<int32_t>* rn) {
  std::vector<int32_t> src;
  h->book.group_sources(g, &src);
  rs->clear();
  rd->clear();
  rn->clear();
  for (size_t i = 0; i < src.size(); ++i) {
    const int32_t d = staging_first + int32_t(i);
    if (!rn->empty() && rs->back() + rn->back() == src[i] && rd->back() + rn->back() == d) {
      ++rn->back();
    } else {
      rs->push_back(src[i]);
      rd->push_back(d);
      rn->push_back(1);
    }
  }
}

static int check_group(const ema_slice* h, int32_t g, int32_t staging_first, const char* what) {
  if (!h->book.slab_mode())
    return fail(EMA_ERR_INVAL, std::string(what) + ": the slice is not in slabs");
  const ema::SlabCfg& c = h->book.slab_cfg();
  if (g < 0 || g >= c.layers / c.group) return fail(EMA_ERR_INVAL, std::string(what) + ": bad group");
  if (staging_first < 0) return fail(EMA_ERR_INVAL, std::string(what) + ": bad staging_first");
  return EMA_OK;
}

int ema_slab_group_runs(ema_slice_t h, int32_t group, int32_t staging_first, int32_t* src_first,
                        int32_t* dst_first, int32_t* run_blocks, int32_t cap,
                        int32_t* n_runs) try {
  if (!h || !n_runs) return fail(EMA_ERR_INVAL, "slab_group_runs: NULL argument");
  int rc = check_group(h, group, staging_first, "slab_group_runs");
  if (rc) return rc;
  std::vector<int32_t> rs, rd, rn;
  slab_runs(h, group, staging_first, &rs, &rd, &rn);
  *n_runs = int32_t(rn.size());
  for (int32_t i = 0; i < int32_t(rn.size()) && i < cap; ++i) {
    if (src_first) src_first[i] = rs[i];
    if (dst_first) dst_first[i] = rd[i];
    if (run_blocks) run_blocks[i] = rn[i];
  }
  return EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slab_prefetch_group(ema_slice_t h, int32_t group, int32_t staging_first, int32_t engine,
                            void* stream) try {
  if (!h) return fail(EMA_ERR_INVAL, "slab_prefetch_group: NULL handle");
  int rc = check_group(h, group, staging_first, "slab_prefetch_group");
  if (rc) return rc;
  if (engine != EMA_ENGINE_KERNEL && engine != EMA_ENGINE_DMA)
    return fail(EMA_ERR_INVAL, "slab_prefetch_group: unknown engine");
  if (engine == EMA_ENGINE_DMA && h->shape.slice_layout != EMA_LAYOUT_ATTN)
    return fail(EMA_ERR_INVAL,
                "slab_prefetch_group: the copy engines need the slice in the local layout");
  const ema::SlabCfg& c = h->book.slab_cfg();
  const int32_t m = int32_t(h->book.borrowed_slabs().size());
  const int64_t count = int64_t(m) * c.group * c.slab_blocks;
  if (staging_first + count > h->book.n_local())
    return fail(EMA_ERR_INVAL, "slab_prefetch_group: staging image past the local pool");
  for (int64_t i = 0; i < count; ++i)
    if (h->book.owner(int32_t(staging_first + i)) != EMA_STAGING)
      return fail(EMA_ERR_INVAL, "slab_prefetch_group: staging image holds a non-staging block");
  if (h->host_only || count == 0) return EMA_OK;
  DeviceScope ds;
  if ((rc = ds.enter(h))) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (engine == EMA_ENGINE_DMA) {
    std::vector<int32_t> rs, rd, rn;
    slab_runs(h, group, staging_first, &rs, &rd, &rn);
    const ema::PoolView pv = pool_view(h);
    for (size_t r = 0; r < rn.size(); ++r) {
      char* d = pv.local + int64_t(rd[r]) * h->bb;
      const char* sp = pv.slice + (int64_t(rs[r]) - pv.n_local) * h->bb;
      HIP_TRY(hipMemcpyAsync(d, sp, size_t(rn[r]) * h->bb, hipMemcpyDeviceToDeviceNoCU, st),
              "slab_prefetch_group copy");
    }
    return EMA_OK;
  }
  {
    std::vector<int32_t> rs, rd, rn;
    slab_runs(h, group, staging_first, &rs, &rd, &rn);
    if (int(rn.size()) <= ema::kArgRuns) {   // few runs: in the launch arguments
      HIP_TRY(ema::launch_block_copy_runs(pool_view(h), rs.data(), rd.data(), rn.data(),
                                          int32_t(rn.size()), h->d_err, st),
              "slab_prefetch_group launch");
      return EMA_OK;
    }
  }
  if (h->slab_built != h->book.slab_version()) {
    // every group's sources, rebuilt only when the set of borrowed slabs changed
    if (size_t(m) * c.layers * c.slab_blocks > h->slab_cap)
      return fail(EMA_ERR_INVAL, "slab_prefetch_group: lists larger than their buffer");
    if (h->slab_up_pending) {
      HIP_TRY(hipEventSynchronize(h->slab_up_ev), "hipEventSynchronize(slab lists)");
      h->slab_up_pending = false;
    }
    if (h->slab_use_pending) HIP_TRY(hipStreamWaitEvent(st, h->slab_use_ev, 0), "hipStreamWaitEvent");
    std::vector<int32_t> src;
    size_t off = 0;
    for (int32_t g = 0; g < c.layers / c.group; ++g) {
      h->book.group_sources(g, &src);
      std::copy(src.begin(), src.end(), h->h_slab + off);
      off += src.size();
    }
    HIP_TRY(hipMemcpyAsync(h->d_slab, h->h_slab, off * 4, hipMemcpyHostToDevice, st),
            "hipMemcpyAsync(slab lists)");
    HIP_TRY(hipEventRecord(h->slab_up_ev, st), "hipEventRecord(slab lists)");
    h->slab_up_pending = true;
    h->slab_built = h->book.slab_version();
    h->slab_m = m;
  }
  HIP_TRY(ema::launch_block_copy(pool_view(h), h->d_slab + size_t(group) * count, nullptr,
                                 int32_t(count), h->d_err, st, true, nullptr, staging_first),
          "slab_prefetch_group launch");
  HIP_TRY(hipEventRecord(h->slab_use_ev, st), "hipEventRecord(slab prefetch)");
  h->slab_use_pending = true;
  return EMA_OK;
} catch (...) {
  return internal_error();
}

int ema_slab_reclaim(ema_slice_t h, int32_t n_slabs, int32_t* canon_tables, int64_t n_entries,
                     void* stream, ema_slab_reclaim_result* result, int32_t* slabs,
                     int32_t slabs_cap, int32_t* victims, int32_t victims_cap) try {
  if (!h || !result) return fail(EMA_ERR_INVAL, "slab_reclaim: NULL handle or result");
  if (n_slabs < 0 || n_entries < 0 || (n_entries > 0 && !canon_tables))
    return fail(EMA_ERR_INVAL, "slab_reclaim: bad count or table pointer");
  if (h->host_only && (canon_tables || n_entries))
    return fail(EMA_ERR_INVAL, "slab_reclaim: host-only slices take no device tables");
  int rc;
  DeviceScope ds;
  if (!h->host_only && (rc = ds.enter(h))) return rc;
  ema::SlabReclaimPlan plan;
  std::string err;
  if ((rc = h->book.slab_reclaim(n_slabs, &plan, &err))) return fail(rc, err);
  result->reclaimed = plan.reclaimed;
  result->n_victims = int32_t(plan.victims.size());
  result->released = int32_t(plan.released.size());
  for (int32_t i = 0; slabs && i < int32_t(plan.slabs.size()) && i < slabs_cap; ++i)
    slabs[i] = plan.slabs[i];
  for (int32_t i = 0; victims && i < result->n_victims && i < victims_cap; ++i)
    victims[i] = plan.victims[i];
  if (h->host_only || n_entries == 0 || plan.released.empty()) return EMA_OK;
  // every released block's table entries become -1 (no data moves: the
  // preempted requests are dropped)
  hipStream_t st = static_cast<hipStream_t>(stream);
  const Bits bits = bit_span(plan.released);
  const size_t need = bits.words;
  if (need > h->h_work_cap || need > h->work_cap)
    return fail(EMA_ERR_INVAL, "slab_reclaim: plan larger than the work buffers");
  if ((rc = begin_upload(h, st))) return rc;
  put_bits(plan.released, bits, reinterpret_cast<uint32_t*>(h->h_work));
  if ((rc = upload(h, need, st))) return rc;
  ema::TableRewrite rw;
  rw.tables = canon_tables;
  rw.n_entries = n_entries;
  rw.released_bits = reinterpret_cast<const uint32_t*>(h->d_work);
  rw.bits_base = bits.base;
  rw.n_bits = bits.n;
  HIP_TRY(ema::launch_block_copy(pool_view(h), nullptr, nullptr, 0, h->d_err, st, true, &rw),
          "slab_reclaim rewrite");
  return end_upload(h, st);
} catch (...) {
  return internal_error();
}

int ema_slice_device_errors(ema_slice_t h, int32_t* count) try {
  if (!h || !count) return fail(EMA_ERR_INVAL, "device_errors: NULL argument");
  *count = 0;
  if (h->host_only) return EMA_OK;
  DeviceScope ds;
  int rc = ds.enter(h);
  if (rc) return rc;
  HIP_TRY(hipDeviceSynchronize(), "hipDeviceSynchronize");
  HIP_TRY(hipMemcpy(count, h->d_err, 4, hipMemcpyDeviceToHost), "hipMemcpy(err)");
  HIP_TRY(hipMemset(h->d_err, 0, 4), "hipMemset(err)");
  return EMA_OK;
} catch (...) {
  return internal_error();
}

}  // extern "C"
