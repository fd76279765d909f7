// Host side of libflowpool: the C ABI of include/flowpool.h.
//
// Pool state (paper Sec. 3.2): this rank's GVA segments for the HBM and DRAM
// tiers, the physical backing of each tier (device chunks; pinned, mapped
// host chunks), the page table GVA page -> physical page (host mirror plus a
// device copy that the kernels walk), the page allocators, the device sample
// table and metadata arena that pair each sample's text ids with its image
// pages (Sec. 3.1), and a small ring of pinned staging buffers for the
// asynchronous metadata uploads.

#include <algorithm>
#include <climits>
#include <cstdarg>
#include <cstddef>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <stdexcept>
#include <numeric>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "flowpool.h"
#include "fp_internal.h"
#include "schedule.h"
#include "allocate.h"

using fp::SampleDesc;

namespace {

thread_local std::string t_err;

fp_status fail(fp_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  t_err = buf;
  return code;
}

#define FP_HIP(call)                                                                  \
  do {                                                                                \
    hipError_t e_ = (call);                                                           \
    if (e_ != hipSuccess) return fail(FP_EHIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

constexpr uint64_t kDefaultGvaStart = 0x0000100000000000ull;
constexpr int64_t kDefaultMaxSamples = 65536;
constexpr int64_t kDefaultMetaBytes = 64ll << 20;
constexpr int64_t kDefaultChunkBytes = 1ll << 30;
constexpr int64_t kMaxSampleRows = 1 << 24;
constexpr int32_t kMaxPlanMicrobatches = 1 << 20;
// A tail chunk must fit the smallest full chunk (2 vectors per thread): the
// pack kernel's threads cover at most that many vectors of a chunk.
static_assert(fp::kTail2Vecs <= fp::kTail1Vecs && fp::kTail1Vecs <= 2 * fp::kPackBlock, "tail chunk sizes");
// 16-byte vectors one pack or one write may move. The kernels index vectors
// with 32-bit integers, and a thread forms the indices of its vectors (up to
// 767 past its chunk's start) before testing them against the chunk's end,
// so the count stays that far below 2^31.
constexpr int64_t kMaxVectors = (1ll << 31) - 1024;
constexpr int kRing = 8;
// Pinned staging buffers are at least this large; pool_create allocates them
// all, so a call that stages no more than this never allocates.
constexpr size_t kStageHostMin = 1 << 20;
// Runs of one pack at most: per sample, a text run before each image and one
// after the last, and an image run per image.
constexpr int kMaxPackRuns = fp::kMaxPackSamples + 2 * fp::kMaxPackImages;
// Streams remembered per sample as its readers without growing host memory.
constexpr size_t kReaders = 8;
// Stands for "no stream" where a stream handle is remembered (no valid
// hipStream_t has this value).
void* const kNoStream = reinterpret_cast<void*>(~uintptr_t(0));

// Device scratch of pack_microbatch_noalloc: the staged run table of a pack
// too large for its kernel arguments goes here instead of into a staging
// buffer the pool allocates. One array per GPU, shared by every pool and
// call on that GPU; each pool records its device's address of it at
// creation. The largest run table (kMaxPackSamples lengths, kMaxPackRuns
// runs, kBuckets bucket runs and entries) fits.
constexpr size_t kScratchBytes = 64 << 10;
static_assert(((4 * (size_t)fp::kMaxPackSamples + 15) & ~(size_t)15) + 16 * (size_t)kMaxPackRuns +
                      18 * (size_t)fp::kBuckets <= kScratchBytes,
              "the largest run table fits the scratch");
}  // namespace

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

// Device address of `scratch` on a device, looked up once per device with the
// device current (the array's name is a host-side stand-in; only this
// address is valid on the GPU). Null and the HIP error on failure.
uint8_t* scratch_address(int device, hipError_t* err) {
  static std::mutex mu;
  static std::unordered_map<int, uint8_t*> addr;
  std::lock_guard<std::mutex> lock(mu);
  auto it = addr.find(device);
  if (it != addr.end()) return it->second;
  void* ptr = nullptr;
  *err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (*err != hipSuccess || !ptr) return nullptr;
  addr.emplace(device, (uint8_t*)ptr);
  return (uint8_t*)ptr;
}

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) == hipSuccess && hipSetDevice(dev) == hipSuccess) ok = true;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

// First-fit allocator over [0, size) with coalescing (metadata arena).
struct RangeAlloc {
  std::map<int64_t, int64_t> free_;  // offset -> length
  void init(int64_t size) {
    free_.clear();
    if (size > 0) free_[0] = size;
  }
  int64_t alloc(int64_t n) {
    for (auto it = free_.begin(); it != free_.end(); ++it) {
      if (it->second >= n) {
        const int64_t off = it->first, len = it->second;
        free_.erase(it);
        if (len > n) free_[off + n] = len - n;
        return off;
      }
    }
    return -1;
  }
  void release(int64_t off, int64_t n) {
    auto next = free_.lower_bound(off);
    if (next != free_.end() && off + n == next->first) {
      n += next->second;
      next = free_.erase(next);
    }
    if (next != free_.begin()) {
      auto prev = std::prev(next);
      if (prev->first + prev->second == off) {
        prev->second += n;
        return;
      }
    }
    free_[off] = n;
  }
};

// Pinned host buffer + device buffer + completion event, reused round-robin.
struct Stage {
  uint8_t* host = nullptr;
  uint8_t* host_dev = nullptr;   // the same pinned buffer as the GPU addresses it
  size_t host_cap = 0;
  uint8_t* dev = nullptr;
  size_t dev_cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};

struct SampleRec {
  int32_t slot;
  int32_t len, n_text, n_img, n_vis;
  int64_t meta_off, meta_len;
  int64_t text_off, page_off;    // metadata-arena offsets of text ids and page GVAs
  int64_t pl_off = -1, pl_len = 0;  // page list moved out of the main block by a migration
  std::vector<uint64_t> pages;   // GVAs in visual-row order
  std::vector<int32_t> img;      // (placeholder position, rows) per image
  // Stream ordering with the GPU work that touches the sample:
  int32_t written = -1;          // event after its write (metadata upload +
                                 // k_write), -1 once seen complete
  void* write_stream = nullptr;  // stream of that write
  std::vector<void*> readers;    // streams that have packed it (capacity kReaders reserved)
  std::vector<int32_t> reader_events;  // events standing in for reader streams the caller
                                       // retired with pool_forget_stream
  int32_t captured = 0;          // packs of it captured into HIP graphs and not yet released
};

// A freed sample whose pages, metadata and slot wait for packs still in
// flight; they return to the allocators once all its events have completed.
struct Deferred {
  std::vector<uint64_t> pages;
  std::vector<std::pair<int64_t, int64_t>> meta;   // metadata ranges (offset, bytes)
  int32_t slot = -1;                               // descriptor slot, or -1
  std::vector<int32_t> events;
};

// Reference-counted, reusable HIP events (timing disabled).
struct EventPool {
  std::vector<hipEvent_t> ev;
  std::vector<int32_t> refs;
  std::vector<int32_t> idle;
  hipError_t acquire(int32_t* out) {
    if (idle.empty()) {
      hipEvent_t e = nullptr;
      hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableTiming);
      if (r != hipSuccess) return r;
      ev.push_back(e);
      refs.push_back(0);
      idle.push_back((int32_t)ev.size() - 1);
    }
    *out = idle.back();
    idle.pop_back();
    refs[(size_t)*out] = 1;
    return hipSuccess;
  }
  void ref(int32_t i) { ++refs[(size_t)i]; }
  void unref(int32_t i) {
    if (--refs[(size_t)i] == 0) idle.push_back(i);
  }
  // Completed (or failed: a failure shows up again at the next synchronising call).
  bool done(int32_t i) {
    const hipError_t r = hipEventQuery(ev[(size_t)i]);
    if (r == hipErrorNotReady) return false;
    if (r != hipSuccess) (void)hipGetLastError();
    return true;
  }
  // Drops the completed events of a list (waiting for each first if `wait`).
  void prune(std::vector<int32_t>* list, bool wait) {
    size_t k = 0;
    for (int32_t i : *list) {
      if (wait) (void)hipEventSynchronize(ev[(size_t)i]);
      if (done(i)) unref(i);
      else (*list)[k++] = i;
    }
    list->resize(k);
  }
};

uint64_t splitmix64(uint64_t& s) {
  uint64_t z = (s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

int64_t align16(int64_t x) { return (x + 15) & ~int64_t(15); }

}  // namespace

struct fp_pool {
  fp_pool_config cfg{};
  std::mutex mu;
  int64_t rb = 0, pb = 0;
  int n_cu = 0;                       // compute units of the device (pack chunk geometry)
  int64_t n_pages[2] = {0, 0};
  uint64_t gva_start = 0;
  uint64_t region_start[2] = {0, 0};
  uint64_t seg_start[2] = {0, 0};
  uint64_t max_size[2] = {0, 0};
  // physical backing
  std::vector<void*> chunks[2];
  int64_t frames_per_chunk[2] = {1, 1};
  bool owned[2] = {true, true};       // false: the caller's backing, never freed here
  std::vector<uint64_t> pte;          // host mirror, index = global vpn
  uint64_t* pte_dev = nullptr;
  // allocators, page index inside the tier's segment
  std::vector<uint8_t> used[2];
  std::vector<int64_t> stack[2];      // scatter: LIFO, back() pops first
  int64_t n_free[2] = {0, 0};
  // samples
  SampleDesc* desc_dev = nullptr;
  std::vector<int32_t> free_slots;
  uint8_t* meta_dev = nullptr;
  RangeAlloc meta;
  std::unordered_map<uint64_t, SampleRec> samples;
  uint64_t next_id = 1;
  EventPool events;
  std::vector<Deferred> deferred;
  int64_t deferred_pages = 0;
  // staging
  Stage ring[kRing];
  int ring_next = 0;
  uint8_t* scratch_dev = nullptr;     // this device's address of `scratch`
  fp::Divisors dv{};                  // division constants of the row, page and GVA sizes
  // Host arrays a pack builds its run table in, sized at creation for the
  // largest pack (kMaxPackSamples samples, kMaxPackRuns runs), so a pack
  // allocates no host memory. Used under `mu`.
  std::vector<SampleRec*> pk_recs;
  std::vector<int32_t> pk_lens;
  std::vector<fp::PackRun> pk_runs, pk_brun;
  std::vector<uint16_t> pk_bucket;

  uint64_t page_gva(int tier, int64_t idx) const { return seg_start[tier] + (uint64_t)idx * (uint64_t)pb; }
  int page_index(uint64_t gva, int64_t* idx) const {
    for (int t = 0; t < 2; ++t) {
      if (gva >= seg_start[t] && gva < seg_start[t] + max_size[t]) {
        *idx = (int64_t)((gva - seg_start[t]) / (uint64_t)pb);
        return t;
      }
    }
    return -1;
  }
};

namespace {

fp_status stage_acquire(fp_pool* p, size_t host_bytes, size_t dev_bytes, Stage** out) {
  Stage& s = p->ring[p->ring_next];
  p->ring_next = (p->ring_next + 1) % kRing;
  if (s.pending) {
    FP_HIP(hipEventSynchronize(s.ev));
    s.pending = false;
  }
  if (host_bytes > s.host_cap) {
    if (s.host) FP_HIP(hipHostFree(s.host));
    s.host = nullptr;
    s.host_dev = nullptr;
    s.host_cap = 0;
    size_t cap = std::max<size_t>(host_bytes, kStageHostMin);
    FP_HIP(hipHostMalloc((void**)&s.host, cap, hipHostMallocDefault));
    s.host_cap = cap;
    void* dptr = nullptr;
    FP_HIP(hipHostGetDevicePointer(&dptr, s.host, 0));
    s.host_dev = (uint8_t*)dptr;
  }
  if (dev_bytes > s.dev_cap) {
    if (s.dev) FP_HIP(hipFree(s.dev));
    s.dev = nullptr;
    s.dev_cap = 0;
    size_t cap = std::max<size_t>(dev_bytes, 1 << 18);
    FP_HIP(hipMalloc((void**)&s.dev, cap));
    s.dev_cap = cap;
  }
  *out = &s;
  return FP_OK;
}

fp_status stage_release(Stage* s, hipStream_t stream) {
  FP_HIP(hipEventRecord(s->ev, stream));
  s->pending = true;
  return FP_OK;
}

void free_all(fp_pool* p) {
  for (hipEvent_t e : p->events.ev) {
    (void)hipEventSynchronize(e);
    (void)hipEventDestroy(e);
  }
  p->events = EventPool{};
  for (auto& s : p->ring) {
    if (s.ev) (void)hipEventSynchronize(s.ev);
    if (s.host) (void)hipHostFree(s.host);
    if (s.dev) (void)hipFree(s.dev);
    if (s.ev) (void)hipEventDestroy(s.ev);
    s = Stage{};
  }
  if (p->owned[0])
    for (void* c : p->chunks[0]) (void)hipFree(c);
  if (p->owned[1])
    for (void* c : p->chunks[1]) (void)hipHostFree(c);
  p->chunks[0].clear();
  p->chunks[1].clear();
  if (p->pte_dev) (void)hipFree(p->pte_dev);
  if (p->desc_dev) (void)hipFree(p->desc_dev);
  if (p->meta_dev) (void)hipFree(p->meta_dev);
  p->pte_dev = nullptr;
  p->desc_dev = nullptr;
  p->meta_dev = nullptr;
}

// Pages for one sample, all-or-nothing. Returns FP_ENOMEM without changes.
fp_status alloc_pages(fp_pool* p, int64_t n, const uint8_t* wish, std::vector<uint64_t>* out) {
  out->clear();
  if (n == 0) return FP_OK;
  if (p->cfg.alloc_policy == FP_ALLOC_CONTIG) {
    for (int t = 0; t < 2; ++t) {
      const std::vector<uint8_t>& used = p->used[t];
      int64_t run = 0;
      for (int64_t i = 0; i < p->n_pages[t]; ++i) {
        run = used[i] ? 0 : run + 1;
        if (run == n) {
          const int64_t first = i - n + 1;
          for (int64_t j = first; j <= i; ++j) {
            p->used[t][j] = 1;
            out->push_back(p->page_gva(t, j));
          }
          p->n_free[t] -= n;
          return FP_OK;
        }
      }
    }
    return fail(FP_ENOMEM, "no run of %lld free pages", (long long)n);
  }
  int64_t left[2] = {(int64_t)p->stack[0].size(), (int64_t)p->stack[1].size()};
  std::vector<uint8_t> tiers((size_t)n);
  for (int64_t j = 0; j < n; ++j) {
    int t = wish ? wish[j] : FP_TIER_HBM;
    if (left[t] == 0) t = 1 - t;
    if (left[t] == 0) return fail(FP_ENOMEM, "%lld pages do not fit", (long long)n);
    --left[t];
    tiers[(size_t)j] = (uint8_t)t;
  }
  for (int64_t j = 0; j < n; ++j) {
    const int t = tiers[(size_t)j];
    const int64_t i = p->stack[t].back();
    p->stack[t].pop_back();
    p->used[t][i] = 1;
    p->n_free[t] -= 1;
    out->push_back(p->page_gva(t, i));
  }
  return FP_OK;
}

void release_pages(fp_pool* p, const std::vector<uint64_t>& pages) {
  for (auto it = pages.rbegin(); it != pages.rend(); ++it) {
    int64_t i = 0;
    const int t = p->page_index(*it, &i);
    p->used[t][i] = 0;
    p->n_free[t] += 1;
    if (p->cfg.alloc_policy == FP_ALLOC_SCATTER) p->stack[t].push_back(i);
  }
}

// Returns what a deferred free holds to the allocators.
void release_deferred(fp_pool* p, Deferred& d) {
  release_pages(p, d.pages);
  for (const auto& m : d.meta)
    if (m.second > 0) p->meta.release(m.first, m.second);
  if (d.slot >= 0) p->free_slots.push_back(d.slot);
}

// Releases at once what no pending event holds, else queues it.
void defer_or_release(fp_pool* p, Deferred&& d) {
  if (d.events.empty()) {
    release_deferred(p, d);
  } else {
    p->deferred_pages += (int64_t)d.pages.size();
    p->deferred.push_back(std::move(d));
  }
}

// Appends to `events` (each with a reference of its own) what follows every
// pack that has read sample r: an event recorded now on each reader stream
// that still has work queued, and the events that stand in for retired reader
// streams.
fp_status mark_readers(fp_pool* p, const SampleRec& r, std::vector<int32_t>* events) {
  for (int32_t e : r.reader_events) {
    p->events.ref(e);
    events->push_back(e);
  }
  for (void* st : r.readers) {
    const hipError_t q = hipStreamQuery((hipStream_t)st);
    if (q == hipSuccess) continue;
    if (q != hipErrorNotReady) return fail(FP_EHIP, "stream query: %s", hipGetErrorString(q));
    int32_t ev = -1;
    hipError_t e = p->events.acquire(&ev);
    if (e == hipSuccess) e = hipEventRecord(p->events.ev[(size_t)ev], (hipStream_t)st);
    if (e != hipSuccess) {
      if (ev >= 0) p->events.unref(ev);
      return fail(FP_EHIP, "reader event: %s", hipGetErrorString(e));
    }
    events->push_back(ev);
  }
  return FP_OK;
}

// Completes the deferred frees whose packs have finished, oldest first
// (waiting for all of them if `wait`).
void reclaim(fp_pool* p, bool wait) {
  size_t k = 0;
  for (size_t i = 0; i < p->deferred.size(); ++i) {
    Deferred& d = p->deferred[i];
    p->events.prune(&d.events, wait);
    if (d.events.empty()) {
      p->deferred_pages -= (int64_t)d.pages.size();
      release_deferred(p, d);
    } else {
      if (k != i) p->deferred[k] = std::move(d);   // never self-move: it would empty the record
      ++k;
    }
  }
  p->deferred.resize(k);
}

// Makes `stream` wait for the writes of the given samples that may still be
// running on another stream (host-side check first: usually they are done).
fp_status order_after_writes(fp_pool* p, SampleRec* const* recs, size_t n, hipStream_t stream) {
  for (size_t i = 0; i < n; ++i) {
    SampleRec* r = recs[i];
    if (r->written < 0) continue;
    if (p->events.done(r->written)) {
      p->events.unref(r->written);
      r->written = -1;
    } else if (r->write_stream != (void*)stream) {
      FP_HIP(hipStreamWaitEvent(stream, p->events.ev[(size_t)r->written], 0));
    }
  }
  return FP_OK;
}

// True while `stream` is being captured into a HIP graph.
bool capturing(hipStream_t stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return cs != hipStreamCaptureStatusNone;
}

// A caller-provided tier backing: 256-byte aligned, at least `bytes` long
// inside one allocation, and of the tier's kind: device memory of `device`
// (HBM tier), or pinned host memory mapped into the GPU at the same address
// (host tier).
fp_status check_backing(int tier, void* ptr, uint64_t bytes, int device) {
  const char* name = tier ? "host_backing" : "hbm_backing";
  if (bytes == 0) return fail(FP_EINVAL, "%s given for a tier without pages", name);
  if ((uintptr_t)ptr % 256) return fail(FP_EALIGN, "%s must be 256-byte aligned", name);
  hipPointerAttribute_t attr{};
  if (hipPointerGetAttributes(&attr, ptr) != hipSuccess) {
    (void)hipGetLastError();
    return fail(FP_EINVAL, "%s is not memory the HIP runtime knows", name);
  }
  if (tier == 0 && (attr.type != hipMemoryTypeDevice || attr.device != device))
    return fail(FP_EINVAL, "hbm_backing must be device memory of device %d", device);
  if (tier == 1) {
    void* dptr = nullptr;
    if (attr.type != hipMemoryTypeHost || hipHostGetDevicePointer(&dptr, ptr, 0) != hipSuccess || dptr != ptr) {
      (void)hipGetLastError();
      return fail(FP_EINVAL, "host_backing must be pinned host memory mapped at the same address");
    }
  }
  void* base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, ptr) != hipSuccess) {
    (void)hipGetLastError();
    return fail(FP_EINVAL, "%s: its allocation's extent is unknown", name);
  }
  if ((uint64_t)(uintptr_t)ptr + bytes > (uint64_t)(uintptr_t)base + (uint64_t)size)
    return fail(FP_EINVAL, "%s: %llu bytes needed, %llu left in its allocation", name, (unsigned long long)bytes,
                (unsigned long long)((uintptr_t)base + size - (uintptr_t)ptr));
  return FP_OK;
}

// Partition by FP_PLAN_LPT or FP_PLAN_ZIGZAG (flowpool.h states both).
// Runs an entry point's body; host memory exhaustion inside it becomes
// ENOMEM instead of an exception crossing the C ABI.
template <class F>
fp_status guarded(F&& body) {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(FP_ENOMEM, "host memory exhausted");
  } catch (const std::exception& e) {
    return fail(FP_EINVAL, "%s", e.what());
  }
}

fp_status greedy(const int32_t* lengths, const int64_t* costs, int32_t n, int32_t capacity,
                 int32_t n_mb, int32_t policy, int32_t* assign, int32_t* mb_tokens, int64_t* mb_cost,
                 int32_t* mb_max) {
  std::vector<int32_t> order((size_t)n);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return costs[a] > costs[b] || (costs[a] == costs[b] && a < b);
  });
  std::vector<int64_t> tok((size_t)n_mb, 0), cst((size_t)n_mb, 0);
  std::vector<int32_t> mx((size_t)n_mb, 0);
  for (int32_t i = 0; i < n; ++i) assign[i] = -1;
  const int64_t period = 2ll * n_mb;
  for (int32_t pos = 0; pos < n; ++pos) {
    const int32_t i = order[(size_t)pos];
    int best = -1;
    if (policy == FP_PLAN_ZIGZAG) {
      for (int64_t q = 0; q < period && best < 0; ++q) {
        const int64_t r = ((int64_t)pos + q) % period;
        const int j = (int)(r < n_mb ? r : period - 1 - r);
        if (tok[(size_t)j] + lengths[i] <= capacity) best = j;
      }
    } else {
      for (int j = 0; j < n_mb; ++j) {
        if (tok[(size_t)j] + lengths[i] <= capacity &&
            (best < 0 || cst[(size_t)j] < cst[(size_t)best]))
          best = j;
      }
    }
    if (best >= 0) {
      assign[i] = best;
      tok[(size_t)best] += lengths[i];
      cst[(size_t)best] += costs[i];
      mx[(size_t)best] = std::max(mx[(size_t)best], lengths[i]);
    }
  }
  for (int j = 0; j < n_mb; ++j) {
    if (mb_tokens) mb_tokens[j] = (int32_t)tok[(size_t)j];
    if (mb_cost) mb_cost[j] = cst[(size_t)j];
    if (mb_max) mb_max[j] = mx[(size_t)j];
  }
  return FP_OK;
}

}  // namespace

extern "C" {

int32_t fp_abi_version(void) { return FP_ABI_VERSION; }

const char* fp_last_error(void) { return t_err.c_str(); }

void fp_config_init(fp_pool_config* cfg) {
  if (!cfg) return;
  std::memset(cfg, 0, sizeof(*cfg));
  cfg->world_size = 1;
}

fp_status pool_create(const fp_pool_config* cfg_in, fp_pool** out) {
  return guarded([&]() -> fp_status {
    if (!cfg_in || !out) return fail(FP_EINVAL, "null argument");
    *out = nullptr;
    fp_pool_config c = *cfg_in;
    if (c.hidden < 8 || ((2ll * c.hidden) % 16) != 0 || c.hidden > (1 << 20))
      return fail(FP_EINVAL, "hidden %d: 2*hidden must be a positive multiple of 16", c.hidden);
    if (c.page_tokens < 1 || c.page_tokens > (1 << 20)) return fail(FP_EINVAL, "page_tokens %d", c.page_tokens);
    if (c.hbm_pages < 0 || c.host_pages < 0 || c.hbm_pages + c.host_pages < 1 ||
        c.hbm_pages + c.host_pages > (1ll << 31))
      return fail(FP_EINVAL, "page counts %lld/%lld", (long long)c.hbm_pages, (long long)c.host_pages);
    if (c.alloc_policy != FP_ALLOC_CONTIG && c.alloc_policy != FP_ALLOC_SCATTER)
      return fail(FP_EINVAL, "alloc_policy %d", c.alloc_policy);
    if (c.world_size != 1 || c.rank != 0)
      return fail(FP_EINVAL, "world_size/rank %d/%d: this library runs one process", c.world_size, c.rank);
    if (c.vocab < 0 || c.vocab > (1ll << 31)) return fail(FP_EINVAL, "vocab %lld", (long long)c.vocab);
    if (c.pack_cus < 0 || c.pack_cus > 65536 || c.reserved != 0) return fail(FP_EINVAL, "pack_cus %d / reserved", c.pack_cus);
    if (c.gva_start == 0) c.gva_start = kDefaultGvaStart;
    if (c.gva_start % 4096) return fail(FP_EINVAL, "gva_start must be a multiple of 4096");
    {
      // The pack kernel divides GVA offsets below 2^52 by the page size.
      const unsigned __int128 span = (unsigned __int128)(c.hbm_pages + c.host_pages) *
                                     (unsigned __int128)(2ll * c.hidden) * (unsigned __int128)c.page_tokens;
      if (span >= ((unsigned __int128)1 << 52) || (unsigned __int128)c.gva_start + span > ~(uint64_t)0)
        return fail(FP_EINVAL, "GVA span of the pool exceeds 2^52 bytes or the address space");
    }
    if (c.max_samples == 0) c.max_samples = kDefaultMaxSamples;
    if (c.max_samples < 1 || c.max_samples > (1ll << 31) - 1) return fail(FP_EINVAL, "max_samples");
    if (c.meta_bytes == 0) c.meta_bytes = kDefaultMetaBytes;
    if (c.meta_bytes < 16 || c.meta_bytes > fp::kMaxMetaBytes) return fail(FP_EINVAL, "meta_bytes");
    if (c.chunk_bytes == 0) c.chunk_bytes = kDefaultChunkBytes;
    if (c.chunk_bytes < 0) return fail(FP_EINVAL, "chunk_bytes");
    int ndev = 0;
    FP_HIP(hipGetDeviceCount(&ndev));
    if (c.device < 0 || c.device >= ndev) return fail(FP_EINVAL, "device %d of %d", c.device, ndev);
    DeviceGuard guard(c.device);
    if (!guard.ok) return fail(FP_EHIP, "hipSetDevice(%d) failed", c.device);

    int n_cu = c.pack_cus;
    if (n_cu == 0) FP_HIP(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, c.device));
    fp_pool* p = new fp_pool();
    p->cfg = c;
    p->n_cu = n_cu;
    p->rb = 2ll * c.hidden;
    p->pb = p->rb * c.page_tokens;
    p->n_pages[0] = c.hbm_pages;
    p->n_pages[1] = c.host_pages;
    p->gva_start = c.gva_start;
    // Sec. 3.2: per tier a region [start, start + world_size*max_size); this
    // rank's segment [start + rank*max_size, start + (rank+1)*max_size); the
    // DRAM region follows the HBM region.
    for (int t = 0; t < 2; ++t) p->max_size[t] = (uint64_t)p->n_pages[t] * (uint64_t)p->pb;
    p->region_start[0] = c.gva_start;
    p->region_start[1] = c.gva_start + (uint64_t)c.world_size * p->max_size[0];
    for (int t = 0; t < 2; ++t) p->seg_start[t] = p->region_start[t] + (uint64_t)c.rank * p->max_size[t];
    p->dv = fp::make_divisors(p->rb, c.page_tokens, (uint64_t)p->pb);

    // Until the pool is handed out, leaving this scope (an error return or an
    // exception) frees everything it holds.
    struct Hold {
      fp_pool* p;
      ~Hold() {
        if (!p) return;
        std::string keep = t_err;
        free_all(p);
        delete p;
        t_err = keep;
      }
    } hold{p};

    // Physical backing: the caller's buffer as one chunk, or library chunks of
    // whole pages.
    void* backing[2] = {c.hbm_backing, c.host_backing};
    for (int t = 0; t < 2; ++t) {
      if (backing[t]) {
        fp_status bs = check_backing(t, backing[t], (uint64_t)p->n_pages[t] * (uint64_t)p->pb, c.device);
        if (bs != FP_OK) return bs;
        p->chunks[t].push_back(backing[t]);
        p->frames_per_chunk[t] = std::max<int64_t>(1, p->n_pages[t]);
        p->owned[t] = false;
        continue;
      }
      p->frames_per_chunk[t] = std::max<int64_t>(1, c.chunk_bytes / p->pb);
      for (int64_t f = 0; f < p->n_pages[t]; f += p->frames_per_chunk[t]) {
        const int64_t frames = std::min(p->frames_per_chunk[t], p->n_pages[t] - f);
        void* ptr = nullptr;
        hipError_t e = (t == 0) ? hipMalloc(&ptr, (size_t)(frames * p->pb))
                                : hipHostMalloc(&ptr, (size_t)(frames * p->pb), hipHostMallocMapped);
        if (e != hipSuccess)
          return fail(FP_EHIP, "allocating %s backing (%lld bytes): %s", t ? "host" : "HBM",
                           (long long)(frames * p->pb), hipGetErrorString(e));
        if (t == 1) {
          void* dptr = nullptr;
          e = hipHostGetDevicePointer(&dptr, ptr, 0);
          if (e != hipSuccess || dptr != ptr) {
            (void)hipHostFree(ptr);
            return fail(FP_EHIP, "host backing is not mapped at the same address");
          }
        }
        p->chunks[t].push_back(ptr);
      }
    }
    // Page table: GVA page (HBM pages, then host pages) -> physical frame.
    const int64_t total = p->n_pages[0] + p->n_pages[1];
    p->pte.resize((size_t)total);
    uint64_t seed = c.frame_shuffle_seed;
    for (int t = 0; t < 2; ++t) {
      std::vector<int64_t> order((size_t)p->n_pages[t]);
      std::iota(order.begin(), order.end(), 0);
      if (seed) {
        for (int64_t i = p->n_pages[t] - 1; i > 0; --i) {
          const int64_t j = (int64_t)(splitmix64(seed) % (uint64_t)(i + 1));
          std::swap(order[(size_t)i], order[(size_t)j]);
        }
      }
      for (int64_t i = 0; i < p->n_pages[t]; ++i) {
        const int64_t f = order[(size_t)i];
        const uint64_t addr = (uint64_t)p->chunks[t][(size_t)(f / p->frames_per_chunk[t])] +
                              (uint64_t)(f % p->frames_per_chunk[t]) * (uint64_t)p->pb;
        const int64_t vpn = (int64_t)((p->page_gva(t, i) - p->gva_start) / (uint64_t)p->pb);
        p->pte[(size_t)vpn] = addr | fp::PTE_VALID | (t ? fp::PTE_HOST : 0);
      }
      p->used[t].assign((size_t)p->n_pages[t], 0);
      p->stack[t].resize((size_t)p->n_pages[t]);
      for (int64_t i = 0; i < p->n_pages[t]; ++i) p->stack[t][(size_t)i] = p->n_pages[t] - 1 - i;
      p->n_free[t] = p->n_pages[t];
    }
    hipError_t e = hipMalloc((void**)&p->pte_dev, sizeof(uint64_t) * (size_t)total);
    if (e == hipSuccess)
      e = hipMemcpy(p->pte_dev, p->pte.data(), sizeof(uint64_t) * (size_t)total, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMalloc((void**)&p->desc_dev, sizeof(SampleDesc) * (size_t)c.max_samples);
    if (e == hipSuccess) e = hipMalloc((void**)&p->meta_dev, (size_t)c.meta_bytes);
    for (int i = 0; e == hipSuccess && i < kRing; ++i)
      e = hipEventCreateWithFlags(&p->ring[i].ev, hipEventDisableTiming);
    if (e != hipSuccess) return fail(FP_EHIP, "pool metadata allocation: %s", hipGetErrorString(e));
    // Every staging slot's pinned buffer now, so that calls staging at most
    // kStageHostMin bytes (plans, pack run tables) never allocate one.
    for (int i = 0; i < kRing; ++i) {
      Stage* sg = nullptr;
      fp_status ss = stage_acquire(p, kStageHostMin, 0, &sg);
      if (ss != FP_OK) return ss;
    }
    {
      hipError_t se = hipSuccess;
      p->scratch_dev = scratch_address(c.device, &se);     // the device is current here
      if (!p->scratch_dev) return fail(FP_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(se));
    }
    p->pk_recs.resize(fp::kMaxPackSamples);
    p->pk_lens.resize(fp::kMaxPackSamples);
    p->pk_runs.resize(kMaxPackRuns);
    p->pk_brun.resize(fp::kBuckets);
    p->pk_bucket.resize(fp::kBuckets);
    p->meta.init(c.meta_bytes);
    p->free_slots.resize((size_t)c.max_samples);
    for (int64_t i = 0; i < c.max_samples; ++i) p->free_slots[(size_t)i] = (int32_t)(c.max_samples - 1 - i);
    hold.p = nullptr;
    *out = p;
    return FP_OK;
  });
}

fp_status pool_destroy(fp_pool* p) {
  return guarded([&]() -> fp_status {
    if (!p) return FP_OK;
    {
      DeviceGuard guard(p->cfg.device);
      free_all(p);
    }
    delete p;
    return FP_OK;
  });
}

fp_status pool_write_sample(fp_pool* p, const int32_t* text_ids, int32_t n_text,
                            const int32_t* img_pos, const int32_t* img_ntok, int32_t n_img,
                            const void* vis_emb, const uint8_t* page_tier_wish, void* stream,
                            uint64_t* out_sample_id) {
  return guarded([&]() -> fp_status {
    if (!p || !out_sample_id) return fail(FP_EINVAL, "null argument");
    std::lock_guard<std::mutex> lock(p->mu);
    if (n_text < 0 || n_img < 0) return fail(FP_EINVAL, "negative count");
    if ((n_text && !text_ids) || (n_img && (!img_pos || !img_ntok))) return fail(FP_EINVAL, "null array");
    int64_t n_vis = 0;
    for (int32_t j = 0; j < n_img; ++j) {
      if (img_ntok[j] < 0) return fail(FP_EINVAL, "image %d has %d rows", j, img_ntok[j]);
      if (img_pos[j] < 0 || img_pos[j] > n_text || (j && img_pos[j] < img_pos[j - 1]))
        return fail(FP_EINVAL, "image %d placeholder %d (text %d)", j, img_pos[j], n_text);
      n_vis += img_ntok[j];
    }
    const int64_t len = n_vis + n_text;
    if (len < 1 || len > kMaxSampleRows) return fail(FP_EINVAL, "sample length %lld", (long long)len);
    if (n_vis * (p->rb / 16) > kMaxVectors)
      return fail(FP_EINVAL, "%lld visual rows of %lld bytes are too many for one write", (long long)n_vis,
                  (long long)p->rb);
    for (int32_t i = 0; i < n_text; ++i)
      if (text_ids[i] < 0 || text_ids[i] >= p->cfg.vocab)
        return fail(FP_EINVAL, "text id %d at %d outside [0, %lld)", text_ids[i], i, (long long)p->cfg.vocab);
    const int64_t n_pages = (n_vis + p->cfg.page_tokens - 1) / p->cfg.page_tokens;
    if (page_tier_wish) {
      if (p->cfg.alloc_policy != FP_ALLOC_SCATTER) return fail(FP_EINVAL, "tier wishes need the scatter policy");
      for (int64_t j = 0; j < n_pages; ++j)
        if (page_tier_wish[j] > 1) return fail(FP_EINVAL, "tier wish %d", page_tier_wish[j]);
    }
    DeviceGuard guard(p->cfg.device);
    if (!guard.ok) return fail(FP_EHIP, "hipSetDevice");
    if (capturing((hipStream_t)stream))
      return fail(FP_ESTATE, "pool_write_sample cannot be captured into a graph (its staging buffers are reused)");
    const uint8_t* vis_dev = nullptr;
    if (vis_emb && n_vis > 0) {
      if ((uintptr_t)vis_emb % 16) return fail(FP_EALIGN, "vis_emb must be 16-byte aligned");
      // Ordinary (unregistered) host memory would fault the write kernel.
      hipPointerAttribute_t attr{};
      if (hipPointerGetAttributes(&attr, vis_emb) != hipSuccess) {
        (void)hipGetLastError();
        return fail(FP_EINVAL, "vis_emb is not device-accessible memory");
      }
      if (attr.type == hipMemoryTypeUnregistered || !attr.devicePointer)
        return fail(FP_EINVAL, "vis_emb is ordinary host memory, not device-accessible");
      if (attr.type == hipMemoryTypeDevice && attr.device != p->cfg.device)
        return fail(FP_EINVAL, "vis_emb is memory of device %d, the pool is on device %d", attr.device,
                    p->cfg.device);
      vis_dev = (const uint8_t*)attr.devicePointer;
    }
    const int64_t meta_len = align16(8 * n_pages) + align16(8ll * n_img) + align16(4ll * n_text);
    int64_t meta_off = 0;
    SampleRec rec;
    fp_status st = FP_OK;
    // Frees deferred behind packs in flight come back first; if that is not
    // enough, wait for those packs (the producer yields to the consumer).
    reclaim(p, false);
    for (int attempt = 0;; ++attempt) {
      st = FP_OK;
      if (p->free_slots.empty()) {
        st = fail(FP_ENOMEM, "all %lld sample slots in use", (long long)p->cfg.max_samples);
      } else if (meta_len > 0 && (meta_off = p->meta.alloc(meta_len)) < 0) {
        st = fail(FP_ENOMEM, "metadata arena full (%lld bytes wanted)", (long long)meta_len);
      } else {
        st = alloc_pages(p, n_pages, page_tier_wish, &rec.pages);
        if (st != FP_OK && meta_len > 0) p->meta.release(meta_off, meta_len);
      }
      if (st == FP_OK) break;
      if (attempt > 0 || p->deferred.empty()) return st;
      reclaim(p, true);
    }
    auto rollback = [&](fp_status s) {
      std::string keep = t_err;
      release_pages(p, rec.pages);
      if (meta_len > 0) p->meta.release(meta_off, meta_len);
      t_err = keep;
      return s;
    };
    hipStream_t hs = (hipStream_t)stream;
    SampleDesc d{};
    d.len = (int32_t)len;
    d.n_text = n_text;
    d.n_img = n_img;
    d.n_vis = (int32_t)n_vis;
    d.n_pages = (int32_t)n_pages;
    d.page_off = meta_off;
    d.img_off = meta_off + align16(8 * n_pages);
    d.text_off = d.img_off + align16(8ll * n_img);
    if (meta_len > 0) {
      Stage* s = nullptr;
      st = stage_acquire(p, (size_t)meta_len, 0, &s);
      if (st != FP_OK) return rollback(st);
      std::memcpy(s->host, rec.pages.data(), 8 * (size_t)n_pages);
      int32_t* img = (int32_t*)(s->host + (d.img_off - meta_off));
      for (int32_t j = 0; j < n_img; ++j) {
        img[2 * j] = img_pos[j];
        img[2 * j + 1] = img_ntok[j];
      }
      if (n_text) std::memcpy(s->host + (d.text_off - meta_off), text_ids, 4 * (size_t)n_text);
      hipError_t e = hipMemcpyAsync(p->meta_dev + meta_off, s->host, (size_t)meta_len,
                                    hipMemcpyHostToDevice, hs);
      if (e != hipSuccess) return rollback(fail(FP_EHIP, "metadata upload: %s", hipGetErrorString(e)));
      st = stage_release(s, hs);
      if (st != FP_OK) return rollback(st);
    }
    const int32_t slot = p->free_slots.back();
    fp::WriteArgs wa{};
    wa.desc = d;
    wa.desc_table = p->desc_dev;
    wa.slot = slot;
    wa.meta = p->meta_dev;
    wa.pte = p->pte_dev;
    wa.gva_start = p->gva_start;
    wa.vis = vis_dev;
    wa.row_bytes = (int32_t)p->rb;
    wa.page_tokens = p->cfg.page_tokens;
    wa.max_chunk_rows = (int32_t)std::min<int64_t>(n_vis, fp::kChunkVecs / (p->rb / 16) + 2);
    wa.dv = p->dv;
    hipError_t e = fp::launch_write(wa, hs);
    if (e != hipSuccess) return rollback(fail(FP_EHIP, "write kernel: %s", hipGetErrorString(e)));
    int32_t ev = -1;
    e = p->events.acquire(&ev);
    if (e == hipSuccess) e = hipEventRecord(p->events.ev[(size_t)ev], hs);
    if (e != hipSuccess) {
      // The write is already queued: wait for it rather than hand out its pages again.
      (void)hipStreamSynchronize(hs);
      if (ev >= 0) p->events.unref(ev);
      return rollback(fail(FP_EHIP, "write event: %s", hipGetErrorString(e)));
    }
    rec.written = ev;
    rec.write_stream = stream;
    p->free_slots.pop_back();
    rec.slot = slot;
    rec.len = (int32_t)len;
    rec.n_text = n_text;
    rec.n_img = n_img;
    rec.n_vis = (int32_t)n_vis;
    rec.meta_off = meta_off;
    rec.meta_len = meta_len;
    rec.text_off = d.text_off;
    rec.page_off = d.page_off;
    rec.readers.reserve(kReaders);
    rec.img.resize(2 * (size_t)n_img);
    for (int32_t j = 0; j < n_img; ++j) {
      rec.img[2 * (size_t)j] = img_pos[j];
      rec.img[2 * (size_t)j + 1] = img_ntok[j];
    }
    const uint64_t id = p->next_id++;
    p->samples.emplace(id, std::move(rec));
    *out_sample_id = id;
    return FP_OK;
  });
}

fp_status pool_free_sample(fp_pool* p, uint64_t sample_id) {
  return guarded([&]() -> fp_status {
    if (!p) return fail(FP_EINVAL, "null pool");
    std::lock_guard<std::mutex> lock(p->mu);
    auto it = p->samples.find(sample_id);
    if (it == p->samples.end()) return fail(FP_ENOENT, "sample %llu", (unsigned long long)sample_id);
    SampleRec& r = it->second;
    if (r.captured > 0)
      return fail(FP_ESTATE, "sample %llu is read by %d captured pack(s): release them with pool_release_captured first",
                  (unsigned long long)sample_id, r.captured);
    DeviceGuard guard(p->cfg.device);
    if (!guard.ok) return fail(FP_EHIP, "hipSetDevice");
    // The sample's own write is waited for here, so that reuse of its pages
    // never races with it on another stream and, without packs in flight,
    // pages return in free order. Packs still reading it defer the release.
    if (r.written >= 0) {
      FP_HIP(hipEventSynchronize(p->events.ev[(size_t)r.written]));
      p->events.unref(r.written);
      r.written = -1;
    }
    Deferred d;
    // An event recorded now on every stream that packed the sample and still
    // has work queued follows those packs; idle streams need none.
    fp_status st = mark_readers(p, r, &d.events);
    if (st != FP_OK) {
      for (int32_t x : d.events) p->events.unref(x);
      return st;
    }
    for (int32_t x : r.reader_events) p->events.unref(x);
    d.pages = std::move(r.pages);
    d.meta.emplace_back(r.meta_off, r.meta_len);
    if (r.pl_off >= 0) d.meta.emplace_back(r.pl_off, r.pl_len);
    d.slot = r.slot;
    p->samples.erase(it);
    defer_or_release(p, std::move(d));
    return FP_OK;
  });
}

fp_status pool_reclaim(fp_pool* p, int32_t wait, int64_t* out_deferred_pages) {
  return guarded([&]() -> fp_status {
    if (!p) return fail(FP_EINVAL, "null pool");
    std::lock_guard<std::mutex> lock(p->mu);
    DeviceGuard guard(p->cfg.device);
    if (!guard.ok) return fail(FP_EHIP, "hipSetDevice");
    reclaim(p, wait != 0);
    // Forget the write events that have completed (or, with wait, all of
    // them), and the completed events of retired reader streams.
    for (auto& kv : p->samples) {
      SampleRec& r = kv.second;
      p->events.prune(&r.reader_events, wait != 0);
      if (r.written < 0) continue;
      if (wait) (void)hipEventSynchronize(p->events.ev[(size_t)r.written]);
      if (p->events.done(r.written)) {
        p->events.unref(r.written);
        r.written = -1;
      }
    }
    if (out_deferred_pages) *out_deferred_pages = p->deferred_pages;
    return FP_OK;
  });
}

fp_status pool_migrate(fp_pool* p, const uint64_t* sample_ids, int32_t n, int32_t tier, void* stream,
                       int64_t* out_pages_moved) {
  return guarded([&]() -> fp_status {
    if (!p) return fail(FP_EINVAL, "null pool");
    std::lock_guard<std::mutex> lock(p->mu);
    if (p->cfg.alloc_policy != FP_ALLOC_SCATTER) return fail(FP_EINVAL, "migration needs the scatter policy");
    if (tier != FP_TIER_HBM && tier != FP_TIER_HOST) return fail(FP_EINVAL, "tier %d", tier);
    if (n < 0 || (n > 0 && !sample_ids)) return fail(FP_EINVAL, "n %d / null sample_ids", n);
    DeviceGuard guard(p->cfg.device);
    if (!guard.ok) return fail(FP_EHIP, "hipSetDevice");
    std::vector<SampleRec*> recs;
    std::vector<std::vector<int32_t>> moving;   // per sample: indices of pages to move
    std::unordered_set<uint64_t> seen;
    int64_t need = 0;
    for (int32_t i = 0; i < n; ++i) {
      auto it = p->samples.find(sample_ids[i]);
      if (it == p->samples.end()) return fail(FP_ENOENT, "sample %llu", (unsigned long long)sample_ids[i]);
      if (!seen.insert(sample_ids[i]).second)
        return fail(FP_EINVAL, "sample %llu listed twice", (unsigned long long)sample_ids[i]);
      if (it->second.captured > 0)
        return fail(FP_ESTATE, "sample %llu is read by %d captured pack(s): its pages cannot move until "
                               "pool_release_captured", (unsigned long long)sample_ids[i], it->second.captured);
      std::vector<int32_t> mv;
      for (size_t k = 0; k < it->second.pages.size(); ++k) {
        int64_t idx = 0;
        if (p->page_index(it->second.pages[k], &idx) != tier) mv.push_back((int32_t)k);
      }
      if (mv.empty()) continue;
      need += (int64_t)mv.size();
      recs.push_back(&it->second);
      moving.push_back(std::move(mv));
    }
    if (out_pages_moved) *out_pages_moved = need;
    if (need == 0) return FP_OK;
    // All-or-nothing: target pages and the new page lists are reserved first.
    reclaim(p, false);
    std::vector<int64_t> pl_off(recs.size(), -1);
    auto unreserve = [&]() {
      for (size_t j = 0; j < recs.size(); ++j)
        if (pl_off[j] >= 0) p->meta.release(pl_off[j], align16(8 * (int64_t)recs[j]->pages.size()));
      std::fill(pl_off.begin(), pl_off.end(), -1);
    };
    for (int attempt = 0;; ++attempt) {
      bool ok = (int64_t)p->stack[tier].size() >= need;
      for (size_t j = 0; ok && j < recs.size(); ++j) {
        pl_off[j] = p->meta.alloc(align16(8 * (int64_t)recs[j]->pages.size()));
        ok = pl_off[j] >= 0;
      }
      if (ok) break;
      unreserve();
      if (attempt > 0 || p->deferred.empty())
        return fail(FP_ENOMEM, "%lld pages (or their page lists) do not fit in tier %d", (long long)need, tier);
      reclaim(p, true);
    }
    hipStream_t hs = (hipStream_t)stream;
    if (capturing(hs)) {
      unreserve();
      return fail(FP_ESTATE, "pool_migrate cannot be captured into a graph (it moves pages now)");
    }
    fp_status st = order_after_writes(p, recs.data(), recs.size(), hs);   // the copies read what the writes wrote
    if (st != FP_OK) {
      unreserve();
      return st;
    }
    // Staging: the new page lists, then each sample's new page_off for its descriptor.
    size_t stage_bytes = 0;
    for (SampleRec* r : recs) stage_bytes += (size_t)align16(8 * (int64_t)r->pages.size()) + 16;
    Stage* sg = nullptr;
    st = stage_acquire(p, stage_bytes, 0, &sg);
    if (st != FP_OK) {
      unreserve();
      return st;
    }
    // From here on nothing fails half-way but a HIP error: take the pages.
    std::vector<std::vector<uint64_t>> new_pages(recs.size());
    std::vector<std::vector<uint64_t>> old_pages(recs.size());
    // Consecutive pages whose old and new frames are both adjacent inside one
    // backing chunk are copied as one run.
    struct Run { uint64_t src, dst, bytes; int src_chunk, dst_chunk; };
    std::vector<Run> runs;
    const int64_t P = p->cfg.page_tokens;
    auto chunk_of = [&](uint64_t addr) {
      int id = 0;
      for (int t = 0; t < 2; ++t) {
        const uint64_t chunk_span = (uint64_t)p->frames_per_chunk[t] * (uint64_t)p->pb;
        for (void* c : p->chunks[t]) {
          if (addr >= (uint64_t)c && addr < (uint64_t)c + chunk_span) return id;
          ++id;
        }
      }
      return -1;
    };
    for (size_t j = 0; j < recs.size(); ++j) {
      SampleRec& r = *recs[j];
      new_pages[j] = r.pages;
      for (int32_t k : moving[j]) {
        const int64_t i = p->stack[tier].back();
        p->stack[tier].pop_back();
        p->used[tier][i] = 1;
        p->n_free[tier] -= 1;
        const uint64_t gva = p->page_gva(tier, i);
        const uint64_t src = p->pte[(size_t)((r.pages[(size_t)k] - p->gva_start) / (uint64_t)p->pb)] & fp::PTE_ADDR_MASK;
        const uint64_t dst = p->pte[(size_t)((gva - p->gva_start) / (uint64_t)p->pb)] & fp::PTE_ADDR_MASK;
        const int64_t rows = std::min<int64_t>(P, r.n_vis - (int64_t)k * P);
        const uint64_t bytes = (uint64_t)(rows * p->rb);
        const int sc = chunk_of(src), dc = chunk_of(dst);
        if (!runs.empty() && runs.back().src + runs.back().bytes == src && runs.back().dst + runs.back().bytes == dst &&
            runs.back().bytes % (uint64_t)p->pb == 0 && runs.back().src_chunk == sc && runs.back().dst_chunk == dc)
          runs.back().bytes += bytes;
        else
          runs.push_back(Run{src, dst, bytes, sc, dc});
        old_pages[j].push_back(r.pages[(size_t)k]);
        new_pages[j][(size_t)k] = gva;
      }
    }
    hipError_t e = hipSuccess;
    for (const Run& run : runs) {
      e = hipMemcpyAsync((void*)run.dst, (const void*)run.src, run.bytes, hipMemcpyDefault, hs);
      if (e != hipSuccess) break;
    }
    size_t at = 0;
    for (size_t j = 0; e == hipSuccess && j < recs.size(); ++j) {
      const size_t nb = 8 * new_pages[j].size();
      std::memcpy(sg->host + at, new_pages[j].data(), nb);
      e = hipMemcpyAsync(p->meta_dev + pl_off[j], sg->host + at, nb, hipMemcpyHostToDevice, hs);
      at += (size_t)align16((int64_t)nb);
      if (e != hipSuccess) break;
      std::memcpy(sg->host + at, &pl_off[j], 8);
      e = hipMemcpyAsync(&p->desc_dev[recs[j]->slot].page_off, sg->host + at, 8, hipMemcpyHostToDevice, hs);
      at += 16;
    }
    int32_t ev = -1;
    if (e == hipSuccess) e = p->events.acquire(&ev);
    if (e == hipSuccess) e = hipEventRecord(p->events.ev[(size_t)ev], hs);
    if (e != hipSuccess) {
      // Queued copies may still run: wait for them, then put everything back.
      (void)hipStreamSynchronize(hs);
      if (ev >= 0) p->events.unref(ev);
      for (size_t j = 0; j < recs.size(); ++j) {
        std::vector<uint64_t> taken;
        for (int32_t k : moving[j]) taken.push_back(new_pages[j][(size_t)k]);
        release_pages(p, taken);
      }
      unreserve();
      return fail(FP_EHIP, "migration copies: %s", hipGetErrorString(e));
    }
    st = stage_release(sg, hs);
    // The pages left behind and the old page lists wait for the copies and for
    // every pack that may still read them.
    for (size_t j = 0; j < recs.size(); ++j) {
      SampleRec& r = *recs[j];
      Deferred d;
      d.pages = std::move(old_pages[j]);
      const int64_t pl_bytes = align16(8 * (int64_t)r.pages.size());
      if (r.pl_off >= 0) {
        d.meta.emplace_back(r.pl_off, r.pl_len);
      } else {
        d.meta.emplace_back(r.meta_off, pl_bytes);     // the head of the main block
        r.meta_off += pl_bytes;
        r.meta_len -= pl_bytes;
      }
      r.pl_off = pl_off[j];
      r.pl_len = pl_bytes;
      r.page_off = pl_off[j];
      r.pages = std::move(new_pages[j]);
      fp_status ms = mark_readers(p, r, &d.events);
      if (ms != FP_OK) {
        // Without an event on every reader, wait for the whole device instead.
        (void)hipDeviceSynchronize();
        if (st == FP_OK) st = ms;
      }
      p->events.ref(ev);
      d.events.push_back(ev);
      if (r.written >= 0) p->events.unref(r.written);
      p->events.ref(ev);
      r.written = ev;
      r.write_stream = stream;
      defer_or_release(p, std::move(d));
    }
    p->events.unref(ev);
    return st;
  });
}

fp_status plan_partition(const int32_t* lengths, const int64_t* costs_scaled, int32_t n,
                         int32_t capacity, int32_t n_mb, int32_t policy, int32_t* out_assign,
                         int32_t* out_mb_tokens, int64_t* out_mb_cost_scaled,
                         int32_t* out_mb_max_len) {
  return guarded([&]() -> fp_status {
    if (n < 0 || n_mb < 1 || n_mb > kMaxPlanMicrobatches || capacity < 1 || capacity > (1 << 28))
      return fail(FP_EINVAL, "n %d, n_mb %d, capacity %d", n, n_mb, capacity);
    if (policy != FP_PLAN_LPT && policy != FP_PLAN_ZIGZAG) return fail(FP_EINVAL, "policy %d", policy);
    if (n && (!lengths || !costs_scaled || !out_assign)) return fail(FP_EINVAL, "null array");
    for (int32_t i = 0; i < n; ++i)
      if (lengths[i] < 1 || costs_scaled[i] < 0) return fail(FP_EINVAL, "sample %d length/cost", i);
    return greedy(lengths, costs_scaled, n, capacity, n_mb, policy, out_assign, out_mb_tokens, out_mb_cost_scaled,
                  out_mb_max_len);
  });
}

fp_status plan_microbatches(fp_pool* p, const uint64_t* sample_ids, int32_t n, int32_t capacity,
                            int32_t n_mb, int32_t cost_k, int32_t policy, int32_t* out_assign,
                            int32_t* out_mb_tokens, int64_t* out_mb_cost_scaled, int32_t* out_mb_max_len,
                            int64_t* out_sample_cost_scaled, void* stream) {
  return guarded([&]() -> fp_status {
    if (!p) return fail(FP_EINVAL, "null pool");
    std::lock_guard<std::mutex> lock(p->mu);
    if (n < 0 || n_mb < 1 || n_mb > kMaxPlanMicrobatches || capacity < 1 || capacity > (1 << 28) || cost_k < 1 ||
        cost_k > (1 << 24))
      return fail(FP_EINVAL, "n %d, n_mb %d, capacity %d, cost_k %d", n, n_mb, capacity, cost_k);
    if (policy != FP_PLAN_LPT && policy != FP_PLAN_ZIGZAG) return fail(FP_EINVAL, "policy %d", policy);
    if (n && (!sample_ids || !out_assign)) return fail(FP_EINVAL, "null array");
    std::vector<int32_t> slots((size_t)n), lens((size_t)n);
    std::vector<SampleRec*> recs((size_t)n);
    std::unordered_set<uint64_t> seen;
    seen.reserve((size_t)n * 2);
    for (int32_t i = 0; i < n; ++i) {
      auto it = p->samples.find(sample_ids[i]);
      if (it == p->samples.end()) return fail(FP_ENOENT, "sample %llu", (unsigned long long)sample_ids[i]);
      if (!seen.insert(sample_ids[i]).second)
        return fail(FP_EINVAL, "sample %llu listed twice", (unsigned long long)sample_ids[i]);
      slots[(size_t)i] = it->second.slot;
      lens[(size_t)i] = it->second.len;
      recs[(size_t)i] = &it->second;
    }
    std::vector<int64_t> costs((size_t)n);
    if (n > 0) {
      DeviceGuard guard(p->cfg.device);
      if (!guard.ok) return fail(FP_EHIP, "hipSetDevice");
      hipStream_t hs = (hipStream_t)stream;
      if (capturing(hs)) return fail(FP_ESTATE, "plan_microbatches waits for its result and cannot be captured");
      // The cost kernel reads the slots from, and writes the costs to, a
      // pinned staging buffer directly: no copy kernels run beside the packs
      // of other streams.
      const size_t slot_bytes = align16(4ll * n);
      Stage* s = nullptr;
      fp_status st = stage_acquire(p, slot_bytes + 8 * (size_t)n, 0, &s);
      if (st != FP_OK) return st;
      std::memcpy(s->host, slots.data(), 4 * (size_t)n);
      st = order_after_writes(p, recs.data(), recs.size(), hs);   // the descriptors come from the writes
      if (st != FP_OK) return st;
      FP_HIP(fp::launch_cost(p->desc_dev, (const int32_t*)s->host_dev, n, cost_k,
                             (int64_t*)(s->host_dev + slot_bytes), hs));
      FP_HIP(hipStreamSynchronize(hs));
      std::memcpy(costs.data(), s->host + slot_bytes, 8 * (size_t)n);
      st = stage_release(s, hs);
      if (st != FP_OK) return st;
    }
    if (out_sample_cost_scaled) std::memcpy(out_sample_cost_scaled, costs.data(), 8 * (size_t)n);
    return greedy(lens.data(), costs.data(), n, capacity, n_mb, policy, out_assign, out_mb_tokens,
                  out_mb_cost_scaled, out_mb_max_len);
  });
}

namespace {

constexpr int32_t kMaxPackingCapacity = 1 << 20;

fp_status packing_outputs(const fp::PackingPlan& plan, int32_t* out_mb_of_seq, int32_t* out_n_mb,
                          int32_t* out_mb_tokens, int32_t* out_mb_max_len, int64_t* out_mb_cost_scaled,
                          int32_t* out_mb_bucket, int32_t* out_mb_rank, int32_t* out_mb_slot) {
  const size_t m = plan.tokens.size();
  if (out_n_mb) *out_n_mb = (int32_t)m;
  if (out_mb_of_seq) std::copy(plan.mb_of_seq.begin(), plan.mb_of_seq.end(), out_mb_of_seq);
  if (out_mb_tokens) std::copy(plan.tokens.begin(), plan.tokens.end(), out_mb_tokens);
  if (out_mb_max_len) std::copy(plan.max_len.begin(), plan.max_len.end(), out_mb_max_len);
  if (out_mb_cost_scaled) std::copy(plan.cost.begin(), plan.cost.end(), out_mb_cost_scaled);
  if (out_mb_bucket) std::copy(plan.bucket.begin(), plan.bucket.end(), out_mb_bucket);
  if (out_mb_rank) std::copy(plan.rank.begin(), plan.rank.end(), out_mb_rank);
  if (out_mb_slot) std::copy(plan.slot.begin(), plan.slot.end(), out_mb_slot);
  return FP_OK;
}

fp_status check_packing_args(int32_t n, int32_t capacity, int32_t n_ranks, int32_t n_buckets) {
  if (n < 0) return fail(FP_EINVAL, "n %d", n);
  if (capacity < 1 || capacity > kMaxPackingCapacity)
    return fail(FP_EINVAL, "capacity %d outside [1, %d]", capacity, kMaxPackingCapacity);
  if (n_ranks < 1 || n_ranks > (1 << 20)) return fail(FP_EINVAL, "n_ranks %d outside [1, 2^20]", n_ranks);
  if (n_buckets < 1) return fail(FP_EINVAL, "n_buckets %d", n_buckets);
  return FP_OK;
}

}  // namespace

fp_status alloc_candidates(int32_t backbone, int32_t devices, int32_t per_node, int32_t global_batch,
                           int32_t layers, int32_t* out_dp, int32_t* out_tp, int32_t* out_pp, int32_t cap,
                           int32_t* out_n) {
  return guarded([&]() -> fp_status {
    if (devices < 1 || per_node < 1 || global_batch < 1 || layers < 0 || devices > (1 << 20) ||
        per_node > 4096 || global_batch > (1 << 24) || layers > 65536)
      return fail(FP_EINVAL, "devices %d, per_node %d, global_batch %d, layers %d", devices, per_node,
                  global_batch, layers);
    if (!out_n) return fail(FP_EINVAL, "null out_n");
    const std::vector<fp::Config> c = fp::prune_candidates(backbone != 0, devices, per_node, global_batch, layers);
    *out_n = (int32_t)c.size();
    if ((int64_t)c.size() > cap) return fail(FP_EINVAL, "%zu candidates, room for %d", c.size(), cap);
    for (size_t i = 0; i < c.size(); ++i) {
      if (out_dp) out_dp[i] = c[i].dp;
      if (out_tp) out_tp[i] = c[i].tp;
      if (out_pp) out_pp[i] = c[i].pp;
    }
    return FP_OK;
  });
}

fp_status plan_allocation(int32_t n_modules, const int32_t* n_configs, const int64_t* tau, const int64_t* cost,
                          int64_t budget, int32_t* out_choice, int64_t* out_G, int64_t* out_F,
                          int64_t* out_devices) {
  return guarded([&]() -> fp_status {
    if (n_modules < 2 || n_modules > 64) return fail(FP_EINVAL, "n_modules %d (encoders + 1 backbone)", n_modules);
    if (!n_configs || !tau || !cost) return fail(FP_EINVAL, "null array");
    if (budget < 0) return fail(FP_EINVAL, "budget %lld", (long long)budget);
    std::vector<std::vector<int64_t>> t((size_t)n_modules), c((size_t)n_modules);
    double combos = 1;
    size_t at = 0;
    for (int32_t i = 0; i < n_modules; ++i) {
      if (n_configs[i] < 1) return fail(FP_EINVAL, "module %d has %d configurations", i, n_configs[i]);
      if (i < n_modules - 1) combos *= n_configs[i];
      for (int32_t k = 0; k < n_configs[i]; ++k, ++at) {
        if (tau[at] < 0 || tau[at] > (1ll << 50) || cost[at] < 0 || cost[at] > (1ll << 40))
          return fail(FP_EINVAL, "module %d configuration %d: tau %lld, cost %lld", i, k, (long long)tau[at],
                      (long long)cost[at]);
        t[(size_t)i].push_back(tau[at]);
        c[(size_t)i].push_back(cost[at]);
      }
    }
    if (combos > (double)(1 << 22)) return fail(FP_EINVAL, "%.0f encoder combinations (at most 2^22)", combos);
    fp::FlowChoice best;
    if (!fp::flow_match(t, c, budget, &best))
      return fail(FP_ECAPACITY, "no choice of configurations fits %lld devices", (long long)budget);
    if (out_choice) std::copy(best.choice.begin(), best.choice.end(), out_choice);
    if (out_G) *out_G = best.G;
    if (out_F) *out_F = best.F;
    if (out_devices) *out_devices = best.devices;
    return FP_OK;
  });
}

fp_status plan_dynamic_packing(const int32_t* lengths, int32_t n, int32_t capacity, int32_t n_ranks,
                               int32_t n_buckets, int32_t* out_mb_of_seq, int32_t* out_n_mb,
                               int32_t* out_mb_tokens, int32_t* out_mb_max_len, int64_t* out_mb_cost_scaled,
                               int32_t* out_mb_bucket, int32_t* out_mb_rank, int32_t* out_mb_slot) {
  return guarded([&]() -> fp_status {
    fp_status st = check_packing_args(n, capacity, n_ranks, n_buckets);
    if (st != FP_OK) return st;
    if (n > 0 && !lengths) return fail(FP_EINVAL, "null lengths");
    for (int32_t i = 0; i < n; ++i)
      if (lengths[i] < 1 || lengths[i] > capacity)
        return fail(FP_EINVAL, "length %d of sequence %d outside [1, %d]", lengths[i], i, capacity);
    fp::PackingPlan plan;
    fp::dynamic_packing(lengths, n, capacity, n_ranks, n_buckets, &plan);
    return packing_outputs(plan, out_mb_of_seq, out_n_mb, out_mb_tokens, out_mb_max_len, out_mb_cost_scaled,
                           out_mb_bucket, out_mb_rank, out_mb_slot);
  });
}

fp_status plan_pool_packing(fp_pool* p, const uint64_t* sample_ids, int32_t n, int32_t capacity,
                            int32_t n_ranks, int32_t n_buckets, int32_t* out_mb_of_seq, int32_t* out_n_mb,
                            int32_t* out_mb_tokens, int32_t* out_mb_max_len, int64_t* out_mb_cost_scaled,
                            int32_t* out_mb_bucket, int32_t* out_mb_rank, int32_t* out_mb_slot) {
  return guarded([&]() -> fp_status {
    if (!p) return fail(FP_EINVAL, "null pool");
    fp_status st = check_packing_args(n, capacity, n_ranks, n_buckets);
    if (st != FP_OK) return st;
    if (n > 0 && !sample_ids) return fail(FP_EINVAL, "null sample_ids");
    std::vector<int32_t> lens((size_t)n);
    {
      std::lock_guard<std::mutex> lock(p->mu);
      for (int32_t i = 0; i < n; ++i) {
        auto it = p->samples.find(sample_ids[i]);
        if (it == p->samples.end()) return fail(FP_ENOENT, "sample %llu", (unsigned long long)sample_ids[i]);
        lens[(size_t)i] = it->second.len;
        if (lens[(size_t)i] > capacity)
          return fail(FP_EINVAL, "sample %llu of length %d exceeds capacity %d",
                      (unsigned long long)sample_ids[i], lens[(size_t)i], capacity);
      }
    }
    fp::PackingPlan plan;
    fp::dynamic_packing(lens.data(), n, capacity, n_ranks, n_buckets, &plan);
    return packing_outputs(plan, out_mb_of_seq, out_n_mb, out_mb_tokens, out_mb_max_len, out_mb_cost_scaled,
                           out_mb_bucket, out_mb_rank, out_mb_slot);
  });
}

// The word of a sample's image runs: its page list's arena word index, or,
// when its pages have consecutive GVAs (a contiguous allocation), -1 - the
// page number of its first page, from which the kernel computes every page's
// number without reading the list. Only rows packed in 12 KiB chunks take
// the shortcut: same-machine A/B, qwen (H 3584) 0.45 % faster per launch,
// video (H 5120, 8 KiB chunks) 0.3 % slower with it.
static int32_t image_word(const fp_pool* p, const SampleRec& r) {
  const size_t n = r.pages.size();
  if (n > 0 && p->rb < fp::kSmallChunkRowBytes) {
    const uint64_t pb = (uint64_t)p->pb;
    const uint64_t first = r.pages[0];
    bool consecutive = true;
    for (size_t k = 1; k < n && consecutive; ++k) consecutive = r.pages[k] == first + k * pb;
    const int64_t vpn0 = (int64_t)((first - p->gva_start) / pb);
    if (consecutive && vpn0 + (int64_t)n < INT32_MAX) return (int32_t)(-1 - vpn0);
  }
  return (int32_t)(r.page_off / 8);
}

// Bucket index of runs covering rows [0, total) (run k starts where run k-1
// ends): at most max_buckets buckets of 2^shift rows; bucket b gets the run
// holding its first row and that run's number. Returns the bucket count.
static int32_t build_buckets(const fp::PackRun* runs, int32_t n_runs, int64_t total, int32_t max_buckets,
                             int32_t* shift_out, fp::PackRun* brun, uint16_t* bucket) {
  int32_t shift = 0;
  while (total > 0 && ((total - 1) >> shift) >= max_buckets) ++shift;
  const int32_t nb = total > 0 ? (int32_t)(((total - 1) >> shift) + 1) : 0;
  for (int32_t b = 0, k = 0; b < nb; ++b) {
    const int64_t first = (int64_t)b << shift;
    while (k + 1 < n_runs && runs[k].end <= first) ++k;
    bucket[b] = (uint16_t)k;
    brun[b] = runs[k];
  }
  *shift_out = shift;
  return nb;
}

// pack_microbatch, and (scratch_dev != null) its variant that stages a large
// run table into the caller-supplied device scratch instead of the pool's
// staging buffers and allocates nothing.
static fp_status pack_impl(fp_pool* p, const uint64_t* sample_ids, int32_t n, const void* embed_table,
                           int64_t vocab, void* out_emb, int64_t out_rows_cap, int32_t* out_cu_seqlens,
                           int32_t* out_position_ids, int32_t* out_n_tokens, int32_t* out_max_seqlen,
                           int32_t tier_mask, void* stream, uint8_t* scratch_dev, size_t scratch_bytes) {
  const bool noalloc = scratch_dev != nullptr;
  if (!p) return fail(FP_EINVAL, "null pool");
  std::lock_guard<std::mutex> lock(p->mu);
  if (n < 0 || n > fp::kMaxPackSamples) return fail(FP_EINVAL, "n %d outside [0, %d]", n, fp::kMaxPackSamples);
  if (n && !sample_ids) return fail(FP_EINVAL, "null sample_ids");
  if (tier_mask < 1 || tier_mask > 3) return fail(FP_EINVAL, "tier_mask %d", tier_mask);
  if (out_rows_cap < 0) return fail(FP_EINVAL, "out_rows_cap");
  if ((uintptr_t)out_emb % 16 || (uintptr_t)embed_table % 16) return fail(FP_EALIGN, "out_emb/embed_table alignment");
  if ((uintptr_t)out_cu_seqlens % 4 || (uintptr_t)out_position_ids % 4) return fail(FP_EALIGN, "cu/pos alignment");
  SampleRec** recs = p->pk_recs.data();
  int64_t total = 0, n_text = 0, n_imgs = 0;
  int32_t mx = 0;
  for (int32_t i = 0; i < n; ++i) {
    auto it = p->samples.find(sample_ids[i]);
    if (it == p->samples.end()) return fail(FP_ENOENT, "sample %llu", (unsigned long long)sample_ids[i]);
    SampleRec& r = it->second;
    recs[i] = &r;
    total += r.len;
    n_text += r.n_text;
    n_imgs += r.n_img;
    mx = std::max(mx, r.len);
  }
  if (n_imgs > fp::kMaxPackImages)
    return fail(FP_EINVAL, "%lld images in one microbatch (at most %d)", (long long)n_imgs, fp::kMaxPackImages);
  if (total > out_rows_cap) return fail(FP_ECAPACITY, "%lld rows > capacity %lld", (long long)total, (long long)out_rows_cap);
  const int64_t vpr = p->rb / 16;
  if (total * vpr > kMaxVectors)
    return fail(FP_EINVAL, "microbatch of %lld rows of %lld bytes is too large", (long long)total, (long long)p->rb);
  if (total > 0 && !out_emb) return fail(FP_EINVAL, "null out_emb");
  if (n_text > 0 && (tier_mask & FP_TIER_MASK_HBM)) {
    if (!embed_table) return fail(FP_EINVAL, "null embed_table with text rows");
    if (vocab < p->cfg.vocab) return fail(FP_EINVAL, "table vocab %lld < pool vocab %lld", (long long)vocab, (long long)p->cfg.vocab);
  }
  if (noalloc) {
    // Remembering a new reader stream must not grow a sample's list.
    for (int32_t i = 0; i < n; ++i) {
      const SampleRec& r = *recs[i];
      if (std::find(r.readers.begin(), r.readers.end(), stream) == r.readers.end() &&
          r.readers.size() >= r.readers.capacity())
        return fail(FP_ESTATE, "sample %llu was packed on %zu other streams, the most this call can record "
                               "without allocating", (unsigned long long)sample_ids[i], r.readers.size());
    }
  }
  DeviceGuard guard(p->cfg.device);
  if (!guard.ok) return fail(FP_EHIP, "hipSetDevice");
  hipStream_t hs = (hipStream_t)stream;
  fp::PackPlan pl{};
  fp::PackArgs& a = pl.a;
  a.meta = p->meta_dev;
  a.pte = p->pte_dev;
  a.gva_start = p->gva_start;
  a.table = (const uint8_t*)embed_table;
  a.out = (uint8_t*)out_emb;
  a.cu = out_cu_seqlens;
  a.pos = out_position_ids;
  a.n = n;
  a.n_tokens = (int32_t)total;
  a.row_bytes = (int32_t)p->rb;
  a.page_tokens = p->cfg.page_tokens;
  const bool plain_table = vocab >= 0 && vocab <= fp::kPlainTableMaxBytes / p->rb;
  a.tier_mask = tier_mask | (plain_table ? fp::kTablePlainLoads : 0);
  a.pt_mul = p->dv.pt_mul;
  a.pt_shift = p->dv.pt_shift;
  a.pb_mul = p->dv.pb_mul;
  a.pb_shift = p->dv.pb_shift;
  pl.div_mul = p->dv.div_mul;
  pl.div_shift = p->dv.div_shift;
  // The run table: sample lengths, then the runs of every sample in row
  // order (a text run per nonempty stretch of text rows, an image run per
  // stretch of images with no text row between them), then the bucket index.
  int32_t* lens = p->pk_lens.data();
  fp::PackRun* runs = p->pk_runs.data();
  int32_t n_runs = 0;
  {
    int32_t row = 0;
    for (int32_t i = 0; i < n; ++i) {
      const SampleRec& r = *recs[i];
      const int32_t s0 = row;
      lens[i] = r.len;
      int32_t ti = 0, vis = 0;
      bool in_image = false;
      auto text_to = [&](int32_t upto) {
        if (upto <= ti) return;
        if (n_runs) runs[n_runs - 1].end = row;
        runs[n_runs++] = fp::PackRun{0, s0 | fp::kTextRun, 0, (int32_t)(r.text_off / 4 + ti - row)};
        row += upto - ti;
        ti = upto;
        in_image = false;
      };
      for (int32_t j = 0; j < r.n_img; ++j) {
        text_to(r.img[2 * (size_t)j]);
        const int32_t nt = r.img[2 * (size_t)j + 1];
        if (nt <= 0) continue;
        if (!in_image) {
          if (n_runs) runs[n_runs - 1].end = row;
          runs[n_runs++] = fp::PackRun{0, s0, vis - row, image_word(p, r)};
          in_image = true;
        }
        row += nt;
        vis += nt;
      }
      text_to(r.n_text);
    }
    if (n_runs) runs[n_runs - 1].end = row;
  }
  // A microbatch of a few samples and runs launches with the compact kernel
  // arguments (less host time per launch), whose bucket index is shorter.
  const bool small = n <= fp::PackArgsSmall::kMaxSamples && n_runs <= fp::PackArgsSmall::kMaxRuns;
  int32_t shift = 0;
  const int32_t n_buckets = build_buckets(runs, n_runs, total, small ? fp::PackArgsSmall::kMaxBuckets : fp::kBuckets,
                                          &shift, p->pk_brun.data(), p->pk_bucket.data());
  const int32_t bucket_len = n_buckets + (n_buckets & 1);
  a.bucket_shift = shift;

  pl.max_chunk_rows = (int32_t)std::min<int64_t>(total, fp::kChunkVecs / vpr + 2);
  pl.small = small;
  pl.n_runs = n_runs;
  pl.n_buckets = n_buckets;
  fp::pack_chunks(&pl, p->n_cu);

  const bool staged = n > fp::kInlineSamples || n_runs > fp::kInlineRuns;
  const bool captured = capturing(hs);
  if (captured) {
    // A captured pack is one kernel whose arguments hold the whole
    // microbatch, so a replay packs the same samples again.
    if (staged)
      return fail(FP_ESTATE, "a pack of more than %d samples or %d runs cannot be captured into a graph",
                  fp::kInlineSamples, fp::kInlineRuns);
    // No event queries during capture: the writes must already be known complete.
    for (int32_t i = 0; i < n; ++i)
      if (recs[i]->written >= 0)
        return fail(FP_ESTATE, "a sample's write is not known complete: synchronize and call pool_reclaim "
                               "before capturing its pack");
  }
  Stage* s = nullptr;
  if (!staged) {
    if (n) std::memcpy(a.lens, lens, 4 * (size_t)n);
    if (n_runs) std::memcpy(a.runs, runs, sizeof(fp::PackRun) * (size_t)n_runs);
    if (n_buckets) std::memcpy(a.bucket, p->pk_bucket.data(), 2 * (size_t)n_buckets);
    if (n_buckets) std::memcpy(a.brun, p->pk_brun.data(), sizeof(fp::PackRun) * (size_t)n_buckets);
    a.off_runs = (int32_t)(offsetof(fp::PackArgs, runs) - offsetof(fp::PackArgs, lens));
    a.off_brun = (int32_t)(offsetof(fp::PackArgs, brun) - offsetof(fp::PackArgs, lens));
    a.off_bucket = (int32_t)(offsetof(fp::PackArgs, bucket) - offsetof(fp::PackArgs, lens));
    pl.staged = nullptr;
  } else {
    const size_t o_runs = ((size_t)4 * n + 15) & ~(size_t)15;
    const size_t o_br = o_runs + sizeof(fp::PackRun) * (size_t)n_runs;
    const size_t o_b = o_br + sizeof(fp::PackRun) * (size_t)n_buckets;
    const size_t bytes = o_b + 2 * (size_t)bucket_len;
    uint8_t* dest = nullptr;
    if (noalloc) {
      if (bytes > scratch_bytes)
        return fail(FP_ECAPACITY, "run table of %zu bytes exceeds the %zu-byte scratch", bytes, scratch_bytes);
      fp_status st = stage_acquire(p, bytes, 0, &s);        // never allocates: buffers hold kStageHostMin
      if (st != FP_OK) return st;
      dest = scratch_dev;
    } else {
      fp_status st = stage_acquire(p, bytes, bytes, &s);
      if (st != FP_OK) return st;
      dest = s->dev;
    }
    std::memset(s->host, 0, bytes);
    if (n) std::memcpy(s->host, lens, 4 * (size_t)n);
    if (n_runs) std::memcpy(s->host + o_runs, runs, sizeof(fp::PackRun) * (size_t)n_runs);
    if (n_buckets) std::memcpy(s->host + o_br, p->pk_brun.data(), sizeof(fp::PackRun) * (size_t)n_buckets);
    if (n_buckets) std::memcpy(s->host + o_b, p->pk_bucket.data(), 2 * (size_t)n_buckets);
    FP_HIP(hipMemcpyAsync(dest, s->host, bytes, hipMemcpyHostToDevice, hs));
    pl.staged = dest;
    a.off_runs = (int32_t)o_runs;
    a.off_brun = (int32_t)o_br;
    a.off_bucket = (int32_t)o_b;
  }
  {
    fp_status st = order_after_writes(p, recs, (size_t)n, hs);
    if (st != FP_OK) return st;
  }
  hipError_t e = fp::launch_pack(pl, hs);
  if (e != hipSuccess) return fail(FP_EHIP, "pack kernel: %s", hipGetErrorString(e));
  if (s) {
    fp_status st = stage_release(s, hs);
    if (st != FP_OK) return st;
  }
  // Remember the stream as a reader of each sample; a free records its event
  // there (no event per pack: events between back-to-back packs slow them).
  for (int32_t i = 0; i < n; ++i) {
    SampleRec* r = recs[i];
    if (std::find(r->readers.begin(), r->readers.end(), stream) == r->readers.end()) r->readers.push_back(stream);
    if (captured) ++r->captured;
  }
  if (out_n_tokens) *out_n_tokens = (int32_t)total;
  if (out_max_seqlen) *out_max_seqlen = mx;
  return FP_OK;
}

fp_status pack_microbatch(fp_pool* p, const uint64_t* sample_ids, int32_t n, const void* embed_table,
                          int64_t vocab, void* out_emb, int64_t out_rows_cap, int32_t* out_cu_seqlens,
                          int32_t* out_position_ids, int32_t* out_n_tokens, int32_t* out_max_seqlen,
                          int32_t tier_mask, void* stream) {
  return guarded([&]() -> fp_status {
    return pack_impl(p, sample_ids, n, embed_table, vocab, out_emb, out_rows_cap, out_cu_seqlens, out_position_ids,
                     out_n_tokens, out_max_seqlen, tier_mask, stream, nullptr, 0);
  });
}

fp_status pack_microbatch_noalloc(fp_pool* p, const uint64_t* sample_ids, int32_t n, const void* embed_table,
                                  int64_t vocab, void* out_emb, int64_t out_rows_cap, int32_t* out_cu_seqlens,
                                  int32_t* out_position_ids, int32_t* out_n_tokens, int32_t* out_max_seqlen,
                                  int32_t tier_mask, void* stream) {
  return guarded([&]() -> fp_status {
    if (!p) return fail(FP_EINVAL, "null pool");
    return pack_impl(p, sample_ids, n, embed_table, vocab, out_emb, out_rows_cap, out_cu_seqlens, out_position_ids,
                     out_n_tokens, out_max_seqlen, tier_mask, stream, p->scratch_dev, kScratchBytes);
  });
}

fp_status pool_forget_stream(fp_pool* p, void* stream) {
  return guarded([&]() -> fp_status {
    if (!p) return fail(FP_EINVAL, "null pool");
    std::lock_guard<std::mutex> lock(p->mu);
    DeviceGuard guard(p->cfg.device);
    if (!guard.ok) return fail(FP_EHIP, "hipSetDevice");
    hipStream_t hs = (hipStream_t)stream;
    if (capturing(hs)) return fail(FP_ESTATE, "pool_forget_stream on a capturing stream");
    // One event after the stream's queued work stands in for it wherever it
    // is a reader (none if the stream is idle).
    int32_t ev = -1;
    const hipError_t q = hipStreamQuery(hs);
    if (q != hipSuccess && q != hipErrorNotReady) return fail(FP_EHIP, "stream query: %s", hipGetErrorString(q));
    bool used = false;
    for (auto& kv : p->samples)
      if (std::find(kv.second.readers.begin(), kv.second.readers.end(), stream) != kv.second.readers.end()) used = true;
    if (used && q == hipErrorNotReady) {
      hipError_t e = p->events.acquire(&ev);
      if (e == hipSuccess) e = hipEventRecord(p->events.ev[(size_t)ev], hs);
      if (e != hipSuccess) {
        if (ev >= 0) p->events.unref(ev);
        return fail(FP_EHIP, "stream event: %s", hipGetErrorString(e));
      }
    }
    for (auto& kv : p->samples) {
      SampleRec& r = kv.second;
      auto it = std::find(r.readers.begin(), r.readers.end(), stream);
      if (it != r.readers.end()) {
        r.readers.erase(it);
        if (ev >= 0) {
          p->events.ref(ev);
          r.reader_events.push_back(ev);
        }
      }
      // A write still running on the stream: its event stays the sample's
      // ordering point, but no later stream may be taken for this one.
      if (r.write_stream == stream) r.write_stream = kNoStream;
    }
    if (ev >= 0) p->events.unref(ev);
    return FP_OK;
  });
}

fp_status pool_release_captured(fp_pool* p, const uint64_t* sample_ids, int32_t n) {
  return guarded([&]() -> fp_status {
    if (!p) return fail(FP_EINVAL, "null pool");
    if (n < 0 || (n > 0 && !sample_ids)) return fail(FP_EINVAL, "n %d / null sample_ids", n);
    std::lock_guard<std::mutex> lock(p->mu);
    // All-or-nothing: every listed occurrence must hold a capture.
    std::unordered_map<uint64_t, int32_t> want;
    for (int32_t i = 0; i < n; ++i) ++want[sample_ids[i]];
    for (const auto& kv : want) {
      auto it = p->samples.find(kv.first);
      if (it == p->samples.end()) return fail(FP_ENOENT, "sample %llu", (unsigned long long)kv.first);
      if (it->second.captured < kv.second)
        return fail(FP_EINVAL, "sample %llu holds %d captured pack(s), %d released", (unsigned long long)kv.first,
                    it->second.captured, kv.second);
    }
    for (const auto& kv : want) p->samples.find(kv.first)->second.captured -= kv.second;
    return FP_OK;
  });
}

// Compute units of the calling thread's current device.
static fp_status current_cus(int* n_cu) {
  int dev = 0;
  FP_HIP(hipGetDevice(&dev));
  FP_HIP(hipDeviceGetAttribute(n_cu, hipDeviceAttributeMultiprocessorCount, dev));
  return FP_OK;
}

fp_status fp_copy_bytes(const void* src, void* dst, int64_t bytes, int32_t row_bytes, void* stream) {
  return guarded([&]() -> fp_status {
    if (bytes < 0 || bytes % 16 || bytes / 16 > kMaxVectors) return fail(FP_EINVAL, "bytes %lld", (long long)bytes);
    if (row_bytes < 16 || row_bytes % 16) return fail(FP_EINVAL, "row_bytes %d", row_bytes);
    if (bytes && (!src || !dst)) return fail(FP_EINVAL, "null buffer");
    if ((uintptr_t)src % 16 || (uintptr_t)dst % 16) return fail(FP_EALIGN, "src/dst must be 16-byte aligned");
    int n_cu = 0;
    fp_status st = current_cus(&n_cu);
    if (st != FP_OK) return st;
    FP_HIP(fp::launch_copy(src, dst, bytes / 16, row_bytes, n_cu, (hipStream_t)stream));
    return FP_OK;
  });
}

fp_status fp_gather_rows(const uint64_t* rows_src, int32_t n_rows, int32_t row_bytes, void* dst, void* stream) {
  return guarded([&]() -> fp_status {
    if (n_rows < 0 || row_bytes < 16 || row_bytes % 16 || (int64_t)n_rows * (row_bytes / 16) > kMaxVectors)
      return fail(FP_EINVAL, "n_rows %d, row_bytes %d", n_rows, row_bytes);
    if (n_rows && (!rows_src || !dst)) return fail(FP_EINVAL, "null buffer");
    if ((uintptr_t)rows_src % 8 || (uintptr_t)dst % 16) return fail(FP_EALIGN, "rows_src/dst alignment");
    int n_cu = 0;
    fp_status st = current_cus(&n_cu);
    if (st != FP_OK) return st;
    FP_HIP(fp::launch_gather(rows_src, n_rows, row_bytes, dst, n_cu, (hipStream_t)stream));
    return FP_OK;
  });
}

fp_status pool_stats(const fp_pool* p, int64_t* free_hbm_pages, int64_t* free_host_pages, int64_t* n_samples) {
  if (!p) return fail(FP_EINVAL, "null pool");
  fp_pool* q = const_cast<fp_pool*>(p);
  std::lock_guard<std::mutex> lock(q->mu);
  if (free_hbm_pages) *free_hbm_pages = p->n_free[0];
  if (free_host_pages) *free_host_pages = p->n_free[1];
  if (n_samples) *n_samples = (int64_t)p->samples.size();
  return FP_OK;
}

fp_status pool_sample_pages(const fp_pool* p, uint64_t sample_id, uint64_t* gvas, int32_t cap, int32_t* n) {
  if (!p) return fail(FP_EINVAL, "null pool");
  fp_pool* q = const_cast<fp_pool*>(p);
  std::lock_guard<std::mutex> lock(q->mu);
  auto it = p->samples.find(sample_id);
  if (it == p->samples.end()) return fail(FP_ENOENT, "sample %llu", (unsigned long long)sample_id);
  const int32_t cnt = (int32_t)it->second.pages.size();
  if (n) *n = cnt;
  if (cap < cnt) return fail(FP_EINVAL, "capacity %d < %d pages", cap, cnt);
  if (cnt && !gvas) return fail(FP_EINVAL, "null gvas");
  if (cnt) std::memcpy(gvas, it->second.pages.data(), 8 * (size_t)cnt);
  return FP_OK;
}

fp_status pool_sample_info(const fp_pool* p, uint64_t sample_id, int32_t* length, int32_t* n_text,
                           int32_t* n_vis) {
  if (!p) return fail(FP_EINVAL, "null pool");
  fp_pool* q = const_cast<fp_pool*>(p);
  std::lock_guard<std::mutex> lock(q->mu);
  auto it = p->samples.find(sample_id);
  if (it == p->samples.end()) return fail(FP_ENOENT, "sample %llu", (unsigned long long)sample_id);
  if (length) *length = it->second.len;
  if (n_text) *n_text = it->second.n_text;
  if (n_vis) *n_vis = it->second.n_vis;
  return FP_OK;
}

fp_status pool_translate(const fp_pool* p, uint64_t gva, int32_t* tier, uint64_t* phys) {
  if (!p) return fail(FP_EINVAL, "null pool");
  int64_t idx = 0;
  const int t = p->page_index(gva, &idx);
  if (t < 0) return fail(FP_EINVAL, "GVA %#llx is not mapped", (unsigned long long)gva);
  const uint64_t page = p->page_gva(t, idx);
  const uint64_t e = p->pte[(size_t)((page - p->gva_start) / (uint64_t)p->pb)];
  if (tier) *tier = (e & fp::PTE_HOST) ? FP_TIER_HOST : FP_TIER_HBM;
  if (phys) *phys = (e & fp::PTE_ADDR_MASK) + (gva - page);
  return FP_OK;
}

fp_status pool_layout(const fp_pool* p, uint64_t* region_start, uint64_t* segment_start, int64_t* page_bytes) {
  if (!p) return fail(FP_EINVAL, "null pool");
  for (int t = 0; t < 2; ++t) {
    if (region_start) region_start[t] = p->region_start[t];
    if (segment_start) segment_start[t] = p->seg_start[t];
  }
  if (page_bytes) *page_bytes = p->pb;
  return FP_OK;
}

}  // extern "C"
