// Error reporting, the device-memory block cache, fills and a device-wide
// exclusive scan used by the rule-book builders.
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <mutex>

#include <map>
#include <tuple>
#include <utility>
#include <vector>
#include "internal.h"

namespace sscn {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

sscn_status fail(sscn_status st, const std::string& msg) {
  set_error(msg);
  return st;
}

sscn_status hip_fail(hipError_t e, const char* what) {
  set_error(std::string(what) + ": " + hipGetErrorString(e));
  return e == hipErrorOutOfMemory ? SSCN_ERR_OOM : SSCN_ERR_DEVICE;
}

// ------------------------------------------------------------------ memory
// Device memory is cached by the library.  A freed block goes to a free
// list keyed by (device, stream, size) and is handed out again only to an
// allocation on the same stream, which the stream orders after the block's
// last use there: the guarantee of stream-ordered allocation, without its
// cost (the runtime's stream-ordered pool took 0.1-0.6 ms per allocation or
// free of tens of MB; a cache hit is a map lookup).  Blocks go back to the
// device only when an allocation fails: then the device is synchronised,
// every cached block of it released, and the allocation tried once more.
namespace {
struct Cache {
  std::mutex mu;
  std::map<void*, std::pair<size_t, int>> owned;  // every block: (bytes, device)
  std::map<std::tuple<int, hipStream_t, size_t>, std::vector<void*>> idle;  // freed blocks
  std::map<int, size_t> held;                     // bytes owned per device
  size_t cap = 0;                                 // per-device cap on `held` (0: none)
  bool cap_read = false;                          // SSCN_DEVICE_MEMORY_CAP looked up
};
Cache& cache() {
  static Cache* c = new Cache;  // never destroyed: frees may run during exit
  return *c;
}
// 512-byte steps up to 1 MiB, 2 MiB steps above
size_t block_bytes(size_t b) {
  if (b <= ((size_t)1 << 20)) return (b + 511) & ~(size_t)511;
  const size_t step = (size_t)2 << 20;
  return (b + step - 1) & ~(step - 1);
}
void release_idle(Cache& c, int dev) {
  (void)hipDeviceSynchronize();
  for (auto it = c.idle.begin(); it != c.idle.end();) {
    if (std::get<0>(it->first) != dev) {
      ++it;
      continue;
    }
    for (void* q : it->second) {
      (void)hipFree(q);
      c.held[dev] -= c.owned[q].first;
      c.owned.erase(q);
    }
    it = c.idle.erase(it);
  }
}
}  // namespace

sscn_status dev_alloc(void** p, size_t bytes, hipStream_t s) {
  *p = nullptr;
  if (bytes == 0) return SSCN_OK;
  int dev = 0;
  SSCN_HIP(hipGetDevice(&dev));
  const size_t want = block_bytes(bytes);
  Cache& c = cache();
  std::lock_guard<std::mutex> lock(c.mu);
  // smallest idle block of this stream that is large enough, if it wastes
  // at most half of the request
  auto it = c.idle.lower_bound(std::make_tuple(dev, s, want));
  if (it != c.idle.end() && std::get<0>(it->first) == dev && std::get<1>(it->first) == s &&
      std::get<2>(it->first) <= want + want / 2) {
    *p = it->second.back();
    it->second.pop_back();
    if (it->second.empty()) c.idle.erase(it);
    return SSCN_OK;
  }
  // The cap (sscn_set_device_memory_cap, or SSCN_DEVICE_MEMORY_CAP in bytes
  // read at the first allocation) makes a new block fail as a real
  // out-of-memory would, after the same release of idle blocks.
  if (!c.cap_read) {
    c.cap_read = true;
    if (const char* env = std::getenv("SSCN_DEVICE_MEMORY_CAP")) c.cap = (size_t)std::strtoull(env, nullptr, 10);
  }
  if (c.cap && c.held[dev] + want > c.cap) {
    release_idle(c, dev);
    if (c.held[dev] + want > c.cap)
      return fail(SSCN_ERR_OOM, std::string("device allocation of ") + std::to_string(bytes) +
                                    " bytes exceeds the library's device memory cap of " + std::to_string(c.cap) +
                                    " bytes");
  }
  hipError_t e = hipMalloc(p, want);
  if (e == hipErrorOutOfMemory) {
    (void)hipGetLastError();
    release_idle(c, dev);
    e = hipMalloc(p, want);
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    *p = nullptr;
    return fail(e == hipErrorOutOfMemory ? SSCN_ERR_OOM : SSCN_ERR_DEVICE,
                std::string("device allocation of ") + std::to_string(bytes) + " bytes failed: " +
                    hipGetErrorString(e));
  }
  c.owned[*p] = std::make_pair(want, dev);
  c.held[dev] += want;
  return SSCN_OK;
}

void set_device_memory_cap(size_t bytes) {
  Cache& c = cache();
  std::lock_guard<std::mutex> lock(c.mu);
  c.cap = bytes;
  c.cap_read = true;
}

static std::atomic<bool> g_deterministic{false};
bool deterministic() { return g_deterministic.load(std::memory_order_relaxed); }
void set_deterministic(bool on) { g_deterministic.store(on, std::memory_order_relaxed); }

static thread_local hipEvent_t t_time_before = nullptr, t_time_after = nullptr;

bool take_launch_timer(hipEvent_t* before, hipEvent_t* after) {
  if (!t_time_before) return false;
  *before = t_time_before;
  *after = t_time_after;
  t_time_before = t_time_after = nullptr;
  return true;
}

static thread_local const NoAlloc* t_no_alloc = nullptr;
const NoAlloc* no_alloc() { return t_no_alloc; }
void set_no_alloc(const NoAlloc* na) { t_no_alloc = na; }

void dev_free(void* p, hipStream_t s) {
  if (!p) return;
  Cache& c = cache();
  std::lock_guard<std::mutex> lock(c.mu);
  auto it = c.owned.find(p);
  if (it == c.owned.end()) return;
  c.idle[std::make_tuple(it->second.second, s, it->second.first)].push_back(p);
}

void occupancy(const void* kern, int block, size_t lds, int* per_cu, int* cus) {
  struct Key {
    int dev;
    const void* kern;
    int block;
    size_t lds;
    bool operator<(const Key& o) const {
      return std::tie(dev, kern, block, lds) < std::tie(o.dev, o.kern, o.block, o.lds);
    }
  };
  static std::mutex mu;
  static std::map<Key, std::pair<int, int>> cache;
  int dev = 0;
  (void)hipGetDevice(&dev);
  const Key k{dev, kern, block, lds};
  {
    std::lock_guard<std::mutex> lock(mu);
    auto it = cache.find(k);
    if (it != cache.end()) {
      *per_cu = it->second.first;
      *cus = it->second.second;
      return;
    }
  }
  int n_cu = 256, n = 1;
  (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, block, lds) != hipSuccess || n < 1) n = 1;
  {
    std::lock_guard<std::mutex> lock(mu);
    cache[k] = {n, n_cu};
  }
  *per_cu = n;
  *cus = n_cu;
}

void RulebookData::note_use(hipStream_t s) {
  if (s == stream) return;
  std::lock_guard<std::mutex> lock(use_mu);
  hipEvent_t ev = nullptr;
  for (auto& u : foreign_uses)
    if (u.first == s) ev = u.second;
  if (!ev) {
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
      // without an event the build stream cannot be ordered after s: wait
      // for s here instead
      (void)hipGetLastError();
      (void)hipStreamSynchronize(s);
      return;
    }
    foreign_uses.emplace_back(s, ev);
  }
  (void)hipEventRecord(ev, s);
}

RulebookData::~RulebookData() {
  int cur = 0;
  (void)hipGetDevice(&cur);
  if (cur != device) (void)hipSetDevice(device);
  for (auto& u : foreign_uses) {
    (void)hipStreamWaitEvent(stream, u.second, 0);
    (void)hipEventDestroy(u.second);
  }
  for (void* p : blocks) dev_free(p, stream);
  if (chunk_ready) (void)hipEventDestroy(chunk_ready);
  if (plan_ready) (void)hipEventDestroy(plan_ready);
  if (order_ready) (void)hipEventDestroy(order_ready);
  if (cur != device) (void)hipSetDevice(cur);
}

// ------------------------------------------------------------------- fills
template <typename T>
__global__ void k_fill(T* __restrict__ p, T v, int64_t count) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (; i < count; i += step) p[i] = v;
}

template <typename T>
static sscn_status fill(T* p, T v, int64_t count, hipStream_t s) {
  if (count <= 0) return SSCN_OK;
  int64_t blocks = ceil_div(count, 256);
  if (blocks > 65536) blocks = 65536;
  k_fill<T><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(p, v, count);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

sscn_status fill_i32(int32_t* p, int32_t v, int64_t count, hipStream_t s) { return fill(p, v, count, s); }
sscn_status fill_u64(uint64_t* p, uint64_t v, int64_t count, hipStream_t s) { return fill(p, v, count, s); }
sscn_status fill_f32(float* p, float v, int64_t count, hipStream_t s) { return fill(p, v, count, s); }

// -------------------------------------------------------------------- scan
// Two-level reduce-then-scan.  A block covers kScanItems * kScanThreads
// consecutive elements; block totals are scanned recursively.
constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int64_t kScanChunk = (int64_t)kScanThreads * kScanItems;

template <typename T>
__device__ T block_exclusive_sum(T v, T* lds_wave, T& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  T x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    T y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) lds_wave[wave] = x;
  __syncthreads();
  T wave_off = 0, tot = 0;
  for (int w = 0; w < kScanThreads / 64; ++w) {
    T t = lds_wave[w];
    if (w < wave) wave_off += t;
    tot += t;
  }
  total = tot;
  __syncthreads();
  return wave_off + x - v;
}

template <typename T>
__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(const T* __restrict__ in, int64_t count,
                                                             T* __restrict__ partial) {
  __shared__ T lds_wave[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk;
  T s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    int64_t idx = base + (int64_t)i * kScanThreads + threadIdx.x;
    if (idx < count) s += in[idx];
  }
  T total;
  (void)block_exclusive_sum<T>(s, lds_wave, total);
  if (threadIdx.x == 0) partial[blockIdx.x] = total;
}

template <typename T>
__global__ __launch_bounds__(kScanThreads) void k_scan_apply(const T* in, int64_t count,
                                                            const T* __restrict__ partial, T* out) {
  __shared__ T tile[kScanChunk];
  __shared__ T lds_wave[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk;
  // coalesced load into LDS
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    int e = i * kScanThreads + threadIdx.x;
    int64_t idx = base + e;
    tile[e] = idx < count ? in[idx] : T(0);
  }
  __syncthreads();
  // each thread owns kScanItems consecutive elements
  T local[kScanItems];
  T s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    local[i] = tile[threadIdx.x * kScanItems + i];
    s += local[i];
  }
  T total;
  const T carry = partial ? partial[blockIdx.x] : T(0);
  T run = block_exclusive_sum<T>(s, lds_wave, total) + carry;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    tile[threadIdx.x * kScanItems + i] = run;
    run += local[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    int e = i * kScanThreads + threadIdx.x;
    int64_t idx = base + e;
    if (idx < count) out[idx] = tile[e];
  }
  // the block holding the last element also writes the grand total
  if (count - 1 < base + kScanChunk && threadIdx.x == 0) out[count] = carry + total;
}

template <typename T>
__global__ void k_scan_store_zero(T* out) { out[0] = 0; }

template <typename T>
static sscn_status exclusive_scan(const T* in, T* out, int64_t count, hipStream_t s) {
  if (count <= 0) {
    k_scan_store_zero<T><<<1, 1, 0, s>>>(out);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  const int64_t blocks = ceil_div(count, kScanChunk);
  if (blocks == 1) {
    k_scan_apply<T><<<1, kScanThreads, 0, s>>>(in, count, nullptr, out);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  T* partial = nullptr;
  sscn_status st = dev_alloc((void**)&partial, sizeof(T) * (blocks + 1), s);
  if (st != SSCN_OK) return st;
  k_scan_reduce<T><<<dim3((unsigned)blocks), kScanThreads, 0, s>>>(in, count, partial);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) {
    st = exclusive_scan<T>(partial, partial, blocks, s);
    if (st == SSCN_OK) {
      k_scan_apply<T><<<dim3((unsigned)blocks), kScanThreads, 0, s>>>(in, count, partial, out);
      e = hipGetLastError();
    }
  }
  dev_free(partial, s);
  if (e != hipSuccess) return hip_fail(e, "scan launch");
  return st;
}

// The recursive call above scans `partial` in place; in-place use is safe
// because every block reads all of its chunk into LDS before writing it and
// the grand total goes to index `count`, past the input.
sscn_status exclusive_scan_i64(const int64_t* in, int64_t* out, int64_t count, hipStream_t s) {
  return exclusive_scan<int64_t>(in, out, count, s);
}
sscn_status exclusive_scan_i32(const int32_t* in, int32_t* out, int64_t count, hipStream_t s) {
  return exclusive_scan<int32_t>(in, out, count, s);
}

}  // namespace sscn

extern "C" const char* sscn_last_error(void) { return sscn::g_last_error.c_str(); }

extern "C" sscn_status sscn_time_next_launch(hipEvent_t before, hipEvent_t after) {
  if ((before == nullptr) != (after == nullptr))
    return sscn::fail(SSCN_ERR_INVALID_ARG, "both events or neither");
  sscn::t_time_before = before;
  sscn::t_time_after = after;
  return SSCN_OK;
}

extern "C" sscn_status sscn_set_device_memory_cap(uint64_t bytes) {
  sscn::set_device_memory_cap((size_t)bytes);
  return SSCN_OK;
}

extern "C" sscn_status sscn_set_deterministic(int32_t on) {
  sscn::set_deterministic(on != 0);
  return SSCN_OK;
}

extern "C" sscn_status sscn_release_cached(void) {
  int dev = 0;
  SSCN_HIP(hipGetDevice(&dev));
  sscn::Cache& c = sscn::cache();
  std::lock_guard<std::mutex> lock(c.mu);
  sscn::release_idle(c, dev);
  return SSCN_OK;
}
