// Internal declarations shared by the translation units of libsscn.so.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <memory>
#include <new>
#include <cstdint>
#include <string>
#include <mutex>
#include <vector>

#include "sscn.h"

namespace sscn {

// Output rows are grouped in tiles of kTile rows; the rule book stores, for
// every (offset o, tile t), one contiguous segment of pairs whose output row
// lies in tile t.  Segments are laid out offset-major: seg[o * n_tiles + t].
constexpr int kTile = 64;
// Output rows per tile of the padded chunk table (a multiple of kTile, at
// most 255 so that a row inside a tile and the padding row fit in a byte).
constexpr int kChunkRows = 128;
constexpr int kWave = 64;
// Output rows per block of the row-block plan (four MFMA row tiles, one
// per wavefront of a workgroup).
constexpr int kPlanRows = 64;
// Bits of the key that orders rows by their offset set.
constexpr int kPlanKeyBits = 15;
// A plan entry packs an input row (kPlanNoRow: none) below the item's offset.
constexpr int kPlanRowBits = 25;  // plan entries: input row | offset << kPlanRowBits (offsets < 128)
constexpr uint32_t kPlanNoRow = (1u << kPlanRowBits) - 1;
constexpr int kPlanMaxK = 96;      // offsets of a rule book that gets a row-block plan
constexpr int kPlanMaskWords = 3;  // words of an offset set of at most kPlanMaxK offsets
__host__ __device__ constexpr int plan_words(int K) { return (K + 31) / 32; }
// Tiles are grouped into this many contiguous ranges, one per XCD of the
// chip (each XCD has its own L2); see the tile order of a rule book.
constexpr int kTileGroups = 8;

constexpr uint64_t kEmptyKey = ~0ull;
constexpr int kMaxBatch = 1 << 15;
constexpr int kMaxExtent = 1 << 16;
constexpr int kMaxDim = 4;

// error flags raised by device code
constexpr int kFlagOutOfRange = 1;
constexpr int kFlagDuplicate = 2;
constexpr int kFlagWideKey = 4;  // a batch index too large for 32-bit SSC keys

// ---------------------------------------------------------------- errors
void set_error(const std::string& msg);
sscn_status fail(sscn_status st, const std::string& msg);
sscn_status hip_fail(hipError_t e, const char* what);

#define SSCN_TRY(expr)              \
  do {                              \
    sscn_status st_ = (expr);       \
    if (st_ != SSCN_OK) return st_; \
  } while (0)

#define SSCN_HIP(call)                                   \
  do {                                                   \
    hipError_t e_ = (call);                              \
    if (e_ != hipSuccess) return ::sscn::hip_fail(e_, #call); \
  } while (0)

// ---------------------------------------------------------------- memory
// Device allocation for work on stream s from the library's block cache: a
// block freed on s is reused only by later allocations on s (stream order
// keeps its previous users first); see runtime.hip.
sscn_status dev_alloc(void** p, size_t bytes, hipStream_t s);
void dev_free(void* p, hipStream_t s);

// Set (on the calling thread) while an entry point that must not allocate
// runs: the rule-book tables built on first use are then an error instead of
// being built, and temporaries come from the caller-provided region.
struct NoAlloc {
  void* scratch = nullptr;  // device address of the temporary region
  size_t bytes = 0;
};
const NoAlloc* no_alloc();
void set_no_alloc(const NoAlloc* na);

// Events the caller asked to have recorded at the start and the end of the
// next launch of a row-block or wgrad kernel on this thread
// (sscn_time_next_launch): the launch takes them (clearing the request) and
// records them with its own dispatch (hipExtLaunchKernelGGL), so that no
// separate event packets idle the GPU between kernels.
bool take_launch_timer(hipEvent_t* before, hipEvent_t* after);

// The cap on the library's device memory per device (0: none), and whether
// wgrad adds its partial blocks in a fixed order (sscn_set_deterministic).
void set_device_memory_cap(size_t bytes);
bool deterministic();
void set_deterministic(bool on);

// One direction of a rule book: tiles over the output rows of that
// direction, offset-major segments, and the pair arrays (pointers into the
// rule book's device blocks).
struct Storage {
  int64_t n_tiles = 0;
  int64_t* seg = nullptr;        // K * n_tiles + 1 entries
  int32_t* in_rows = nullptr;    // n_pairs
  int32_t* out_rows = nullptr;   // n_pairs
  int32_t* order = nullptr;      // n_tiles: per tile group (contiguous range), tiles by decreasing work
  bool order_built = false;      // `order` is filled on first use (ensure_order)
  // The same pairs as a padded chunk table: output rows cut into tiles of
  // kChunkRows rows; within a tile, per offset, the pairs in chunks of 16
  // (the last chunk padded).  Chunks are numbered tile-major, then by offset.
  int64_t n_ctiles = 0;
  int32_t* ctile = nullptr;      // K * n_ctiles + 1: first chunk of (tile, offset); last entry = chunk count
  int32_t* c_in = nullptr;       // 16 per chunk: input row, -1 for padding
  uint8_t* c_out = nullptr;      // 16 per chunk: output row - tile start, kChunkRows for padding
  int32_t* c_off = nullptr;      // per chunk: offset (as stored)
  // Row-block plan (K <= kPlanMaxK): the output rows ordered by the set of offsets
  // that reach them (rows with similar sets side by side) and cut into
  // blocks of kPlanRows; per block, one item per offset that reaches any of
  // its rows, holding each row's input row for that offset (-1 if none).
  uint32_t* row_mask = nullptr;  // n_rows x plan_words(K) when the build provides it: offsets reaching each output row
  int64_t n_blocks = 0;
  int32_t* perm = nullptr;       // kPlanRows * n_blocks: output row at each position, -1 past the end
  int32_t* b_first = nullptr;    // n_blocks + 1: first item of each block
  int4* b_rec = nullptr;         // n_blocks: blocks by decreasing item count, as (block, first item, items, 0)
  uint32_t* items = nullptr;     // kPlanRows per item: input row | offset (as stored) << kPlanRowBits
};

struct RulebookData {
  std::atomic<int> refs{1};
  int device = 0;
  hipStream_t stream = nullptr;  // build stream (used to release storage)
  int f = 0, stride = 1, K = 0;
  bool submanifold = false;
  int64_t n_in = 0, n_out = 0, n_pairs = 0;
  int dim = 3;                   // spatial dimensions d: coordinates are n x (d + 1)
  int32_t in_size[4] = {0, 0, 0, 0}, out_size[4] = {0, 0, 0, 0};
  std::vector<int64_t> pairs_per_offset;  // host copy, K entries
  Storage fwd;                   // tiles over output rows
  Storage bwd;                   // tiles over input rows (SC only; SSC mirrors fwd)
  int32_t* out_coords = nullptr; // n_out x (d + 1)
  int32_t* in_coords = nullptr;  // n_in x (d + 1) (SC only; an SSC's input sites are its output sites)
  std::vector<void*> blocks;     // device allocations owning all of the above
  // The chunk tables are built on first use (by the kernels that read
  // them) on the build stream; when work on another stream needs one,
  // `chunk_ready` is recorded on the build stream then (after the tables'
  // kernels) and that stream waits for it.
  std::mutex chunk_mu;
  hipEvent_t chunk_ready = nullptr;
  hipEvent_t plan_ready = nullptr;   // the same for the row-block plans
  hipEvent_t order_ready = nullptr;  // and for the tile orders
  // Work that reads the rule book on streams other than the build stream:
  // per such stream, an event recorded after its latest use.  The storage
  // goes back to the block cache on the build stream, so the destructor
  // first makes the build stream wait for each of these events; later
  // allocations on the build stream are then ordered after every reader.
  std::mutex use_mu;
  std::vector<std::pair<hipStream_t, hipEvent_t>> foreign_uses;
  void note_use(hipStream_t s);
  ~RulebookData();
};

// Records, when it goes out of scope, that work reading `d` was queued on
// `s` (see RulebookData::foreign_uses).
struct UseNote {
  RulebookData* d;
  hipStream_t s;
  ~UseNote() {
    if (d) d->note_use(s);
  }
};

}  // namespace sscn

struct sscn_rulebook_s {
  sscn::RulebookData* d;
  bool transposed;
};

namespace sscn {

// What a kernel needs to run one direction of a rule book.
struct View {
  const Storage* st;
  int K;
  bool mirror;        // segment for offset o is stored under K-1-o
  int64_t n_in, n_out;
  int64_t n_pairs;
  RulebookData* owner;
};

// Builds the padded chunk table of the view's storage if it is not there
// yet and makes `s` wait for it.
sscn_status ensure_chunks(const View& v, hipStream_t s);
// The same for the row-block plan (K <= kPlanMaxK).
sscn_status ensure_plan(const View& v, hipStream_t s);
// The same for the tile order of the view's storage.
sscn_status ensure_order(const View& v, hipStream_t s);

inline View view_of(const sscn_rulebook_s* rb) {
  const RulebookData* d = rb->d;
  View v;
  v.K = d->K;
  v.n_pairs = d->n_pairs;
  v.owner = rb->d;
  if (!rb->transposed) {
    v.st = &d->fwd; v.mirror = false; v.n_in = d->n_in; v.n_out = d->n_out;
  } else if (d->submanifold) {
    v.st = &d->fwd; v.mirror = true; v.n_in = d->n_out; v.n_out = d->n_in;
  } else {
    v.st = &d->bwd; v.mirror = false; v.n_in = d->n_out; v.n_out = d->n_in;
  }
  return v;
}

// Device-wide exclusive scan: out[i] = sum_{q<i} in[q], out[count] = total.
// `in` and `out` may alias.  Temporary storage is allocated on `s`.
sscn_status exclusive_scan_i64(const int64_t* in, int64_t* out, int64_t count, hipStream_t s);
sscn_status exclusive_scan_i32(const int32_t* in, int32_t* out, int64_t count, hipStream_t s);

// Resident workgroups of `kern` per CU (block threads, dynamic LDS bytes) and
// the CU count of the current device; cached per (device, kernel, shape).
void occupancy(const void* kern, int block, size_t lds, int* per_cu, int* cus);

// Fill helpers (graph-capture safe: kernels, not memset nodes).
sscn_status fill_i32(int32_t* p, int32_t v, int64_t count, hipStream_t s);
sscn_status fill_u64(uint64_t* p, uint64_t v, int64_t count, hipStream_t s);
sscn_status fill_f32(float* p, float v, int64_t count, hipStream_t s);

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Workgroup i of a launch is dispatched to XCD i % kTileGroups.  Renumber a
// grid of n workgroups so that each XCD takes one contiguous range of logical
// items (bijective on [0, n)).
__device__ inline int64_t xcd_remap(int64_t bid, int64_t n) {
  const int64_t per = n / kTileGroups, rem = n % kTileGroups;
  const int64_t x = bid % kTileGroups, k = bid / kTileGroups;
  return x * per + (x < rem ? x : rem) + k;
}

}  // namespace sscn
