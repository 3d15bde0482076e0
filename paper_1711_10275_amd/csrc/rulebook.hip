// Rule-book construction on the GPU (Sec. 4.2 of the paper).
//
// Dictionary: open addressing with linear probing in HBM.  SSC builds key a
// location by its linear index ((b L0 + x0) L1 + x1) L2 + x2 whenever every
// batch index present keeps it below 2^32 - 1, and store it by group: a
// 16-byte slot holds the group key (linear key / 3) and the rows of the
// group's 3 consecutive linear keys, so that the x2 neighbours of nearby
// sites share slots.  The insert flags a batch index beyond that limit and
// the build is redone with 16-byte slots {64-bit key, row} (16 bits per
// field, b < 2^15 so no key equals the empty marker), which the SC builds
// always use.  Capacity is a power of two >= 2n slots (load <= 1/2).
//
// Rule book layout: output rows are cut into tiles of kTile = 64 rows (one
// wavefront); for every offset o and tile t the pairs whose output row lies
// in t form one contiguous segment, segments ordered offset-major, and
// within a segment pairs are in increasing output row.  A kernel that owns
// a range of output tiles therefore finds all of its pairs for offset o in
// one contiguous range, and the whole array is already sorted by
// (offset, out row, in row) for export.
//
// SSC (Sec. 4.1, Sec. 4.2 last paragraph): the input dictionary is the
// output dictionary; one wavefront per tile probes the f^3 neighbours of
// its 64 sites, a ballot per offset counts the hits, a device-wide scan of
// the (offset, tile) counts gives segment starts, and a second pass writes
// each hit at its segment start + its rank among the wave's hits.
//
// SC (Sec. 4.1, Sec. 4.2 step 1): every input x visits the outputs y with
// x = s*y + i; an output dictionary records, per output location, the
// smallest visit index v = j*K + o (atomicMin).  The output rows are the
// ranks of those first visits (a scan over visit flags), which numbers the
// outputs in first-visit order with the inputs taken in row order.  From
// the per-visit output rows an output-major neighbour map is written and
// compacted exactly like the SSC one; the input-major map gives the
// transposed (DC / dgrad) direction.
#include <algorithm>
#include <cstring>
#include <type_traits>

#include "internal.h"

namespace sscn {

// ------------------------------------------------------------- dictionary
__device__ __forceinline__ uint64_t pack_key(int b, int x0, int x1, int x2) {
  return ((uint64_t)(uint32_t)b << 48) | ((uint64_t)(uint32_t)x0 << 32) |
         ((uint64_t)(uint32_t)x1 << 16) | (uint64_t)(uint32_t)x2;
}

// 64-bit finaliser of MurmurHash3 (public domain): spreads nearby locations
// over the table.
__device__ __forceinline__ uint64_t mix64(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return k;
}

struct __align__(16) Slot {
  uint64_t key;
  int32_t row;
  int32_t pad;
};

__device__ __forceinline__ int32_t table_lookup(const Slot* __restrict__ table, uint64_t mask, uint64_t key) {
  uint64_t slot = mix64(key) & mask;
  while (true) {
    const Slot v = table[slot];
    if (v.key == key) return v.row;
    if (v.key == kEmptyKey) return -1;
    slot = (slot + 1) & mask;
  }
}

// Every slot empty; the row field starts at row_init (INT32_MAX for the
// first-visit minimum of the SC output dictionary).
// Also zeroes the first n_zero words of `zero` (the build's counters).
__global__ void k_fill_slots(Slot* __restrict__ table, uint64_t cap, int32_t row_init,
                             unsigned long long* __restrict__ zero, int n_zero) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_zero; i += (int64_t)gridDim.x * blockDim.x)
    zero[i] = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < cap;
       i += (uint64_t)gridDim.x * blockDim.x) {
    Slot v;
    v.key = kEmptyKey;
    v.row = row_init;
    v.pad = 0;
    table[i] = v;
  }
}

__device__ __forceinline__ bool in_grid(int x0, int x1, int x2, int L0, int L1, int L2) {
  return (unsigned)x0 < (unsigned)L0 && (unsigned)x1 < (unsigned)L1 && (unsigned)x2 < (unsigned)L2;
}

// 8-byte slots: key in the low word, row in the high word; all ones = empty.
constexpr uint32_t kEmptyKey32 = ~0u;

__device__ __forceinline__ uint32_t pack_key32(int b, int x0, int x1, int x2, int L0, int L1, int L2) {
  return (((uint32_t)b * (uint32_t)L0 + (uint32_t)x0) * (uint32_t)L1 + (uint32_t)x1) * (uint32_t)L2 +
         (uint32_t)x2;
}

// 32-bit finaliser of MurmurHash3 (public domain).
__device__ __forceinline__ uint32_t mix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85ebca6bu;
  h ^= h >> 13;
  h *= 0xc2b2ae35u;
  h ^= h >> 16;
  return h;
}

// Grouped slots of the 32-bit keys: word 0 the group key (all ones =
// empty), words 1..3 the rows of keys 3 g .. 3 g + 2 (all ones = -1 =
// absent).  A wavefront's 64 consecutive surface sites and three offsets
// along x2 touch about 60 such slots, against about 125 when every key has
// a slot of its own (storing runs of consecutive keys in consecutive slots
// of such a table instead clusters it, which made inserts and lookups
// slower).  Measured on 2M scene sites: the probe 232 -> 184 us and the
// insert 104 -> 82 us, against a fill of twice the bytes (9 -> 13 us);
// groups of 7 in 32-byte slots touch fewer slots (about 44) but took longer
// (probe 200 us, fill 22 us), and lower or higher loads did not help.
constexpr uint32_t kGroupKeys = 3;
constexpr int kGroupWords = 4;  // 16 bytes per slot

__device__ __forceinline__ uint32_t group_home(uint32_t group, uint32_t mask) { return mix32(group) & mask; }

// Every word all ones (empty group keys, absent rows); zeroes the first
// n_zero words of `zero`.
__global__ void k_fill_slots8(uint4* __restrict__ table, uint64_t pieces,
                              unsigned long long* __restrict__ zero, int n_zero) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_zero; i += (int64_t)gridDim.x * blockDim.x)
    zero[i] = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < pieces;
       i += (uint64_t)gridDim.x * blockDim.x)
    table[i] = make_uint4(~0u, ~0u, ~0u, ~0u);
}

// Insert into the grouped slots, in two passes so that most sites need no
// atomic (device-wide atomics are far slower than stores):
//  1. every site stores its group key into the group's home slot with a
//     plain store; of the groups that share a home slot one key remains;
//  2. every site reads its home slot back: its own group key means the
//     group holds the slot (all its sites agree); otherwise the site probes
//     on from the home slot with a CAS per slot, as an ordinary
//     linear-probing insert (a slot that holds its group key already was
//     claimed by another site of the group).  The site then stores its row
//     in the slot.
// Slots never become empty again, so every slot between a group's home slot
// and the slot that holds it is occupied, which is what lookups rely on.  A
// repeated location stores its row in the same word as the first; the probe
// finds that (a site whose own lookup returns another row).
// batch_lim: batch indices below it keep every key of their sample below
// the empty marker; a larger one raises kFlagWideKey and inserts nothing.
__device__ __forceinline__ int site_check8(const int4& c, int L0, int L1, int L2, uint32_t batch_lim) {
  if ((unsigned)c.x >= (unsigned)kMaxBatch || !in_grid(c.y, c.z, c.w, L0, L1, L2)) return kFlagOutOfRange;
  if ((uint32_t)c.x >= batch_lim) return kFlagWideKey;
  return 0;
}

__global__ __launch_bounds__(256) void k_insert8_store(const int4* __restrict__ coords, int64_t n, int L0, int L1,
                                                       int L2, uint32_t batch_lim, uint32_t* __restrict__ table,
                                                       uint32_t mask, unsigned long long* __restrict__ flags,
                                                       int4* __restrict__ copy) {
  int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  int4 c = coords[j];
  if (copy) copy[j] = c;
  const int bad = site_check8(c, L0, L1, L2, batch_lim);
  if (bad) {
    atomicOr(flags, (unsigned long long)bad);
    return;
  }
  const uint32_t group = pack_key32(c.x, c.y, c.z, c.w, L0, L1, L2) / kGroupKeys;
  table[(size_t)group_home(group, mask) * kGroupWords] = group;
}

__global__ __launch_bounds__(256) void k_insert8_fix(const int4* __restrict__ coords, int64_t n, int L0, int L1,
                                                     int L2, uint32_t batch_lim, uint32_t* __restrict__ table,
                                                     uint32_t mask) {
  int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  const int4 c = coords[j];
  if (site_check8(c, L0, L1, L2, batch_lim)) return;
  const uint32_t key = pack_key32(c.x, c.y, c.z, c.w, L0, L1, L2);
  const uint32_t group = key / kGroupKeys;
  uint32_t slot = group_home(group, mask);
  if (table[(size_t)slot * kGroupWords] != group) {
    while (true) {
      slot = (slot + 1) & mask;
      const uint32_t prev = atomicCAS(&table[(size_t)slot * kGroupWords], kEmptyKey32, group);
      if (prev == kEmptyKey32 || prev == group) break;
    }
  }
  table[(size_t)slot * kGroupWords + 1 + key % kGroupKeys] = (uint32_t)j;
}

// Insert every site; flag coordinates outside the grid and repeated
// locations.  copy (if not NULL) receives the coordinates.
__global__ __launch_bounds__(256) void k_insert(const int4* __restrict__ coords, int64_t n, int L0,
                                                int L1, int L2, Slot* __restrict__ table, uint64_t mask,
                                                unsigned long long* __restrict__ flags, int4* __restrict__ copy) {
  int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  int4 c = coords[j];
  if (copy) copy[j] = c;
  if ((unsigned)c.x >= (unsigned)kMaxBatch || !in_grid(c.y, c.z, c.w, L0, L1, L2)) {
    atomicOr(flags, (unsigned long long)kFlagOutOfRange);
    return;
  }
  uint64_t key = pack_key(c.x, c.y, c.z, c.w);
  uint64_t slot = mix64(key) & mask;
  while (true) {
    unsigned long long prev =
        atomicCAS((unsigned long long*)&table[slot].key, (unsigned long long)kEmptyKey,
                  (unsigned long long)key);
    if (prev == kEmptyKey) {
      table[slot].row = (int32_t)j;
      return;
    }
    if (prev == key) {
      atomicOr(flags, (unsigned long long)kFlagDuplicate);
      return;
    }
    slot = (slot + 1) & mask;
  }
}

// ---------------------------------------------------------------- SSC probe
// One wavefront per (tile of 64 output sites, slice of P consecutive
// offsets).  Many small wavefronts keep enough independent lookups in flight
// (the probe is bound by the table reads).  nbr is offset-major [K][n]:
// nbr[o*n + k] = row of the site at x_k + i_o - (f-1)/2, or -1.
// With `mirror`, only the offsets below the centre c = (K-1)/2 are looked
// up: site j is the neighbour of site k at offset o exactly when k is the
// neighbour of j at the mirror offset K-1-o (i_{K-1-o} - (f-1)/2 =
// -(i_o - (f-1)/2)), so each hit also fills nbr[K-1-o][j] = k (those rows
// start at -1), and nbr[c][k] = k; counts[o*n_tiles + t] = hits of tile t
// at offset o (ballot) for o < c, the other offsets are counted afterwards
// (k_count_nbr).  Without it every offset is looked up and counted here
// (fewer launches: better for small inputs).
// Inputs from this many sites on use the mirrored SSC probe.
constexpr int64_t kMirrorProbeMin = 1 << 18;

template <int P, bool NARROW>
__global__ __launch_bounds__(256) void k_ssc_probe(
    const int4* __restrict__ coords, int64_t n, int L0, int L1, int L2, int f,
    const void* __restrict__ table_v, uint64_t mask, int32_t* __restrict__ nbr, int64_t* __restrict__ counts,
    int64_t n_tiles, int mirror, uint32_t batch_lim, unsigned long long* __restrict__ flags) {
  const int lane = threadIdx.x & 63;
  const int plane = f * f, K = f * f * f;
  // Workgroup = 4 tiles x one slice of P offsets.  Logical order: tile
  // groups major, slices minor, and each XCD takes a contiguous run of it,
  // so the lookups that the slices of neighbouring sites share stay in that
  // XCD's L2.
  const int ctr = (K - 1) / 2;
  const int o_end = mirror ? ctr : K;  // offsets looked up
  const int slices = max((o_end + P - 1) / P, 1);
  const int64_t lb = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t t = (lb / slices) * (blockDim.x / 64) + (threadIdx.x >> 6);
  if (t >= n_tiles) return;  // uniform per wavefront
  const int64_t k = t * kTile + lane;
  const bool valid = k < n;
  const int4 c = valid ? coords[k] : make_int4(0, 0, 0, 0);
  const bool site_ok = valid && (unsigned)c.x < (unsigned)kMaxBatch && in_grid(c.y, c.z, c.w, L0, L1, L2);
  const int h = (f - 1) / 2;
  const int o0 = (int)(lb % slices) * P;
  if (mirror && o0 == 0 && valid) nbr[(int64_t)ctr * n + k] = site_ok ? (int32_t)k : -1;
  int32_t rows[P];
  if constexpr (NARROW) {
    // Grouped slots: a lookup reads the group's home slot whole (one 16-byte
    // load: the group key and the rows; one round trip unless the slot holds
    // another group), and walks on slot by slot to the group or to an empty
    // slot.  (Two 4-byte loads, the key and the row word: 190 us instead of
    // 184 for the 2M-site scenes.)
    static_assert(kGroupWords == 4, "one 16-byte load per slot");
    const uint32_t* tb = reinterpret_cast<const uint32_t*>(table_v);
    uint32_t grp[P], sub[P], slot[P], gw[P], rw[P];
    bool live[P];
    auto read_slot = [&](int q) {
      const uint4 v = *reinterpret_cast<const uint4*>(tb + (size_t)slot[q] * kGroupWords);
      gw[q] = v.x;
      rw[q] = sub[q] == 0 ? v.y : (sub[q] == 1 ? v.z : v.w);
    };
#pragma unroll
    for (int q = 0; q < P; ++q) {
      const int o = o0 + q;
      const int i0 = o / plane, i1 = (o / f) % f, i2 = o % f;
      const int y0 = c.y + i0 - h, y1 = c.z + i1 - h, y2 = c.w + i2 - h;
      live[q] = o < o_end && site_ok && in_grid(y0, y1, y2, L0, L1, L2);
      const uint32_t key = pack_key32(c.x, y0, y1, y2, L0, L1, L2);
      grp[q] = key / kGroupKeys;
      sub[q] = key % kGroupKeys;
      slot[q] = group_home(grp[q], (uint32_t)mask);
      if (live[q]) read_slot(q);
    }
#pragma unroll
    for (int q = 0; q < P; ++q) {
      rows[q] = -1;
      bool done = !live[q];
      while (!done) {
        if (gw[q] == grp[q]) {
          rows[q] = (int32_t)rw[q];
          done = true;
        } else if (gw[q] == kEmptyKey32) {
          done = true;
        } else {
          slot[q] = (slot[q] + 1) & (uint32_t)mask;
          read_slot(q);
        }
      }
    }
    // A repeated location stored its row in the same word as the first: the
    // site whose own lookup returns another row reports it (one slice per
    // site; sites past the batch limit were not inserted).
    if (o0 == 0 && site_ok && (uint32_t)c.x < batch_lim) {
      const uint32_t key = pack_key32(c.x, c.y, c.z, c.w, L0, L1, L2);
      const uint32_t g0 = key / kGroupKeys, s0 = key % kGroupKeys;
      uint32_t sl = group_home(g0, (uint32_t)mask);
      while (tb[(size_t)sl * kGroupWords] != g0) sl = (sl + 1) & (uint32_t)mask;  // present: inserted
      if (tb[(size_t)sl * kGroupWords + 1 + s0] != (uint32_t)k) atomicOr(flags, (unsigned long long)kFlagDuplicate);
    }
  } else {
    // 16-byte slots: a lookup reads the aligned window of 4 slots (64 bytes)
    // that holds its first slot, and the following windows while the probe
    // sequence runs on (stop at the key or at an empty slot), so most
    // lookups take a single round trip.
    uint64_t key[P], slot[P];
    bool live[P];
    uint64_t vk[P][4];
    int32_t vr[P][4];
    auto window = [&](uint64_t sl) -> uint64_t { return sl & ~3ull; };
    auto read_window = [&](int q) {
      const Slot* tw = reinterpret_cast<const Slot*>(table_v) + window(slot[q]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const Slot e = tw[j];
        vk[q][j] = e.key;
        vr[q][j] = e.row;
      }
    };
#pragma unroll
    for (int q = 0; q < P; ++q) {
      const int o = o0 + q;
      const int i0 = o / plane, i1 = (o / f) % f, i2 = o % f;
      const int y0 = c.y + i0 - h, y1 = c.z + i1 - h, y2 = c.w + i2 - h;
      live[q] = o < o_end && site_ok && in_grid(y0, y1, y2, L0, L1, L2);
      key[q] = pack_key(c.x, y0, y1, y2);
      slot[q] = mix64(key[q]) & mask;
      if (live[q]) read_window(q);
    }
#pragma unroll
    for (int q = 0; q < P; ++q) {
      rows[q] = -1;
      bool done = !live[q];
      while (!done) {
        const int from = (int)(slot[q] - window(slot[q]));
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (!done && j >= from) {
            if (vk[q][j] == key[q]) {
              rows[q] = vr[q][j];
              done = true;
            } else if (vk[q][j] == kEmptyKey) {
              done = true;
            }
          }
        }
        if (!done) {
          slot[q] = (window(slot[q]) + 4) & mask;  // first slot of the next window
          read_window(q);
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < P; ++q) {
    const int o = o0 + q;
    if (o >= o_end) break;  // uniform
    const int32_t row = rows[q];
    if (valid) nbr[(int64_t)o * n + k] = row;
    if (mirror && row >= 0) nbr[(int64_t)(K - 1 - o) * n + row] = (int32_t)k;
    const unsigned long long bal = __ballot(row >= 0);
    if (lane == 0) counts[(int64_t)o * n_tiles + t] = __popcll(bal);
  }
}

// stats[1 + o] = |R_o| = seg[(o+1) T] - seg[o T] after the scan.
__global__ void k_offset_totals(const int64_t* __restrict__ seg, int64_t n_tiles, int K,
                                unsigned long long* __restrict__ stats) {
  const int o = blockIdx.x * blockDim.x + threadIdx.x;
  if (o < K) stats[1 + o] = (unsigned long long)(seg[(int64_t)(o + 1) * n_tiles] - seg[(int64_t)o * n_tiles]);
}

// Count, per (offset, tile), the present entries of an offset-major
// neighbour map for offsets [o_first, K) (the SC directions; the SSC
// offsets from the centre on).
__global__ __launch_bounds__(256) void k_count_nbr(const int32_t* __restrict__ nbr, int64_t n_rows,
                                                   int K, int64_t* __restrict__ counts,
                                                   int64_t n_tiles, int o_first = 0) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  if (t >= n_tiles) return;
  const int64_t k = t * kTile + lane;
  const bool valid = k < n_rows;
  for (int o = o_first; o < K; ++o) {
    const int32_t row = valid ? nbr[(int64_t)o * n_rows + k] : -1;
    const unsigned long long m = __ballot(row >= 0);
    if (lane == 0) counts[(int64_t)o * n_tiles + t] = __popcll(m);
  }
}

// Write every present entry at its segment start + its rank among the
// wavefront's present entries (so segments are sorted by output row).  With
// row_mask (K <= kPlanMaxK), also the set of offsets present for each row
// (plan_words(K) words per row, offset o as bit o % 32 of word o / 32).  One
// workgroup per tile: wavefront w takes the offsets o = w mod 4 (four times
// the wavefronts of one per tile, to keep more reads in flight), and the
// row masks of the four are combined in LDS.
// host_stats (if not NULL, pinned host memory): workgroup 0 also copies
// the n_stats words of stats there (sizes and flags, final before this
// kernel), in place of a separate copy to the host.
__global__ __launch_bounds__(256) void k_compact(const int32_t* __restrict__ nbr, int64_t n_rows, int K,
                                                 const int64_t* __restrict__ seg, int64_t n_tiles,
                                                 int32_t* __restrict__ in_rows,
                                                 int32_t* __restrict__ out_rows,
                                                 uint32_t* __restrict__ row_mask,
                                                 const unsigned long long* __restrict__ stats,
                                                 unsigned long long* __restrict__ host_stats, int n_stats) {
  __shared__ uint32_t part[kPlanMaskWords][4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // one workgroup per tile, consecutive tiles on one XCD: the runs of
  // neighbouring tiles meet inside cache lines, merged in that XCD's L2
  const int64_t t = xcd_remap(blockIdx.x, gridDim.x);
  if (host_stats && blockIdx.x == 0)
    for (int i = threadIdx.x; i < n_stats; i += blockDim.x) host_stats[i] = stats[i];
  const int64_t k = t * kTile + lane;
  const bool valid = k < n_rows;
  const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  // the tile's segment starts, offset o in lane o % 64 of word o / 64 (one
  // round trip instead of one per offset; K <= 128, else read in the loop)
  const bool seg_regs = K <= 128;
  int64_t s_lo = 0, s_hi = 0;
  if (seg_regs) {
    if (lane < K) s_lo = seg[(int64_t)lane * n_tiles + t];
    if (lane + 64 < K) s_hi = seg[(int64_t)(lane + 64) * n_tiles + t];
  }
  uint32_t present[kPlanMaskWords] = {0u, 0u, 0u};
  // the rows of up to 8 of the wavefront's offsets are requested together
  // (one round trip per 8)
  constexpr int B = 8;
  int32_t rows[B];
  for (int i = 0, o = wave; o < K; ++i, o += 4) {
    if (i % B == 0) {
#pragma unroll
      for (int q = 0; q < B; ++q)
        rows[q] = (valid && o + 4 * q < K) ? nbr[(int64_t)(o + 4 * q) * n_rows + k] : -1;
    }
    int32_t row = rows[0];
#pragma unroll
    for (int q = 1; q < B; ++q)
      if (i % B == q) row = rows[q];
    const unsigned long long m = __ballot(row >= 0);
    int64_t start;
    if (seg_regs) {
      const int64_t w = o < 64 ? s_lo : s_hi;
      const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)w, o & 63);
      const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(w >> 32), o & 63);
      start = (int64_t)(((uint64_t)hi << 32) | lo);
    } else {
      start = m ? seg[(int64_t)o * n_tiles + t] : 0;
    }
    if (row >= 0) {
      const int64_t pos = start + __popcll(m & below);
      in_rows[pos] = row;
      out_rows[pos] = (int32_t)k;
      const uint32_t bit = 1u << (o & 31);
      present[0] |= o < 32 ? bit : 0u;
      present[1] |= o >= 32 && o < 64 ? bit : 0u;
      present[2] |= o >= 64 ? bit : 0u;
    }
  }
  if (!row_mask) return;  // uniform
  const int W = plan_words(K);
#pragma unroll
  for (int i = 0; i < kPlanMaskWords; ++i) part[i][wave][lane] = present[i];
  __syncthreads();
  if (wave == 0 && valid)
    for (int i = 0; i < W; ++i)
      row_mask[k * W + i] = part[i][0][lane] | part[i][1][lane] | part[i][2][lane] | part[i][3][lane];
}

// ------------------------------------------------------------- tile order
// Work of a tile = number of 16-pair chunks over all offsets.  The tiles are
// cut into kTileGroups contiguous index ranges (group g = t * groups / T,
// one per XCD, so that neighbouring tiles share an L2) and listed group by
// group, each group by decreasing work (a counting sort), so that the
// workgroups dealing out a group's tiles finish on its smallest ones.
__global__ void k_tile_work(const int64_t* __restrict__ seg, int64_t n_tiles, int K, int max_key,
                            int32_t* __restrict__ key, int32_t* __restrict__ hist) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_tiles) return;
  int chunks = 0;
  for (int o = 0; o < K; ++o) {
    const int64_t n = seg[(int64_t)o * n_tiles + t + 1] - seg[(int64_t)o * n_tiles + t];
    chunks += (int)((n + 15) >> 4);
  }
  const int grp = (int)(t * kTileGroups / n_tiles);
  const int k = grp * (max_key + 1) + max_key - min(chunks, max_key);  // larger work -> smaller key
  key[t] = k;
  atomicAdd(&hist[k], 1);
}

__global__ void k_tile_scatter(const int32_t* __restrict__ key, int64_t n_tiles, int32_t* __restrict__ cursor,
                               int32_t* __restrict__ order) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_tiles) return;
  order[atomicAdd(&cursor[key[t]], 1)] = (int32_t)t;
}

// --------------------------------------------------- one-workgroup passes
// For the small arrays of a build a single workgroup of 1024 threads does a
// whole pass in one launch (launches dominate such passes).
constexpr int kOneBlock = 1024;
constexpr int64_t kOneBlockScanMax = 1 << 17;     // elements
constexpr int64_t kOneBlockSegMax = 1 << 15;      // elements, for the in-place segment scans of compaction

// Exclusive prefix of the per-thread values `v` over the workgroup (1024
// threads = 16 wavefronts); returns the total through `total`.
__device__ int64_t block_exclusive_scan(int64_t v, int64_t* wave_tot, int64_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) wave_tot[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t run = 0;
    for (int w = 0; w < kOneBlock / 64; ++w) {
      const int64_t t = wave_tot[w];
      wave_tot[w] = run;
      run += t;
    }
    wave_tot[kOneBlock / 64] = run;
  }
  __syncthreads();
  total = wave_tot[kOneBlock / 64];
  return wave_tot[wave] + x - v;
}

// Inclusive prefix sum over the 64 lanes of a wavefront with DPP moves (no
// LDS round trips): shifts by 1, 2, 4, 8 inside each row of 16 lanes, then
// the row totals are carried into the following rows.
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false); // row_bcast:15 into rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false); // row_bcast:31 into rows 2, 3
  return x;
}

// seg = exclusive scan of counts (count entries; seg[count] = total).  If
// stats is not NULL, stats[1 + o] = seg[(o+1) T] - seg[o T] (pairs per
// offset) for o < K.  One workgroup of kOneBlock threads: each wavefront
// scans a contiguous range in coalesced 64-element chunks (16 chunks loaded
// per round), twice: once for its total, once to write the prefix.
__global__ __launch_bounds__(kOneBlock) void k_scan_one_block(const int64_t* counts,  // may alias seg
                                                              int64_t* seg, int64_t count,
                                                              int64_t n_tiles, int K,
                                                              unsigned long long* __restrict__ stats) {
  constexpr int U = 16;
  constexpr int NW = kOneBlock / 64;
  __shared__ int64_t wave_base[NW + 1];
  extern __shared__ int64_t bound[];  // K + 1 entries: seg[o T]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t per = (count + NW - 1) / NW;
  const int64_t lo = min<int64_t>((int64_t)wave * per, count), hi = min<int64_t>(lo + per, count);
  // pass 1: the wave's total
  int64_t part = 0;
  for (int64_t i0 = lo; i0 < hi; i0 += 64 * U) {
    int64_t v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + 64 * u + lane;
      v[u] = i < hi ? counts[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) part += v[u];
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) part += __shfl_xor(part, d, 64);
  if (lane == 0) wave_base[wave] = part;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t run = 0;
    for (int w = 0; w < NW; ++w) {
      const int64_t t = wave_base[w];
      wave_base[w] = run;
      run += t;
    }
    wave_base[NW] = run;
  }
  __syncthreads();
  // pass 2: prefix within 64-element chunks plus a running carry
  int64_t carry = wave_base[wave];
  for (int64_t i0 = lo; i0 < hi; i0 += 64 * U) {
    int64_t v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + 64 * u + lane;
      v[u] = i < hi ? counts[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // an element counts the pairs of one (offset, tile): at most kTile, so
      // a chunk of 64 fits 32-bit arithmetic
      const int x = wave_inclusive_scan((int)v[u]);
      const int64_t i = i0 + 64 * u + lane;
      const int64_t ex = carry + x - v[u];
      if (i < hi) {
        seg[i] = ex;
        if (stats && i % n_tiles == 0) bound[i / n_tiles] = ex;
      }
      carry += __builtin_amdgcn_readlane(x, 63);
    }
  }
  if (threadIdx.x == 0) {
    seg[count] = wave_base[NW];
    if (stats) bound[K] = wave_base[NW];
  }
  __syncthreads();
  if (stats)
    for (int o = threadIdx.x; o < K; o += blockDim.x) stats[1 + o] = (unsigned long long)(bound[o + 1] - bound[o]);
}

// The same scan with the whole array in registers (each element counts the
// pairs of one (offset, tile): at most kTile, so 32-bit arithmetic inside a
// wavefront): wavefront w holds chunks of 64 elements [64 C w, 64 C (w + 1)),
// loaded coalesced in one round trip; one pass gives the wavefront totals,
// a second scans the chunks with DPP.  count <= 16 * 64 * C.
template <int C>
__global__ __launch_bounds__(kOneBlock) void k_scan_seg_regs(const int64_t* counts,  // may alias seg
                                                             int64_t* seg, int64_t count, int64_t n_tiles, int K,
                                                             unsigned long long* __restrict__ stats) {
  constexpr int NW = kOneBlock / 64;
  __shared__ int64_t wsum[NW + 1];
  extern __shared__ int64_t bound[];  // K + 1 entries: seg[o T]
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t base = (int64_t)wave * 64 * C;
  // low words through a buffer resource: one lane offset, the chunk in the
  // scalar offset; elements past the end read zero
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int64_t*>(counts), (short)0, (int)(count * sizeof(int64_t)), 0x00020000);
  const int voff = (int)((base + lane) * sizeof(int64_t));
  int v[C], tot = 0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    v[c] = __builtin_amdgcn_raw_buffer_load_b32(rc, voff, c * 64 * (int)sizeof(int64_t), 0);
    tot += v[c];
  }
  const int wtot = __builtin_amdgcn_readlane(wave_inclusive_scan(tot), 63);
  if (lane == 0) wsum[wave] = wtot;
  __syncthreads();
  if (t == 0) {
    int64_t run = 0;
    for (int w = 0; w < NW; ++w) {
      const int64_t x = wsum[w];
      wsum[w] = run;
      run += x;
    }
    wsum[NW] = run;
  }
  __syncthreads();
  int64_t carry = wsum[wave];
  // i mod T and i / T, advanced by 64 = q64 T + r64 per chunk with one
  // compare (a loop here is turned into a 64-bit division per chunk by the
  // compiler); an empty rule book has no tiles.  count < 2^17, so 32 bits.
  const uint32_t T = (uint32_t)(n_tiles > 0 ? n_tiles : 1);
  const uint32_t q64 = 64u / T, r64 = 64u % T;
  uint32_t rem = (uint32_t)(base + lane) % T, quo = (uint32_t)(base + lane) / T;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int x = wave_inclusive_scan(v[c]);
    const int64_t i = base + 64 * c + lane;
    const int64_t ex = carry + x - v[c];
    if (i < count) {
      seg[i] = ex;
      if (stats && rem == 0) bound[quo] = ex;
    }
    carry += __builtin_amdgcn_readlane(x, 63);
    rem += r64;
    quo += q64;
    if (rem >= T) {
      rem -= T;
      ++quo;
    }
  }
  if (t == 0) {
    seg[count] = wsum[NW];
    if (stats) bound[K] = wsum[NW];
  }
  __syncthreads();
  if (stats)
    for (int o = t; o < K; o += blockDim.x) stats[1 + o] = (unsigned long long)(bound[o + 1] - bound[o]);
}

// seg from per-(offset, tile) counts (offset-major, K x T, not aliasing
// seg) with one workgroup per offset: workgroup o first sums the counts of
// all offsets before it (every workgroup reads them again; they are few and
// L2-resident), then scans its own T counts from that base.  stats[1 + o]
// (if not NULL) = pairs of offset o.  Used where K x T is small, so that the
// whole scan is one launch spread over K CUs.
__global__ __launch_bounds__(kOneBlock) void k_scan_seg_offsets(const int64_t* __restrict__ counts,
                                                                int64_t* __restrict__ seg, int64_t T, int K,
                                                                unsigned long long* __restrict__ stats) {
  __shared__ int64_t wave_tot[kOneBlock / 64 + 1];
  const int o = blockIdx.x;
  const int t = threadIdx.x;
  const int64_t first = (int64_t)o * T;
  // two counts per 16-byte load, 16 loads in flight per thread
  int64_t part = 0;
  const longlong2* c2 = reinterpret_cast<const longlong2*>(counts);
  const int64_t n2 = first / 2;
#pragma unroll 16
  for (int64_t q = t; q < n2; q += kOneBlock) {
    const longlong2 v = c2[q];
    part += v.x + v.y;
  }
  if ((first & 1) && t == 0) part += counts[first - 1];
  int64_t base;
  (void)block_exclusive_scan(part, wave_tot, base);
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < T; c0 += kOneBlock) {
    const int64_t i = c0 + t;
    const int64_t v = i < T ? counts[first + i] : 0;
    int64_t total;
    const int64_t ex = block_exclusive_scan(v, wave_tot, total);
    if (i < T) seg[first + i] = base + carry + ex;
    carry += total;
  }
  if (t == 0) {
    if (o == K - 1) seg[(int64_t)K * T] = base + carry;
    if (stats) stats[1 + o] = (unsigned long long)carry;
  }
}

// seg from counts in one launch where that fits (see k_scan_one_block).
static void launch_seg_scan_one(const int64_t* counts, int64_t* seg, int64_t count, int64_t n_tiles, int K,
                                unsigned long long* stats, hipStream_t s) {
  const size_t lds = sizeof(int64_t) * (K + 1);
  if (counts != seg && K > 1 && count == K * n_tiles)
    k_scan_seg_offsets<<<K, kOneBlock, 0, s>>>(counts, seg, n_tiles, K, stats);
  else if (count <= 16 * 64 * 32)
    k_scan_seg_regs<32><<<1, kOneBlock, lds, s>>>(counts, seg, count, n_tiles, K, stats);
  else if (count <= 16 * 64 * 48)
    k_scan_seg_regs<48><<<1, kOneBlock, lds, s>>>(counts, seg, count, n_tiles, K, stats);
  else if (count <= 16 * 64 * 96)
    k_scan_seg_regs<96><<<1, kOneBlock, lds, s>>>(counts, seg, count, n_tiles, K, stats);
  else
    k_scan_one_block<<<1, kOneBlock, lds, s>>>(counts, seg, count, n_tiles, K, stats);
}

// The tile order (see build_tile_order) in one workgroup: keys from the
// chunk counts (kept in LDS), then a counting sort in LDS.
// (one workgroup reads K seg entries per tile: beyond a few thousand tiles
// the multi-workgroup passes are faster)
constexpr int64_t kOneBlockOrderMax = 1 << 12;    // tiles
__global__ __launch_bounds__(kOneBlock) void k_tile_order_one_block(const int64_t* __restrict__ seg,
                                                                    int64_t n_tiles, int K, int max_key,
                                                                    int32_t* __restrict__ order) {
  extern __shared__ int32_t hist[];  // bins = kTileGroups (max_key + 1), then n_tiles 16-bit keys
  __shared__ int64_t wave_tot[kOneBlock / 64 + 1];
  const int bins = kTileGroups * (max_key + 1);
  uint16_t* keys = reinterpret_cast<uint16_t*>(hist + bins);
  for (int i = threadIdx.x; i < bins; i += blockDim.x) hist[i] = 0;
  __syncthreads();
  for (int64_t t = threadIdx.x; t < n_tiles; t += blockDim.x) {
    int chunks = 0;
#pragma unroll 9
    for (int o = 0; o < K; ++o) {
      const int64_t n = seg[(int64_t)o * n_tiles + t + 1] - seg[(int64_t)o * n_tiles + t];
      chunks += (int)((n + 15) >> 4);
    }
    const int grp = (int)(t * kTileGroups / n_tiles);
    const int key = grp * (max_key + 1) + max_key - min(chunks, max_key);  // larger work -> smaller key
    keys[t] = (uint16_t)key;
    atomicAdd(&hist[key], 1);
  }
  __syncthreads();
  // exclusive scan of the bins: each thread a contiguous run
  const int per = (bins + kOneBlock - 1) / kOneBlock;
  const int lo = min((int)threadIdx.x * per, bins), hi = min(lo + per, bins);
  int64_t sum = 0;
  for (int i = lo; i < hi; ++i) sum += hist[i];
  int64_t total;
  int64_t run = block_exclusive_scan(sum, wave_tot, total);
  for (int i = lo; i < hi; ++i) {
    const int c = hist[i];
    hist[i] = (int)run;
    run += c;
  }
  __syncthreads();
  for (int64_t t = threadIdx.x; t < n_tiles; t += blockDim.x) order[atomicAdd(&hist[keys[t]], 1)] = (int32_t)t;
}

// ----------------------------------------------------------------- SC build
struct ScGeom {
  int f, s, K;
  int L0, L1, L2;     // input extents
  int M0, M1, M2;     // output extents
};

// Output location seen by input c at offset o, if any.
__device__ __forceinline__ bool sc_target(const ScGeom& g, int4 c, int o, int& y0, int& y1, int& y2) {
  const int i0 = o / (g.f * g.f), i1 = (o / g.f) % g.f, i2 = o % g.f;
  const int t0 = c.y - i0, t1 = c.z - i1, t2 = c.w - i2;
  if (t0 < 0 || t1 < 0 || t2 < 0) return false;
  if (t0 % g.s || t1 % g.s || t2 % g.s) return false;
  y0 = t0 / g.s; y1 = t1 / g.s; y2 = t2 / g.s;
  return y0 < g.M0 && y1 < g.M1 && y2 < g.M2;
}

__device__ __forceinline__ bool site_in_range(int4 c, const ScGeom& g) {
  return (unsigned)c.x < (unsigned)kMaxBatch && in_grid(c.y, c.z, c.w, g.L0, g.L1, g.L2);
}

// Record the first visit (smallest j*K + o) of every output location.
// With `check` (K <= 32 and f >= s: every input in range has a target),
// also flag inputs outside the grid and repeated locations: two inputs at
// one location visit the same (output, offset), which two distinct inputs
// never do, so the output slot keeps the offsets visited so far (its pad
// word) and a second visit of one is a repeated location.  `copy` (if not
// NULL) receives the coordinates.
__global__ __launch_bounds__(256) void k_sc_visit(const int4* __restrict__ coords, int64_t n, ScGeom g,
                                                  Slot* __restrict__ otable, uint64_t omask, int check,
                                                  unsigned long long* __restrict__ flags,
                                                  int4* __restrict__ copy) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  const int4 c = coords[j];
  if (copy) copy[j] = c;
  if (!site_in_range(c, g)) {
    if (check) atomicOr(flags, (unsigned long long)kFlagOutOfRange);
    return;
  }
  for (int o = 0; o < g.K; ++o) {
    int y0, y1, y2;
    if (!sc_target(g, c, o, y0, y1, y2)) continue;
    const uint64_t key = pack_key(c.x, y0, y1, y2);
    uint64_t slot = mix64(key) & omask;
    while (true) {
      unsigned long long prev =
          atomicCAS((unsigned long long*)&otable[slot].key, (unsigned long long)kEmptyKey,
                    (unsigned long long)key);
      if (prev == kEmptyKey || prev == key) break;
      slot = (slot + 1) & omask;
    }
    atomicMin(&otable[slot].row, (int32_t)(j * g.K + o));
    if (check) {
      const int32_t bit = (int32_t)(1u << o);
      if (atomicOr(&otable[slot].pad, bit) & bit) atomicOr(flags, (unsigned long long)kFlagDuplicate);
    }
  }
}

// Where every input sees at most one output (f <= s): its offset o (the
// position i = x mod s per dimension, when that is below f) and its output
// y = x div s.  Same result as sc_target over all offsets.
__device__ __forceinline__ bool sc_target1(const ScGeom& g, int4 c, bool in_range, int& o, int& y0, int& y1,
                                           int& y2) {
  const int i0 = c.y % g.s, i1 = c.z % g.s, i2 = c.w % g.s;
  o = (i0 * g.f + i1) * g.f + i2;
  y0 = c.y / g.s; y1 = c.z / g.s; y2 = c.w / g.s;
  return in_range && i0 < g.f && i1 < g.f && i2 < g.f && y0 < g.M0 && y1 < g.M1 && y2 < g.M2;
}

// Group the hit lanes of a wavefront by output key (one pass per distinct
// key): the lowest lane of each group, its leader, gets the group's lanes in
// peers (0 elsewhere); every hit lane gets its leader's lane (-1 elsewhere).
// Lanes follow the rows, so the leader holds the group's smallest visit.
__device__ __forceinline__ void sc_group(bool hit, uint64_t key, int lane, uint64_t& peers, int& leader) {
  uint64_t todo = __ballot(hit);
  peers = 0;
  leader = -1;
  while (todo) {
    const int l = __ffsll((unsigned long long)todo) - 1;
    const uint64_t lk = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(key >> 32), l) << 32) |
                        (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)key, l);
    const uint64_t p = __ballot(hit && key == lk);
    if (lane == l) peers = p;
    if ((p >> lane) & 1) leader = l;
    todo &= ~p;
  }
}

// unsorted[0] = 1 unless the rows are strictly increasing in (batch, x0,
// x1, x2): such rows hold no location twice (one plain store per
// wavefront that finds a pair out of order; no atomics).
__global__ __launch_bounds__(256) void k_sc_order(const int4* __restrict__ coords, int64_t n,
                                                  int* __restrict__ unsorted) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  if (j >= 1 && j < n) {
    const int4 a = coords[j - 1], b = coords[j];
    const bool less = a.x != b.x ? a.x < b.x : a.y != b.y ? a.y < b.y : a.z != b.z ? a.z < b.z : a.w < b.w;
    bad = !less;
  }
  const unsigned long long m = __ballot(bad);
  if (m && (threadIdx.x & 63) == __ffsll(m) - 1) unsorted[0] = 1;
}

// k_sc_visit where every input sees at most one output (f <= s: offset
// i = x mod s per dimension, when that is below f) and K <= 32.  The lanes
// of a wavefront whose inputs share an output (neighbouring rows of sorted
// coordinates often do: about half of the surface sites of 2^3 cells) are
// grouped first, and one lane per output does the atomics for its group:
// the lowest lane, whose visit is the group's smallest (lanes follow the
// rows), with the group's offsets in one OR.  Two lanes of a group with the
// same offset are one location twice.
__global__ __launch_bounds__(256) void k_sc_visit1(const int4* __restrict__ coords, int64_t n, ScGeom g,
                                                   Slot* __restrict__ otable, uint64_t omask, int check,
                                                   unsigned long long* __restrict__ flags,
                                                   int4* __restrict__ copy, const int* __restrict__ unsorted) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int lane = threadIdx.x & 63;
  const bool valid = j < n;
  const int4 c = valid ? coords[j] : make_int4(0, 0, 0, 0);
  if (valid && copy) copy[j] = c;
  const bool in_range = valid && site_in_range(c, g);
  if (valid && !in_range && check) atomicOr(flags, (unsigned long long)kFlagOutOfRange);
  int o, y0, y1, y2;
  const bool hit = sc_target1(g, c, in_range, o, y0, y1, y2);
  const uint64_t key = hit ? pack_key(c.x, y0, y1, y2) : kEmptyKey;
  uint64_t peers;
  int leader;
  sc_group(hit, key, lane, peers, leader);
  // offsets of each group: one ballot per offset
  uint32_t bits = 0;
  for (int b = 0; b < g.K; ++b)
    if (__ballot(hit && o == b) & peers) bits |= 1u << b;
  if (!peers) return;
  if (check && __popc(bits) != __popcll(peers)) atomicOr(flags, (unsigned long long)kFlagDuplicate);
  const bool collect = check && *unsorted;
  const int32_t v = (int32_t)(j * g.K + o);
  uint64_t slot = mix64(key) & omask;
  if (!collect) {
    // a slot that already holds the key with a smaller first visit needs no
    // atomics (its minimum only falls; a stale copy only shows an earlier,
    // larger state); else the insert starts where this probe stopped
    while (true) {
      const Slot e = otable[slot];
      if (e.key == key) {
        if (e.row < v) return;
        break;
      }
      if (e.key == kEmptyKey) break;
      slot = (slot + 1) & omask;
    }
  }
  while (true) {
    const unsigned long long prev =
        atomicCAS((unsigned long long*)&otable[slot].key, (unsigned long long)kEmptyKey, (unsigned long long)key);
    if (prev == kEmptyKey || prev == key) break;
    slot = (slot + 1) & omask;
  }
  atomicMin(&otable[slot].row, v);
  // rows in strictly increasing order hold no location twice: the offsets
  // are only collected (an atomic per group) for other rows
  if (collect && (atomicOr(&otable[slot].pad, (int32_t)bits) & (int32_t)bits))
    atomicOr(flags, (unsigned long long)kFlagDuplicate);
}

// first[v] = 1 iff visit v is the first visit of its output; count pairs
// per offset (wave ballots summed in LDS, one global atomic per block and
// offset).
__global__ __launch_bounds__(256) void k_sc_mark(const int4* __restrict__ coords, int64_t n, ScGeom g,
                                                 const Slot* __restrict__ otable, uint64_t omask,
                                                 int32_t* __restrict__ first,
                                                 unsigned long long* __restrict__ per_offset) {
  __shared__ unsigned int cnt[512];
  for (int o = threadIdx.x; o < g.K; o += blockDim.x) cnt[o] = 0;
  __syncthreads();
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool valid = j < n;
  const int4 c = valid ? coords[j] : make_int4(0, 0, 0, 0);
  const bool ok = valid && site_in_range(c, g);
  const int lane = threadIdx.x & 63;
  for (int o = 0; o < g.K; ++o) {
    int y0, y1, y2;
    int32_t is_first = 0;
    const bool hit = ok && sc_target(g, c, o, y0, y1, y2);
    if (hit) {
      const int32_t v = (int32_t)(j * g.K + o);
      is_first = table_lookup(otable, omask, pack_key(c.x, y0, y1, y2)) == v;
    }
    if (valid) first[j * g.K + o] = is_first;
    const unsigned long long m = __ballot(hit);
    if (lane == 0 && m) atomicAdd(&cnt[o], (unsigned int)__popcll(m));
  }
  __syncthreads();
  for (int o = threadIdx.x; o < g.K; o += blockDim.x)
    if (cnt[o]) atomicAdd(&per_offset[o], (unsigned long long)cnt[o]);
}

// k_sc_mark where every input sees at most one output: first[j] = 1 iff
// input j makes the first visit of its output.  Only a group leader (see
// sc_group) can: it looks up its output's first visit, the other lanes of
// its group are later rows of the same output.  The workgroup's pair count
// per offset goes to part[o][workgroup] (summed by k_offset_sums: global
// atomics on K words from every workgroup serialise).
__global__ __launch_bounds__(256) void k_sc_mark1(const int4* __restrict__ coords, int64_t n, ScGeom g,
                                                  const Slot* __restrict__ otable, uint64_t omask,
                                                  int32_t* __restrict__ first, uint32_t* __restrict__ part) {
  __shared__ unsigned int cnt[32];
  if (threadIdx.x < 32) cnt[threadIdx.x] = 0;
  __syncthreads();
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int lane = threadIdx.x & 63;
  const bool valid = j < n;
  const int4 c = valid ? coords[j] : make_int4(0, 0, 0, 0);
  int o, y0, y1, y2;
  const bool hit = sc_target1(g, c, valid && site_in_range(c, g), o, y0, y1, y2);
  const uint64_t key = hit ? pack_key(c.x, y0, y1, y2) : kEmptyKey;
  uint64_t peers;
  int leader;
  sc_group(hit, key, lane, peers, leader);
  int32_t is_first = 0;
  if (hit && leader == lane) is_first = table_lookup(otable, omask, key) == (int32_t)(j * g.K + o);
  if (valid) first[j] = is_first;
  for (int b = 0; b < g.K; ++b) {
    const unsigned long long m = __ballot(hit && o == b);
    if (lane == 0 && m) atomicAdd(&cnt[b], (unsigned int)__popcll(m));
  }
  __syncthreads();
  if (threadIdx.x < g.K) part[(int64_t)threadIdx.x * gridDim.x + blockIdx.x] = cnt[threadIdx.x];
}

// per_offset[o] = sum of part[o][0 .. n_parts), one workgroup per offset.
__global__ __launch_bounds__(kOneBlock) void k_offset_sums(const uint32_t* __restrict__ part, int64_t n_parts,
                                                           unsigned long long* __restrict__ per_offset) {
  __shared__ int64_t wave_tot[kOneBlock / 64 + 1];
  const uint32_t* row = part + (int64_t)blockIdx.x * n_parts;
  int64_t v = 0;
  for (int64_t i = threadIdx.x; i < n_parts; i += blockDim.x) v += row[i];
  int64_t total;
  (void)block_exclusive_scan(v, wave_tot, total);
  if (threadIdx.x == 0) per_offset[blockIdx.x] = (unsigned long long)total;
}

// Per visit: output row = rank of its output's first visit.  Writes the
// output-major map nbr_out[o][k] = j, the input-major map nbr_in[o][j] = k,
// and the output coordinates (by the first visitor).
__global__ __launch_bounds__(256) void k_sc_assign(const int4* __restrict__ coords, int64_t n, ScGeom g,
                                                   const Slot* __restrict__ otable, uint64_t omask,
                                                   const int32_t* __restrict__ rank, int64_t n_out,
                                                   int32_t* __restrict__ nbr_out,
                                                   int32_t* __restrict__ nbr_in,
                                                   int4* __restrict__ out_coords) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  const int4 c = coords[j];
  if (!site_in_range(c, g)) return;
  for (int o = 0; o < g.K; ++o) {
    int y0, y1, y2;
    if (!sc_target(g, c, o, y0, y1, y2)) continue;
    const int32_t vmin = table_lookup(otable, omask, pack_key(c.x, y0, y1, y2));
    const int32_t k = rank[vmin];
    nbr_out[(int64_t)o * n_out + k] = (int32_t)j;
    nbr_in[(int64_t)o * n + j] = k;
    if (vmin == (int32_t)(j * g.K + o)) out_coords[k] = make_int4(c.x, y0, y1, y2);
  }
}

// k_sc_assign for one_target (every input sees at most one output): besides
// nbr_out and the output coordinates, the input-major direction is kept as one
// record per input, tgt[j] = {k, o} ({-1, -1} for an input of no output), and
// its pair count per (offset, tile of kTile inputs) goes to counts[o][t] for
// every offset, so that no K x n map is filled, counted and compacted.
__global__ __launch_bounds__(256) void k_sc_assign1(const int4* __restrict__ coords, int64_t n, ScGeom g,
                                                    const Slot* __restrict__ otable, uint64_t omask,
                                                    const int32_t* __restrict__ rank, int64_t n_out,
                                                    int32_t* __restrict__ nbr_out, int2* __restrict__ tgt,
                                                    int64_t* __restrict__ counts, int64_t n_tiles,
                                                    int4* __restrict__ out_coords) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = j / kTile;  // one tile per wavefront
  if (t >= n_tiles) return;     // whole wavefronts
  const int lane = threadIdx.x & 63;
  const bool valid = j < n;
  const int4 c = valid ? coords[j] : make_int4(0, 0, 0, 0);
  int o, y0, y1, y2;
  const bool hit = sc_target1(g, c, valid && site_in_range(c, g), o, y0, y1, y2);
  const uint64_t key = hit ? pack_key(c.x, y0, y1, y2) : kEmptyKey;
  uint64_t peers;
  int leader;
  sc_group(hit, key, lane, peers, leader);
  // the leader looks up the output row for its group
  int32_t vmin = -1, k = -1;
  if (hit && leader == lane) {
    vmin = table_lookup(otable, omask, key);
    k = rank[vmin / g.K];
  }
  k = __shfl(k, hit ? leader : lane);
  const int32_t oj = hit ? o : -1;
  if (hit) {
    nbr_out[(int64_t)o * n_out + k] = (int32_t)j;
    if (vmin == (int32_t)(j * g.K + o)) out_coords[k] = make_int4(c.x, y0, y1, y2);
  }
  if (valid) tgt[j] = make_int2(hit ? k : -1, oj);
  for (int b = 0; b < g.K; ++b) {
    const unsigned long long m = __ballot(oj == b);
    if (lane == 0) counts[(int64_t)b * n_tiles + t] = __popcll(m);
  }
}

// Pairs and row masks of the input-major direction from the records of
// k_sc_assign1 (counts already scanned into seg): input j of tile t with
// offset o goes to seg[o][t] + its rank among the tile's inputs of offset o,
// the order k_compact gives; its row mask is the one bit of o (K <= 32).
__global__ __launch_bounds__(256) void k_compact1(const int2* __restrict__ tgt, int64_t n, int K,
                                                  const int64_t* __restrict__ seg, int64_t n_tiles,
                                                  int32_t* __restrict__ in_rows, int32_t* __restrict__ out_rows,
                                                  uint32_t* __restrict__ row_mask) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = j / kTile;
  if (t >= n_tiles) return;  // whole wavefronts
  const int lane = threadIdx.x & 63;
  const bool valid = j < n;
  const int2 r = valid ? tgt[j] : make_int2(-1, -1);
  unsigned long long peers = 0;
  for (int o = 0; o < K; ++o) {
    const unsigned long long m = __ballot(r.y == o);
    if (r.y == o) peers = m;
  }
  if (r.y >= 0) {
    const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t pos = seg[(int64_t)r.y * n_tiles + t] + __popcll(peers & below);
    in_rows[pos] = r.x;
    out_rows[pos] = (int32_t)j;
  }
  if (row_mask && valid) row_mask[j] = r.y >= 0 ? 1u << r.y : 0u;
}

// ------------------------------------------------------------- host helpers
static uint64_t table_capacity(int64_t n) {
  uint64_t cap = 64;
  while (cap < (uint64_t)(2 * n)) cap <<= 1;
  return cap;
}

static inline unsigned grid_for(int64_t threads, int block) {
  return (unsigned)std::max<int64_t>(1, ceil_div(threads, block));
}


// ------------------------------------------------------- chunk table
// Chunks per (tile, offset) of the padded chunk table.  A tile without any
// pair gets one padding chunk, so that its output rows are still written.
__global__ void k_chunk_count(const int64_t* __restrict__ seg, int64_t n_tiles, int K, int64_t n_ct,
                              int32_t* __restrict__ cnt) {
  const int64_t tt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tt >= n_ct) return;
  constexpr int S = kChunkRows / kTile;
  const int64_t t_lo = tt * S, t_hi = min<int64_t>(t_lo + S, n_tiles);
  int total = 0;
  for (int o = 0; o < K; ++o) {
    const int64_t c = seg[o * n_tiles + t_hi] - seg[o * n_tiles + t_lo];
    const int ch = (int)((c + 15) >> 4);
    cnt[tt * K + o] = ch;
    total += ch;
  }
  if (total == 0) cnt[tt * K] = 1;
}

// One thread per pair of offset blockIdx.y: its chunk and slot follow from
// its rank inside the (tile, offset) segment; the segment's last pair pads
// the rest of its chunk.
__global__ void k_chunk_fill(const int64_t* __restrict__ seg, int64_t n_tiles, int K,
                             const int32_t* __restrict__ in_rows, const int32_t* __restrict__ out_rows,
                             const int32_t* __restrict__ ctile, int32_t* __restrict__ c_in,
                             uint8_t* __restrict__ c_out, int32_t* __restrict__ c_off) {
  constexpr int S = kChunkRows / kTile;
  const int o = blockIdx.y;
  const int64_t p = seg[(int64_t)o * n_tiles] + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= seg[(int64_t)(o + 1) * n_tiles]) return;
  const int32_t orow = out_rows[p];
  const int64_t tt = orow / kChunkRows;
  const int64_t base = seg[o * n_tiles + tt * S];
  const int64_t end = seg[o * n_tiles + min<int64_t>(tt * S + S, n_tiles)];
  const int64_t q = p - base;
  const int64_t ch = ctile[tt * K + o] + (q >> 4);
  const int slot = (int)(q & 15);
  c_in[ch * 16 + slot] = in_rows[p];
  c_out[ch * 16 + slot] = (uint8_t)(orow - tt * kChunkRows);
  if (slot == 0) c_off[ch] = o;
  if (p + 1 == end)
    for (int e = slot + 1; e < 16; ++e) {
      c_in[ch * 16 + e] = -1;
      c_out[ch * 16 + e] = (uint8_t)kChunkRows;
    }
}

// The padding chunk of a tile without pairs.
__global__ void k_chunk_pad(const int64_t* __restrict__ seg, int64_t n_tiles, int K, int64_t n_ct,
                            const int32_t* __restrict__ ctile, int32_t* __restrict__ c_in,
                            uint8_t* __restrict__ c_out, int32_t* __restrict__ c_off) {
  const int64_t tt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tt >= n_ct) return;
  constexpr int S = kChunkRows / kTile;
  const int64_t t_lo = tt * S, t_hi = min<int64_t>(t_lo + S, n_tiles);
  int64_t pairs = 0;
  for (int o = 0; o < K; ++o) pairs += seg[o * n_tiles + t_hi] - seg[o * n_tiles + t_lo];
  if (pairs != 0) return;
  const int64_t ch = ctile[tt * K];
  for (int e = 0; e < 16; ++e) {
    c_in[ch * 16 + e] = -1;
    c_out[ch * 16 + e] = (uint8_t)kChunkRows;
  }
  c_off[ch] = 0;
}

// One device allocation carved into 256-byte aligned parts.
struct Arena {
  size_t total = 0;
  std::vector<std::pair<void**, size_t>> parts;
  template <typename T>
  void add(T** p, size_t count) {
    parts.push_back({(void**)p, total});
    total += (std::max<size_t>(count, 1) * sizeof(T) + 255) & ~(size_t)255;
  }
  sscn_status alloc(void** base, hipStream_t s) {
    SSCN_TRY(dev_alloc(base, total, s));
    for (auto& pr : parts) *pr.first = (char*)*base + pr.second;
    return SSCN_OK;
  }
};

// Stream-ordered temporaries released (after the queued work) on every exit path.
struct Temps {
  hipStream_t s;
  std::vector<void*> ptrs;
  explicit Temps(hipStream_t st) : s(st) {}
  sscn_status alloc(Arena& a) {
    void* base = nullptr;
    SSCN_TRY(a.alloc(&base, s));
    ptrs.push_back(base);
    return SSCN_OK;
  }
  ~Temps() {
    for (void* p : ptrs) dev_free(p, s);
  }
};

static sscn_status owned_alloc(RulebookData* d, Arena& a, hipStream_t s) {
  void* base = nullptr;
  SSCN_TRY(a.alloc(&base, s));
  d->blocks.push_back(base);
  return SSCN_OK;
}

// The single readback of a build, through pinned host staging, in two
// halves: readback_begin queues the copy and an event behind it, so that
// more work can be queued after it before readback_end waits for the copy
// alone (the GPU then runs that work while the host returns to its caller).
// One readback in flight per host thread.
struct ReadbackState {
  void* pinned = nullptr;
  size_t bytes = 0;
  hipEvent_t done = nullptr;
};
static thread_local ReadbackState t_readback;

// The staging buffer (at least `bytes`), for a kernel to write into
// directly (then readback_begin with dev = NULL only records the event).
static sscn_status readback_staging(size_t bytes, void** host) {
  ReadbackState& r = t_readback;
  if (r.bytes < bytes) {
    if (r.pinned) (void)hipHostFree(r.pinned);
    r.pinned = nullptr;
    r.bytes = 0;
    SSCN_HIP(hipHostMalloc(&r.pinned, std::max<size_t>(bytes, 4096), hipHostMallocCoherent));
    r.bytes = std::max<size_t>(bytes, 4096);
  }
  *host = r.pinned;
  return SSCN_OK;
}

static sscn_status readback_begin(const void* dev, size_t bytes, hipStream_t s) {
  ReadbackState& r = t_readback;
  void* staging = nullptr;
  SSCN_TRY(readback_staging(bytes, &staging));
  if (!r.done) SSCN_HIP(hipEventCreateWithFlags(&r.done, hipEventDisableTiming));
  if (dev) SSCN_HIP(hipMemcpyAsync(staging, dev, bytes, hipMemcpyDeviceToHost, s));
  SSCN_HIP(hipEventRecord(r.done, s));
  return SSCN_OK;
}

static sscn_status readback_end(void* host, size_t bytes) {
  SSCN_HIP(hipEventSynchronize(t_readback.done));
  std::memcpy(host, t_readback.pinned, bytes);
  return SSCN_OK;
}

static sscn_status readback(void* host, const void* dev, size_t bytes, hipStream_t s) {
  SSCN_TRY(readback_begin(dev, bytes, s));
  return readback_end(host, bytes);
}

static sscn_status launch_fill_slots(Slot* t, uint64_t cap, int32_t row_init, hipStream_t s,
                                     unsigned long long* zero = nullptr, int n_zero = 0) {
  k_fill_slots<<<(unsigned)std::min<uint64_t>((cap + 255) / 256, 16384), 256, 0, s>>>(t, cap, row_init, zero,
                                                                                       n_zero);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

// Segment table of one direction from its pair counts per (offset, tile),
// in place.
static sscn_status scan_seg(Storage& st, int K, hipStream_t s) {
  // one workgroup up to 32k counts (its time grows with the count: ~10 us
  // at 32k, ~27 us at 67k), the multi-workgroup scan beyond
  if (K * st.n_tiles <= kOneBlockSegMax) {
    launch_seg_scan_one(st.seg, st.seg, K * st.n_tiles, std::max<int64_t>(st.n_tiles, 1), K, nullptr, s);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  return exclusive_scan_i64(st.seg, st.seg, K * st.n_tiles, s);
}

// Segment table and pair arrays of one direction from an offset-major
// neighbour map (st.seg, st.in_rows and st.out_rows already allocated).
static sscn_status compact_storage(const int32_t* nbr, int64_t n_rows, int K, Storage& st, hipStream_t s,
                                   bool counted, uint32_t* row_mask = nullptr,
                                   const unsigned long long* stats = nullptr,
                                   unsigned long long* host_stats = nullptr, int n_stats = 0) {
  if (!counted && st.n_tiles > 0) {
    k_count_nbr<<<grid_for(st.n_tiles * 64, 256), 256, 0, s>>>(nbr, n_rows, K, st.seg, st.n_tiles);
    SSCN_HIP(hipGetLastError());
  }
  if (!counted) SSCN_TRY(scan_seg(st, K, s));
  if (st.n_tiles > 0) {
    k_compact<<<(unsigned)st.n_tiles, 256, 0, s>>>(nbr, n_rows, K, st.seg, st.n_tiles, st.in_rows,
                                                             st.out_rows, K <= kPlanMaxK ? row_mask : nullptr,
                                                             stats, host_stats, n_stats);
    SSCN_HIP(hipGetLastError());
  }
  return SSCN_OK;
}

// st.order from st.seg (st.order already allocated, n_tiles entries).
static sscn_status build_tile_order(Storage& st, int K, hipStream_t s) {
  if (st.n_tiles == 0) return SSCN_OK;
  const int max_key = K * (kTile / 16 + 1);
  const int bins = kTileGroups * (max_key + 1);
  const size_t lds = sizeof(int32_t) * bins + sizeof(uint16_t) * st.n_tiles;
  if (st.n_tiles <= kOneBlockOrderMax && bins <= 65536 && lds <= 128 * 1024) {
    k_tile_order_one_block<<<1, kOneBlock, lds, s>>>(st.seg, st.n_tiles, K, max_key, st.order);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  Temps tmp(s);
  int32_t* key; int32_t* hist;
  Arena a;
  a.add(&key, st.n_tiles);
  a.add(&hist, bins + 1);
  SSCN_TRY(tmp.alloc(a));
  SSCN_TRY(fill_i32(hist, 0, bins + 1, s));
  k_tile_work<<<grid_for(st.n_tiles, 256), 256, 0, s>>>(st.seg, st.n_tiles, K, max_key, key, hist);
  SSCN_HIP(hipGetLastError());
  SSCN_TRY(exclusive_scan_i32(hist, hist, bins, s));
  k_tile_scatter<<<grid_for(st.n_tiles, 256), 256, 0, s>>>(key, st.n_tiles, hist, st.order);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

// Padded chunk table of one direction (seg and pair arrays complete).
// Allocated in the rule book's own blocks.
static sscn_status build_chunks(RulebookData* d, Storage& st, int64_t n_rows, int K, hipStream_t s) {
  const int64_t n_ct = ceil_div(n_rows, kChunkRows);
  st.n_ctiles = n_ct;
  const int64_t cap = ceil_div(d->n_pairs, 16) + n_ct * (K + 1);
  Arena a;
  a.add(&st.ctile, (size_t)K * n_ct + 1);
  a.add(&st.c_in, (size_t)cap * 16);
  a.add(&st.c_out, (size_t)cap * 16);
  a.add(&st.c_off, (size_t)cap);
  SSCN_TRY(owned_alloc(d, a, s));
  if (n_ct == 0) return fill_i32(st.ctile, 0, 1, s);
  k_chunk_count<<<grid_for(n_ct, 256), 256, 0, s>>>(st.seg, st.n_tiles, K, n_ct, st.ctile);
  SSCN_HIP(hipGetLastError());
  SSCN_TRY(exclusive_scan_i32(st.ctile, st.ctile, (int64_t)K * n_ct, s));
  int64_t max_ppo = 0;
  for (int64_t c : d->pairs_per_offset) max_ppo = std::max(max_ppo, c);
  if (max_ppo > 0) {
    k_chunk_fill<<<dim3((unsigned)ceil_div(max_ppo, 256), (unsigned)K), 256, 0, s>>>(
        st.seg, st.n_tiles, K, st.in_rows, st.out_rows, st.ctile, st.c_in, st.c_out, st.c_off);
    SSCN_HIP(hipGetLastError());
  }
  k_chunk_pad<<<grid_for(n_ct, 256), 256, 0, s>>>(st.seg, st.n_tiles, K, n_ct, st.ctile, st.c_in, st.c_out,
                                                   st.c_off);
  SSCN_HIP(hipGetLastError());
  return SSCN_OK;
}

// Orders work on stream s behind a table built on first use: its kernels
// were queued on the rule book's own stream, and an event recorded there
// now follows them.  Events are recorded only when another stream asks (an
// event packet between two kernels of one stream idles the GPU for some
// microseconds).  Called with chunk_mu held.
static sscn_status follow_rulebook_stream(RulebookData* d, hipEvent_t& ev, hipStream_t s) {
  if (s == d->stream) return SSCN_OK;
  if (!ev) SSCN_HIP(hipEventCreateWithFlags(&ev, hipEventDisableTiming));
  SSCN_HIP(hipEventRecord(ev, d->stream));
  SSCN_HIP(hipStreamWaitEvent(s, ev, 0));
  return SSCN_OK;
}

sscn_status ensure_chunks(const View& v, hipStream_t s) {
  RulebookData* d = v.owner;
  Storage& st = v.st == &d->fwd ? d->fwd : d->bwd;
  {
    std::lock_guard<std::mutex> lock(d->chunk_mu);
    if (st.ctile == nullptr) {
      if (no_alloc())
        return fail(SSCN_ERR_INVALID_ARG,
                    "the rule book's chunk table is not built yet and this call may not allocate: run "
                    "sparse_conv_forward or sparse_conv_backward on it once first");
      int cur = 0;
      SSCN_HIP(hipGetDevice(&cur));
      if (cur != d->device) return fail(SSCN_ERR_INVALID_ARG, "rule book used on another device");
      const int64_t n_rows = &st == &d->fwd ? d->n_out : d->n_in;
      SSCN_TRY(build_chunks(d, st, n_rows, d->K, d->stream));
    }
    return follow_rulebook_stream(d, d->chunk_ready, s);
  }
}

sscn_status ensure_order(const View& v, hipStream_t s) {
  RulebookData* d = v.owner;
  Storage& st = v.st == &d->fwd ? d->fwd : d->bwd;
  {
    std::lock_guard<std::mutex> lock(d->chunk_mu);
    if (!st.order_built) {
      if (no_alloc())
        return fail(SSCN_ERR_INVALID_ARG,
                    "the rule book's tile order is not built yet and this call may not allocate: run "
                    "sparse_conv_forward or sparse_conv_backward on it once first");
      int cur = 0;
      SSCN_HIP(hipGetDevice(&cur));
      if (cur != d->device) return fail(SSCN_ERR_INVALID_ARG, "rule book used on another device");
      SSCN_TRY(build_tile_order(st, d->K, d->stream));
      st.order_built = true;
    }
    return follow_rulebook_stream(d, d->order_ready, s);
  }
}

// ------------------------------------------------------ row-block plan
// Offset set of every output row as a bit mask of W words (offset o is bit
// o % 32 of word o / 32).  One thread per pair of offset blockIdx.y (pairs
// of one offset have distinct output rows).
__global__ void k_plan_mask(const int64_t* __restrict__ seg, int64_t n_tiles,
                            const int32_t* __restrict__ out_rows, int W, uint32_t* __restrict__ mask) {
  const int o = blockIdx.y;
  const int64_t p = seg[(int64_t)o * n_tiles] + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= seg[(int64_t)(o + 1) * n_tiles]) return;
  atomicOr(&mask[(int64_t)out_rows[p] * W + (o >> 5)], 1u << (o & 31));
}

// A row's offset set (W <= kPlanMaskWords words; the rest zero).
struct RowSet {
  uint32_t w[kPlanMaskWords];
};
__device__ __forceinline__ RowSet load_set(const uint32_t* __restrict__ mask, int64_t r, int W, bool ok) {
  RowSet m;
#pragma unroll
  for (int i = 0; i < kPlanMaskWords; ++i) m.w[i] = ok && i < W ? mask[r * W + i] : 0u;
  return m;
}
// The sort key's offsets for more than 32 offsets (chosen on the host).
struct KeySel {
  uint8_t o[kPlanKeyBits];
};

// Sort key of an offset set: the set itself when it has at most
// kPlanKeyBits offsets; for 3^3 filters the 12 edge neighbours and 3 of the
// 6 face neighbours (o = 9 i0 + 3 i1 + i2; the centre is in nearly every
// set and the corners vary least between neighbouring surface sites);
// up to 32 offsets otherwise, the highest kPlanKeyBits; beyond 32 the
// offsets of sel (the host takes those displaced along exactly two axes).
__device__ __forceinline__ uint32_t plan_key(const RowSet& s, int K, const KeySel& sel) {
  if (K > 32) {
    uint32_t k = 0;
#pragma unroll
    for (int i = 0; i < kPlanKeyBits; ++i) {
      const int o = sel.o[i];
      const uint32_t w = o < 32 ? s.w[0] : (o < 64 ? s.w[1] : s.w[2]);
      k = (k << 1) | ((w >> (o & 31)) & 1u);
    }
    return k;
  }
  const uint32_t m = s.w[0];
  if (K <= kPlanKeyBits) return m;
  if (K == 27) {
    constexpr int sel[kPlanKeyBits] = {1, 3, 5, 7, 9, 11, 15, 17, 19, 21, 23, 25, 10, 12, 14};
    uint32_t k = 0;
#pragma unroll
    for (int i = 0; i < kPlanKeyBits; ++i) k = (k << 1) | ((m >> sel[i]) & 1u);
    return k;
  }
  return m >> (K - kPlanKeyBits);
}

// Adds one to counter[key] for every active lane with one atomic per distinct
// key of the wavefront (offset sets repeat a lot: a plain atomic per row
// serialises on the common ones) and returns the counter's value before this
// lane's increment.  Lanes find the lanes with the same key by one ballot
// per key bit, so all of the wavefront's atomics are issued at once.
template <int BITS = kPlanKeyBits>
__device__ __forceinline__ int wave_count(int32_t* counter, uint32_t key, bool active) {
  const int lane = threadIdx.x & 63;
  uint64_t peers = __ballot(active);
#pragma unroll
  for (int bit = 0; bit < BITS; ++bit) {
    const bool set = (key >> bit) & 1u;
    const uint64_t x = __ballot(set);
    peers &= set ? x : ~x;
  }
  const int leader = peers ? __ffsll((unsigned long long)peers) - 1 : lane;
  int base = 0;
  if (active && lane == leader) base = atomicAdd(&counter[key], __popcll(peers));
  base = __shfl(base, leader, 64);
  return base + __popcll(peers & ((1ull << lane) - 1ull));
}

// The counting sort's passes take 256 RPT rows per workgroup of 256 and
// count in LDS first (one LDS atomic per distinct key per wavefront, then
// one global atomic per distinct key per workgroup): the keys of surface
// rows are few and popular, and one global atomic per wavefront on the
// same few counters serialised the passes (60 us each at 2M rows).  LDS:
// one counter per key (at most 2^kPlanKeyBits = 128 KB), and the list of
// the keys the workgroup holds, so that only those are flushed.  RPT (rows
// per thread) grows with the row count so that there are about 256
// workgroups (one per CU: the counters take up to 128 KB).
constexpr int kSortMaxRows = 256 * 16;

struct SortLds {
  int32_t* cnt;        // bins counters (a multiple of 4)
  uint16_t* keys;      // distinct keys of the workgroup, in order of first sight
  int32_t* n_keys;
};
__device__ __forceinline__ SortLds sort_lds(char* base, int bins) {
  const int words = (bins + 3) & ~3;
  SortLds l;
  l.cnt = reinterpret_cast<int32_t*>(base);
  l.n_keys = l.cnt + words;
  l.keys = reinterpret_cast<uint16_t*>(l.n_keys + 4);
  // zero the counters (16 bytes per store) and the key count
  int4* c4 = reinterpret_cast<int4*>(l.cnt);
  for (int b = threadIdx.x; b < words / 4; b += blockDim.x) c4[b] = make_int4(0, 0, 0, 0);
  if (threadIdx.x == 0) *l.n_keys = 0;
  __syncthreads();
  return l;
}
static size_t sort_lds_bytes(int bins) {
  return sizeof(int32_t) * (((bins + 3) & ~3) + 4) + sizeof(uint16_t) * kSortMaxRows;
}

// wave_count on the workgroup's LDS counters; a key seen for the first time
// in the workgroup joins its key list.
__device__ __forceinline__ int count_in_lds(const SortLds& l, uint32_t key, bool active) {
  const int lane = threadIdx.x & 63;
  uint64_t peers = __ballot(active);
#pragma unroll
  for (int bit = 0; bit < kPlanKeyBits; ++bit) {
    const bool set = (key >> bit) & 1u;
    const uint64_t x = __ballot(set);
    peers &= set ? x : ~x;
  }
  const int leader = peers ? __ffsll((unsigned long long)peers) - 1 : lane;
  int base = 0;
  if (active && lane == leader) {
    base = atomicAdd(&l.cnt[key], __popcll(peers));
    if (base == 0) l.keys[atomicAdd(l.n_keys, 1)] = (uint16_t)key;
  }
  base = __shfl(base, leader, 64);
  return base + __popcll(peers & ((1ull << lane) - 1ull));
}

template <int RPT>
__global__ __launch_bounds__(256) void k_plan_hist(const uint32_t* __restrict__ mask, int64_t n, int K, int W,
                                                   KeySel sel, int bins, int32_t* __restrict__ hist) {
  static_assert(256 * RPT <= kSortMaxRows, "key list");
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const SortLds l = sort_lds(lds, bins);
  const int64_t r0 = (int64_t)blockIdx.x * (256 * RPT) + threadIdx.x;
  uint32_t key[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = r0 + 256 * i;
    key[i] = plan_key(load_set(mask, r, W, r < n), K, sel);
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const bool ok = r0 + 256 * i < n;
    (void)count_in_lds(l, ok ? key[i] : 0u, ok);
  }
  __syncthreads();
  for (int j = threadIdx.x; j < *l.n_keys; j += 256) {
    const int key = l.keys[j];
    atomicAdd(&hist[key], l.cnt[key]);
  }
}

// Counting sort by key (the order inside one key is arbitrary: it changes
// which rows share a block, never a row's result): a workgroup ranks its
// rows per key in LDS, reserves one range per key it holds, then places
// its rows.
template <int RPT>
__global__ __launch_bounds__(256) void k_plan_sort(const uint32_t* __restrict__ mask, int64_t n, int K, int W,
                                                   KeySel sel, int bins, int32_t* __restrict__ cursor,
                                                   int32_t* __restrict__ perm, int32_t* __restrict__ pos_of) {
  static_assert(256 * RPT <= kSortMaxRows, "key list");
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const SortLds l = sort_lds(lds, bins);
  const int64_t r0 = (int64_t)blockIdx.x * (256 * RPT) + threadIdx.x;
  uint32_t key[RPT];
  int32_t rank[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = r0 + 256 * i;
    key[i] = r < n ? plan_key(load_set(mask, r, W, true), K, sel) : 0u;
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) rank[i] = count_in_lds(l, key[i], r0 + 256 * i < n);
  __syncthreads();
  for (int j = threadIdx.x; j < *l.n_keys; j += 256) {
    const int k = l.keys[j];
    l.cnt[k] = atomicAdd(&cursor[k], l.cnt[k]);  // the workgroup's first position for key k
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int64_t r = r0 + 256 * i;
    if (r < n) {
      const int32_t p = l.cnt[key[i]] + rank[i];
      perm[p] = (int32_t)r;
      pos_of[r] = p;
    }
  }
}

// One wavefront per block: union of the offset sets of its rows and its item
// count; the positions past the last row are marked empty.
static_assert(kPlanRows == 64, "one wavefront per plan block");
__global__ void k_plan_blocks(const uint32_t* __restrict__ mask, int W, int32_t* __restrict__ perm, int64_t n,
                              int64_t n_blocks, uint32_t* __restrict__ bmask, int32_t* __restrict__ cnt) {
  const int64_t b = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (b >= n_blocks) return;
  const int64_t p = b * kPlanRows + lane;
  RowSet u;
  if (p < n) {
    u = load_set(mask, perm[p], W, true);
  } else {
    u = load_set(mask, 0, W, false);
    perm[p] = -1;
  }
  int c = 0;
#pragma unroll
  for (int i = 0; i < kPlanMaskWords; ++i) {
    if (i >= W) break;  // uniform
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) u.w[i] |= (uint32_t)__shfl_xor((int)u.w[i], d, 64);
    if (lane == 0) bmask[b * W + i] = u.w[i];
    c += __popc(u.w[i]);
  }
  if (lane == 0) cnt[b] = c;
}

// Thread (block, slot): marks its slot of every item of the block empty
// (items in ascending offset order).
__global__ void k_plan_items(const uint32_t* __restrict__ bmask, int W, const int32_t* __restrict__ b_first,
                             int64_t n_blocks, uint32_t* __restrict__ items) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t b = t / kPlanRows;
  const int m = (int)(t % kPlanRows);
  if (b >= n_blocks) return;
  int64_t item = b_first[b];
  for (int i = 0; i < W; ++i) {
    uint32_t u = bmask[b * W + i];
    while (u) {
      const uint32_t o = 32u * (uint32_t)i + (uint32_t)(__ffs(u) - 1);
      u &= u - 1;
      items[item * kPlanRows + m] = kPlanNoRow | (o << kPlanRowBits);
      ++item;
    }
  }
}

// Every pair into its block's item for its offset, at its row's slot.
__global__ void k_plan_pairs(const int64_t* __restrict__ seg, int64_t n_tiles, const int32_t* __restrict__ in_rows,
                             const int32_t* __restrict__ out_rows, const int32_t* __restrict__ pos_of,
                             const uint32_t* __restrict__ bmask, int W, const int32_t* __restrict__ b_first,
                             uint32_t* __restrict__ items) {
  const int o = blockIdx.y;
  const int64_t p = seg[(int64_t)o * n_tiles] + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= seg[(int64_t)(o + 1) * n_tiles]) return;
  const int32_t pos = pos_of[out_rows[p]];
  const int64_t b = pos / kPlanRows;
  // items before offset o's: the block's offsets below o
  int64_t item = b_first[b] + __popc(bmask[b * W + (o >> 5)] & ((1u << (o & 31)) - 1u));
  for (int i = 0; i < (o >> 5); ++i) item += __popc(bmask[b * W + i]);
  items[item * kPlanRows + pos % kPlanRows] = (uint32_t)in_rows[p] | ((uint32_t)o << kPlanRowBits);
}

// Blocks by decreasing item count, for more blocks than one workgroup takes
// in a launch: a counting sort over the K + 1 possible counts in two
// passes.  k_order_hist counts the blocks per count (LDS counters, one
// global atomic per count per workgroup); k_order_place ranks each
// workgroup's blocks per count in LDS, reserves one range per count with one
// global atomic, and writes their (block, first item, items, 0) records
// (the order inside one count is arbitrary).  kOrderPerWg blocks per
// workgroup; kOrderBins counters (item counts 0 .. K <= kPlanMaxK).
constexpr int kOrderPerWg = 4096;
constexpr int kOrderBins = 128;
static_assert(kPlanMaxK < kOrderBins, "one bin per item count");
__global__ __launch_bounds__(256) void k_order_hist(const int32_t* __restrict__ b_first, int64_t nb, int K,
                                                    int32_t* __restrict__ ohist) {
  __shared__ int32_t cnt[kOrderBins];
  if (threadIdx.x < kOrderBins) cnt[threadIdx.x] = 0;
  __syncthreads();
  const int64_t b0 = (int64_t)blockIdx.x * kOrderPerWg;
  for (int i = threadIdx.x; i < kOrderPerWg; i += 256) {
    const int64_t b = b0 + i;
    const bool ok = b < nb;
    (void)wave_count<7>(cnt, ok ? (uint32_t)(K - (b_first[b + 1] - b_first[b])) : 0u, ok);
  }
  __syncthreads();
  if (threadIdx.x <= K && cnt[threadIdx.x] > 0) atomicAdd(&ohist[threadIdx.x], cnt[threadIdx.x]);
}

__global__ __launch_bounds__(256) void k_order_place(const int32_t* __restrict__ b_first, int64_t nb, int K,
                                                     const int32_t* __restrict__ ohist, int32_t* __restrict__ ocur,
                                                     int4* __restrict__ order) {
  __shared__ int32_t cnt[kOrderBins], base[kOrderBins];
  if (threadIdx.x < kOrderBins) cnt[threadIdx.x] = 0;
  __syncthreads();
  const int64_t b0 = (int64_t)blockIdx.x * kOrderPerWg;
  constexpr int PER = kOrderPerWg / 256;
  int rank[PER];
  uint32_t key[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int64_t b = b0 + threadIdx.x + 256 * i;
    const bool ok = b < nb;
    key[i] = ok ? (uint32_t)(K - (b_first[b + 1] - b_first[b])) : 0u;
    rank[i] = wave_count<7>(cnt, key[i], ok);
  }
  __syncthreads();
  if (threadIdx.x <= K) {
    int start = 0;  // blocks of larger counts come first
    for (int c = 0; c < (int)threadIdx.x; ++c) start += ohist[c];
    base[threadIdx.x] = cnt[threadIdx.x] > 0 ? start + atomicAdd(&ocur[threadIdx.x], cnt[threadIdx.x]) : 0;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int64_t b = b0 + threadIdx.x + 256 * i;
    if (b < nb) order[base[key[i]] + rank[i]] = make_int4((int32_t)b, b_first[b], K - (int)key[i], 0);
  }
}

// Exclusive scan of at most kSmallScanMax int32 values in one launch (out
// may alias in; out[count] = total).  Wavefront w holds elements
// [2048 w, 2048 w + 2048) in registers, loaded in coalesced chunks of 64;
// one pass gives the wavefront totals, a second scans the chunks with DPP.
constexpr int kSmallScanMax = kOneBlock * 32;
__global__ __launch_bounds__(kOneBlock) void k_scan_small(const int32_t* in, int32_t* out, int count) {
  constexpr int NW = kOneBlock / 64;
  __shared__ int wsum[NW + 1];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int base = wave * 2048;
  int v[32], tot = 0;
#pragma unroll
  for (int c = 0; c < 32; ++c) {
    const int i = base + 64 * c + lane;
    v[c] = i < count ? in[i] : 0;
    tot += v[c];
  }
  const int wtot = __builtin_amdgcn_readlane(wave_inclusive_scan(tot), 63);
  if (lane == 0) wsum[wave] = wtot;
  __syncthreads();
  if (t == 0) {
    int run = 0;
    for (int w = 0; w < NW; ++w) {
      const int x = wsum[w];
      wsum[w] = run;
      run += x;
    }
    wsum[NW] = run;
  }
  __syncthreads();
  int carry = wsum[wave];
#pragma unroll
  for (int c = 0; c < 32; ++c) {
    const int x = wave_inclusive_scan(v[c]);
    const int i = base + 64 * c + lane;
    if (i < count) out[i] = carry + x - v[c];
    carry += __builtin_amdgcn_readlane(x, 63);
  }
  if (t == 0) out[count] = wsum[NW];
}

static sscn_status scan_i32(int32_t* p, int64_t count, hipStream_t s) {
  if (count <= kSmallScanMax) {
    k_scan_small<<<1, kOneBlock, 0, s>>>(p, p, (int)count);
    SSCN_HIP(hipGetLastError());
    return SSCN_OK;
  }
  return exclusive_scan_i32(p, p, count, s);
}

// Blocks by decreasing item count, with the scan of the item counts before
// it, in one workgroup (nb <= kScanOrderMax): cnt[b] (items of block b)
// becomes b_first (exclusive scan, b_first[nb] = total) and order lists the
// blocks by decreasing count as (block, first item, items, 0) records (a
// counting sort over the K + 1 possible counts; the order inside one count
// is arbitrary).  The counts stay in
// LDS for the second pass.  Beyond kScanOrderMax blocks the scan and the
// two passes of k_order_hist / k_order_place run wider.
constexpr int64_t kScanOrderMax = 8192;
__global__ __launch_bounds__(kOneBlock) void k_plan_scan_order(int32_t* __restrict__ cnt, int64_t nb, int K,
                                                               int4* __restrict__ order) {
  constexpr int NW = kOneBlock / 64;
  __shared__ uint8_t c8[kScanOrderMax];
  __shared__ int32_t hist[kOrderBins], cur[kOrderBins], wsum[NW];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  if (t < kOrderBins) hist[t] = 0;
  __syncthreads();
  int carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += kOneBlock) {
    const int64_t b = b0 + t;
    const bool ok = b < nb;
    const int v = ok ? cnt[b] : 0;
    if (ok) c8[b] = (uint8_t)v;
    const int inc = wave_inclusive_scan(v);
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int before = carry, total = 0;
    for (int w = 0; w < NW; ++w) {
      const int x = wsum[w];
      before += w < wave ? x : 0;
      total += x;
    }
    if (ok) cnt[b] = before + inc - v;
    carry += total;
    (void)wave_count<7>(hist, ok ? (uint32_t)(K - v) : 0u, ok);
    __syncthreads();  // wsum is rewritten by the next chunk
  }
  if (t == 0) {
    cnt[nb] = carry;
    int run = 0;
    for (int c = 0; c <= K; ++c) {
      cur[c] = run;
      run += hist[c];
    }
  }
  __syncthreads();
  for (int64_t b0 = 0; b0 < nb; b0 += kOneBlock) {
    const int64_t b = b0 + t;
    const bool ok = b < nb;
    const int p = wave_count<7>(cur, ok ? (uint32_t)(K - c8[b]) : 0u, ok);
    if (ok) order[p] = make_int4((int32_t)b, cnt[b], (int32_t)c8[b], 0);
  }
}

// Row-block plan of one direction (seg and pair arrays complete), in the
// rule book's own blocks.  ppo_bound >= 0: the pair counts are not on the
// host yet (the plan is queued inside the build); at most ppo_bound pairs
// per offset, and room for nb K items.  hist0: plan_hist_words(K) zeroed
// words for the key histogram, or NULL.
// The key histogram (bins + 1 words), then the block-count histogram and
// cursor of the block order (kOrderBins words each).
static int64_t plan_hist_words(int K) { return (1 << std::min(K, kPlanKeyBits)) + 1 + 2 * kOrderBins; }

// Sort-key offsets for more than 32 offsets: those displaced from the
// filter's middle along exactly two axes, in increasing o, then the others
// (the d-dimensional counterpart of the 3^3 filter's edge neighbours).
static KeySel plan_key_sel(int K, int f, int dim) {
  KeySel sel{};
  int n = 0;
  for (int pass = 0; pass < 2 && n < kPlanKeyBits; ++pass)
    for (int o = 0; o < K && n < kPlanKeyBits; ++o) {
      int nz = 0;
      for (int q = 0, r = o; q < dim; ++q, r /= f) nz += (r % f) != (f - 1) / 2;
      if ((nz == 2) == (pass == 0)) sel.o[n++] = (uint8_t)o;
    }
  return sel;
}

static sscn_status build_plan(RulebookData* d, Storage& st, int64_t n_rows, int K, hipStream_t s,
                              int64_t ppo_bound = -1, int32_t* hist0 = nullptr) {
  const int64_t nb = ceil_div(n_rows, kPlanRows);
  st.n_blocks = nb;
  const int64_t cap =
      std::max<int64_t>(1, ppo_bound >= 0 ? nb * K : std::min<int64_t>(d->n_pairs, nb * K));
  Arena a;
  a.add(&st.perm, (size_t)nb * kPlanRows);
  a.add(&st.b_first, (size_t)nb + 1);
  a.add(&st.b_rec, (size_t)nb);
  a.add(&st.items, (size_t)cap * kPlanRows);
  SSCN_TRY(owned_alloc(d, a, s));
  if (nb == 0) return fill_i32(st.b_first, 0, 1, s);
  const int bins = 1 << std::min(K, kPlanKeyBits);
  Temps tmp(s);
  const int W = plan_words(K);
  const KeySel sel = plan_key_sel(K, d->f, d->dim);
  uint32_t* mask = st.row_mask; uint32_t* bmask; int32_t* hist = nullptr; int32_t* pos_of;
  Arena t;
  if (!(hist0 && mask)) t.add(&hist, (size_t)plan_hist_words(K));
  if (!mask) t.add(&mask, (size_t)n_rows * W);  // right after hist: one fill clears both
  t.add(&bmask, (size_t)nb * W);
  t.add(&pos_of, (size_t)n_rows);
  SSCN_TRY(tmp.alloc(t));
  int64_t max_ppo = ppo_bound;
  if (ppo_bound < 0)
    for (int64_t c : d->pairs_per_offset) max_ppo = std::max(max_ppo, c);
  if (st.row_mask) {
    if (hist0) hist = hist0;
    else SSCN_TRY(fill_i32(hist, 0, plan_hist_words(K), s));
  } else {
    SSCN_TRY(fill_i32(hist, 0, (int32_t*)(mask + n_rows * W) - hist, s));
    if (max_ppo > 0) {
      k_plan_mask<<<dim3((unsigned)ceil_div(max_ppo, 256), (unsigned)K), 256, 0, s>>>(st.seg, st.n_tiles,
                                                                                      st.out_rows, W, mask);
      SSCN_HIP(hipGetLastError());
    }
  }
  const int64_t per_wg = ceil_div(n_rows, 256);  // rows per workgroup for 256 workgroups
  const int rpt = per_wg <= 256 ? 1 : per_wg <= 512 ? 2 : per_wg <= 1024 ? 4 : per_wg <= 2048 ? 8 : 16;
  const unsigned sort_wgs = (unsigned)ceil_div(n_rows, 256 * rpt);
  const size_t sort_lds = sort_lds_bytes(bins);
  auto hist_k = rpt == 1 ? k_plan_hist<1> : rpt == 2 ? k_plan_hist<2> : rpt == 4 ? k_plan_hist<4>
              : rpt == 8 ? k_plan_hist<8> : k_plan_hist<16>;
  auto sort_k = rpt == 1 ? k_plan_sort<1> : rpt == 2 ? k_plan_sort<2> : rpt == 4 ? k_plan_sort<4>
              : rpt == 8 ? k_plan_sort<8> : k_plan_sort<16>;
  hist_k<<<sort_wgs, 256, sort_lds, s>>>(mask, n_rows, K, W, sel, bins, hist);
  SSCN_HIP(hipGetLastError());
  SSCN_TRY(scan_i32(hist, bins, s));
  sort_k<<<sort_wgs, 256, sort_lds, s>>>(mask, n_rows, K, W, sel, bins, hist, st.perm, pos_of);
  SSCN_HIP(hipGetLastError());
  k_plan_blocks<<<grid_for(nb * 64, 256), 256, 0, s>>>(mask, W, st.perm, n_rows, nb, bmask, st.b_first);
  SSCN_HIP(hipGetLastError());
  if (nb <= kScanOrderMax) {
    k_plan_scan_order<<<1, kOneBlock, 0, s>>>(st.b_first, nb, K, st.b_rec);
  } else {
    SSCN_TRY(scan_i32(st.b_first, nb, s));
    int32_t* ohist = hist + bins + 1;
    const unsigned owgs = (unsigned)ceil_div(nb, kOrderPerWg);
    k_order_hist<<<owgs, 256, 0, s>>>(st.b_first, nb, K, ohist);
    SSCN_HIP(hipGetLastError());
    k_order_place<<<owgs, 256, 0, s>>>(st.b_first, nb, K, ohist, ohist + kOrderBins, st.b_rec);
  }
  SSCN_HIP(hipGetLastError());
  k_plan_items<<<grid_for(nb * kPlanRows, 256), 256, 0, s>>>(bmask, W, st.b_first, nb, st.items);
  SSCN_HIP(hipGetLastError());
  if (max_ppo > 0) {
    k_plan_pairs<<<dim3((unsigned)ceil_div(max_ppo, 256), (unsigned)K), 256, 0, s>>>(
        st.seg, st.n_tiles, st.in_rows, st.out_rows, pos_of, bmask, W, st.b_first, st.items);
    SSCN_HIP(hipGetLastError());
  }
  return SSCN_OK;
}

sscn_status ensure_plan(const View& v, hipStream_t s) {
  RulebookData* d = v.owner;
  if (d->K > kPlanMaxK || std::max(d->n_in, d->n_out) >= (int64_t)kPlanNoRow)
    return fail(SSCN_ERR_INVALID_ARG, "row-block plan needs at most 96 offsets and fewer than 2^25 - 1 rows");
  Storage& st = v.st == &d->fwd ? d->fwd : d->bwd;
  {
    std::lock_guard<std::mutex> lock(d->chunk_mu);
    if (st.b_first == nullptr) {
      if (no_alloc())
        return fail(SSCN_ERR_INVALID_ARG,
                    "the rule book's row-block plan is not built yet and this call may not allocate: run "
                    "sparse_conv_forward or sparse_conv_backward on it once first");
      int cur = 0;
      SSCN_HIP(hipGetDevice(&cur));
      if (cur != d->device) return fail(SSCN_ERR_INVALID_ARG, "rule book used on another device");
      const int64_t n_rows = &st == &d->fwd ? d->n_out : d->n_in;
      SSCN_TRY(build_plan(d, st, n_rows, d->K, d->stream));
    }
    return follow_rulebook_stream(d, d->plan_ready, s);
  }
}

static sscn_status check_common(const int32_t* coords, int64_t n, const int32_t* spatial_size,
                                int32_t f, sscn_rulebook* out) {
  if (!out) return fail(SSCN_ERR_INVALID_ARG, "out handle pointer is NULL");
  if (!spatial_size) return fail(SSCN_ERR_INVALID_ARG, "spatial_size is NULL");
  if (n < 0) return fail(SSCN_ERR_INVALID_ARG, "n < 0");
  if (n > 0 && !coords) return fail(SSCN_ERR_INVALID_ARG, "coords is NULL with n > 0");
  if (n > 0 && ((uintptr_t)coords & 15)) return fail(SSCN_ERR_INVALID_ARG, "coords must be 16-byte aligned");
  if (f < 1 || f > 8) return fail(SSCN_ERR_INVALID_ARG, "filter_size must be in [1, 8]");
  for (int d = 0; d < 3; ++d)
    if (spatial_size[d] < 1 || spatial_size[d] > kMaxExtent)
      return fail(SSCN_ERR_INVALID_ARG, "spatial_size entries must be in [1, 65536]");
  const int64_t K = (int64_t)f * f * f;
  if (n * K >= (int64_t)INT32_MAX) return fail(SSCN_ERR_INVALID_ARG, "n * f^3 must be below 2^31");
  return SSCN_OK;
}

static sscn_status flags_error(unsigned long long flags) {
  if (flags & kFlagOutOfRange)
    return fail(SSCN_ERR_OUT_OF_RANGE, "a coordinate lies outside the grid or the batch index outside [0, 32768)");
  if (flags & kFlagDuplicate) return fail(SSCN_ERR_DUPLICATE, "two rows share one location");
  return SSCN_OK;
}

static sscn_status new_handle(RulebookData* d, sscn_rulebook* out) {
  sscn_rulebook_s* h = new (std::nothrow) sscn_rulebook_s;
  if (!h) {
    delete d;
    return fail(SSCN_ERR_OOM, "host allocation failed");
  }
  h->d = d;
  h->transposed = false;
  *out = h;
  return SSCN_OK;
}

// SSC build with 8-byte dictionary slots (batch_lim > 0: batch indices
// below batch_lim keep the 32-bit keys below the empty marker) or 16-byte
// ones (batch_lim == 0).  Sets *wide and returns no rule book (its queued
// work is discarded) when a batch index reaches batch_lim.
static sscn_status ssc_build(const int32_t* coords, int64_t n, const int32_t* spatial_size, int32_t filter_size,
                             hipStream_t stream, uint32_t batch_lim, bool* wide, sscn_rulebook* out) {
  const int f = filter_size, K = f * f * f;
  const int L0 = spatial_size[0], L1 = spatial_size[1], L2 = spatial_size[2];
  const bool narrow = batch_lim > 0;
  hipStream_t s = stream;

  RulebookData* d = new (std::nothrow) RulebookData;
  if (!d) return fail(SSCN_ERR_OOM, "host allocation failed");
  std::unique_ptr<RulebookData> guard(d);
  (void)hipGetDevice(&d->device);
  d->stream = s;
  d->f = f; d->stride = 1; d->K = K; d->submanifold = true;
  d->n_in = d->n_out = n;
  for (int i = 0; i < 3; ++i) d->in_size[i] = d->out_size[i] = spatial_size[i];
  d->pairs_per_offset.assign(K, 0);
  const int64_t n_tiles = ceil_div(n, kTile);
  d->fwd.n_tiles = n_tiles;

  {
    Temps tmp(s);
    const uint64_t cap = table_capacity(n);
    Slot* table = nullptr; uint32_t* table8 = nullptr;  // table8: grouped slots of kGroupWords words
    int32_t* nbr; int64_t* counts; unsigned long long* stats; int32_t* hist = nullptr;
    // With K <= kPlanMaxK the row-block plan is queued before the readback too: its
    // launches overlap the build's kernels and the host waits once.
    const bool one_phase = (uint64_t)K * (uint64_t)n * 8u <= (512ull << 20);
    const bool eager_plan = one_phase && n > 0 && K <= kPlanMaxK && n < (int64_t)kPlanNoRow;
    Arena ta;
    if (narrow) ta.add(&table8, cap * kGroupWords); else ta.add(&table, cap);
    ta.add(&nbr, (size_t)K * n);
    ta.add(&counts, (size_t)K * n_tiles + 1);
    ta.add(&stats, 1 + K);
    if (eager_plan) ta.add(&hist, (size_t)plan_hist_words(K));  // right after stats: one fill clears both
    SSCN_TRY(tmp.alloc(ta));
    const int n_zero =
        (int)ceil_div(hist ? (char*)(hist + plan_hist_words(K)) - (char*)stats : (int64_t)(1 + K) * 8, 8);
    // Pair storage for the worst case (every offset of every site) when that
    // is modest (one_phase): then it shares one allocation with the rest of
    // the rule book, compaction is queued before the one readback, and the
    // host waits once.  Otherwise the exact size comes from the readback first.
    auto add_pairs = [&](Arena& pa, int64_t cap_pairs) {
      pa.add(&d->fwd.in_rows, cap_pairs);
      pa.add(&d->fwd.out_rows, cap_pairs);
      pa.add(&d->fwd.order, n_tiles);
      if (K <= kPlanMaxK) pa.add(&d->fwd.row_mask, (size_t)n * plan_words(K));
    };
    Arena oa;  // owned by the rule book, needed before the readback
    oa.add(&d->fwd.seg, (size_t)K * n_tiles + 1);
    oa.add(&d->out_coords, (size_t)4 * n);
    if (one_phase) add_pairs(oa, (int64_t)K * n);
    SSCN_TRY(owned_alloc(d, oa, s));

    if (narrow) {
      const uint64_t pieces = cap * kGroupWords / 4;  // 16-byte stores
      k_fill_slots8<<<(unsigned)std::min<uint64_t>((pieces + 255) / 256, 16384), 256, 0, s>>>(
          (uint4*)table8, pieces, stats, n_zero);
      SSCN_HIP(hipGetLastError());
    } else {
      SSCN_TRY(launch_fill_slots(table, cap, -1, s, stats, n_zero));
    }
    if (n > 0) {
      if (narrow) {
        k_insert8_store<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, L0, L1, L2, batch_lim, table8,
                                                        (uint32_t)(cap - 1), stats, (int4*)d->out_coords);
        SSCN_HIP(hipGetLastError());
        k_insert8_fix<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, L0, L1, L2, batch_lim, table8,
                                                      (uint32_t)(cap - 1));
      } else
        k_insert<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, L0, L1, L2, table, cap - 1, stats,
                                                 (int4*)d->out_coords);
      SSCN_HIP(hipGetLastError());
      constexpr int P = 3;  // lookups per wavefront
      // mirrored lookups halve the table reads; they cost two more launches,
      // which only pays off on larger inputs
      const bool mirror = n >= kMirrorProbeMin && K > 1;
      const int c = (K - 1) / 2;  // centre offset
      if (mirror) SSCN_TRY(fill_i32(nbr + (int64_t)(c + 1) * n, -1, (int64_t)(K - 1 - c) * n, s));
      const int64_t slices = std::max<int64_t>(ceil_div(mirror ? c : K, P), 1);
      const unsigned grid = (unsigned)(grid_for(n_tiles * 64, 256) * slices);
      if (narrow)
        k_ssc_probe<P, true><<<grid, 256, 0, s>>>((const int4*)coords, n, L0, L1, L2, f, table8, cap - 1, nbr,
                                                   counts, n_tiles, mirror ? 1 : 0, batch_lim, stats);
      else
        k_ssc_probe<P, false><<<grid, 256, 0, s>>>((const int4*)coords, n, L0, L1, L2, f, table, cap - 1, nbr,
                                                    counts, n_tiles, mirror ? 1 : 0, 0u, stats);
      SSCN_HIP(hipGetLastError());
      if (mirror) {
        k_count_nbr<<<grid_for(n_tiles * 64, 256), 256, 0, s>>>(nbr, n, K, counts, n_tiles, c);
        SSCN_HIP(hipGetLastError());
      }
    }
    if (K * n_tiles <= kOneBlockScanMax) {
      launch_seg_scan_one(counts, d->fwd.seg, K * n_tiles, std::max<int64_t>(n_tiles, 1), K, n > 0 ? stats : nullptr,
                          s);
      SSCN_HIP(hipGetLastError());
    } else {
      SSCN_TRY(exclusive_scan_i64(counts, d->fwd.seg, K * n_tiles, s));
      if (n > 0) {
        k_offset_totals<<<grid_for(K, 256), 256, 0, s>>>(d->fwd.seg, n_tiles, K, stats);
        SSCN_HIP(hipGetLastError());
      }
    }
    const size_t stat_bytes = sizeof(unsigned long long) * (1 + K);
    // Before the readback, the compaction's first workgroup copies the sizes
    // and flags to the pinned staging buffer itself (no copy launch).
    void* staging = nullptr;
    const bool direct = one_phase && n > 0;
    if (direct) SSCN_TRY(readback_staging(stat_bytes, &staging));
    auto compact = [&](bool to_host) -> sscn_status {
      if (n > 0)
        SSCN_TRY(compact_storage(nbr, n, K, d->fwd, s, /*counted=*/true, d->fwd.row_mask, stats,
                                 to_host ? (unsigned long long*)staging : nullptr, 1 + K));
      return SSCN_OK;
    };
    if (one_phase) SSCN_TRY(compact(direct));
    // The sizes and flags are final here.  The plan is queued behind their
    // readback: the host waits for that alone, and the plan's kernels run
    // while it returns (a use of the plan on another stream waits for the
    // rule book's stream).
    SSCN_TRY(readback_begin(direct ? nullptr : stats, stat_bytes, s));
    if (eager_plan) SSCN_TRY(build_plan(d, d->fwd, n, K, s, /*a site has one neighbour per offset*/ n, hist));
    std::vector<unsigned long long> host(1 + K);
    SSCN_TRY(readback_end(host.data(), stat_bytes));
    if (!(host[0] & kFlagOutOfRange) && (host[0] & kFlagWideKey)) {
      *wide = true;  // the queued work is discarded with d and the temporaries
      return SSCN_OK;
    }
    SSCN_TRY(flags_error(host[0]));
    int64_t total = 0;
    for (int o = 0; o < K; ++o) total += (d->pairs_per_offset[o] = (int64_t)host[1 + o]);
    d->n_pairs = total;
    if (!one_phase) {
      Arena pa;
      add_pairs(pa, total);
      SSCN_TRY(owned_alloc(d, pa, s));
      SSCN_TRY(compact(false));
    }
  }
  guard.release();
  return new_handle(d, out);
}

}  // namespace sscn

using namespace sscn;

extern "C" sscn_status ssc_rulebook_build(const int32_t* coords, int64_t n, const int32_t* spatial_size,
                                          int32_t filter_size, hipStream_t stream, sscn_rulebook* out) {
  SSCN_TRY(check_common(coords, n, spatial_size, filter_size, out));
  if (filter_size % 2 == 0) return fail(SSCN_ERR_INVALID_ARG, "SSC needs an odd filter_size");
  // 32-bit keys while one sample's keys stay below the empty marker 2^32 - 1
  const uint64_t vol = (uint64_t)spatial_size[0] * (uint64_t)spatial_size[1] * (uint64_t)spatial_size[2];
  const uint64_t lim = 0xFFFFFFFFull / vol;
  bool wide = false;
  if (lim > 0) {
    SSCN_TRY(ssc_build(coords, n, spatial_size, filter_size, stream, (uint32_t)std::min<uint64_t>(lim, kMaxBatch),
                       &wide, out));
    if (!wide) return SSCN_OK;
  }
  return ssc_build(coords, n, spatial_size, filter_size, stream, 0, &wide, out);
}

extern "C" sscn_status sc_rulebook_build(const int32_t* coords, int64_t n, const int32_t* spatial_size,
                                         int32_t filter_size, int32_t stride, hipStream_t stream,
                                         sscn_rulebook* out) {
  SSCN_TRY(check_common(coords, n, spatial_size, filter_size, out));
  if (stride < 1 || stride > 8) return fail(SSCN_ERR_INVALID_ARG, "stride must be in [1, 8]");
  const int f = filter_size, s_ = stride, K = f * f * f;
  ScGeom g;
  g.f = f; g.s = s_; g.K = K;
  g.L0 = spatial_size[0]; g.L1 = spatial_size[1]; g.L2 = spatial_size[2];
  int M[3];
  for (int dd = 0; dd < 3; ++dd) {
    const int L = spatial_size[dd];
    if (L < f || (L - f) % s_ != 0)
      return fail(SSCN_ERR_SHAPE, "SC needs L >= f and (L - f) divisible by the stride in every dimension");
    M[dd] = (L - f + s_) / s_;
  }
  g.M0 = M[0]; g.M1 = M[1]; g.M2 = M[2];
  hipStream_t s = stream;

  RulebookData* d = new (std::nothrow) RulebookData;
  if (!d) return fail(SSCN_ERR_OOM, "host allocation failed");
  std::unique_ptr<RulebookData> guard(d);
  (void)hipGetDevice(&d->device);
  d->stream = s;
  d->f = f; d->stride = s_; d->K = K; d->submanifold = false;
  d->n_in = n;
  for (int i = 0; i < 3; ++i) { d->in_size[i] = spatial_size[i]; d->out_size[i] = M[i]; }
  d->pairs_per_offset.assign(K, 0);

  {
    Temps tmp(s);
    // outputs seen per input: prod over d of ceil(f / s) (at most K)
    const int per_dim = (f + s_ - 1) / s_;
    const int64_t max_out = n * (int64_t)per_dim * per_dim * per_dim;
    const uint64_t cap = table_capacity(n), ocap = table_capacity(max_out);
    Slot* table = nullptr; Slot* otable; unsigned long long* stats; int32_t* first; int32_t* rank;
    // Repeated locations and range errors: found while visiting the outputs
    // where every input has one (K <= 32, f >= s), else by an input
    // dictionary.
    const bool visit_checks = K <= 32 && f >= s_;
    Arena ta;
    if (!visit_checks) ta.add(&table, cap);
    ta.add(&otable, ocap);
    ta.add(&stats, 3 + K);  // flags, pairs per offset, n_out, rows out of order
    // every input sees at most one output (f <= s): the visits are grouped
    // per output inside each wavefront first, and first / rank hold one
    // entry per input
    const bool one_target = per_dim == 1 && K <= 32;
    ta.add(&first, (size_t)n * (one_target ? 1 : K));
    ta.add(&rank, (size_t)n * (one_target ? 1 : K) + 1);
    uint32_t* mark_part = nullptr;  // one_target: pair counts per (offset, workgroup of k_sc_mark1)
    if (one_target) ta.add(&mark_part, (size_t)K * grid_for(std::max<int64_t>(n, 1), 256));
    SSCN_TRY(tmp.alloc(ta));
    Arena ia;
    ia.add(&d->in_coords, (size_t)4 * n);
    SSCN_TRY(owned_alloc(d, ia, s));

    int* unsorted = (int*)(stats + 2 + K);
    if (visit_checks) {
      SSCN_TRY(launch_fill_slots(otable, ocap, INT32_MAX, s, stats, 3 + K));
      if (n > 0 && one_target) {
        k_sc_order<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, unsorted);
        SSCN_HIP(hipGetLastError());
        k_sc_visit1<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, g, otable, ocap - 1, 1, stats,
                                                     (int4*)d->in_coords, unsorted);
        SSCN_HIP(hipGetLastError());
      } else if (n > 0) {
        k_sc_visit<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, g, otable, ocap - 1, 1, stats,
                                                    (int4*)d->in_coords);
        SSCN_HIP(hipGetLastError());
      }
    } else {
      SSCN_TRY(launch_fill_slots(table, cap, -1, s, stats, 3 + K));
      if (n > 0) {
        SSCN_TRY(launch_fill_slots(otable, ocap, INT32_MAX, s));
        k_insert<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, g.L0, g.L1, g.L2, table, cap - 1, stats,
                                                 (int4*)d->in_coords);
        SSCN_HIP(hipGetLastError());
        if (one_target)
          k_sc_visit1<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, g, otable, ocap - 1, 0, stats,
                                                       nullptr, unsorted);
        else
          k_sc_visit<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, g, otable, ocap - 1, 0, stats,
                                                      nullptr);
        SSCN_HIP(hipGetLastError());
      }
    }
    if (n > 0) {
      if (one_target) {
        const unsigned nb = grid_for(n, 256);
        k_sc_mark1<<<nb, 256, 0, s>>>((const int4*)coords, n, g, otable, ocap - 1, first, mark_part);
        SSCN_HIP(hipGetLastError());
        k_offset_sums<<<K, kOneBlock, 0, s>>>(mark_part, nb, stats + 1);
      } else
        k_sc_mark<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, g, otable, ocap - 1, first, stats + 1);
      SSCN_HIP(hipGetLastError());
      const int64_t n_visits = one_target ? n : n * K;  // entries of first / rank
      SSCN_TRY(exclusive_scan_i32(first, rank, n_visits, s));
      // n_out = rank[n_visits] joins the readback
      SSCN_HIP(hipMemcpyAsync(stats + 1 + K, rank + (size_t)n_visits, sizeof(int32_t), hipMemcpyDeviceToDevice, s));

    }
    std::vector<unsigned long long> host(2 + K);
    SSCN_TRY(readback(host.data(), stats, sizeof(unsigned long long) * (2 + K), s));
    SSCN_TRY(flags_error(host[0]));
    int64_t total = 0;
    for (int o = 0; o < K; ++o) total += (d->pairs_per_offset[o] = (int64_t)host[1 + o]);
    d->n_pairs = total;
    const int64_t n_out = (int64_t)(uint32_t)(host[1 + K] & 0xffffffffull);
    d->n_out = n_out;
    d->fwd.n_tiles = ceil_div(n_out, kTile);
    d->bwd.n_tiles = ceil_div(n, kTile);

    Arena oa;
    oa.add(&d->out_coords, (size_t)4 * n_out);
    oa.add(&d->fwd.seg, (size_t)K * d->fwd.n_tiles + 1);
    oa.add(&d->bwd.seg, (size_t)K * d->bwd.n_tiles + 1);
    oa.add(&d->fwd.in_rows, total);
    oa.add(&d->fwd.out_rows, total);
    oa.add(&d->bwd.in_rows, total);
    oa.add(&d->bwd.out_rows, total);
    oa.add(&d->fwd.order, d->fwd.n_tiles);
    oa.add(&d->bwd.order, d->bwd.n_tiles);
    if (K <= kPlanMaxK && n > 0) {
      oa.add(&d->fwd.row_mask, (size_t)n_out * plan_words(K));
      oa.add(&d->bwd.row_mask, (size_t)n * plan_words(K));
    }
    SSCN_TRY(owned_alloc(d, oa, s));
    if (n > 0 && one_target) {
      int32_t* nbr_out; int2* tgt;
      Arena na;
      na.add(&nbr_out, (size_t)K * n_out);
      na.add(&tgt, (size_t)n);
      SSCN_TRY(tmp.alloc(na));
      SSCN_TRY(fill_i32(nbr_out, -1, (int64_t)K * n_out, s));
      k_sc_assign1<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, g, otable, ocap - 1, rank, n_out,
                                                    nbr_out, tgt, d->bwd.seg, d->bwd.n_tiles,
                                                    (int4*)d->out_coords);
      SSCN_HIP(hipGetLastError());
      SSCN_TRY(compact_storage(nbr_out, n_out, K, d->fwd, s, false, d->fwd.row_mask));
      SSCN_TRY(scan_seg(d->bwd, K, s));
      k_compact1<<<grid_for(n, 256), 256, 0, s>>>(tgt, n, K, d->bwd.seg, d->bwd.n_tiles, d->bwd.in_rows,
                                                  d->bwd.out_rows, d->bwd.row_mask);
      SSCN_HIP(hipGetLastError());
    } else if (n > 0) {
      int32_t* nbr_out; int32_t* nbr_in;
      Arena na;
      na.add(&nbr_out, (size_t)K * n_out);
      na.add(&nbr_in, (size_t)K * n);
      SSCN_TRY(tmp.alloc(na));
      SSCN_TRY(fill_i32(nbr_out, -1, (int64_t)K * n_out, s));
      SSCN_TRY(fill_i32(nbr_in, -1, (int64_t)K * n, s));
      k_sc_assign<<<grid_for(n, 256), 256, 0, s>>>((const int4*)coords, n, g, otable, ocap - 1, rank, n_out,
                                                   nbr_out, nbr_in, (int4*)d->out_coords);
      SSCN_HIP(hipGetLastError());
      SSCN_TRY(compact_storage(nbr_out, n_out, K, d->fwd, s, false, d->fwd.row_mask));
      SSCN_TRY(compact_storage(nbr_in, n, K, d->bwd, s, false, d->bwd.row_mask));
    } else {
      SSCN_TRY(exclusive_scan_i64(d->fwd.seg, d->fwd.seg, 0, s));
      SSCN_TRY(exclusive_scan_i64(d->bwd.seg, d->bwd.seg, 0, s));
    }
  }
  guard.release();
  return new_handle(d, out);
}

extern "C" sscn_status sscn_rulebook_transpose(sscn_rulebook rb, sscn_rulebook* out) {
  if (!rb || !out) return fail(SSCN_ERR_INVALID_ARG, "NULL rule book or out pointer");
  sscn_rulebook_s* h = new (std::nothrow) sscn_rulebook_s;
  if (!h) return fail(SSCN_ERR_OOM, "host allocation failed");
  rb->d->refs.fetch_add(1);
  h->d = rb->d;
  h->transposed = !rb->transposed;
  *out = h;
  return SSCN_OK;
}

extern "C" sscn_status sscn_rulebook_query(sscn_rulebook rb, sscn_rulebook_info* info, int64_t* ppo) {
  if (!rb || !info) return fail(SSCN_ERR_INVALID_ARG, "NULL rule book or info pointer");
  const RulebookData* d = rb->d;
  const bool t = rb->transposed;
  info->n_in = t ? d->n_out : d->n_in;
  info->n_out = t ? d->n_in : d->n_out;
  info->n_pairs = d->n_pairs;
  info->filter_size = d->f;
  info->stride = d->stride;
  info->submanifold = d->submanifold ? 1 : 0;
  info->transposed = t ? 1 : 0;
  info->n_offsets = d->K;
  info->dim = d->dim;
  for (int i = 0; i < kMaxDim; ++i) {
    info->in_size[i] = t ? d->out_size[i] : d->in_size[i];
    info->out_size[i] = t ? d->in_size[i] : d->out_size[i];
  }
  if (ppo) {
    for (int o = 0; o < d->K; ++o) {
      // a transposed SSC view holds R_{K-1-o} under offset o (same sizes by symmetry)
      const int so = (t && d->submanifold) ? d->K - 1 - o : o;
      ppo[o] = d->pairs_per_offset[so];
    }
  }
  return SSCN_OK;
}

extern "C" sscn_status sscn_rulebook_out_coords(sscn_rulebook rb, int32_t* out_coords, hipStream_t s) {
  if (!rb) return fail(SSCN_ERR_INVALID_ARG, "NULL rule book");
  const RulebookData* d = rb->d;
  const int64_t n_out = rb->transposed ? d->n_in : d->n_out;
  if (n_out == 0) return SSCN_OK;
  if (!out_coords) return fail(SSCN_ERR_INVALID_ARG, "out_coords is NULL");
  // a transposed SC view outputs at the SC's input sites
  const int32_t* src = (rb->transposed && !d->submanifold) ? d->in_coords : d->out_coords;
  UseNote note{rb->d, s};
  SSCN_HIP(hipMemcpyAsync(out_coords, src, sizeof(int32_t) * (d->dim + 1) * n_out, hipMemcpyDeviceToDevice, s));
  return SSCN_OK;
}

extern "C" sscn_status sscn_rulebook_export(sscn_rulebook rb, int32_t* in_rows, int32_t* out_rows,
                                            int32_t* offsets, hipStream_t s) {
  if (!rb) return fail(SSCN_ERR_INVALID_ARG, "NULL rule book");
  const RulebookData* d = rb->d;
  if (d->n_pairs == 0) return SSCN_OK;
  if (!in_rows || !out_rows || !offsets) return fail(SSCN_ERR_INVALID_ARG, "NULL export array");
  const View v = view_of(rb);
  UseNote note{rb->d, s};
  // stored segment boundaries per offset: seg[o * n_tiles], read on the host
  std::vector<int64_t> start(d->K + 1);
  int64_t acc = 0;
  for (int o = 0; o < d->K; ++o) { start[o] = acc; acc += d->pairs_per_offset[o]; }
  start[d->K] = acc;
  int64_t pos = 0;
  for (int o = 0; o < d->K; ++o) {
    const int so = v.mirror ? d->K - 1 - o : o;
    const int64_t cnt = d->pairs_per_offset[so];
    if (!cnt) continue;
    SSCN_HIP(hipMemcpyAsync(in_rows + pos, v.st->in_rows + start[so], sizeof(int32_t) * cnt,
                            hipMemcpyDeviceToDevice, s));
    SSCN_HIP(hipMemcpyAsync(out_rows + pos, v.st->out_rows + start[so], sizeof(int32_t) * cnt,
                            hipMemcpyDeviceToDevice, s));
    SSCN_TRY(fill_i32(offsets + pos, o, cnt, s));
    pos += cnt;
  }
  return SSCN_OK;
}

extern "C" void sscn_rulebook_free(sscn_rulebook rb) {
  if (!rb) return;
  if (rb->d->refs.fetch_sub(1) == 1) delete rb->d;
  delete rb;
}

// ========================================================== any dimension
// Rule books of d-dimensional layers for d = 1, 2, 4 (d = 3 takes the tuned
// builders above).  The method is the same in every dimension (Sec. 3
// defines the layers on d-dimensional grids; Sec. 1: 4-D data such as RGB-D
// video): sites are rows (b, x_0, .., x_{d-1}) of an n x (d + 1) int32
// array, F = {0..f-1}^d is enumerated with the first coordinate most
// significant, keys are the linear index ((b L_0 + x_0) L_1 + ..) in 64
// bits.  The dictionary is the 16-byte-slot table, the SSC probe looks up
// every (offset, site) pair (one lane each, offset-major so that a
// wavefront reads consecutive sites), and the SC outputs are numbered by
// first visit exactly as in three dimensions; both directions are then
// compacted into the same storage as the 3-D builders produce, so the
// convolution, pooling and export calls are unchanged.
namespace sscn {
namespace {

template <int DD>
struct GeomN {
  int32_t L[DD];  // input extents
  int32_t M[DD];  // output extents (SC)
  int f, s, K;
};

// Reads site j; false if it lies outside the grid (or the batch range).
template <int DD>
__device__ __forceinline__ bool site_n(const int32_t* __restrict__ coords, int64_t j, const GeomN<DD>& g, int& b,
                                       int (&x)[DD]) {
  const int32_t* r = coords + j * (DD + 1);
  b = r[0];
  bool ok = (unsigned)b < (unsigned)kMaxBatch;
#pragma unroll
  for (int q = 0; q < DD; ++q) {
    x[q] = r[1 + q];
    ok = ok && (unsigned)x[q] < (unsigned)g.L[q];
  }
  return ok;
}

template <int DD>
__device__ __forceinline__ uint64_t key_n(int b, const int (&x)[DD], const int32_t (&ext)[DD]) {
  uint64_t k = (uint64_t)(uint32_t)b;
#pragma unroll
  for (int q = 0; q < DD; ++q) k = k * (uint64_t)(uint32_t)ext[q] + (uint64_t)(uint32_t)x[q];
  return k;
}

// Offset o -> its filter position (first coordinate most significant).
template <int DD>
__device__ __forceinline__ void digits_n(int o, int f, int (&i)[DD]) {
#pragma unroll
  for (int q = DD - 1; q >= 0; --q) {
    i[q] = o % f;
    o /= f;
  }
}

template <int DD>
__global__ __launch_bounds__(256) void k_insert_n(const int32_t* __restrict__ coords, int64_t n, GeomN<DD> g,
                                                  Slot* __restrict__ table, uint64_t mask,
                                                  unsigned long long* __restrict__ flags, int32_t* __restrict__ copy) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  if (copy)
    for (int q = 0; q <= DD; ++q) copy[j * (DD + 1) + q] = coords[j * (DD + 1) + q];
  int b, x[DD];
  if (!site_n<DD>(coords, j, g, b, x)) {
    atomicOr(flags, (unsigned long long)kFlagOutOfRange);
    return;
  }
  const uint64_t key = key_n<DD>(b, x, g.L);
  uint64_t slot = mix64(key) & mask;
  while (true) {
    const unsigned long long prev = atomicCAS((unsigned long long*)&table[slot].key, (unsigned long long)kEmptyKey,
                                              (unsigned long long)key);
    if (prev == kEmptyKey) {
      table[slot].row = (int32_t)j;
      return;
    }
    if (prev == key) {
      atomicOr(flags, (unsigned long long)kFlagDuplicate);
      return;
    }
    slot = (slot + 1) & mask;
  }
}

// nbr[o n + k] = row of the site at x_k + i_o - (f-1)/2, or -1 (sites
// outside the grid were flagged by the insert; the build then fails).
template <int DD>
__global__ __launch_bounds__(256) void k_probe_n(const int32_t* __restrict__ coords, int64_t n, GeomN<DD> g,
                                                 const Slot* __restrict__ table, uint64_t mask,
                                                 int32_t* __restrict__ nbr) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n * g.K) return;
  const int o = (int)(idx / n);
  const int64_t k = idx - (int64_t)o * n;
  int b, x[DD], i[DD];
  int32_t j = -1;
  if (site_n<DD>(coords, k, g, b, x)) {
    digits_n<DD>(o, g.f, i);
    const int c = (g.f - 1) / 2;
    bool in = true;
#pragma unroll
    for (int q = 0; q < DD; ++q) {
      x[q] += i[q] - c;
      in = in && (unsigned)x[q] < (unsigned)g.L[q];
    }
    if (in) j = table_lookup(table, mask, key_n<DD>(b, x, g.L));
  }
  nbr[idx] = j;
}

// Output location that input x reaches through offset o, if any.
template <int DD>
__device__ __forceinline__ bool sc_target_n(const GeomN<DD>& g, const int (&x)[DD], int o, int (&y)[DD]) {
  int i[DD];
  digits_n<DD>(o, g.f, i);
  bool ok = true;
#pragma unroll
  for (int q = 0; q < DD; ++q) {
    const int t = x[q] - i[q];
    ok = ok && t >= 0 && t % g.s == 0;
    y[q] = t / g.s;
    ok = ok && y[q] < g.M[q];
  }
  return ok;
}

template <int DD>
__global__ __launch_bounds__(256) void k_sc_visit_n(const int32_t* __restrict__ coords, int64_t n, GeomN<DD> g,
                                                    Slot* __restrict__ otable, uint64_t omask) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  int b, x[DD];
  if (!site_n<DD>(coords, j, g, b, x)) return;
  for (int o = 0; o < g.K; ++o) {
    int y[DD];
    if (!sc_target_n<DD>(g, x, o, y)) continue;
    const uint64_t key = key_n<DD>(b, y, g.M);
    uint64_t slot = mix64(key) & omask;
    while (true) {
      const unsigned long long prev = atomicCAS((unsigned long long*)&otable[slot].key,
                                                (unsigned long long)kEmptyKey, (unsigned long long)key);
      if (prev == kEmptyKey || prev == key) break;
      slot = (slot + 1) & omask;
    }
    atomicMin(&otable[slot].row, (int32_t)(j * g.K + o));
  }
}

// first[j K + o] = 1 iff visit (j, o) is the first of its output;
// per_offset[o] += visits through o.
template <int DD>
__global__ __launch_bounds__(256) void k_sc_mark_n(const int32_t* __restrict__ coords, int64_t n, GeomN<DD> g,
                                                   const Slot* __restrict__ otable, uint64_t omask,
                                                   int32_t* __restrict__ first,
                                                   unsigned long long* __restrict__ per_offset) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n * g.K) return;
  const int64_t j = idx / g.K;
  const int o = (int)(idx - j * g.K);
  int b, x[DD], y[DD];
  int32_t is_first = 0;
  if (site_n<DD>(coords, j, g, b, x) && sc_target_n<DD>(g, x, o, y)) {
    is_first = table_lookup(otable, omask, key_n<DD>(b, y, g.M)) == (int32_t)idx;
    atomicAdd(&per_offset[o], 1ull);
  }
  first[idx] = is_first;
}

template <int DD>
__global__ __launch_bounds__(256) void k_sc_assign_n(const int32_t* __restrict__ coords, int64_t n, GeomN<DD> g,
                                                     const Slot* __restrict__ otable, uint64_t omask,
                                                     const int32_t* __restrict__ rank, int64_t n_out,
                                                     int32_t* __restrict__ nbr_out, int32_t* __restrict__ nbr_in,
                                                     int32_t* __restrict__ out_coords) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n * g.K) return;
  const int64_t j = idx / g.K;
  const int o = (int)(idx - j * g.K);
  int b, x[DD], y[DD];
  if (!site_n<DD>(coords, j, g, b, x) || !sc_target_n<DD>(g, x, o, y)) return;
  const int32_t vmin = table_lookup(otable, omask, key_n<DD>(b, y, g.M));
  const int32_t k = rank[vmin];
  nbr_out[(int64_t)o * n_out + k] = (int32_t)j;
  nbr_in[(int64_t)o * n + j] = k;
  if (vmin == (int32_t)idx) {
    out_coords[(int64_t)k * (DD + 1)] = b;
#pragma unroll
    for (int q = 0; q < DD; ++q) out_coords[(int64_t)k * (DD + 1) + 1 + q] = y[q];
  }
}

template <int DD>
sscn_status build_nd(const int32_t* coords, int64_t n, const int32_t* size, int f, int stride, bool sub,
                     hipStream_t s, sscn_rulebook* out) {
  int K = 1;
  for (int q = 0; q < DD; ++q) K *= f;
  GeomN<DD> g;
  g.f = f; g.s = stride; g.K = K;
  for (int q = 0; q < DD; ++q) {
    g.L[q] = size[q];
    if (sub) {
      g.M[q] = size[q];
    } else {
      if (size[q] < f || (size[q] - f) % stride != 0)
        return fail(SSCN_ERR_SHAPE, "SC needs L >= f and (L - f) divisible by the stride in every dimension");
      g.M[q] = (size[q] - f + stride) / stride;
    }
  }
  RulebookData* d = new (std::nothrow) RulebookData;
  if (!d) return fail(SSCN_ERR_OOM, "host allocation failed");
  std::unique_ptr<RulebookData> guard(d);
  (void)hipGetDevice(&d->device);
  d->stream = s;
  d->dim = DD;
  d->f = f; d->stride = sub ? 1 : stride; d->K = K; d->submanifold = sub;
  d->n_in = n;
  for (int q = 0; q < DD; ++q) { d->in_size[q] = g.L[q]; d->out_size[q] = g.M[q]; }
  d->pairs_per_offset.assign(K, 0);
  {
    Temps tmp(s);
    const uint64_t cap = table_capacity(n);
    Slot* table; unsigned long long* stats;
    Arena ta;
    ta.add(&table, cap);
    ta.add(&stats, 2 + K);
    SSCN_TRY(tmp.alloc(ta));
    SSCN_TRY(launch_fill_slots(table, cap, -1, s, stats, 2 + K));
    if (sub) {
      d->n_out = n;
      d->fwd.n_tiles = ceil_div(n, kTile);
      int32_t* nbr;
      Arena na;
      na.add(&nbr, (size_t)K * n);
      SSCN_TRY(tmp.alloc(na));
      Arena oa;
      oa.add(&d->out_coords, (size_t)(DD + 1) * n);
      oa.add(&d->fwd.seg, (size_t)K * d->fwd.n_tiles + 1);
      SSCN_TRY(owned_alloc(d, oa, s));
      if (n > 0) {
        k_insert_n<DD><<<grid_for(n, 256), 256, 0, s>>>(coords, n, g, table, cap - 1, stats, d->out_coords);
        SSCN_HIP(hipGetLastError());
        k_probe_n<DD><<<grid_for(n * K, 256), 256, 0, s>>>(coords, n, g, table, cap - 1, nbr);
        SSCN_HIP(hipGetLastError());
        k_count_nbr<<<grid_for(d->fwd.n_tiles * 64, 256), 256, 0, s>>>(nbr, n, K, d->fwd.seg, d->fwd.n_tiles);
        SSCN_HIP(hipGetLastError());
      }
      SSCN_TRY(exclusive_scan_i64(d->fwd.seg, d->fwd.seg, K * d->fwd.n_tiles, s));
      if (n > 0) {
        k_offset_totals<<<grid_for(K, 256), 256, 0, s>>>(d->fwd.seg, d->fwd.n_tiles, K, stats);
        SSCN_HIP(hipGetLastError());
      }
      std::vector<unsigned long long> host(2 + K);
      SSCN_TRY(readback(host.data(), stats, sizeof(unsigned long long) * (2 + K), s));
      SSCN_TRY(flags_error(host[0]));
      int64_t total = 0;
      for (int o = 0; o < K; ++o) total += (d->pairs_per_offset[o] = (int64_t)host[1 + o]);
      d->n_pairs = total;
      Arena pa;
      pa.add(&d->fwd.in_rows, total);
      pa.add(&d->fwd.out_rows, total);
      pa.add(&d->fwd.order, d->fwd.n_tiles);
      if (K <= kPlanMaxK && n > 0) pa.add(&d->fwd.row_mask, (size_t)n * plan_words(K));
      SSCN_TRY(owned_alloc(d, pa, s));
      if (n > 0) SSCN_TRY(compact_storage(nbr, n, K, d->fwd, s, /*counted=*/true, d->fwd.row_mask));
    } else {
      // every input reaches at most prod_q ceil(f / s) outputs
      const int per = (f + stride - 1) / stride;
      int64_t max_out = n;
      for (int q = 0; q < DD; ++q) max_out *= per;
      const uint64_t ocap = table_capacity(max_out);
      Slot* otable; int32_t* first; int32_t* rank;
      Arena sa;
      sa.add(&otable, ocap);
      sa.add(&first, (size_t)n * K);
      sa.add(&rank, (size_t)n * K + 1);
      SSCN_TRY(tmp.alloc(sa));
      Arena ia;
      ia.add(&d->in_coords, (size_t)(DD + 1) * n);
      SSCN_TRY(owned_alloc(d, ia, s));
      if (n > 0) {
        SSCN_TRY(launch_fill_slots(otable, ocap, INT32_MAX, s));
        k_insert_n<DD><<<grid_for(n, 256), 256, 0, s>>>(coords, n, g, table, cap - 1, stats, d->in_coords);
        SSCN_HIP(hipGetLastError());
        k_sc_visit_n<DD><<<grid_for(n, 256), 256, 0, s>>>(coords, n, g, otable, ocap - 1);
        SSCN_HIP(hipGetLastError());
        k_sc_mark_n<DD><<<grid_for(n * K, 256), 256, 0, s>>>(coords, n, g, otable, ocap - 1, first, stats + 1);
        SSCN_HIP(hipGetLastError());
        SSCN_TRY(exclusive_scan_i32(first, rank, n * K, s));
        SSCN_HIP(hipMemcpyAsync(stats + 1 + K, rank + (size_t)n * K, sizeof(int32_t), hipMemcpyDeviceToDevice, s));
      }
      std::vector<unsigned long long> host(2 + K);
      SSCN_TRY(readback(host.data(), stats, sizeof(unsigned long long) * (2 + K), s));
      SSCN_TRY(flags_error(host[0]));
      int64_t total = 0;
      for (int o = 0; o < K; ++o) total += (d->pairs_per_offset[o] = (int64_t)host[1 + o]);
      d->n_pairs = total;
      const int64_t n_out = n > 0 ? (int64_t)(uint32_t)(host[1 + K] & 0xffffffffull) : 0;
      d->n_out = n_out;
      d->fwd.n_tiles = ceil_div(n_out, kTile);
      d->bwd.n_tiles = ceil_div(n, kTile);
      Arena oa;
      oa.add(&d->out_coords, (size_t)(DD + 1) * n_out);
      oa.add(&d->fwd.seg, (size_t)K * d->fwd.n_tiles + 1);
      oa.add(&d->bwd.seg, (size_t)K * d->bwd.n_tiles + 1);
      oa.add(&d->fwd.in_rows, total);
      oa.add(&d->fwd.out_rows, total);
      oa.add(&d->bwd.in_rows, total);
      oa.add(&d->bwd.out_rows, total);
      oa.add(&d->fwd.order, d->fwd.n_tiles);
      oa.add(&d->bwd.order, d->bwd.n_tiles);
      SSCN_TRY(owned_alloc(d, oa, s));
      if (n > 0) {
        int32_t* nbr_out; int32_t* nbr_in;
        Arena na;
        na.add(&nbr_out, (size_t)K * n_out);
        na.add(&nbr_in, (size_t)K * n);
        SSCN_TRY(tmp.alloc(na));
        SSCN_TRY(fill_i32(nbr_out, -1, (int64_t)K * n_out, s));
        SSCN_TRY(fill_i32(nbr_in, -1, (int64_t)K * n, s));
        k_sc_assign_n<DD><<<grid_for(n * K, 256), 256, 0, s>>>(coords, n, g, otable, ocap - 1, rank, n_out, nbr_out,
                                                               nbr_in, d->out_coords);
        SSCN_HIP(hipGetLastError());
        SSCN_TRY(compact_storage(nbr_out, n_out, K, d->fwd, s, false));
        SSCN_TRY(compact_storage(nbr_in, n, K, d->bwd, s, false));
      } else {
        SSCN_TRY(exclusive_scan_i64(d->fwd.seg, d->fwd.seg, 0, s));
        SSCN_TRY(exclusive_scan_i64(d->bwd.seg, d->bwd.seg, 0, s));
      }
    }
  }
  guard.release();
  return new_handle(d, out);
}

}  // namespace
}  // namespace sscn

extern "C" sscn_status sscn_rulebook_build_nd(const int32_t* coords, int64_t n, int32_t dim,
                                              const int32_t* spatial_size, int32_t filter_size, int32_t stride,
                                              int32_t submanifold, hipStream_t stream, sscn_rulebook* out) {
  if (!out) return fail(SSCN_ERR_INVALID_ARG, "out handle pointer is NULL");
  if (dim < 1 || dim > kMaxDim) return fail(SSCN_ERR_INVALID_ARG, "dim must be in [1, 4]");
  if (!spatial_size) return fail(SSCN_ERR_INVALID_ARG, "spatial_size is NULL");
  if (submanifold && filter_size % 2 == 0) return fail(SSCN_ERR_INVALID_ARG, "SSC needs an odd filter_size");
  if (submanifold && stride != 1) return fail(SSCN_ERR_INVALID_ARG, "SSC has stride 1");
  if (dim == 3) {
    return submanifold ? ssc_rulebook_build(coords, n, spatial_size, filter_size, stream, out)
                       : sc_rulebook_build(coords, n, spatial_size, filter_size, stride, stream, out);
  }
  if (n < 0) return fail(SSCN_ERR_INVALID_ARG, "n < 0");
  if (n > 0 && !coords) return fail(SSCN_ERR_INVALID_ARG, "coords is NULL with n > 0");
  if (n > 0 && ((uintptr_t)coords & 3)) return fail(SSCN_ERR_INVALID_ARG, "coords must be 4-byte aligned");
  if (filter_size < 1 || filter_size > 8) return fail(SSCN_ERR_INVALID_ARG, "filter_size must be in [1, 8]");
  if (stride < 1 || stride > 8) return fail(SSCN_ERR_INVALID_ARG, "stride must be in [1, 8]");
  // keys: kMaxBatch * prod L must stay below 2^63 (and differ from the empty marker)
  long double vol = (long double)kMaxBatch;
  int64_t K = 1;
  for (int q = 0; q < dim; ++q) {
    if (spatial_size[q] < 1 || spatial_size[q] > kMaxExtent)
      return fail(SSCN_ERR_INVALID_ARG, "spatial_size entries must be in [1, 65536]");
    vol *= (long double)spatial_size[q];
    K *= filter_size;
  }
  if (vol >= 9.2e18L) return fail(SSCN_ERR_INVALID_ARG, "32768 * prod(spatial_size) must stay below 2^63");
  if (K > 512) return fail(SSCN_ERR_INVALID_ARG, "filter_size^dim must be at most 512");
  if (n * K >= (int64_t)INT32_MAX) return fail(SSCN_ERR_INVALID_ARG, "n * filter_size^dim must be below 2^31");
  const bool sub = submanifold != 0;
  switch (dim) {
    case 1: return build_nd<1>(coords, n, spatial_size, filter_size, stride, sub, stream, out);
    case 2: return build_nd<2>(coords, n, spatial_size, filter_size, stride, sub, stream, out);
    default: return build_nd<4>(coords, n, spatial_size, filter_size, stride, sub, stream, out);
  }
}
