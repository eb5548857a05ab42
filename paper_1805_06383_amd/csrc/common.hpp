// Shared device/host definitions of the fstc library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <stdexcept>
#include <string>

#include "fstc.h"

namespace fstc {

using u16 = uint16_t;
using u32 = uint32_t;
using u64 = uint64_t;

constexpr int kWave = 64;

// Device-side error bits, OR-ed into a status word and checked by the host.
enum : u32 {
  kErrBadArc = 1u,      // an input arc's state or label out of range
  kErrHashFull = 2u,    // visited table probe wrapped around (never expected)
  kErrBounds = 4u,      // an internal index check failed
  kErrNewList = 8u,     // more new states than the new-state list holds
  kErrTileSize = 16u,   // a merge tile exceeded its LDS capacity
  kErrScan = 32u,       // a single-pass scan waited too long for a predecessor tile
};

constexpr u64 kEmptyKey = ~0ull;
// Set in a merged arc's visited-table slot when its insert claimed the slot
// (visited-table capacity is at most 2^31 slots).
constexpr u32 kNewFlag = 0x80000000u;
// A product-merge temp entry whose target already had an id (dense visited
// array only: ids and slots are below kDenseMaxPairs = 2^30) holds that id
// with this flag instead of the slot, so the result append needs no
// visited-array lookup.  Hash-table slots reach bit 30 and never carry it.
constexpr u32 kIdFlag = 0x40000000u;
// Dense visited array entries (ids stay below both).
constexpr u32 kUnvisited = 0xffffffffu;
constexpr u32 kClaimed = 0xfffffffeu;
constexpr u64 kMaxHashCap = 1ull << 31;
// Largest pair space |Q1| |Q2| whose visited set is a dense array (4 bytes a
// pair) from the start; up to kDenseMaxPairs the hash table is moved into
// such an array once it would need as many bytes.
constexpr u64 kDensePairs = 1ull << 26;
constexpr u64 kDenseMaxPairs = 1ull << 30;
static_assert(kDenseMaxPairs <= kIdFlag, "dense slots and ids stay below kIdFlag");

// ---------------------------------------------------------------------------
// Host-side error plumbing (exceptions stay inside the library).
struct Error : std::runtime_error {
  int code;
  Error(int c, const std::string &m) : std::runtime_error(m), code(c) {}
};

#define FSTC_HIP(call)                                                              \
  do {                                                                              \
    hipError_t e_ = (call);                                                         \
    if (e_ != hipSuccess)                                                           \
      throw ::fstc::Error(FSTC_ERR_HIP, std::string(#call) + ": " + hipGetErrorString(e_)); \
  } while (0)

inline unsigned bits_for(u64 max_value) {  // bits needed to hold 0..max_value
  unsigned b = 0;
  while (b < 64 && (max_value >> b) != 0) ++b;
  return b;
}

inline u64 ceil_div(u64 a, u64 b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------------------
// Wave64 primitives.
__device__ __forceinline__ u32 lane_id() { return __lane_id(); }

// Number of set bits of `mask` in lanes below the calling lane.
__device__ __forceinline__ u32 count_below(u64 mask) {
  return __builtin_amdgcn_mbcnt_hi((u32)(mask >> 32), __builtin_amdgcn_mbcnt_lo((u32)mask, 0u));
}

template <class T>
__device__ __forceinline__ T wave_inclusive_sum(T x) {
  const u32 lane = lane_id();
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    T y = __shfl_up(x, d, kWave);
    if (lane >= (u32)d) x += y;
  }
  return x;
}

template <class T>
__device__ __forceinline__ T wave_sum(T x) {
#pragma unroll
  for (int d = kWave / 2; d > 0; d >>= 1) x += __shfl_xor(x, d, kWave);
  return x;
}

// Sum of x over the 64 lanes of a wave whose lanes are all active, returned
// to every lane: window sums by DPP row shifts (lane 15 of each row of 16
// ends with the row's sum), rows combined by the row broadcasts of lane 15
// and lane 31, the total read from lane 63.  No LDS traffic.
__device__ __forceinline__ u32 wave_total(u32 x) {
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return (u32)__builtin_amdgcn_readlane((int)x, 63);
}

// Inclusive prefix sum of x over the 64 lanes of a wave whose lanes are all
// active: prefixes within each row of 16 by DPP row shifts (zeros shifted
// in), then the row totals carried by the broadcasts of lane 15 (to rows 1
// and 3) and lane 31 (to rows 2 and 3).
__device__ __forceinline__ u32 wave_inclusive_total(u32 x) {
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// Bitwise OR of x over the 64 lanes of a wave whose lanes are all active,
// returned to every lane (the pattern of wave_total).
__device__ __forceinline__ u32 wave_or(u32 x) {
  x |= (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x |= (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x |= (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x |= (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x |= (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x |= (u32)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return (u32)__builtin_amdgcn_readlane((int)x, 63);
}

template <class T>
__device__ __forceinline__ T wave_max(T x) {
#pragma unroll
  for (int d = kWave / 2; d > 0; d >>= 1) {
    T y = __shfl_xor(x, d, kWave);
    x = y > x ? y : x;
  }
  return x;
}

// Exclusive sum over the threads of a block (NT threads, NT % 64 == 0).
// `scratch` holds NT/64 values of T.  Returns this thread's exclusive prefix
// and writes the block total to *total.  Contains barriers: every thread of
// the block must call it.
template <int NT, class T>
__device__ __forceinline__ T block_exclusive_sum(T x, T *scratch, T *total) {
  constexpr int NW = NT / kWave;
  const u32 lane = lane_id();
  const u32 wid = threadIdx.x / kWave;
  T inc = wave_inclusive_sum(x);
  __syncthreads();
  if (lane == kWave - 1) scratch[wid] = inc;
  __syncthreads();
  if (wid == 0) {
    T v = lane < (u32)NW ? scratch[lane] : T(0);
    v = wave_inclusive_sum(v);
    if (lane < (u32)NW) scratch[lane] = v;
  }
  __syncthreads();
  const T base = wid ? scratch[wid - 1] : T(0);
  *total = scratch[NW - 1];
  return base + inc - x;
}

// Sum over the threads of a block; result valid in every thread.
template <int NT, class T>
__device__ __forceinline__ T block_sum(T x, T *scratch) {
  T total;
  (void)block_exclusive_sum<NT, T>(x, scratch, &total);
  return total;
}

// Index of the last element of sorted a[0..n) that is <= v, assuming
// n >= 1 and a[0] <= v.
template <class T>
__device__ __forceinline__ u64 last_le(const T *a, u64 n, T v) {
  u64 lo = 0, hi = n;  // invariant: a[lo] <= v, answer in [lo, hi)
  while (hi - lo > 1) {
    u64 mid = (lo + hi) >> 1;
    if (a[mid] <= v) lo = mid; else hi = mid;
  }
  return lo;
}

// First index i in [0, n] with a[i] >= v (a sorted ascending).
template <class T>
__device__ __forceinline__ u64 lower_bound_dev(const T *a, u64 n, T v) {
  u64 lo = 0, hi = n;
  while (lo < hi) {
    u64 mid = (lo + hi) >> 1;
    if (a[mid] < v) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// splitmix64 finalizer (Steele, Lea & Flood 2014), used to spread pair keys
// over the visited table.
__device__ __forceinline__ u64 mix64(u64 x) {
  x ^= x >> 30;
  x *= 0xbf58476d1ce4e5b9ull;
  x ^= x >> 27;
  x *= 0x94d049bb133111ebull;
  x ^= x >> 31;
  return x;
}

__device__ __forceinline__ void set_error(u32 *err, u32 bits) { atomicOr(err, bits); }

// Appends `value` to list[] for every lane with pred set, one atomic per
// wave; entries at or beyond `cap` are dropped and flag kErrBounds.  Every
// lane of the wave must call it.
__device__ __forceinline__ void wave_append(bool pred, u32 value, u32 *list, u32 *counter,
                                            u64 cap = ~0ull, u32 *err = nullptr,
                                            u32 err_bits = 4u) {
  const u64 m = __ballot(pred);
  if (!m) return;
  const u32 leader = __ffsll((unsigned long long)m) - 1;
  u32 base = 0;
  if (lane_id() == leader) base = atomicAdd(counter, (u32)__popcll(m));
  base = __shfl(base, leader, kWave);
  if (pred) {
    const u64 pos = (u64)base + count_below(m);
    if (pos < cap) list[pos] = value;
    else if (err) set_error(err, err_bits);
  }
}

// Bits needed to hold 0..v on the device.
__device__ __forceinline__ int bits_for_dev(u32 v) { return v ? 32 - __clz(v) : 0; }

// ---------------------------------------------------------------------------
// Launch helpers shared by the translation units.
// Compute units of the current device (queried once per device).
int compute_units();
void fill_u32(u32 *p, u32 v, u64 n, hipStream_t s);
void fill_u64(u64 *p, u64 v, u64 n, hipStream_t s);

// Exclusive scans: out[i] = sum_{j<i} in[j], i in [0, n]; out has n + 1
// entries.  `temp` must hold scan_temp_bytes(n) bytes.
size_t scan_temp_bytes(u64 n);
void exclusive_scan(const u64 *in, u64 *out, u64 n, void *temp, hipStream_t s);
void exclusive_scan(const u32 *in, u64 *out, u64 n, void *temp, hipStream_t s);
void exclusive_scan(const u32 *in, u32 *out, u64 n, void *temp, hipStream_t s);
// Single-pass exclusive scans (decoupled look-back) of up to four arrays of
// the same length n at once, one launch: in[k] holds u64 when wide[k], else
// u32; out[k] has n + 1 entries (u64).  `state` is scan_lb_state_bytes(n)
// bytes that no other code writes and that were zero-filled once when
// allocated; `ctr` is a device word that is 0 before the call (the call
// leaves it 0); scan failures set kErrScan in *err.
struct ScanJob {
  const void *in;
  bool wide;
  u64 *out;
  bool narrow_out = false;    // out holds u32 (sums must fit)
  const u64 *sub = nullptr;   // scans in[i] - sub[i] (in wide)
  bool total_only = false;    // writes out[n] alone
  u64 *total_to = nullptr;    // the total is also stored here (less *total_minus,
  const u64 *total_minus = nullptr;  // when given; as a u32, saturated, when
  bool total_narrow = false;         // total_narrow)
};
// After the last tile has stored the totals: `words` 32-bit words copied
// from src to dst (host memory the device can write) except word seq_word,
// a system-scope fence, then dst[seq_word] = seq (a publication the host
// can wait for); then the words i of src with bit i of clear_mask set are
// zeroed (words < 64).  when_skipped: a scan skipped by its skip_if word
// still publishes src as it is (and clears nothing).
struct ScanPublish {
  const void *src;
  void *dst;
  u32 words, seq_word, seq;
  u64 clear_mask = 0;
  bool when_skipped = false;
};
size_t scan_lb_state_bytes(u64 n);
// skip_if (may be NULL): a device word read by every workgroup first; when it
// is nonzero the scan does nothing (a scan enqueued before the host knows
// whether it is needed) but the publication asked for with when_skipped.
void exclusive_scan_lb(const ScanJob *jobs, int k, u64 n, void *state, u32 *ctr, u32 *err,
                       hipStream_t s, const ScanPublish *pub = nullptr,
                       const u64 *skip_if = nullptr);

// Stable LSD radix sort of (u64 key, u32 value) on key bits [lo, hi).
// keys/vals hold the input; keys_alt/vals_alt are scratch of the same size;
// `temp` must hold radix_temp_bytes(n) bytes.  The sorted data ends in
// keys/vals.
size_t radix_temp_bytes(u64 n);
void radix_sort_pairs(u64 *keys, u32 *vals, u64 *keys_alt, u32 *vals_alt, u64 n, int lo,
                      int hi, void *temp, hipStream_t s);
// One or two independent sorts of the same kind run together: each pass's
// histogram, scan and scatter are one launch for all the jobs still sorting
// (when every job's digit histogram fits one workgroup's scan, n <= 2^20;
// otherwise the sorts run one after the other).
// A job whose *unsorted word differs from `epoch` when its passes run is
// already in order (the caller's check): its passes copy instead of sorting.
struct SortJob {
  u64 *keys, *keys_alt;
  u32 *vals, *vals_alt;
  u64 n;
  int lo, hi;
  void *temp;  // radix_temp_bytes(n) bytes
  const u32 *unsorted = nullptr;
  u32 epoch = 0;
};
void radix_sort_pairs_batch(const SortJob *jobs, int nj, hipStream_t s);

}  // namespace fstc
