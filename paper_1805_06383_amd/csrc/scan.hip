// Device-wide exclusive prefix sums and fills.
//
// The per-level offsets of the frontier expansion (records per source,
// matches per source, merged arcs per source) are exclusive prefix sums, as in
// the two-stage expansion the paper adopts from Merrill et al. (section 3.4,
// "Updating frontier and visited set").  Reduce-then-scan: one pass reduces
// tiles of 4096 elements, the tile sums are scanned recursively, and a second
// pass scans each tile with its offset.  A single tile is one launch.
#include <atomic>
#include <type_traits>

#include "common.hpp"

namespace fstc {
namespace {

constexpr int kScanNT = 256;
constexpr int kScanIT = 16;
constexpr int kScanTile = kScanNT * kScanIT;

template <class T>
__global__ void k_fill(T *p, T v, u64 n) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x)
    p[i] = v;
}

template <class TI, class TO>
__global__ __launch_bounds__(kScanNT) void k_tile_reduce(const TI *in, u64 n, TO *tile_sums) {
  __shared__ TO scratch[kScanNT / kWave];
  const u64 base = (u64)blockIdx.x * kScanTile;
  TO s = 0;
  // every load issued before the first is used (indices clamped, n >= 1)
  TI v[kScanIT];
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) v[j] = in[min<u64>(base + (u64)j * kScanNT + threadIdx.x, n - 1)];
#pragma unroll
  for (int j = 0; j < kScanIT; ++j)
    if (base + (u64)j * kScanNT + threadIdx.x < n) s += (TO)v[j];
  s = block_sum<kScanNT, TO>(s, scratch);
  if (threadIdx.x == 0) tile_sums[blockIdx.x] = s;
}

// Scans tile blockIdx.x of `in` into `out`, adding tile_offsets[blockIdx.x]
// (or 0).  The last tile also writes out[n] = total.
template <class TI, class TO>
__global__ __launch_bounds__(kScanNT) void k_tile_scan(const TI *in, TO *out, u64 n,
                                                       const TO *tile_offsets) {
  __shared__ TO tile[kScanTile];
  __shared__ TO scratch[kScanNT / kWave];
  const u64 base = (u64)blockIdx.x * kScanTile;
  // coalesced load, blocked re-read
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) {
    u64 i = base + (u64)j * kScanNT + threadIdx.x;
    tile[j * kScanNT + threadIdx.x] = i < n ? (TO)in[i] : TO(0);
  }
  __syncthreads();
  TO local[kScanIT];
  TO run = 0;
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) {
    local[j] = run;
    run += tile[threadIdx.x * kScanIT + j];
  }
  TO total;
  TO excl = block_exclusive_sum<kScanNT, TO>(run, scratch, &total);
  const TO off = tile_offsets ? tile_offsets[blockIdx.x] : TO(0);
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) tile[threadIdx.x * kScanIT + j] = local[j] + excl + off;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) {
    u64 i = base + (u64)j * kScanNT + threadIdx.x;
    if (i < n) out[i] = tile[j * kScanNT + threadIdx.x];
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) out[n] = off + total;
}

// ---------------------------------------------------------------------------
// Single-pass scan with decoupled look-back (Merrill & Garland, "Single-pass
// Parallel Prefix Scan with Decoupled Look-back", 2016).  A workgroup takes
// the next tile number from a counter, so every lower tile belongs to a
// workgroup already running; it publishes its tile total ("aggregate"),
// then wave 0 reads the status words of the 64 tiles below it at once and
// adds aggregates down to the nearest tile that has published its
// inclusive prefix, publishes its own inclusive prefix, and the workgroup
// writes its tile offset by that.
//
// Published values need no memory fences: every 64-bit state word carries
// the call's epoch in its high half, and is written and read with relaxed
// device-scope atomics, which the chip's eight L2 caches keep coherent (a
// release store or acquire load would instead write back or invalidate the
// whole L2 of an XCD, once per tile).  A tile has one status word (epoch,
// bit 0: aggregate published, bit 1: inclusive prefix published), stored
// after the values it announces, in an array of its own so that a wave
// polls 64 neighbouring words; each value is two words (epoch and one half
// of the value each).  A reader polls status words only, then reads the
// values it needs once and takes them if every word carries the current
// epoch (the value stores may become visible after the status store): words
// of other calls never match, and no word depends on the order in which
// another becomes visible.  Failed polls back off; waits are bounded
// (kLbSpins polls of a window): past that, kErrScan.
constexpr int kLbNT = 256;
constexpr int kLbIT = 8;
constexpr int kLbTile = kLbNT * kLbIT;
constexpr u32 kLbSpins = 1u << 22;
constexpr int kLbMax = 4;
// Value words per tile: [kLbMax values][aggregate, inclusive][lo, hi].
constexpr int kLbWords = kLbMax * 4;
constexpr u32 kLbAgg = 1u, kLbInc = 2u;

struct LbArgs {
  const void *in[kLbMax];
  u64 *out[kLbMax];
  u32 wide;    // bit k: in[k] holds u64
  u32 narrow;  // bit k: out[k] holds u32
  u32 tonly;   // bit k: only out[k][n] is written
  u32 tnarrow;  // bit k: total_to[k] holds a u32
  const u64 *sub[kLbMax];
  u64 *total_to[kLbMax];
  const u64 *tminus[kLbMax];
  ScanPublish pub;  // pub.dst == NULL: none
  u64 n;
  u32 nb, epoch;
  u64 *status;  // [nb] status words
  u64 *vals;    // [nb * kLbWords] value words
  u32 *ctr, *err;
  const u64 *skip_if;  // nonzero *skip_if: nothing to do
};

// Publishes value v of array k of tile t as its aggregate (which = 0) or
// inclusive prefix (which = 1).
__device__ __forceinline__ void lb_put(const LbArgs &p, u32 t, int k, int which, u64 v) {
  u64 *w = p.vals + (u64)t * kLbWords + k * 4 + which * 2;
  const u64 tag = (u64)p.epoch << 32;
  __hip_atomic_store(&w[0], tag | (v & 0xffffffffull), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&w[1], tag | (v >> 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Publishes the K aggregates (which = 0) or inclusive prefixes (which = 1)
// of tile t, then its status.
template <int K>
__device__ __forceinline__ void lb_publish(const LbArgs &p, u32 t, int which, const u64 (&v)[K]) {
#pragma unroll
  for (int k = 0; k < K; ++k) lb_put(p, t, k, which, v[k]);
  const u64 st = ((u64)p.epoch << 32) | (which ? (kLbAgg | kLbInc) : kLbAgg);
  __hip_atomic_store(&p.status[t], st, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Reads value `which` of array k of tile j; false unless both words carry
// this call's epoch.
__device__ __forceinline__ bool lb_get(const LbArgs &p, u64 j, int k, int which, u64 *v) {
  const u64 *w = p.vals + j * kLbWords + k * 4 + which * 2;
  const u64 a = __hip_atomic_load(&w[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const u64 b = __hip_atomic_load(&w[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  *v = (a & 0xffffffffull) | (b << 32);
  return (u32)(a >> 32) == p.epoch && (u32)(b >> 32) == p.epoch;
}

// LDS slot of tile element e (a permutation of the tile): the five low bits
// of e flipped by bits 3 to 7, so that both the blocked rows (e = thread
// kLbIT + j: without it every other thread's row starts on the same banks)
// and the striped accesses (e = r kLbNT + thread) spread over all banks.
static_assert(kLbIT == 8 && kLbTile % 256 == 0, "swizzle for rows of eight u64");
__device__ __forceinline__ u32 lb_slot(u32 e) { return e ^ ((e >> 3) & 31u); }

// Exclusive sums over the workgroup of K values at once (one barrier for
// all K); tot[k]: the workgroup's total of array k.  scratch is read after
// the barrier, so a caller that reuses it needs another barrier first.
template <int K>
__device__ __forceinline__ void block_exclusive_sums(u64 (&v)[K], u64 (*scratch)[kLbNT / kWave],
                                                     u64 (&tot)[K]) {
  constexpr int NW = kLbNT / kWave;
  const u32 lane = lane_id(), wid = threadIdx.x / kWave;
  u64 inc[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    inc[k] = wave_inclusive_sum(v[k]);
    if (lane == kWave - 1) scratch[k][wid] = inc[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; ++k) {
    u64 base = 0, all = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const u64 s = scratch[k][w];
      base += (u32)w < wid ? s : 0ull;
      all += s;
    }
    v[k] = base + inc[k] - v[k];
    tot[k] = all;
  }
}

// The publication of p.pub by one wave, after the stores it announces (see
// ScanPublish): lane i copies word i (once lane 0's total stores are
// visible to the wave), then one lane writes the publication number once
// every lane's copy has completed; then, when `clear`, the lanes zero the
// words of clear_mask (each its own words, after copying them).
__device__ __forceinline__ void lb_publish_counters(const LbArgs &p, bool clear) {
  const u32 lane = lane_id();
  u32 *src = const_cast<u32 *>(static_cast<const u32 *>(p.pub.src));
  u32 *dst = static_cast<u32 *>(p.pub.dst);
  __threadfence();
  for (u32 i = lane; i < p.pub.words; i += kWave)
    if (i != p.pub.seq_word) dst[i] = src[i];
  __threadfence_system();
  __builtin_amdgcn_wave_barrier();
  if (lane == 0)
    __hip_atomic_store(&dst[p.pub.seq_word], p.pub.seq, __ATOMIC_RELEASE,
                       __HIP_MEMORY_SCOPE_SYSTEM);
  if (clear && p.pub.clear_mask) {
    for (u32 i = lane; i < p.pub.words && i < 64u; i += kWave)
      if ((p.pub.clear_mask >> i) & 1ull) src[i] = 0u;
  }
}

// out[k][n] = total, and the total (less *tminus[k]) at total_to[k].
__device__ __forceinline__ void lb_store_total(const LbArgs &p, int k, u64 total) {
  if ((p.narrow >> k) & 1u) reinterpret_cast<u32 *>(p.out[k])[p.n] = (u32)total;
  else p.out[k][p.n] = total;
  if (p.total_to[k]) {
    const u64 v = total - (p.tminus[k] ? *p.tminus[k] : 0ull);
    if ((p.tnarrow >> k) & 1u)
      *reinterpret_cast<u32 *>(p.total_to[k]) = (u32)min<u64>(v, 0xffffffffull);
    else
      *p.total_to[k] = v;
  }
}

// Loads element pos(r) of each of the K arrays for r < kLbIT, every load
// issued before the first is used: indices clamped into the arrays, values
// zeroed past their end.  WM / SM: the wide and subtracted arrays as bit
// masks when known at compile time (-1: read from p), so that no load sits
// behind a branch (a branch around a load makes the compiler wait for
// every earlier one).
template <int K, int WM, int SM, class Pos>
__device__ __forceinline__ void lb_load(const LbArgs &p, Pos pos, u64 (&x)[K][kLbIT]) {
  if (p.n == 0) {  // uniform
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int r = 0; r < kLbIT; ++r) x[k][r] = 0;
    return;
  }
  const u64 last = p.n - 1;
  const u32 wide = WM >= 0 ? (u32)WM : p.wide;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    if ((wide >> k) & 1u) {
      const u64 *in = static_cast<const u64 *>(p.in[k]);
#pragma unroll
      for (int r = 0; r < kLbIT; ++r) x[k][r] = in[min<u64>(pos(r), last)];
    } else {
      const u32 *in = static_cast<const u32 *>(p.in[k]);
#pragma unroll
      for (int r = 0; r < kLbIT; ++r) x[k][r] = in[min<u64>(pos(r), last)];
    }
  }
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const u64 *sub = p.sub[k];
    if (SM >= 0 ? ((SM >> k) & 1) != 0 : sub != nullptr) {
#pragma unroll
      for (int r = 0; r < kLbIT; ++r) x[k][r] -= sub[min<u64>(pos(r), last)];
    }
  }
#pragma unroll
  for (int k = 0; k < K; ++k)
#pragma unroll
    for (int r = 0; r < kLbIT; ++r)
      if (pos(r) > last) x[k][r] = 0;
}

// A scan of one tile (n <= kLbTile): each thread loads, scans and stores
// its own kLbIT consecutive elements (no LDS staging, no look-back).
template <int K, int WM, int SM>
__global__ __launch_bounds__(kLbNT) void k_scan_one(LbArgs p) {
  __shared__ u64 scratch[kLbMax][kLbNT / kWave];
  const u32 lane = lane_id();
  if (p.skip_if && *p.skip_if != 0) {  // uniform
    if (threadIdx.x < (u32)kWave && p.pub.dst && p.pub.when_skipped) lb_publish_counters(p, false);
    return;
  }
  const u64 base = (u64)threadIdx.x * kLbIT;
  u64 x[K][kLbIT];
  lb_load<K, WM, SM>(p, [&](int j) { return base + (u64)j; }, x);
  u64 ex[K], tot[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    u64 run = 0;
#pragma unroll
    for (int j = 0; j < kLbIT; ++j) {
      const u64 v = x[k][j];
      x[k][j] = run;
      run += v;
    }
    ex[k] = run;
  }
  block_exclusive_sums<K>(ex, scratch, tot);
  if (threadIdx.x < (u32)kWave) {
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < K; ++k) lb_store_total(p, k, tot[k]);
    }
    if (p.pub.dst) lb_publish_counters(p, true);
  }
#pragma unroll
  for (int k = 0; k < K; ++k) {
    if ((p.tonly >> k) & 1u) continue;  // uniform
    const bool narrow = (p.narrow >> k) & 1u;
#pragma unroll
    for (int j = 0; j < kLbIT; ++j) {
      const u64 i = base + j;
      if (i < p.n) {
        if (narrow) reinterpret_cast<u32 *>(p.out[k])[i] = (u32)(ex[k] + x[k][j]);
        else p.out[k][i] = ex[k] + x[k][j];
      }
    }
  }
}

// Tile loads and stores are striped across the workgroup and pass through
// LDS (full coalescing); each thread scans kLbIT consecutive elements.
template <int K, int WM, int SM>
__global__ __launch_bounds__(kLbNT) void k_scan_lb(LbArgs p) {
  constexpr int NW = kLbNT / kWave;
  __shared__ u32 s_t;
  __shared__ u64 s_off[kLbMax];
  __shared__ u64 scratch[kLbMax][NW];
  __shared__ u64 s_x[kLbTile];  // one array of the tile, transposed
  const u32 lane = lane_id();
  if (p.skip_if && *p.skip_if != 0) {  // uniform: every workgroup leaves before the counter
    if (blockIdx.x == 0 && threadIdx.x < (u32)kWave && p.pub.dst && p.pub.when_skipped)
      lb_publish_counters(p, false);
    return;
  }
  // tile numbers from the counter (a single tile needs none)
  if (threadIdx.x == 0 && p.nb > 1) {
    const u32 t = atomicAdd(p.ctr, 1u);
    if (t == p.nb - 1) atomicExch(p.ctr, 0u);  // the last number is taken: ready for the next call
    s_t = t;
  }
  if (p.nb > 1) __syncthreads();
  const u32 t = p.nb > 1 ? s_t : 0u;
  const u64 tbase = (u64)t * kLbTile;
  // element r of this thread in the striped layout: tile position r kLbNT + thread
  u64 x[K][kLbIT];
  lb_load<K, WM, SM>(p, [&](int r) { return tbase + (u64)r * kLbNT + threadIdx.x; }, x);
  // to the blocked layout (thread i: elements kLbIT i .. kLbIT i + kLbIT - 1),
  // then x[k][j] becomes the exclusive sum within the thread's elements
  u64 ex[K], tot[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
#pragma unroll
    for (int r = 0; r < kLbIT; ++r) s_x[lb_slot((u32)r * kLbNT + threadIdx.x)] = x[k][r];
    __syncthreads();
    u64 run = 0;
#pragma unroll
    for (int j = 0; j < kLbIT; ++j) {
      const u64 v = s_x[lb_slot(threadIdx.x * kLbIT + j)];
      x[k][j] = run;
      run += v;
    }
    ex[k] = run;
    __syncthreads();  // s_x reused
  }
  block_exclusive_sums<K>(ex, scratch, tot);
  if (threadIdx.x < (u32)kWave) {
    u64 off[K];
#pragma unroll
    for (int k = 0; k < K; ++k) off[k] = 0;
    if (t == 0) {
      if (lane == 0 && p.nb > 1) lb_publish<K>(p, 0, 1, tot);  // a single tile has no successor
    } else {
      if (lane == 0) lb_publish<K>(p, t, 0, tot);
      long long hi = (long long)t - 1;  // nearest predecessor of the window
      u32 spins = 0, nap = 1;
      bool failed = false;
      while (true) {
        const long long j = hi - (long long)lane;
        // lane's tile j: below tile 0, an empty inclusive prefix
        u32 fl = kLbAgg | kLbInc;
        if (j >= 0) {
          const u64 st = __hip_atomic_load(&p.status[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          fl = (u32)(st >> 32) == p.epoch ? (u32)st : 0u;
        }
        const u64 pm = __ballot((fl & kLbInc) != 0), rm = __ballot(fl != 0);
        const u32 lp = pm ? (u32)__builtin_ctzll(pm) : (u32)kWave;  // nearest inclusive prefix
        const u64 need = lp < (u32)kWave ? (lp == 63 ? ~0ull : (2ull << lp) - 1ull) : ~0ull;
        bool ok = (rm & need) == need;  // uniform
        u64 v[K];
        if (ok) {
          // values of lanes below lp (aggregates) and of lane lp (its
          // inclusive prefix); taken once every word carries the epoch
          bool good = true;
#pragma unroll
          for (int k = 0; k < K; ++k) {
            v[k] = 0;
            if (j >= 0 && lane <= lp) good = lb_get(p, (u64)j, k, lane == lp ? 1 : 0, &v[k]) && good;
          }
          ok = __ballot(!good) == 0;
        }
        if (!ok) {  // a tile in between has not published yet
          if (++spins > kLbSpins) {
            failed = true;
            break;
          }
          for (u32 i = 0; i < nap; ++i) __builtin_amdgcn_s_sleep(1);
          nap = min(nap + 1, 32u);
          continue;
        }
#pragma unroll
        for (int k = 0; k < K; ++k) off[k] += wave_sum(v[k]);
        if (lp < (u32)kWave) break;
        hi -= kWave;
      }
      if (failed && lane == 0) atomicOr(p.err, kErrScan);
      if (lane == 0) {
        u64 inc[K];
#pragma unroll
        for (int k = 0; k < K; ++k) inc[k] = off[k] + tot[k];
        lb_publish<K>(p, t, 1, inc);
      }
    }
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < K; ++k) {
        s_off[k] = off[k];
        if (t == p.nb - 1) lb_store_total(p, k, off[k] + tot[k]);
      }
    }
    // every other tile has published its inclusive prefix: the totals are final
    if (t == p.nb - 1 && p.pub.dst) lb_publish_counters(p, true);
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; ++k) {
    if ((p.tonly >> k) & 1u) continue;  // uniform
    const u64 o = s_off[k] + ex[k];
#pragma unroll
    for (int j = 0; j < kLbIT; ++j) s_x[lb_slot(threadIdx.x * kLbIT + j)] = o + x[k][j];
    __syncthreads();
    const bool narrow = (p.narrow >> k) & 1u;
#pragma unroll
    for (int r = 0; r < kLbIT; ++r) {
      const u32 e = (u32)r * kLbNT + threadIdx.x;
      const u64 i = tbase + e;
      if (i < p.n) {
        if (narrow) reinterpret_cast<u32 *>(p.out[k])[i] = (u32)s_x[lb_slot(e)];
        else p.out[k][i] = s_x[lb_slot(e)];
      }
    }
    __syncthreads();
  }
}

template <class TO>
size_t temp_elems(u64 n) {
  size_t t = 0;
  u64 nb = ceil_div(n, kScanTile);
  while (nb > 1) {
    t += nb + (nb + 1);  // tile sums + their scan
    nb = ceil_div(nb, kScanTile);
  }
  return t;
}

template <class TI, class TO>
void scan_impl(const TI *in, TO *out, u64 n, TO *temp, hipStream_t s) {
  if (n == 0) {
    hipLaunchKernelGGL((k_fill<TO>), dim3(1), dim3(64), 0, s, out, TO(0), (u64)1);
    return;
  }
  const u64 nb = ceil_div(n, kScanTile);
  if (nb == 1) {
    hipLaunchKernelGGL((k_tile_scan<TI, TO>), dim3(1), dim3(kScanNT), 0, s, in, out, n,
                       (const TO *)nullptr);
    return;
  }
  TO *sums = temp;
  TO *offs = temp + nb;
  hipLaunchKernelGGL((k_tile_reduce<TI, TO>), dim3((unsigned)nb), dim3(kScanNT), 0, s, in, n,
                     sums);
  scan_impl<TO, TO>(sums, offs, nb, temp + nb + (nb + 1), s);
  hipLaunchKernelGGL((k_tile_scan<TI, TO>), dim3((unsigned)nb), dim3(kScanNT), 0, s, in, out,
                     n, (const TO *)offs);
}

}  // namespace

int compute_units() {
  static std::atomic<int> cache[64];
  int dev = 0;
  FSTC_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) dev = 0;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    FSTC_HIP(hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev));
    n = std::max(n, 1);
    cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

void fill_u32(u32 *p, u32 v, u64 n, hipStream_t s) {
  if (!n) return;
  unsigned g = (unsigned)std::min<u64>(ceil_div(n, 256), 4096);
  hipLaunchKernelGGL((k_fill<u32>), dim3(g), dim3(256), 0, s, p, v, n);
}

void fill_u64(u64 *p, u64 v, u64 n, hipStream_t s) {
  if (!n) return;
  unsigned g = (unsigned)std::min<u64>(ceil_div(n, 256), 4096);
  hipLaunchKernelGGL((k_fill<u64>), dim3(g), dim3(256), 0, s, p, v, n);
}

size_t scan_temp_bytes(u64 n) { return temp_elems<u64>(n) * sizeof(u64) + 256; }

// Status words (rounded up to whole 256-byte lines), then value words.
static u64 lb_status_words(u64 nb) { return (nb + 31) / 32 * 32; }

size_t scan_lb_state_bytes(u64 n) {
  const u64 nb = std::max<u64>(1, ceil_div(n, kLbTile));
  return (size_t)(lb_status_words(nb) + nb * kLbWords) * 8 + 256;
}

void exclusive_scan_lb(const ScanJob *jobs, int k, u64 n, void *state, u32 *ctr, u32 *err,
                       hipStream_t s, const ScanPublish *pub, const u64 *skip_if) {
  static std::atomic<u32> epochs{0};
  const u64 nb = std::max<u64>(1, ceil_div(n, kLbTile));
  if (nb >= (1ull << 31)) throw Error(FSTC_ERR_CAPACITY, "scan too large for one launch");
  LbArgs p{};
  p.wide = 0;
  p.narrow = 0;
  p.tonly = 0;
  p.tnarrow = 0;
  for (int i = 0; i < k; ++i) {
    p.in[i] = jobs[i].in;
    p.out[i] = jobs[i].out;
    p.wide |= (jobs[i].wide ? 1u : 0u) << i;
    p.narrow |= (jobs[i].narrow_out ? 1u : 0u) << i;
    p.tonly |= (jobs[i].total_only ? 1u : 0u) << i;
    p.sub[i] = jobs[i].sub;
    p.total_to[i] = jobs[i].total_to;
    p.tminus[i] = jobs[i].total_minus;
    p.tnarrow |= (jobs[i].total_narrow ? 1u : 0u) << i;
  }
  if (pub) p.pub = *pub;
  p.n = n;
  p.nb = (u32)nb;
  u32 e = epochs.fetch_add(1, std::memory_order_relaxed) + 1;
  p.epoch = e ? e : 1u;  // state words of zero-filled memory never match
  p.status = static_cast<u64 *>(state);
  p.vals = p.status + lb_status_words(nb);
  p.ctr = ctr;
  p.err = err;
  p.skip_if = skip_if;
  u32 subm = 0;
  for (int i = 0; i < k; ++i) subm |= (p.sub[i] ? 1u : 0u) << i;
  const dim3 g((unsigned)nb), bl(kLbNT);
  // the column forms of the level scans compiled in (loads without
  // branches); any other form reads them from the arguments
  auto go = [&](auto kk, auto wm, auto sm) {
    constexpr int K = decltype(kk)::value, WM = decltype(wm)::value, SM = decltype(sm)::value;
    if (nb == 1) hipLaunchKernelGGL((k_scan_one<K, WM, SM>), g, bl, 0, s, p);
    else hipLaunchKernelGGL((k_scan_lb<K, WM, SM>), g, bl, 0, s, p);
  };
  using I = std::integral_constant<int, -1>;
  if (k == 4 && p.wide == 0b1001u && subm == 0)
    go(std::integral_constant<int, 4>(), std::integral_constant<int, 0b1001>(), std::integral_constant<int, 0>());
  else if (k == 3 && p.wide == 0b110u && subm == 0b100u)
    go(std::integral_constant<int, 3>(), std::integral_constant<int, 0b110>(), std::integral_constant<int, 0b100>());
  else if (k == 1 && p.wide == 1u && subm == 0)
    go(std::integral_constant<int, 1>(), std::integral_constant<int, 1>(), std::integral_constant<int, 0>());
  else if (k == 1) go(std::integral_constant<int, 1>(), I(), I());
  else if (k == 2) go(std::integral_constant<int, 2>(), I(), I());
  else if (k == 3) go(std::integral_constant<int, 3>(), I(), I());
  else go(std::integral_constant<int, 4>(), I(), I());
}

void exclusive_scan(const u64 *in, u64 *out, u64 n, void *temp, hipStream_t s) {
  scan_impl<u64, u64>(in, out, n, (u64 *)temp, s);
}
void exclusive_scan(const u32 *in, u64 *out, u64 n, void *temp, hipStream_t s) {
  scan_impl<u32, u64>(in, out, n, (u64 *)temp, s);
}
void exclusive_scan(const u32 *in, u32 *out, u64 n, void *temp, hipStream_t s) {
  scan_impl<u32, u32>(in, out, n, (u32 *)temp, s);
}

}  // namespace fstc
