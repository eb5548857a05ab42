// Frontier expansion of one breadth-first level: join counting, match
// emission and the arc-pair write pass.
//
// For a popped pair q1q2 the paper composes every M1 arc of q1 with output b
// with every M2 arc of q2 with input b, for all b, producing n1 * n2 arcs per
// symbol (section 3.4, "Generating transitions", Algorithm 2).  Here a whole
// level of pairs is expanded at once:
//   1. count:  per source, intersect its two sorted segment lists (symbols
//              present at q1 as output and at q2 as input) and count matched
//              symbols and sum_b n1(b) * n2(b) composed arcs;
//   2. (scan:  exclusive sums give every source its match and arc offsets);
//   3. emit:   write one descriptor per matched symbol (arc ranges of both
//              sides and the first output record);
//   4. write:  every workgroup produces a fixed 2048-record window of the
//              level's composed arcs, whatever the fan-out of the sources
//              inside it, so work is balanced across the chip and every
//              store is coalesced.
// Joins are done per thread, per wavefront or per workgroup depending on the
// length of the shorter segment list (kWideMin / kHeavyMin).
#include "level.hpp"

namespace fstc {
namespace {

// Calls f(s1, s2) for every pair of segments with the same symbol, s1 in
// [b1, e1) of sym1 and s2 in [b2, e2) of sym2, in increasing symbol order.
// Walks the shorter list and binary-searches the longer one with a moving
// lower bound.
template <class F>
__device__ __forceinline__ void intersect_serial(const u32 *sym1, u32 b1, u32 e1, const u32 *sym2,
                                                 u32 b2, u32 e2, F &&f) {
  if (e1 - b1 <= e2 - b2) {
    u32 lo = b2;
    for (u32 i = b1; i < e1 && lo < e2; ++i) {
      const u32 sym = sym1[i];
      u32 l = lo, h = e2;
      while (l < h) {
        const u32 m = (l + h) >> 1;
        if (sym2[m] < sym) l = m + 1; else h = m;
      }
      if (l < e2 && sym2[l] == sym) { f(i, l); lo = l + 1; } else lo = l;
    }
  } else {
    u32 lo = b1;
    for (u32 i = b2; i < e2 && lo < e1; ++i) {
      const u32 sym = sym2[i];
      u32 l = lo, h = e1;
      while (l < h) {
        const u32 m = (l + h) >> 1;
        if (sym1[m] < sym) l = m + 1; else h = m;
      }
      if (l < e1 && sym1[l] == sym) { f(l, i); lo = l + 1; } else lo = l;
    }
  }
}

__device__ __forceinline__ u32 lower_bound_u32(const u32 *a, u32 l, u32 h, u32 v) {
  while (l < h) {
    const u32 m = (l + h) >> 1;
    if (a[m] < v) l = m + 1; else h = m;
  }
  return l;
}

struct Ranges {
  u32 b1, e1, b2, e2;
};

__device__ __forceinline__ Ranges source_ranges(const LevelArgs &a, u32 u) {
  const u32 sid = a.lo + u;
  const u32 q1 = a.sq1[sid], q2 = a.sq2[sid];
  return Ranges{a.c1.row[q1], a.c1.row[q1 + 1], a.c2.row[q2], a.c2.row[q2 + 1]};
}

__device__ __forceinline__ u32 seg_len(const u32 *seg_off, u32 s) { return seg_off[s + 1] - seg_off[s]; }

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_count_small(LevelArgs a) {
  const u64 u = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  bool wide = false, heavy = false;
  if (u < a.nsrc) {
    const Ranges r = source_ranges(a, (u32)u);
    const u32 mn = min(r.e1 - r.b1, r.e2 - r.b2);
    if (mn > kHeavyMin) {
      heavy = true;
    } else if (mn > kWideMin) {
      wide = true;
    } else {
      u64 cnt = 0;
      u32 mc = 0;
      intersect_serial(a.c1.seg_sym, r.b1, r.e1, a.c2.seg_sym, r.b2, r.e2, [&](u32 s1, u32 s2) {
        cnt += (u64)seg_len(a.c1.seg_off, s1) * seg_len(a.c2.seg_off, s2);
        ++mc;
      });
      a.cnt[u] = cnt;
      a.mc[u] = mc;
    }
  }
  wave_append(wide, (u32)u, a.wide, &a.st->nwide);
  wave_append(heavy, (u32)u, a.heavy, &a.st->nheavy);
}

// One lane's share of a cooperative join: element idx of the shorter list.
struct Hit {
  bool found;
  u32 s1, s2;
};

__device__ __forceinline__ Hit probe_one(const LevelArgs &a, const Ranges &r, bool one_short,
                                         u32 idx) {
  Hit h{false, 0, 0};
  if (one_short) {
    if (idx < r.e1) {
      const u32 sym = a.c1.seg_sym[idx];
      const u32 l = lower_bound_u32(a.c2.seg_sym, r.b2, r.e2, sym);
      if (l < r.e2 && a.c2.seg_sym[l] == sym) h = Hit{true, idx, l};
    }
  } else {
    if (idx < r.e2) {
      const u32 sym = a.c2.seg_sym[idx];
      const u32 l = lower_bound_u32(a.c1.seg_sym, r.b1, r.e1, sym);
      if (l < r.e1 && a.c1.seg_sym[l] == sym) h = Hit{true, l, idx};
    }
  }
  return h;
}

// Wavefront per source (grid-stride over the wide list).
__global__ __launch_bounds__(256) void k_count_wide(LevelArgs a) {
  const u32 lane = lane_id();
  const u32 gw = (blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const u32 nw = gridDim.x * blockDim.x / kWave;
  const u32 n = a.st->nwide;
  for (u32 i = gw; i < n; i += nw) {
    const u32 u = a.wide[i];
    const Ranges r = source_ranges(a, u);
    const bool one_short = (r.e1 - r.b1) <= (r.e2 - r.b2);
    const u32 bs = one_short ? r.b1 : r.b2, es = one_short ? r.e1 : r.e2;
    u64 cnt = 0;
    u32 mc = 0;
    for (u32 base = bs; base < es; base += kWave) {
      const Hit h = probe_one(a, r, one_short, base + lane);
      if (h.found) {
        cnt += (u64)seg_len(a.c1.seg_off, h.s1) * seg_len(a.c2.seg_off, h.s2);
        ++mc;
      }
    }
    cnt = wave_sum(cnt);
    mc = wave_sum(mc);
    if (lane == 0) {
      a.cnt[u] = cnt;
      a.mc[u] = mc;
    }
  }
}

// Workgroup per source (grid-stride over the heavy list).
constexpr int kHeavyNT = 512;

__global__ __launch_bounds__(kHeavyNT) void k_count_heavy(LevelArgs a) {
  __shared__ u64 s64[kHeavyNT / kWave];
  __shared__ u32 s32[kHeavyNT / kWave];
  const u32 n = a.st->nheavy;
  for (u32 i = blockIdx.x; i < n; i += gridDim.x) {
    const u32 u = a.heavy[i];
    const Ranges r = source_ranges(a, u);
    const bool one_short = (r.e1 - r.b1) <= (r.e2 - r.b2);
    const u32 bs = one_short ? r.b1 : r.b2, es = one_short ? r.e1 : r.e2;
    u64 cnt = 0;
    u32 mc = 0;
    for (u32 base = bs; base < es; base += kHeavyNT) {
      const Hit h = probe_one(a, r, one_short, base + threadIdx.x);
      if (h.found) {
        cnt += (u64)seg_len(a.c1.seg_off, h.s1) * seg_len(a.c2.seg_off, h.s2);
        ++mc;
      }
    }
    cnt = block_sum<kHeavyNT, u64>(cnt, s64);
    mc = block_sum<kHeavyNT, u32>(mc, s32);
    if (threadIdx.x == 0) {
      a.cnt[u] = cnt;
      a.mc[u] = mc;
    }
  }
}

// ---------------------------------------------------------------------------
__device__ __forceinline__ void put_match(const LevelArgs &a, u64 k, u32 s1, u32 s2, u64 rbase) {
  const u32 a1 = a.c1.seg_off[s1], n1 = a.c1.seg_off[s1 + 1] - a1;
  const u32 a2 = a.c2.seg_off[s2], n2 = a.c2.seg_off[s2 + 1] - a2;
  a.match[k] = make_uint4(a1, a2, n1, n2);
  a.mrbase[k] = rbase;
}

__global__ __launch_bounds__(256) void k_emit_small(LevelArgs a) {
  const u64 u = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= a.nsrc) return;
  const Ranges r = source_ranges(a, (u32)u);
  if (min(r.e1 - r.b1, r.e2 - r.b2) > kWideMin) return;
  u64 k = a.moff[u], rb = a.roff[u];
  intersect_serial(a.c1.seg_sym, r.b1, r.e1, a.c2.seg_sym, r.b2, r.e2, [&](u32 s1, u32 s2) {
    put_match(a, k, s1, s2, rb);
    rb += (u64)seg_len(a.c1.seg_off, s1) * seg_len(a.c2.seg_off, s2);
    ++k;
  });
}

__global__ __launch_bounds__(256) void k_emit_wide(LevelArgs a) {
  const u32 lane = lane_id();
  const u32 gw = (blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const u32 nw = gridDim.x * blockDim.x / kWave;
  const u32 n = a.st->nwide;
  for (u32 i = gw; i < n; i += nw) {
    const u32 u = a.wide[i];
    const Ranges r = source_ranges(a, u);
    const bool one_short = (r.e1 - r.b1) <= (r.e2 - r.b2);
    const u32 bs = one_short ? r.b1 : r.b2, es = one_short ? r.e1 : r.e2;
    u64 k = a.moff[u], rb = a.roff[u];
    for (u32 base = bs; base < es; base += kWave) {
      const Hit h = probe_one(a, r, one_short, base + lane);
      const u64 prod = h.found ? (u64)seg_len(a.c1.seg_off, h.s1) * seg_len(a.c2.seg_off, h.s2) : 0;
      const u64 fm = __ballot(h.found);
      const u64 incl = wave_inclusive_sum(prod);
      const u64 total = __shfl(incl, kWave - 1, kWave);
      if (h.found) put_match(a, k + count_below(fm), h.s1, h.s2, rb + incl - prod);
      k += (u64)__popcll(fm);
      rb += total;
    }
  }
}

__global__ __launch_bounds__(kHeavyNT) void k_emit_heavy(LevelArgs a) {
  __shared__ u64 s64[kHeavyNT / kWave];
  __shared__ u32 s32[kHeavyNT / kWave];
  const u32 n = a.st->nheavy;
  for (u32 i = blockIdx.x; i < n; i += gridDim.x) {
    const u32 u = a.heavy[i];
    const Ranges r = source_ranges(a, u);
    const bool one_short = (r.e1 - r.b1) <= (r.e2 - r.b2);
    const u32 bs = one_short ? r.b1 : r.b2, es = one_short ? r.e1 : r.e2;
    u64 k = a.moff[u], rb = a.roff[u];
    for (u32 base = bs; base < es; base += kHeavyNT) {
      const Hit h = probe_one(a, r, one_short, base + threadIdx.x);
      const u64 prod = h.found ? (u64)seg_len(a.c1.seg_off, h.s1) * seg_len(a.c2.seg_off, h.s2) : 0;
      u32 ftot;
      u64 ptot;
      const u32 fex = block_exclusive_sum<kHeavyNT, u32>(h.found ? 1u : 0u, s32, &ftot);
      const u64 pex = block_exclusive_sum<kHeavyNT, u64>(prod, s64, &ptot);
      if (h.found) put_match(a, k + fex, h.s1, h.s2, rb + pex);
      k += ftot;
      rb += ptot;
    }
  }
}

// 8 consecutive record keys with 16-byte stores (p is 32-byte aligned).
// A lane writes kRun consecutive records per run; the lanes of a wave write
// consecutive runs, so every vector store of a wave covers one contiguous
// span (64 * 16 bytes for u32 keys and for weights).
constexpr int kRun = 4;
constexpr int kRuns = kExpandIT / kRun;  // runs per thread
static_assert(kExpandIT % kRun == 0, "whole runs per thread");

// Records are written once and read once by the merge, long after they
// have left the caches at the sizes that matter: streaming stores.
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef u64 u64x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void store_run(u32 *p, const u32 (&k)[kRun]) {
  const u32x4 v = {k[0], k[1], k[2], k[3]};
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(p));
}
__device__ __forceinline__ void store_run(u64 *p, const u64 (&k)[kRun]) {
  const u64x2 v0 = {k[0], k[1]}, v1 = {k[2], k[3]};
  __builtin_nontemporal_store(v0, reinterpret_cast<u64x2 *>(p));
  __builtin_nontemporal_store(v1, reinterpret_cast<u64x2 *>(p) + 1);
}
__device__ __forceinline__ void store_run(float *p, const float (&w)[kRun]) {
  const f32x4 v = {w[0], w[1], w[2], w[3]};
  __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(p));
}

// ---------------------------------------------------------------------------
// Arc-pair write pass.  Workgroup b produces the records of write tiles
// kExpandGroup*b .. kExpandGroup*(b+1) - 1: the matches overlapping them are
// staged in LDS (all tiles at once when they fit, else one tile after the
// other).  Wave w writes the wave span [w*64*kExpandIT, (w+1)*64*kExpandIT)
// of the group as kRuns passes of 64 lanes x kRun consecutive records; for
// each run a lane finds the match of its first record by binary search in
// LDS, takes (i, j) = divmod(offset, n2) to select the M1 and M2 arcs, and
// steps through the run.  Record = (part1 << b2 | part2, p1 * p2).
template <class KT>
__global__ __launch_bounds__(kExpandNT) void k_expand(const uint4 *match, const u64 *mrbase, u64 M,
                                                      u64 R, const uint2 *arcs1,
                                                      const uint2 *arcs2, int b2, KT *rec_key,
                                                      float *rec_w, const ExpandTile *tiles,
                                                      u64 ntiles, u32 *err) {
  __shared__ u32 s_rel[kExpandTile];
  __shared__ uint4 s_m[kExpandTile];
  constexpr u32 kSpan = kWave * kExpandIT;                      // records per wave
  constexpr u32 kWavesPerTile = (u32)(kExpandTile / kSpan);
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const u64 g0 = (u64)blockIdx.x * kExpandGroup;
  const u64 ng = min(kExpandGroup, ntiles - g0);
  const u64 r0 = g0 * kExpandTile;
  const ExpandTile ta = tiles[g0], tb = tiles[g0 + ng - 1];
  // one staging for the whole group when its matches fit, else per tile
  const bool one = tb.kend - ta.k0 <= kExpandTile;
  const u32 passes = one ? 1u : (u32)ng;
  for (u32 pass = 0; pass < passes; ++pass) {
    const ExpandTile ti = one ? ExpandTile{ta.k0, tb.kend, ta.base0, 0} : tiles[g0 + pass];
    const u64 rs = one ? r0 : r0 + pass * kExpandTile;  // record origin of s_rel
    const u64 k0 = ti.k0, nm = ti.kend - ti.k0;
    if (ti.kend <= k0 || ti.kend > M || nm > kExpandTile) {  // impossible: >= 1 record per match
      if (threadIdx.x == 0) set_error(err, kErrBounds);
      return;
    }
    if (pass) __syncthreads();  // previous tile's LDS fully read
    for (u32 i = threadIdx.x; i < nm; i += kExpandNT) {
      s_rel[i] = i == 0 ? 0u : (u32)(mrbase[k0 + i] - rs);
      s_m[i] = match[k0 + i];
    }
    __syncthreads();
    if (!one && w / kWavesPerTile != pass) continue;
#pragma unroll
    for (int h = 0; h < kRuns; ++h) {
      const u64 rfirst = r0 + w * kSpan + h * (kWave * kRun) + lane * kRun;
      if (rfirst >= R) break;
      const u32 cnt = (u32)min<u64>(kRun, R - rfirst);
      const u32 rel = (u32)(rfirst - rs);
      u32 mi = (u32)last_le<u32>(s_rel, nm, rel);
      uint4 m = s_m[mi];
      const u64 t = mi == 0 ? rfirst - ti.base0 : (u64)(rel - s_rel[mi]);
      u32 i1, i2;
      if (t < (1ull << 32)) {
        const u32 tt = (u32)t;
        i1 = tt / m.w;
        i2 = tt - i1 * m.w;
      } else {
        const u64 q = t / m.w;
        i1 = (u32)q;
        i2 = (u32)(t - q * m.w);
      }
      KT key[kRun];
      float wt[kRun];
#pragma unroll
      for (int j = 0; j < kRun; ++j) {
        key[j] = 0;
        wt[j] = 0.f;
        if ((u32)j < cnt) {
          const uint2 A1 = arcs1[m.x + i1];
          const uint2 A2 = arcs2[m.y + i2];
          key[j] = (KT)(((u64)A1.x << b2) | (u64)A2.x);
          wt[j] = __uint_as_float(A1.y) * __uint_as_float(A2.y);
          if (++i2 == m.w) {
            i2 = 0;
            if (++i1 == m.z && (u32)j + 1 < cnt) {
              i1 = 0;
              m = s_m[++mi];
            }
          }
        }
      }
      if (cnt == kRun) {
        store_run(rec_key + rfirst, key);
        store_run(rec_w + rfirst, wt);
      } else {
        for (u32 j = 0; j < cnt; ++j) {
          rec_key[rfirst + j] = key[j];
          rec_w[rfirst + j] = wt[j];
        }
      }
    }
  }
}

__global__ void k_tile_matches(const u64 *mrbase, u64 M, u64 R, u64 ntiles, ExpandTile *tiles) {
  for (u64 t = (u64)blockIdx.x * blockDim.x + threadIdx.x; t < ntiles; t += (u64)gridDim.x * blockDim.x) {
    const u64 r0 = t * kExpandTile;
    const u64 k0 = last_le<u64>(mrbase, M, r0);
    tiles[t] = ExpandTile{k0, lower_bound_dev<u64>(mrbase, M, min(r0 + kExpandTile, R)),
                          mrbase[k0], 0};
  }
}

}  // namespace

void launch_count(const LevelArgs &a, hipStream_t s) {
  const unsigned g = (unsigned)ceil_div(a.nsrc, 256);
  hipLaunchKernelGGL(k_count_small, dim3(g), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_count_wide, dim3(2048), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_count_heavy, dim3(512), dim3(kHeavyNT), 0, s, a);
}

void launch_emit(const LevelArgs &a, hipStream_t s) {
  const unsigned g = (unsigned)ceil_div(a.nsrc, 256);
  hipLaunchKernelGGL(k_emit_small, dim3(g), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_emit_wide, dim3(2048), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_emit_heavy, dim3(512), dim3(kHeavyNT), 0, s, a);
}

void launch_expand(const uint4 *match, const u64 *mrbase, u64 M, u64 R, const CsrView &c1,
                   const CsrView &c2, int b2, bool wide_keys, void *rec_key, float *rec_w,
                   ExpandTile *tiles, u32 *err, hipStream_t s) {
  if (R == 0) return;
  const u64 g = ceil_div(R, kExpandTile);
  if (g >= (1ull << 31)) throw Error(FSTC_ERR_CAPACITY, "level too large for one launch");
  const unsigned gs = (unsigned)std::min<u64>(ceil_div(g, 256), 1u << 20);
  hipLaunchKernelGGL(k_tile_matches, dim3(gs), dim3(256), 0, s, mrbase, M, R, g, tiles);
  const unsigned gw = (unsigned)ceil_div(g, kExpandGroup);
  if (wide_keys)
    hipLaunchKernelGGL((k_expand<u64>), dim3(gw), dim3(kExpandNT), 0, s, match, mrbase, M, R,
                       c1.arcs, c2.arcs, b2, (u64 *)rec_key, rec_w, tiles, g, err);
  else
    hipLaunchKernelGGL((k_expand<u32>), dim3(gw), dim3(kExpandNT), 0, s, match, mrbase, M, R,
                       c1.arcs, c2.arcs, b2, (u32 *)rec_key, rec_w, tiles, g, err);
}

}  // namespace fstc
