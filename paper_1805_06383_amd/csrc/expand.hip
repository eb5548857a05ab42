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
// Joins are done per thread, per 16-lane group, per wavefront or per
// workgroup depending on the lengths of the two segment lists (the rules
// beside kThreadSteps).
#include "level.hpp"
#include "product.hpp"

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


__device__ __forceinline__ Ranges source_ranges(const LevelArgs &a, u32 u) {
  const u32 sid = a.lo + u;
  const u32 q1 = a.sq1[sid], q2 = a.sq2[sid];
  return Ranges{a.c1.row[q1], a.c1.row[q1 + 1], a.c2.row[q2], a.c2.row[q2 + 1]};
}

__device__ __forceinline__ u32 seg_len(const u32 *seg_off, u32 s) { return seg_off[s + 1] - seg_off[s]; }

// ---------------------------------------------------------------------------
// Sources of more than kMergeSmall unmerged arcs are merged by the
// multi-block path (a.big); the largest count among the others sizes the
// merge window (st->max_small).  Both are gathered by the count kernels.
constexpr int kCountNT = 256;

// How source ranges r are joined (the rules beside kThreadSteps; sources
// of more than kHeavyMin symbols on the shorter list are classified before);
// the count and emit kernels classify alike.
enum : u32 { kJoinThread = 0, kJoinGroup = 1, kJoinWide = 2 };
__device__ __forceinline__ u32 join_class(const Ranges &r) {
  const u32 n1 = r.e1 - r.b1, n2 = r.e2 - r.b2;
  const u32 mn = min(n1, n2), mx = max(n1, n2);
  if (mn * (32u - __clz(mx)) <= kThreadSteps) return kJoinThread;
  if (mn <= kGroupMax && mx <= kGroupLong) return kJoinGroup;
  return kJoinWide;
}

// Thread per source: selects the product-merge sources (no records, no
// matches; pk = their entry count, pflag their flags for the level scan),
// joins the other short ones, lists the rest for the wavefront / workgroup
// joins.  List appends and the window maximum are aggregated per workgroup
// in LDS: one device atomic per list per block.
__global__ __launch_bounds__(kCountNT) void k_count_small(LevelArgs a) {
  constexpr int kLists = 5;
  __shared__ u32 s_n[kLists], s_base[kLists], s_max, s_unfit;
  const u32 lane = lane_id();
  const u64 u = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  if (threadIdx.x < kLists) s_n[threadIdx.x] = 0;
  if (threadIdx.x == 0) s_max = s_unfit = 0;
  // a source of a shape the one-workgroup small-level kernel declines
  // (group joins: decided by their count); counted per level
  bool unfit = false;
  // wide, heavy, big, one-per-wave product, 16-lane join
  bool pred[kLists] = {false, false, false, false, false};
  u64 cnt = 0;
  u32 pk = 0;
  bool mf = false;
  Ranges r{0, 0, 0, 0};
  if (u < a.nsrc) {
    const u32 sid = a.lo + (u32)u;
    const u32 q1 = a.sq1[sid], q2 = a.sq2[sid];
    a.tstart[u] = 0;
    a.mend[u] = 0;
    a.newc[u] = 0;
    r = Ranges{a.c1.row[q1], a.c1.row[q1 + 1], a.c2.row[q2], a.c2.row[q2 + 1]};
    const u32 mn = min(r.e1 - r.b1, r.e2 - r.b2);
    unfit = mn > kSmallShortList || max(r.e1 - r.b1, r.e2 - r.b2) > kSmallLongList;
    if (a.prod && mn >= kProdMinSymbols && mn <= (u32)kWave) pk = select_product(a, (u32)u, q1, q2, r, mf);
    if (pk && a.unred && !(a.quad && (a.phdr[2 * u].w & 4u))) pk = 0;  // records
    a.pk[u] = pk;
    a.pflag[u] = pk ? 1ull | ((u64)mf << 32) : 0ull;
    if (pk) {
      a.cnt[u] = 0;
      a.mc[u] = 0;
      unfit = true;
      // strided sources go to the four-source kernel when it runs
      pred[3] = !(a.quad && (a.phdr[2 * u].w & 4u));
    } else if (mn > kHeavyMin) {
      pred[1] = true;
      unfit = true;
    } else if (join_class(r) == kJoinWide) {
      pred[0] = true;
      unfit = true;
    } else if (join_class(r) == kJoinGroup) {
      pred[4] = true;
    } else {
      u32 mc = 0;
      intersect_serial(a.c1.seg_sym, r.b1, r.e1, a.c2.seg_sym, r.b2, r.e2, [&](u32 s1, u32 s2) {
        cnt += (u64)seg_len(a.c1.seg_off, s1) * seg_len(a.c2.seg_off, s2);
        ++mc;
      });
      a.cnt[u] = cnt;
      a.mc[u] = mc;
      pred[2] = cnt > kMergeSmall;
      unfit = unfit || cnt > kSmallPerSource;
    }
  }
  const u32 small_max = wave_max((u32)(pred[2] ? 0 : cnt));
  const u32 nunfit = (u32)__popcll(__ballot(unfit));
  __syncthreads();
  if (lane == 0 && nunfit) atomicAdd(&s_unfit, nunfit);
  u64 m[kLists];
  u32 woff[kLists];
#pragma unroll
  for (int l = 0; l < kLists; ++l) {
    m[l] = __ballot(pred[l]);
    woff[l] = 0;
    if (m[l]) {
      const u32 leader = __ffsll((unsigned long long)m[l]) - 1;
      if (lane == leader) woff[l] = atomicAdd(&s_n[l], (u32)__popcll(m[l]));
      woff[l] = __shfl(woff[l], leader, kWave);
    }
  }
  if (lane == 0 && small_max) atomicMax(&s_max, small_max);
  __syncthreads();
  u32 *const counters[kLists] = {&a.st->nwide, &a.st->nheavy, &a.st->nbig, &a.st->ngen,
                                 &a.st->ngrp};
  if (threadIdx.x < kLists && s_n[threadIdx.x])
    s_base[threadIdx.x] = atomicAdd(counters[threadIdx.x], s_n[threadIdx.x]);
  if (threadIdx.x == kLists && s_max) atomicMax(&a.st->max_small, s_max);
  if (threadIdx.x == kLists + 1 && s_unfit) atomicAdd(&a.st->unfit, s_unfit);
  __syncthreads();
  u32 *const lists[kLists] = {a.wide, a.heavy, a.big, a.glist, a.grp};
#pragma unroll
  for (int l = 0; l < kLists; ++l) {
    if (!pred[l]) continue;
    const u32 pos = s_base[l] + woff[l] + count_below(m[l]);
    lists[l][pos] = (u32)u;
    // saves the listed joins two dependent loads
    if (l == 0) a.wrange[pos] = make_uint4(r.b1, r.e1, r.b2, r.e2);
    if (l == 4) a.wrange[a.nsrc - 1 - pos] = make_uint4(r.b1, r.e1, r.b2, r.e2);
  }
}

// Big-source append and window maximum of one joined source (lane 0 of the
// joining wave or thread 0 of the joining block): big sources are rare, the
// maximum is kept in `run_max` and published once per block.
__device__ __forceinline__ void note_count(const LevelArgs &a, u32 u, u64 cnt, u32 &run_max) {
  if (cnt > kMergeSmall) a.big[atomicAdd(&a.st->nbig, 1u)] = u;
  else run_max = max(run_max, (u32)cnt);
}

template <int NT>
__device__ __forceinline__ void publish_max(const LevelArgs &a, u32 run_max, u32 *s_max) {
  if (threadIdx.x == 0) *s_max = 0;
  __syncthreads();
  run_max = wave_max(run_max);
  if (lane_id() == 0 && run_max) atomicMax(s_max, run_max);
  __syncthreads();
  if (threadIdx.x == 0 && *s_max) atomicMax(&a.st->max_small, *s_max);
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

// Wave-cooperative probe of short-list elements base + lane against the
// longer list, both sorted with distinct symbols: 64-symbol chunks of the
// longer list are loaded into the lanes (one coalesced load each) and
// searched by a 6-step binary search over lane shuffles.  `lp` is the first
// chunk start of the longer list that can still match; it only moves
// forward, so the next call (the next 64 short elements) resumes there.
// All arguments but idx-dependent ones are wave-uniform.
__device__ __forceinline__ Hit wave_probe(const LevelArgs &a, const Ranges &r, bool one_short,
                                          u32 base, u32 es, u32 &lp) {
  const u32 *ssym = one_short ? a.c1.seg_sym : a.c2.seg_sym;
  const u32 *lsym = one_short ? a.c2.seg_sym : a.c1.seg_sym;
  const u32 le = one_short ? r.e2 : r.e1;
  const u32 lane = lane_id();
  const u32 idx = base + lane;
  const bool valid = idx < es;
  const u32 sym = valid ? ssym[idx] : 0xffffffffu;  // labels are below 2^32 - 1
  const u32 last = min(es - base, (u32)kWave) - 1;
  const u32 smax = __shfl(sym, (int)last, kWave);
  u32 fpos = 0xffffffffu;
  if (le - lp > 4u * kWave) {
    // a long remainder: each lane binary-searches its symbol (fewer
    // dependent loads than walking the chunks)
    u32 l = lp;
    if (valid) {
      l = lower_bound_u32(lsym, lp, le, sym);
      if (l < le && lsym[l] == sym) fpos = l;
    }
    lp = __shfl(l, (int)last, kWave);  // later short symbols are above smax
    if (fpos == 0xffffffffu) return Hit{false, 0, 0};
    return one_short ? Hit{true, idx, fpos} : Hit{true, fpos, idx};
  }
  for (u32 c = lp; c < le; c += kWave) {
    const u32 len = min(le - c, (u32)kWave);
    const u32 lv = lane < len ? lsym[c + lane] : 0xffffffffu;
    if (__shfl(lv, 0, kWave) > smax) break;  // this chunk and later ones are past the short chunk
    u32 pos = 0;  // elements of the chunk below sym (at most 63: then lane 63 decides)
#pragma unroll
    for (u32 step = kWave / 2; step; step >>= 1) {
      const u32 v = __shfl(lv, (int)(pos + step - 1), kWave);
      pos = v < sym ? pos + step : pos;
    }
    const u32 at = __shfl(lv, (int)pos, kWave);
    if (valid && at == sym) fpos = c + pos;
    if (__shfl(lv, (int)(len - 1), kWave) >= smax) {  // later short symbols start in this chunk
      lp = c;
      break;
    }
    lp = c + kWave;
  }
  if (fpos == 0xffffffffu) return Hit{false, 0, 0};
  return one_short ? Hit{true, idx, fpos} : Hit{true, fpos, idx};
}

// The joins of the listed sources, one launch of kListNT-thread blocks:
// blocks [0, gw) take the wide list with a wavefront per source, the others
// the heavy list with the whole block per source (both grid-stride over
// their list, whose length the small-source kernel left in *st).
constexpr int kListNT = 512;
constexpr int kHeavyNT = kListNT;

__device__ __forceinline__ void count_wide_sources(const LevelArgs &a, u32 blk, u32 nblk,
                                                   u32 &run_max) {
  const u32 lane = lane_id();
  const u32 gw = (blk * kListNT + threadIdx.x) / kWave;
  const u32 nw = nblk * kListNT / kWave;
  const u32 n = a.st->nwide;
  for (u32 i = gw; i < n; i += nw) {
    const u32 u = a.wide[i];
    const uint4 wr = a.wrange[i];
    const Ranges r{wr.x, wr.y, wr.z, wr.w};
    const bool one_short = (r.e1 - r.b1) <= (r.e2 - r.b2);
    const u32 bs = one_short ? r.b1 : r.b2, es = one_short ? r.e1 : r.e2;
    u64 cnt = 0;
    u32 mc = 0;
    u32 lp = one_short ? r.b2 : r.b1;
    for (u32 base = bs; base < es; base += kWave) {
      const Hit h = wave_probe(a, r, one_short, base, es, lp);
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
      note_count(a, u, cnt, run_max);
    }
  }
}

__device__ __forceinline__ void count_heavy_sources(const LevelArgs &a, u32 blk, u32 nblk,
                                                    u32 &run_max, u64 *s64, u32 *s32) {
  const u32 n = a.st->nheavy;
  for (u32 i = blk; i < n; i += nblk) {
    const u32 u = a.heavy[i];
    const Ranges r = source_ranges(a, u);
    const bool one_short = (r.e1 - r.b1) <= (r.e2 - r.b2);
    const u32 bs = one_short ? r.b1 : r.b2, es = one_short ? r.e1 : r.e2;
    u64 cnt = 0;
    u32 mc = 0;
    for (u32 base = bs; base < es; base += kListNT) {
      const Hit h = probe_one(a, r, one_short, base + threadIdx.x);
      if (h.found) {
        cnt += (u64)seg_len(a.c1.seg_off, h.s1) * seg_len(a.c2.seg_off, h.s2);
        ++mc;
      }
    }
    cnt = block_sum<kListNT, u64>(cnt, s64);
    mc = block_sum<kListNT, u32>(mc, s32);
    if (threadIdx.x == 0) {
      a.cnt[u] = cnt;
      a.mc[u] = mc;
      note_count(a, u, cnt, run_max);
    }
  }
}

// Join of one source by a group of kGroupLanes lanes (group-uniform
// control flow; the group's lanes are all active): chunks of 16 symbols of
// the shorter list, each searched by a 4-step binary search over lane
// shuffles in 16-symbol chunks of the longer list, starting from the first
// chunk that can still match (it only moves forward).  Calls f(s1, s2, m,
// j) once per chunk of the shorter list, in increasing symbol order, with
// (s1, s2) this lane's match (m: whether it has one) and j its group lane.
template <class F>
__device__ __forceinline__ void group_join(const LevelArgs &a, const Ranges &r, F &&f) {
  constexpr int G = kGroupLanes;
  const u32 j = lane_id() % G;
  const bool one_short = (r.e1 - r.b1) <= (r.e2 - r.b2);
  const u32 *ssym = one_short ? a.c1.seg_sym : a.c2.seg_sym;
  const u32 *lsym = one_short ? a.c2.seg_sym : a.c1.seg_sym;
  const u32 bs = one_short ? r.b1 : r.b2, es = one_short ? r.e1 : r.e2;
  const u32 le = one_short ? r.e2 : r.e1;
  u32 lp = one_short ? r.b2 : r.b1;
  for (u32 base = bs; base < es; base += G) {
    const u32 idx = base + j;
    const bool valid = idx < es;
    const u32 sym = valid ? ssym[idx] : 0xffffffffu;  // labels are below 2^32 - 1
    const u32 last = min(es - base, (u32)G) - 1;
    const u32 smax = __shfl(sym, (int)last, G);
    u32 fpos = 0xffffffffu;
    for (u32 c = lp; c < le; c += G) {
      const u32 len = min(le - c, (u32)G);
      const u32 lv = j < len ? lsym[c + j] : 0xffffffffu;
      if (__shfl(lv, 0, G) > smax) break;  // this chunk and later ones are past the short chunk
      u32 pos = 0;  // elements of the chunk below sym (at most 15)
#pragma unroll
      for (u32 step = G / 2; step; step >>= 1) {
        const u32 v = __shfl(lv, (int)(pos + step - 1), G);
        pos = v < sym ? pos + step : pos;
      }
      const u32 at = __shfl(lv, (int)pos, G);
      if (valid && at == sym) fpos = c + pos;
      if (__shfl(lv, (int)(len - 1), G) >= smax) {  // later short symbols start in this chunk
        lp = c;
        break;
      }
      lp = c + G;
    }
    const bool m = fpos != 0xffffffffu;
    f(one_short ? idx : fpos, one_short ? fpos : idx, m, j);
  }
}

// Sum over the kGroupLanes lanes of this lane's group.
template <class T>
__device__ __forceinline__ T group_sum(T x) {
#pragma unroll
  for (int d = kGroupLanes / 2; d > 0; d >>= 1) x += __shfl_xor(x, d, kGroupLanes);
  return x;
}

// Inclusive prefix sum over the lanes of this lane's group.
template <class T>
__device__ __forceinline__ T group_inclusive_sum(T x) {
  const u32 j = lane_id() % kGroupLanes;
#pragma unroll
  for (u32 d = 1; d < kGroupLanes; d <<= 1) {
    const T y = __shfl_up(x, d, kGroupLanes);
    if (j >= d) x += y;
  }
  return x;
}

__device__ __forceinline__ void count_group_sources(const LevelArgs &a, u32 blk, u32 nblk,
                                                    u32 &run_max) {
  constexpr u32 G = kGroupLanes;
  const u32 gi = (blk * kListNT + threadIdx.x) / G;
  const u32 ng = nblk * kListNT / G;
  const u32 n = a.st->ngrp;
  // every group of a wave runs the same number of rounds, so that the
  // wave's lanes stay together; a group past the list idles
  const u32 gw0 = gi - (threadIdx.x % kWave) / G;  // first group of this wave
  for (u32 i0 = gw0; i0 < n; i0 += ng) {
    const u32 i = i0 + (threadIdx.x % kWave) / G;
    const bool have = i < n;
    const u32 u = have ? a.grp[i] : 0u;
    u64 cnt = 0;
    u32 mc = 0;
    if (have) {
      const uint4 wr = a.wrange[a.nsrc - 1 - i];
      const Ranges r{wr.x, wr.y, wr.z, wr.w};
      group_join(a, r, [&](u32 s1, u32 s2, bool m, u32) {
        if (m) {
          cnt += (u64)seg_len(a.c1.seg_off, s1) * seg_len(a.c2.seg_off, s2);
          ++mc;
        }
      });
    }
    cnt = group_sum(cnt);
    mc = group_sum(mc);
    if (have && threadIdx.x % G == 0) {
      a.cnt[u] = cnt;
      a.mc[u] = mc;
      note_count(a, u, cnt, run_max);
    }
    // one atomic per wave for the sources the small-level kernel declines
    const u64 big_join = __ballot(have && threadIdx.x % G == 0 && cnt > kSmallPerSource);
    if (big_join && lane_id() == (u32)__builtin_ctzll(big_join))
      atomicAdd(&a.st->unfit, (u32)__popcll(big_join));
  }
}

// The listed joins: blocks [0, gg) the 16-lane joins, [gg, gg + gw) the
// wavefront joins, the rest the workgroup joins (each grid-stride over its
// list).
__global__ __launch_bounds__(kListNT) void k_count_lists(LevelArgs a, u32 gg, u32 gw) {
  __shared__ u64 s64[kListNT / kWave];
  __shared__ u32 s32[kListNT / kWave];
  __shared__ u32 s_max;
  u32 run_max = 0;
  if (blockIdx.x < gg)
    count_group_sources(a, blockIdx.x, gg, run_max);
  else if (blockIdx.x < gg + gw)
    count_wide_sources(a, blockIdx.x - gg, gw, run_max);
  else
    count_heavy_sources(a, blockIdx.x - gg - gw, gridDim.x - gg - gw, run_max, s64, s32);
  publish_max<kListNT>(a, run_max, &s_max);
}

// ---------------------------------------------------------------------------
__device__ __forceinline__ void put_match(const LevelArgs &a, u64 k, u32 s1, u32 s2, u64 rbase) {
  const u32 a1 = a.c1.seg_off[s1], n1 = a.c1.seg_off[s1 + 1] - a1;
  const u32 a2 = a.c2.seg_off[s2], n2 = a.c2.seg_off[s2 + 1] - a2;
  a.match[k] = make_uint4(a1, a2, n1, n2);
  a.mrbase[k] = rbase;
  // entries of the write tiles whose first record lies in this match
  const u64 end = rbase + (u64)n1 * n2;
  for (u64 t = (rbase + kExpandTile - 1) / kExpandTile; t * kExpandTile < end; ++t)
    a.tiles[t] = ExpandTile{k, rbase};
}

__global__ __launch_bounds__(256) void k_emit_small(LevelArgs a) {
  const u64 u = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= a.nsrc) return;
  if (a.pk[u]) return;  // product merge: no matches, no records
  const Ranges r = source_ranges(a, (u32)u);
  if (join_class(r) != kJoinThread) return;  // listed (heavy sources are never thread joins)
  u64 k = a.moff[u], rb = a.roff[u];
  intersect_serial(a.c1.seg_sym, r.b1, r.e1, a.c2.seg_sym, r.b2, r.e2, [&](u32 s1, u32 s2) {
    put_match(a, k, s1, s2, rb);
    rb += (u64)seg_len(a.c1.seg_off, s1) * seg_len(a.c2.seg_off, s2);
    ++k;
  });
}

// The listed 16-lane joins: each group writes its source's match
// descriptors in symbol order.
__global__ __launch_bounds__(256) void k_emit_group(LevelArgs a) {
  constexpr u32 G = kGroupLanes;
  const u32 gi = (blockIdx.x * blockDim.x + threadIdx.x) / G;
  const u32 ng = gridDim.x * blockDim.x / G;
  const u32 n = a.st->ngrp;
  const u32 gw0 = gi - (threadIdx.x % kWave) / G;  // first group of this wave
  const u64 gmask = 0xffffull << (lane_id() & ~(G - 1));
  for (u32 i0 = gw0; i0 < n; i0 += ng) {
    const u32 i = i0 + (threadIdx.x % kWave) / G;
    if (i >= n) continue;  // group-uniform; shuffles stay within groups
    const u32 u = a.grp[i];  // never a product source
    const uint4 wr = a.wrange[a.nsrc - 1 - i];
    const Ranges r{wr.x, wr.y, wr.z, wr.w};
    u64 k = a.moff[u], rb = a.roff[u];
    group_join(a, r, [&](u32 s1, u32 s2, bool m, u32) {
      const u64 prod = m ? (u64)seg_len(a.c1.seg_off, s1) * seg_len(a.c2.seg_off, s2) : 0;
      const u64 fm = __ballot(m) & gmask;
      const u64 incl = group_inclusive_sum(prod);
      const u64 total = __shfl(incl, (int)(G - 1), G);
      if (m) put_match(a, k + count_below(fm), s1, s2, rb + incl - prod);
      k += (u64)__popcll(fm);
      rb += total;
    });
  }
}

__global__ __launch_bounds__(256) void k_emit_wide(LevelArgs a) {
  const u32 gw = (blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const u32 nw = gridDim.x * blockDim.x / kWave;
  const u32 n = a.st->nwide;
  for (u32 i = gw; i < n; i += nw) {
    const u32 u = a.wide[i];
    if (a.pk[u]) continue;  // product merge
    const uint4 wr = a.wrange[i];
    const Ranges r{wr.x, wr.y, wr.z, wr.w};
    const bool one_short = (r.e1 - r.b1) <= (r.e2 - r.b2);
    const u32 bs = one_short ? r.b1 : r.b2, es = one_short ? r.e1 : r.e2;
    u64 k = a.moff[u], rb = a.roff[u];
    u32 lp = one_short ? r.b2 : r.b1;
    for (u32 base = bs; base < es; base += kWave) {
      const Hit h = wave_probe(a, r, one_short, base, es, lp);
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
    if (a.pk[u]) continue;  // product merge
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

// Records are written once and read once by the merge, long after they
// have left the caches at the sizes that matter: streaming stores of kRun
// consecutive records per lane (the lanes of a wave write consecutive runs,
// so every pair of vector stores of a wave covers one contiguous span).
constexpr int kRun = kExpandIT;
typedef u32 u32x4 __attribute__((ext_vector_type(4)));
typedef u64 u64x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void store_run(u32 *p, const u32 (&k)[kRun]) {
#pragma unroll
  for (int i = 0; i < kRun; i += 4) {
    const u32x4 v = {k[i], k[i + 1], k[i + 2], k[i + 3]};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(p + i));
  }
}
__device__ __forceinline__ void store_run(u64 *p, const u64 (&k)[kRun]) {
#pragma unroll
  for (int i = 0; i < kRun; i += 2) {
    const u64x2 v = {k[i], k[i + 1]};
    __builtin_nontemporal_store(v, reinterpret_cast<u64x2 *>(p + i));
  }
}
__device__ __forceinline__ void store_run(float *p, const float (&w)[kRun]) {
#pragma unroll
  for (int i = 0; i < kRun; i += 4) {
    const f32x4 v = {w[i], w[i + 1], w[i + 2], w[i + 3]};
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(p + i));
  }
}

// Arc j of a CSR arc array.  With NARROW, j < 2^29 and the byte offset is a
// 32-bit value added to the array base (one address operation per load).
template <bool NARROW>
__device__ __forceinline__ uint2 load_arc(const uint2 *arcs, u32 j) {
  if (NARROW) return *reinterpret_cast<const uint2 *>(reinterpret_cast<const char *>(arcs) + (j << 3));
  return arcs[j];
}

// ---------------------------------------------------------------------------
// Arc-pair write pass.  Workgroup b produces the records of write tiles
// kExpandGroup*b .. kExpandGroup*(b+1) - 1: the matches overlapping them are
// staged in LDS (all tiles at once when they fit, else one tile after the
// other) with a bitmap of their first records, so that the match holding a
// record is a prefix popcount away.  Lane l of wave w writes the run of kRun
// consecutive records starting at w*64*kRun + l*kRun of the group: it finds
// the match of the run's first record, its offset t in the match gives
// (i, j) = divmod(t, n2) (M1 arc i, M2 arc j of the match), and the next
// records step through the match and into the following ones.  All arc
// loads of the run are issued before any is used, and the records are
// stored last, so loads are not queued behind the wave's own stores.
// Record = (part1 << b2 | part2, p1 * p2).
constexpr u32 kSpanRecs = kExpandNT * kExpandIT;  // records per workgroup
constexpr u32 kSpanWords = kSpanRecs / 32;         // bitmap words
static_assert(kSpanWords == 2 * kWave, "two bitmap words per lane of one wave");
static_assert(kExpandTile % kExpandNT == 0, "whole staging rounds");
static_assert(kRun % 4 == 0, "runs of whole 16-byte stores");

template <class KT, bool NARROW>
__global__ __launch_bounds__(kExpandNT) void k_expand(const uint4 *match, const u64 *mrbase, u64 M,
                                                      u64 R, const uint2 *arcs1,
                                                      const uint2 *arcs2, int b2, KT *rec_key,
                                                      float *rec_w, const ExpandTile *tiles,
                                                      u64 ntiles, u32 *err) {
  __shared__ u32 s_rel[kExpandTile + 1];  // first record of each match, relative; sentinel
  __shared__ u32 s_a1[kExpandTile];       // first M1 arc of the match
  __shared__ u32 s_a2[kExpandTile];       // first M2 arc
  __shared__ u32 s_n2[kExpandTile];       // M2 arcs of the match
  __shared__ u32 s_bits[kSpanWords];      // bit r: a match starts at relative record r
  __shared__ u32 s_pre[kSpanWords];       // set bits in the words before
  constexpr u32 kSpan = kWave * kRun;     // records per wave
  constexpr u32 kWavesPerTile = (u32)(kExpandTile / kSpan);
  constexpr int kStage = (int)(kExpandTile / kExpandNT);
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const u64 g0 = (u64)blockIdx.x * kExpandGroup;
  const u64 ng = min(kExpandGroup, ntiles - g0);
  const u64 r0 = g0 * kExpandTile;
  // matches of tile t: k0(t) .. kend(t) - 1
  auto kend_of = [&](u64 t) -> u64 {
    if (t + 1 >= ntiles) return M;
    const ExpandTile nx = tiles[t + 1];
    return nx.base0 == (t + 1) * kExpandTile ? nx.k0 : nx.k0 + 1;
  };
  const ExpandTile ta = tiles[g0];
  const u64 gend = kend_of(g0 + ng - 1);
  // one staging for the whole group when its matches fit, else per tile
  const bool one = gend - ta.k0 <= kExpandTile;
  const u32 passes = one ? 1u : (u32)ng;
  for (u32 pass = 0; pass < passes; ++pass) {
    const ExpandTile ti = one ? ta : tiles[g0 + pass];
    const u64 kend = one ? gend : kend_of(g0 + pass);
    const u64 rs = one ? r0 : r0 + pass * kExpandTile;  // record origin of s_rel
    const u64 k0 = ti.k0, nm = kend - ti.k0;
    if (kend <= k0 || kend > M || nm > kExpandTile) {  // impossible: >= 1 record per match
      if (threadIdx.x == 0) set_error(err, kErrBounds);
      return;
    }
    if (pass) __syncthreads();  // previous tile's LDS fully read
    if (threadIdx.x < kSpanWords) s_bits[threadIdx.x] = 0;
    if (threadIdx.x == 0) s_rel[nm] = 0xffffffffu;  // no record reaches it
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kStage; ++q) {
      if ((u64)q * kExpandNT >= nm) break;  // uniform
      const u32 i = threadIdx.x + q * kExpandNT;
      const u64 k = k0 + min<u64>(i, nm - 1);  // in bounds
      const u64 rb = mrbase[k];
      const uint4 mm = match[k];
      if (i < nm) {
        // matches start inside the staged span, match k0 at or before it
        const u32 rel = i == 0 ? 0u : (u32)(rb - rs);
        s_rel[i] = rel;
        s_a1[i] = mm.x;
        s_a2[i] = mm.y;
        s_n2[i] = mm.w;
        atomicOr(&s_bits[rel >> 5], 1u << (rel & 31));
      }
    }
    __syncthreads();
    if (w == 0) {
      const u32 c0 = __popc(s_bits[2 * lane]), c1 = __popc(s_bits[2 * lane + 1]);
      const u32 inc = wave_inclusive_sum(c0 + c1);
      s_pre[2 * lane] = inc - c0 - c1;
      s_pre[2 * lane + 1] = inc - c1;
    }
    __syncthreads();
    if (!one && w / kWavesPerTile != pass) continue;

    // 1. M1 / M2 arc index of every record of the run (in bounds even for
    //    records past R: those repeat the run's first record, whose match is
    //    match 0 when the run is empty)
    const u64 rfirst = r0 + w * kSpan + lane * kRun;
    const u32 cnt = rfirst < R ? (u32)min<u64>(kRun, R - rfirst) : 0u;
    u32 p = cnt ? (u32)(rfirst - rs) : 0u;
    const u32 wd = p >> 5;
    u32 mi = s_pre[wd] + __popc(s_bits[wd] & ((2u << (p & 31)) - 1u)) - 1u;
    u32 a1 = s_a1[mi], a2 = s_a2[mi], n2 = s_n2[mi], nxt = s_rel[mi + 1];
    const u64 t = !cnt ? 0 : mi == 0 ? rfirst - ti.base0 : (u64)(p - s_rel[mi]);
    u32 i1, i2;
    if (t < (1ull << 32)) {
      const u32 tt = (u32)t;
      i1 = tt / n2;
      i2 = tt - i1 * n2;
    } else {
      const u64 q = t / n2;
      i1 = (u32)q;
      i2 = (u32)(t - q * n2);
    }
    u32 ix1[kRun], ix2[kRun];
    ix1[0] = a1 + i1;
    ix2[0] = a2 + i2;
#pragma unroll
    for (int j = 1; j < kRun; ++j) {
      ++p;
      ++i2;
      const bool wrap = i2 == n2;
      i2 = wrap ? 0u : i2;
      i1 += wrap ? 1u : 0u;
      if (p == nxt && (u32)j < cnt) {  // record j opens the next match
        ++mi;
        a1 = s_a1[mi];
        a2 = s_a2[mi];
        n2 = s_n2[mi];
        nxt = s_rel[mi + 1];
        i1 = i2 = 0;
      }
      const bool v = (u32)j < cnt;
      ix1[j] = v ? a1 + i1 : ix1[0];
      ix2[j] = v ? a2 + i2 : ix2[0];
    }
    // 2. every arc load of the run in flight at once
    uint2 A1[kRun], A2[kRun];
#pragma unroll
    for (int j = 0; j < kRun; ++j) {
      A1[j] = load_arc<NARROW>(arcs1, ix1[j]);
      A2[j] = load_arc<NARROW>(arcs2, ix2[j]);
    }
    // 3. records, stored last (both branches use every loaded arc, so the
    //    loads stay ahead of them)
    KT key[kRun];
    float wt[kRun];
#pragma unroll
    for (int j = 0; j < kRun; ++j) {
      key[j] = (KT)(((u64)A1[j].x << b2) | (u64)A2[j].x);
      wt[j] = __uint_as_float(A1[j].y) * __uint_as_float(A2[j].y);
    }
    if (cnt == (u32)kRun) {
      store_run(rec_key + rfirst, key);
      store_run(rec_w + rfirst, wt);
    } else {
#pragma unroll
      for (int j = 0; j < kRun; ++j) {
        if ((u32)j < cnt) {
          rec_key[rfirst + j] = key[j];
          rec_w[rfirst + j] = wt[j];
        }
      }
    }
  }
}

}  // namespace

// Grids of the wavefront and workgroup joins: at most one wave (block) per
// listed source, whose number is bounded by the frontier before the count
// and known exactly after it.
static unsigned wide_grid(u64 n) { return (unsigned)std::min<u64>(2048, ceil_div(n, 256 / kWave)); }
static unsigned heavy_grid(u64 n) { return (unsigned)std::min<u64>(512, n); }

// Workgroups of each list kernel when the lists are expected empty.
constexpr unsigned kLeanGrid = 64;

void launch_count(const LevelArgs &a, hipStream_t s, bool lean) {
  const unsigned g = (unsigned)ceil_div(a.nsrc, kCountNT);
  hipLaunchKernelGGL(k_count_small, dim3(g), dim3(kCountNT), 0, s, a);
  // 16-lane joins: at most one group per source, at most as many waves as
  // the chip holds (they loop over the list); wide: at most one wave per
  // source (1024 blocks of 8 waves at most); heavy: one block per source
  // (512 blocks at most)
  const u64 n = a.nsrc;
  unsigned gg = (unsigned)std::min<u64>((u64)compute_units() * 4,
                                        ceil_div(n, kListNT / kGroupLanes));
  unsigned gw = (unsigned)std::min<u64>(1024, ceil_div(n, kListNT / kWave));
  unsigned gh = (unsigned)std::min<u64>(512, n);
  if (lean) {
    gg = std::min(gg, kLeanGrid);
    gw = std::min(gw, kLeanGrid);
    gh = std::min(gh, kLeanGrid);
  }
  hipLaunchKernelGGL(k_count_lists, dim3(gg + gw + gh), dim3(kListNT), 0, s, a, gg, gw);
}

void launch_emit(const LevelArgs &a, u32 nwide, u32 nheavy, u32 ngrp, hipStream_t s) {
  const unsigned g = (unsigned)ceil_div(a.nsrc, 256);
  hipLaunchKernelGGL(k_emit_small, dim3(g), dim3(256), 0, s, a);
  if (ngrp) {
    const unsigned gg = (unsigned)std::min<u64>((u64)compute_units() * 8,
                                                ceil_div((u64)ngrp, 256 / kGroupLanes));
    hipLaunchKernelGGL(k_emit_group, dim3(gg), dim3(256), 0, s, a);
  }
  if (nwide) hipLaunchKernelGGL(k_emit_wide, dim3(wide_grid(nwide)), dim3(256), 0, s, a);
  if (nheavy) hipLaunchKernelGGL(k_emit_heavy, dim3(heavy_grid(nheavy)), dim3(kHeavyNT), 0, s, a);
}

void launch_expand(const uint4 *match, const u64 *mrbase, u64 M, u64 R, const CsrView &c1,
                   const CsrView &c2, int b2, bool wide_keys, void *rec_key, float *rec_w,
                   ExpandTile *tiles, u32 *err, hipStream_t s) {
  if (R == 0) return;
  const u64 g = ceil_div(R, kExpandTile);
  if (g >= (1ull << 31)) throw Error(FSTC_ERR_CAPACITY, "level too large for one launch");
  const unsigned gw = (unsigned)ceil_div(g, kExpandGroup);
  // 32-bit byte offsets into the arc arrays when both hold fewer than 2^29 arcs
  const bool narrow = std::max(c1.num_arcs, c2.num_arcs) < (1ull << 29);
  auto go = [&](auto kt, auto nar) {
    using KT = decltype(kt);
    hipLaunchKernelGGL((k_expand<KT, decltype(nar)::value>), dim3(gw), dim3(kExpandNT), 0, s, match,
                       mrbase, M, R, c1.arcs, c2.arcs, b2, (KT *)rec_key, rec_w, tiles, g, err);
  };
  if (wide_keys) {
    if (narrow) go(u64{}, std::true_type{}); else go(u64{}, std::false_type{});
  } else {
    if (narrow) go(u32{}, std::true_type{}); else go(u32{}, std::false_type{});
  }
}

}  // namespace fstc
