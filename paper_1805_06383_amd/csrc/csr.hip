// Device build of the (state, inner symbol) transducer layout.
//
// Section 3.3 stores a transducer as offsets R[q m + b] into arrays of
// targets T, outer symbols O and weights P, with arcs sorted by inner symbol,
// and section 3.4 sorts on the host before copying to the device.  A dense
// R of |Q| m + 1 entries does not fit large inputs (10^6 states x 10^5 inner
// symbols), so the layout here is two-level: per state a run of segments,
// one per distinct inner symbol present, each pointing at its arcs.  The
// sort runs on the device (radix_sort.hip).
//
// Each arc also carries the rank of its (target, outer symbol) pair among
// the distinct pairs of its source state ("part").  A composed arc's
// (target pair, input, output) is then fixed by the two parts it joins, so
// the merge sorts short part-rank keys instead of full labels.
#include "internal.hpp"
#include "radix_rank.hpp"

#include <atomic>
#include <initializer_list>

namespace fstc {
namespace {

constexpr int kNT = 256;

inline unsigned grid_for(u64 n) { return (unsigned)std::max<u64>(1, std::min<u64>(ceil_div(n, kNT), 1u << 20)); }

__global__ void k_csr_pack(const u32 *src, const u32 *dst, const u32 *il, const u32 *ol, u64 n,
                           u32 nq, u32 nis, u32 nos, int by_output, int bq, int bo, int bi,
                           u64 *kp, u64 *kc, u32 *v1, u32 *v2, u32 *err) {
  for (u64 e = (u64)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (u64)gridDim.x * blockDim.x) {
    u32 s = src[e], d = dst[e], a = il[e], b = ol[e];
    if (s >= nq || d >= nq || a >= nis || b >= nos) {
      set_error(err, kErrBadArc);
      s = d = a = b = 0;
    }
    const u64 inner = by_output ? b : a;
    const u64 outer = by_output ? a : b;
    kp[e] = ((u64)s << (bq + bo)) | ((u64)d << bo) | outer;
    kc[e] = ((u64)s << bi) | inner;
    v1[e] = (u32)e;
    v2[e] = (u32)e;
  }
}

// keys[i] = kc[perm[i]], vals[i] = perm[i]: the segment keys of the arcs in
// part order.
__global__ void k_gather_keys(const u64 *kc, const u32 *perm, u64 n, u64 *keys, u32 *vals) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x) {
    const u32 e = perm[i];
    keys[i] = kc[e];
    vals[i] = e;
  }
}

__global__ void k_head_flags(const u64 *keys, u64 n, u32 *flags) {
  for (u64 k = (u64)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (u64)gridDim.x * blockDim.x)
    flags[k] = (k == 0 || keys[k] != keys[k - 1]) ? 1u : 0u;
}

__global__ void k_parts(const u64 *kp, const u32 *perm, const u32 *flags, const u32 *ex, u64 n,
                        int bq, int bo, uint2 *parts, u32 *part_state, u32 *arc_part_global) {
  const u64 dmask = bq ? ((1ull << bq) - 1) : 0, omask = bo ? ((1ull << bo) - 1) : 0;
  for (u64 k = (u64)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (u64)gridDim.x * blockDim.x) {
    const u32 g = ex[k] + flags[k] - 1u;
    const u64 key = kp[k];
    if (flags[k]) {
      parts[g] = make_uint2((u32)((key >> bo) & dmask), (u32)(key & omask));
      part_state[g] = (u32)(key >> (bq + bo));
    }
    arc_part_global[perm[k]] = g;
  }
}

// row[q] = first index i in [0, K] with state[i] >= q, for q in [0, nq].
__global__ void k_state_offsets(const u32 *state, u64 K, u32 nq, u32 *row) {
  for (u64 q = (u64)blockIdx.x * blockDim.x + threadIdx.x; q <= nq; q += (u64)gridDim.x * blockDim.x)
    row[q] = (u32)lower_bound_dev<u32>(state, K, (u32)q);
}

__global__ void k_max_gap(const u32 *base, u32 nq, u64 *out) {
  u32 m = 0;
  for (u64 q = (u64)blockIdx.x * blockDim.x + threadIdx.x; q < nq; q += (u64)gridDim.x * blockDim.x)
    m = max(m, base[q + 1] - base[q]);
  m = wave_max(m);
  if (lane_id() == 0 && m) atomicMax((unsigned long long *)out, (unsigned long long)m);
}

__global__ void k_segments(const u64 *kc, const u32 *perm, const u32 *flags, const u32 *ex, u64 n,
                           int bi, const u32 *arc_part_global, const u32 *part_base,
                           const float *w, u32 *seg_sym, u32 *seg_off, u32 *seg_state,
                           uint2 *arcs) {
  const u64 imask = bi ? ((1ull << bi) - 1) : 0;
  for (u64 k = (u64)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (u64)gridDim.x * blockDim.x) {
    const u64 key = kc[k];
    const u32 st = (u32)(key >> bi);
    const u32 sidx = ex[k] + flags[k] - 1u;
    if (flags[k]) {
      seg_sym[sidx] = (u32)(key & imask);
      seg_off[sidx] = (u32)k;
      seg_state[sidx] = st;
    }
    if (k == n - 1) seg_off[sidx + 1] = (u32)n;
    const u32 e = perm[k];
    arcs[k] = make_uint2(arc_part_global[e] - part_base[st], __float_as_uint(w[e]));
  }
}

__global__ void k_copy_count(const u32 *src, u64 *dst) { *dst = *src; }

// Wave per state; lane l checks segments row[q] + l, + 64, ...: a segment
// of more arcs than kProdParts, or whose arcs' parts are not all distinct
// (a 64-bit mask of the parts), flags the state (bit 0).  For the other
// states the word also summarises the arcs' weights (kCellSpecial: a
// non-finite or subnormal weight; the largest biased float32 exponent of a
// nonzero weight at kCellEmaxShift, the smallest at kCellEminShift) and
// marks a state of P parts, S segments and P S arcs kCellDense (no segment
// has more than P arcs, so each has exactly P), and kCellIdent as well when
// arc i of every segment has part i; kCellContig when its segment symbols
// are consecutive (the first plus the segment index).
// The arcs' weight words as an array of their own (the product merge's
// operand loads then fetch weights alone), zeros after the last arc.
// One launch: blocks [0, gw) copy the arcs' weight words into wts (zeros
// after the last arc); the others set the cell flags, a wave per state.
// Workgroup blk of nblk.
__device__ __forceinline__ void cell_flags_body(const u32 *row, const u32 *seg_sym,
                                                const u32 *seg_off, const uint2 *arcs,
                                                const u32 *part_base, u32 nq, u32 *flag,
                                                u64 narcs, u32 *wts, u32 gw, u32 blk, u32 nblk) {
  if (blk < gw) {
    for (u64 j = (u64)blk * blockDim.x + threadIdx.x; j < narcs + kArcTail;
         j += (u64)gw * blockDim.x)
      wts[j] = j < narcs ? arcs[j].y : 0u;
    return;
  }
  const u32 lane = lane_id();
  const u64 nw = (u64)(nblk - gw) * blockDim.x / kWave;
  for (u64 q = ((u64)(blk - gw) * blockDim.x + threadIdx.x) / kWave; q < nq; q += nw) {
    bool bad = part_base[q + 1] - part_base[q] > kProdParts, special = false, shuffled = false;
    bool gap = false;  // a symbol other than the first plus its segment index
    u32 emax = 0, emin = 255;
    if (!bad) {
      const u32 sym0 = row[q] < row[q + 1] ? seg_sym[row[q]] : 0u;
      for (u32 sg = row[q] + lane; sg < row[q + 1]; sg += kWave) {
        gap |= seg_sym[sg] != sym0 + (sg - row[q]);
        const u32 a0 = seg_off[sg], n = seg_off[sg + 1] - a0;
        if (n > kProdParts) {
          bad = true;
          continue;
        }
        u64 m = 0;
        auto take = [&](const uint2 x, u32 i) {
          m |= 1ull << (x.x & 63u);
          shuffled |= x.x != i;
          const u32 mag = x.y & 0x7fffffffu, e = mag >> 23;
          special |= e == 255u || (e == 0u && mag != 0u);
          if (mag) {
            emax = max(emax, e);
            emin = min(emin, e);
          }
        };
        // the segment's first kArcTail arcs loaded at once (the arc array
        // has kArcTail spare entries after its last arc), the rest one by one
        uint2 x[kArcTail];
#pragma unroll
        for (u32 i = 0; i < kArcTail; ++i) x[i] = arcs[a0 + i];
#pragma unroll
        for (u32 i = 0; i < kArcTail; ++i)
          if (i < n) take(x[i], i);
        for (u32 i = kArcTail; i < n; ++i) take(arcs[a0 + i], i);
        bad |= (u32)__popcll(m) != n;
      }
    }
    const bool any = __ballot(bad) != 0, spec = __ballot(special) != 0;
    const bool ident = __ballot(shuffled) == 0, contig = __ballot(gap) == 0;
    emax = wave_max(emax);
    emin = 255u - wave_max(255u - emin);
    const u32 P = part_base[q + 1] - part_base[q], r0 = row[q], r1 = row[q + 1];
    const bool dense = (u64)(seg_off[r1] - seg_off[r0]) == (u64)P * (r1 - r0);
    if (lane == 0)
      flag[q] = any ? kCellBad
                    : (spec ? kCellSpecial : 0u) | (dense ? kCellDense : 0u) |
                          (dense && ident ? kCellIdent : 0u) | (contig ? kCellContig : 0u) |
                          (emax << kCellEmaxShift) | (emin << kCellEminShift);
  }
}

__global__ void k_cell_flags(const u32 *row, const u32 *seg_sym, const u32 *seg_off,
                             const uint2 *arcs, const u32 *part_base, u32 nq, u32 *flag, u64 narcs,
                             u32 *wts, u32 gw) {
  cell_flags_body(row, seg_sym, seg_off, arcs, part_base, nq, flag, narcs, wts, gw, blockIdx.x,
                  gridDim.x);
}

// a[i] = v for i in [*count, n).
__global__ void k_fill_tail(u32 *a, const u32 *count, u64 n, u32 v) {
  const u64 c = *count;
  for (u64 i = c + (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x)
    a[i] = v;
}

// ---------------------------------------------------------------------------
// Per-state build.  After one stable sort of the arcs by source state, each
// state's arcs (in input order) are sorted inside one workgroup: by
// (target, outer symbol) to rank its parts, and then, in that part order,
// stably by inner symbol to lay out its segments (so a segment's arcs are
// ordered by part).  A state's parts and segments are first written at
// its own arc offset (a state has at most as many of each as arcs); a scan
// of the per-state counts then gives part_base and row, and a last pass
// moves them to their final places.  Same layout as the global sorts.

// Size classes of the per-state build: groups of 16 and of 64 lanes of a
// wavefront per state up to 16 and kWave arcs, then workgroups of 256
// threads with 1 and 4 items per thread, and of 1024 threads with 8 items
// per thread (several tiles per sort pass beyond 8192 arcs).
constexpr int kLocClasses = 5;
__host__ __device__ constexpr u32 loc_class(u32 d) {
  return d <= 16u ? 0u : d <= (u32)kWave ? 1u : d <= 256u ? 2u : d <= 1024u ? 3u : 4u;
}

struct LocalArgs {
  const u64 *skey;     // [n] source state of each position (sorted)
  const u32 *order;    // [n] arc index at each position (input order within a state)
  const u32 *abase;    // [nq + 1] first position of each state
  const u32 *dst, *inner, *outer;
  const float *w;
  int bo, bp, bi;      // outer-symbol bits, part-key bits, inner-symbol bits
  u64 *ka, *kb;        // [n] sort keys (two buffers)
  u32 *ia, *ib;        // [n] element numbers within the state (two buffers)
  u32 *part_of;        // [n] part rank of element i of a state at abase + i
  uint2 *ptmp;         // [n] parts of a state at its arc offset
  u32 *ssym, *soff;    // [n] segments of a state at its arc offset
  uint2 *arcs;         // [n] the CSR arcs
  u32 *pcnt, *scnt;    // [nq] parts / segments per state
  u64 *maxp;           // largest part count
};

// Raises *m to v.  Same-address atomics serialise, so the current value is
// read first and only a larger v issues one (a handful per launch).
__device__ __forceinline__ void note_max(u64 *m, u64 v) {
  if (v > __hip_atomic_load(m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
    atomicMax((unsigned long long *)m, (unsigned long long)v);
}

// Stable LSD sort of the d keys at a0 (8-bit digits, `bits` key bits) in
// tiles of NT * IT elements; bucket bases come from a histogram over the
// state when it spans more than one tile.  On return kin / iin hold the
// sorted keys and element numbers.
template <int NT, int IT>
__device__ void local_sort(u64 *&kin, u32 *&iin, u64 *&kout, u32 *&iout, u32 a0, u32 d,
                           int bits, u32 *s_cnt, u32 *s_base, u32 *s_tmp, u32 *s_run) {
  constexpr u32 kTile = NT * IT;
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const bool multi = d > kTile;
  for (int shift = 0; shift < bits; shift += 8) {
    const int db = min(8, bits - shift);
    const u32 mask = (1u << db) - 1u;
    if (multi) {
      if (threadIdx.x < 256) s_run[threadIdx.x] = 0;
      __syncthreads();
      for (u32 i = threadIdx.x; i < d; i += NT)
        atomicAdd(&s_run[(u32)(kin[a0 + i] >> shift) & mask], 1u);
      __syncthreads();
      u32 tot;
      const u32 ex = block_exclusive_sum<NT, u32>(threadIdx.x < 256 ? s_run[threadIdx.x] : 0u,
                                                  s_tmp, &tot);
      __syncthreads();
      if (threadIdx.x < 256) s_run[threadIdx.x] = ex;
      __syncthreads();
    }
    for (u32 t0 = 0; t0 < d; t0 += kTile) {
      u64 key[IT];
      u32 val[IT], dig[IT], rid[IT];
      u32 valid = 0;
#pragma unroll
      for (int j = 0; j < IT; ++j) {
        const u32 i = t0 + w * (kWave * IT) + j * kWave + lane;
        const bool v = i < d;
        valid |= (v ? 1u : 0u) << j;
        key[j] = v ? kin[a0 + i] : 0;
        val[j] = v ? iin[a0 + i] : 0;
        dig[j] = (u32)(key[j] >> shift) & mask;
      }
      block_rank_digits<NT, IT>(dig, valid, db, rid, s_cnt, s_base, s_tmp);
#pragma unroll
      for (int j = 0; j < IT; ++j) {
        if (!((valid >> j) & 1u)) continue;
        const u32 pos = (multi ? s_run[dig[j]] : s_base[dig[j]]) + rid[j];
        kout[a0 + pos] = key[j];
        iout[a0 + pos] = val[j];
      }
      if (multi) {
        __syncthreads();  // every s_run read of this tile is done
        const u32 nv = min(d - t0, kTile);
        const u32 t = threadIdx.x;
        if (t < 256) s_run[t] += (t + 1 < 256u ? s_base[t + 1] : nv) - s_base[t];
        __syncthreads();
      }
    }
    __syncthreads();  // kout complete before it is read
    u64 *tk = kin; kin = kout; kout = tk;
    u32 *tv = iin; iin = iout; iout = tv;
  }
}

// Run heads of the sorted keys at a0: calls f(i, run, is_head) for every
// position i with its run number; returns the number of runs.
template <int NT, class F>
__device__ u32 local_runs(const u64 *k, u32 a0, u32 d, u32 *s_tmp, F &&f) {
  u32 carry = 0;
  for (u32 t0 = 0; t0 < d; t0 += NT) {
    const u32 i = t0 + threadIdx.x;
    const bool v = i < d;
    const bool head = v && (i == 0 || k[a0 + i] != k[a0 + i - 1]);
    u32 tot;
    const u32 ex = block_exclusive_sum<NT, u32>(head ? 1u : 0u, s_tmp, &tot);
    if (v) f(i, carry + ex + (head ? 1u : 0u) - 1u, head);
    carry += tot;
  }
  return carry;
}

// One workgroup per listed state: workgroup blk of nblk (stride over the
// list).
template <int NT, int IT>
__device__ __forceinline__ void state_local(const LocalArgs &a, const u32 *list,
                                            const u32 *list_len, u32 blk, u32 nblk) {
  __shared__ u32 s_cnt[(NT / kWave) * 256];
  __shared__ u32 s_base[256];
  __shared__ u32 s_run[256];
  __shared__ u32 s_tmp[NT / kWave];
  const u32 nlist = *list_len;
  const u64 omask = a.bo ? ((1ull << a.bo) - 1) : 0;
  for (u32 li = blk; li < nlist; li += nblk) {
    const u32 q = list[li];
    const u32 a0 = a.abase[q], d = a.abase[q + 1] - a0;
    // parts: ranks of the distinct (target, outer) keys
    for (u32 i = threadIdx.x; i < d; i += NT) {
      const u32 e = a.order[a0 + i];
      a.ka[a0 + i] = ((u64)a.dst[e] << a.bo) | a.outer[e];
      a.ia[a0 + i] = i;
    }
    __syncthreads();
    u64 *kin = a.ka, *kout = a.kb;
    u32 *iin = a.ia, *iout = a.ib;
    local_sort<NT, IT>(kin, iin, kout, iout, a0, d, a.bp, s_cnt, s_base, s_tmp, s_run);
    const u32 np = local_runs<NT>(kin, a0, d, s_tmp, [&](u32 i, u32 r, bool head) {
      a.part_of[a0 + iin[a0 + i]] = r;
      if (head) {
        const u64 k = kin[a0 + i];
        a.ptmp[a0 + r] = make_uint2((u32)(k >> a.bo), (u32)(k & omask));
      }
    });
    __syncthreads();  // part_of complete
    // segments: stable sort by inner symbol of the elements in part order,
    // so that the arcs of a segment are ordered by part (iin holds the
    // elements in part order; kout / iout are free)
    for (u32 i = threadIdx.x; i < d; i += NT) {
      const u32 el = iin[a0 + i];
      kout[a0 + i] = a.inner[a.order[a0 + el]];
      iout[a0 + i] = el;
    }
    __syncthreads();
    {
      u64 *tk = kin; kin = kout; kout = tk;
      u32 *tv = iin; iin = iout; iout = tv;
    }
    local_sort<NT, IT>(kin, iin, kout, iout, a0, d, a.bi, s_cnt, s_base, s_tmp, s_run);
    const u32 ns = local_runs<NT>(kin, a0, d, s_tmp, [&](u32 i, u32 r, bool head) {
      const u32 el = iin[a0 + i];
      a.arcs[a0 + i] = make_uint2(a.part_of[a0 + el], __float_as_uint(a.w[a.order[a0 + el]]));
      if (head) {
        a.ssym[a0 + r] = (u32)kin[a0 + i];
        a.soff[a0 + r] = a0 + i;
      }
    });
    if (threadIdx.x == 0) {
      a.pcnt[q] = np;
      a.scnt[q] = ns;
      note_max(a.maxp, np);
    }
    __syncthreads();  // shared arrays free for the next state
  }
}

// One workgroup per listed state of at most NT IT arcs, every step in LDS:
// the same two stable sorts and runs as state_local, with the state's arcs
// gathered once (order, then targets, symbols and weights) and only the
// results written to memory.  Items are wave-striped as block_rank_digits
// takes them: item j of lane l of wave w is element w (64 IT) + 64 j + l.
template <int IT>
struct LdsState {
  static constexpr int T = 256 * IT;
  u64 key[T];     // sort keys by position
  u32 el[T];      // element at each position
  u32 inner[T];   // per element: inner symbol, weight bits, part rank
  u32 wbits[T];
  u32 part[T];
  u32 cnt[(256 / kWave) * 256];  // block_rank_digits
  u32 base[256];
  u32 tmp[256 / kWave];
  u32 wtot[256 / kWave];
};

template <int IT>
__device__ __forceinline__ void lds_sort(LdsState<IT> &S, u64 (&key)[IT], u32 (&el)[IT],
                                         u32 valid, int bits) {
  constexpr u32 NT = 256;
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  for (int shift = 0; shift < bits; shift += 8) {
    const int db = min(8, bits - shift);
    const u32 mask = (1u << db) - 1u;
    u32 dig[IT], rid[IT];
#pragma unroll
    for (int j = 0; j < IT; ++j) dig[j] = (u32)(key[j] >> shift) & mask;
    block_rank_digits<NT, IT>(dig, valid, db, rid, S.cnt, S.base, S.tmp);
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      if ((valid >> j) & 1u) {
        const u32 pos = S.base[dig[j]] + rid[j];
        S.key[pos] = key[j];
        S.el[pos] = el[j];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const u32 i = w * (kWave * IT) + j * kWave + lane;
      if ((valid >> j) & 1u) {
        key[j] = S.key[i];
        el[j] = S.el[i];
      }
    }
    __syncthreads();  // S.key / S.el free for the next pass
  }
}

// Run heads of the keys in position order: rank[j] = the number of heads at
// or before item j's position, less one; returns the number of runs.  The
// sorted keys are in S.key (written here for positions of valid items).
template <int IT>
__device__ __forceinline__ u32 lds_runs(LdsState<IT> &S, const u64 (&key)[IT], u32 valid,
                                        bool (&head)[IT], u32 (&rank)[IT]) {
  constexpr u32 NW = 256 / kWave;
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const u32 i = w * (kWave * IT) + j * kWave + lane;
    if ((valid >> j) & 1u) S.key[i] = key[j];
  }
  __syncthreads();
  u32 wc = 0;
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const u32 i = w * (kWave * IT) + j * kWave + lane;
    head[j] = ((valid >> j) & 1u) && (i == 0 || S.key[i - 1] != key[j]);
    const u64 m = __ballot(head[j]);
    rank[j] = wc + count_below(m) + (head[j] ? 1u : 0u);
    wc += (u32)__popcll(m);
  }
  if (lane == 0) S.wtot[w] = wc;
  __syncthreads();
  u32 before = 0, all = 0;
#pragma unroll
  for (u32 v = 0; v < NW; ++v) {
    const u32 c = S.wtot[v];
    before += v < w ? c : 0u;
    all += c;
  }
#pragma unroll
  for (int j = 0; j < IT; ++j) rank[j] += before - 1u;
  __syncthreads();  // S.wtot and S.key reads done
  return all;
}

template <int IT>
__device__ __forceinline__ void state_lds(const LocalArgs &a, const u32 *list, const u32 *list_len,
                                          u32 blk, u32 nblk, LdsState<IT> &S) {
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const u32 nlist = *list_len;
  const u64 omask = a.bo ? ((1ull << a.bo) - 1) : 0;
  for (u32 li = blk; li < nlist; li += nblk) {
    const u32 q = list[li];
    const u32 a0 = a.abase[q], d = a.abase[q + 1] - a0;
    // the state's arcs: order, then their fields, every load issued first
    u32 valid = 0, e[IT];
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const u32 i = w * (kWave * IT) + j * kWave + lane;
      valid |= (i < d ? 1u : 0u) << j;
      e[j] = a.order[a0 + min(i, d - 1)];
    }
    u64 key[IT];
    u32 el[IT];
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const u32 i = w * (kWave * IT) + j * kWave + lane;
      const u32 t = a.dst[e[j]], o = a.outer[e[j]], in = a.inner[e[j]];
      const u32 wb = __float_as_uint(a.w[e[j]]);
      key[j] = ((u64)t << a.bo) | o;
      el[j] = i;
      if ((valid >> j) & 1u) {
        S.inner[i] = in;
        S.wbits[i] = wb;
      }
    }
    // parts: ranks of the distinct (target, outer) keys
    lds_sort<IT>(S, key, el, valid, a.bp);
    bool head[IT];
    u32 rank[IT];
    const u32 np = lds_runs<IT>(S, key, valid, head, rank);
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      if (!((valid >> j) & 1u)) continue;
      S.part[el[j]] = rank[j];
      if (head[j])
        a.ptmp[a0 + rank[j]] = make_uint2((u32)(key[j] >> a.bo), (u32)(key[j] & omask));
    }
    __syncthreads();  // S.part complete
    // segments: the elements in part order, stably by inner symbol
#pragma unroll
    for (int j = 0; j < IT; ++j) key[j] = ((valid >> j) & 1u) ? (u64)S.inner[el[j]] : 0ull;
    lds_sort<IT>(S, key, el, valid, a.bi);
    const u32 ns = lds_runs<IT>(S, key, valid, head, rank);
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      if (!((valid >> j) & 1u)) continue;
      const u32 i = w * (kWave * IT) + j * kWave + lane;
      a.arcs[a0 + i] = make_uint2(S.part[el[j]], S.wbits[el[j]]);
      if (head[j]) {
        a.ssym[a0 + rank[j]] = (u32)key[j];
        a.soff[a0 + rank[j]] = a0 + i;
      }
    }
    if (threadIdx.x == 0) {
      a.pcnt[q] = np;
      a.scnt[q] = ns;
      note_max(a.maxp, np);
    }
    __syncthreads();  // shared arrays free for the next state
  }
}

// Bitonic sort of one (key, element) pair per lane within each group of G
// lanes, ascending by key and then element number (so equal keys keep their
// element order).
template <int G>
__device__ __forceinline__ void group_sort(u64 &k, u32 &i) {
  const u32 lane = lane_id();
#pragma unroll
  for (u32 size = 2; size <= (u32)G; size <<= 1) {
#pragma unroll
    for (u32 j = size >> 1; j > 0; j >>= 1) {
      const u64 ok = __shfl_xor(k, (int)j, kWave);
      const u32 oi = __shfl_xor(i, (int)j, kWave);
      const bool up = (lane & size) == 0 || size == (u32)G;  // this run ascends
      const bool low = (lane & j) == 0;                       // lower lane of the pair
      const bool other_less = ok < k || (ok == k && oi < i);
      if ((low == up) == other_less) {
        k = ok;
        i = oi;
      }
    }
  }
}

// A group of G lanes per listed state of at most G arcs (group lane =
// element): the same two sorts as state_local, in registers; workgroup blk
// of nblk (256 threads each).
template <int G>
__device__ __forceinline__ void state_group(const LocalArgs &a, const u32 *list,
                                            const u32 *list_len, u32 blk, u32 nblk) {
  constexpr u32 kPer = kWave / G;  // states per wavefront
  const u32 lane = lane_id(), gl = lane % G, gb = lane - gl;
  const u64 gmask = (G == kWave) ? ~0ull : (((1ull << G) - 1) << gb);
  const u32 nlist = *list_len;
  const u64 omask = a.bo ? ((1ull << a.bo) - 1) : 0;
  const u32 nw = nblk * (256 / kWave);
  for (u32 wi = blk * (256 / kWave) + threadIdx.x / kWave; wi * kPer < nlist; wi += nw) {
    const u32 li = wi * kPer + lane / G;
    const u32 q = li < nlist ? list[li] : 0u;
    const u32 a0 = li < nlist ? a.abase[q] : 0u;
    const u32 d = li < nlist ? a.abase[q + 1] - a0 : 0u;
    const bool v = gl < d;
    const u32 e = v ? a.order[a0 + gl] : 0u;
    // parts
    u64 k = v ? (((u64)a.dst[e] << a.bo) | a.outer[e]) : ~0ull;
    u32 el = gl;
    group_sort<G>(k, el);
    const u64 kprev = __shfl(k, (int)(lane ? lane - 1 : 0), kWave);
    bool head = v && (gl == 0 || k != kprev);
    u64 hm = __ballot(head) & gmask;
    const u32 np = (u32)__popcll(hm);
    const u32 prank = count_below(hm) + (head ? 1u : 0u) - 1u;  // rank of sorted lane
    if (head) a.ptmp[a0 + prank] = make_uint2((u32)(k >> a.bo), (u32)(k & omask));
    // element el receives its part rank (each group holds a permutation)
    const u32 my_part = (u32)__builtin_amdgcn_ds_permute((int)((gb + el) * 4u), (int)prank);
    // segments: by inner symbol, then part, then element (the arcs of a
    // segment ordered by part); the element is the low 6 bits of the
    // tie-break word
    k = v ? (u64)a.inner[e] : ~0ull;
    el = (my_part << 6) | gl;
    group_sort<G>(k, el);
    el &= 63u;
    const u64 sprev = __shfl(k, (int)(lane ? lane - 1 : 0), kWave);
    head = v && (gl == 0 || k != sprev);
    hm = __ballot(head) & gmask;
    const u32 srank = count_below(hm) + (head ? 1u : 0u) - 1u;
    const u32 part = __shfl(my_part, (int)(gb + el), kWave);
    const u32 ee = __shfl(e, (int)(gb + el), kWave);
    if (v) {
      a.arcs[a0 + gl] = make_uint2(part, __float_as_uint(a.w[ee]));
      if (head) {
        a.ssym[a0 + srank] = (u32)k;
        a.soff[a0 + srank] = a0 + gl;
      }
    }
    if (gl == 0 && d) {
      a.pcnt[q] = np;
      a.scnt[q] = (u32)__popcll(hm);
      note_max(a.maxp, np);
    }
  }
}

// One input of the per-state build as its kernels take it.  The build runs
// one or two inputs (the two sides of a composition) in the same launches:
// workgroups [0, split) of a launch take the first input, the rest the
// second, so two short sequences of launches become one.
struct LocalJob {
  LocalArgs a;
  u64 *skey;           // [n] source state of each position (a.skey, writable)
  u32 *order;          // [n] arc index at each position (a.order, writable)
  u32 *abase;          // [nq + 1] first position of each state (a.abase, writable)
  const u32 *src, *il, *ol;  // input arcs (a.dst the targets)
  u64 n;
  u32 nq, nis, nos;
  u32 *lists;          // [kLocClasses nq] states by size class
  u32 *list_len;       // [kLocClasses] list lengths
  u64 *counts;         // [3] segments, parts, largest part count (a.maxp)
  u32 *row, *part_base, *seg_sym, *seg_off;
  uint2 *parts;
  uint4 gs;            // workgroups of the size classes 0..3 (k_loc_small)
  u32 *cell_flag, *wts;  // cell flags and weight words (k_loc_flags)
  u32 gw;              // workgroups of k_loc_flags copying the weights
  // set to `epoch` by the key pass when an arc's source state is below its
  // predecessor's (arcs not grouped by state: the state sort runs)
  u32 *unsorted;
  u32 epoch;
};
struct LocalPair {
  LocalJob j[2];
};

__device__ __forceinline__ const LocalJob &local_job(const LocalPair &p, u32 split, u32 &blk,
                                                     u32 &nblk) {
  if (blockIdx.x < split) {
    blk = blockIdx.x;
    nblk = split;
    return p.j[0];
  }
  blk = blockIdx.x - split;
  nblk = gridDim.x - split;
  return p.j[1];
}

// Sort keys (the source state) and the identity order; checks every arc's
// ids, notes arcs not grouped by state (J.unsorted), and clears the job's
// counters and list lengths.  Inputs stored state by state (as FST files
// keep them) are already in the order the stable state sort gives.
__global__ void k_loc_keys(LocalPair p, u32 split, u32 *err) {
  u32 blk, nblk;
  const LocalJob &J = local_job(p, split, blk, nblk);
  if (blk == 0) {
    if (threadIdx.x < 3) J.counts[threadIdx.x] = 0;
    if (threadIdx.x < (u32)kLocClasses) J.list_len[threadIdx.x] = 0;
  }
  bool down = false;
  for (u64 e = (u64)blk * blockDim.x + threadIdx.x; e < J.n; e += (u64)nblk * blockDim.x) {
    u32 s = J.src[e];
    down |= e > 0 && J.src[e - 1] > s;
    if (s >= J.nq || J.a.dst[e] >= J.nq || J.il[e] >= J.nis || J.ol[e] >= J.nos) {
      set_error(err, kErrBadArc);
      s = 0;
    }
    J.skey[e] = s;
    J.order[e] = (u32)e;
  }
  if (__ballot(down) != 0 && lane_id() == 0) *J.unsorted = J.epoch;
}

// First index i of the sorted keys a[0..n) with a[i] >= v (n when none),
// searched outward from the guess g: a galloping search brackets the answer,
// then a binary search finds it.  A good guess (states of even size) takes
// two loads instead of the log2(n) dependent loads of a plain binary search.
__device__ __forceinline__ u64 lower_bound_near(const u64 *a, u64 n, u64 v, u64 g) {
  g = min(g, n);
  u64 L, R;  // the answer lies in [L, R]
  if (g == n || a[g] >= v) {
    R = g;
    u64 step = 1;
    while (true) {
      if (R < step) {
        L = 0;
        break;
      }
      const u64 q = R - step;
      if (a[q] < v) {
        L = q + 1;
        break;
      }
      R = q;
      step <<= 1;
    }
  } else {
    L = g + 1;
    u64 step = 1;
    while (true) {
      const u64 q = L + step - 1;
      if (q >= n) {
        R = n;
        break;
      }
      if (a[q] >= v) {
        R = q;
        break;
      }
      L = q + 1;
      step <<= 1;
    }
  }
  while (L < R) {
    const u64 mid = (L + R) >> 1;
    if (a[mid] < v) L = mid + 1;
    else R = mid;
  }
  return L;
}

// First position of every state in the sorted state keys; states with arcs
// are listed for the per-state kernels by size class (lists[c nq ..],
// loc_class); states without arcs get zero counts.  One thread per state
// and one for nq; the searches start from the position of a state of
// average size.
__global__ __launch_bounds__(256) void k_loc_lists(LocalPair p, u32 split) {
  __shared__ u32 s_n[kLocClasses], s_base[kLocClasses];
  u32 blk, nblk;
  const LocalJob &J = local_job(p, split, blk, nblk);
  const u32 lane = lane_id(), nq = J.nq;
  const u64 q = (u64)blk * blockDim.x + threadIdx.x;
  if (threadIdx.x < (u32)kLocClasses) s_n[threadIdx.x] = 0;
  u32 d = 0;
  if (q <= nq) {
    const u64 lo = lower_bound_near(J.skey, J.n, q, q * J.n / nq);
    J.abase[q] = (u32)lo;
    if (q < nq) {
      d = (u32)(lower_bound_near(J.skey, J.n, q + 1, (q + 1) * J.n / nq) - lo);
      if (d == 0) J.a.pcnt[q] = J.a.scnt[q] = 0;
    }
  }
  __syncthreads();
  // appends aggregated per wave, then per block: one device atomic per class
  u64 m[kLocClasses];
  u32 woff[kLocClasses];
#pragma unroll
  for (int l = 0; l < kLocClasses; ++l) {
    m[l] = __ballot(d > 0 && loc_class(d) == (u32)l);
    woff[l] = 0;
    if (m[l]) {
      const u32 leader = __ffsll((unsigned long long)m[l]) - 1;
      if (lane == leader) woff[l] = atomicAdd(&s_n[l], (u32)__popcll(m[l]));
      woff[l] = __shfl(woff[l], leader, kWave);
    }
  }
  __syncthreads();
  if (threadIdx.x < (u32)kLocClasses && s_n[threadIdx.x])
    s_base[threadIdx.x] = atomicAdd(&J.list_len[threadIdx.x], s_n[threadIdx.x]);
  __syncthreads();
  if (d > 0) {
    const u32 l = loc_class(d);
    J.lists[(u64)l * nq + s_base[l] + woff[l] + count_below(m[l])] = (u32)q;
  }
}

// The four size classes of 256-thread workgroups in one launch: a job's
// workgroups [0, g.x) the groups of 16 lanes, then g.y of groups of 64
// lanes, g.z workgroups with one item per thread and g.w with four (the
// lists of classes 0 to 3, each nq entries apart).
__global__ __launch_bounds__(256) void k_loc_small(LocalPair p, u32 split) {
  u32 b, nblk;
  const LocalJob &J = local_job(p, split, b, nblk);
  const uint4 g = J.gs;
  const u32 nq = J.nq;
  __shared__ LdsState<4> s_state;  // classes 2 and 3 (class 2 uses its first quarter)
  if (b < g.x) return state_group<16>(J.a, J.lists, J.list_len, b, g.x);
  b -= g.x;
  if (b < g.y) return state_group<kWave>(J.a, J.lists + nq, J.list_len + 1, b, g.y);
  b -= g.y;
  if (b < g.z)
    return state_lds<1>(J.a, J.lists + 2 * (u64)nq, J.list_len + 2, b, g.z,
                        *reinterpret_cast<LdsState<1> *>(&s_state));
  b -= g.z;
  state_lds<4>(J.a, J.lists + 3 * (u64)nq, J.list_len + 3, b, g.w, s_state);
}

// Class 4: workgroups of 1024 threads with eight items per thread.
__global__ __launch_bounds__(1024) void k_loc_large(LocalPair p, u32 split) {
  u32 blk, nblk;
  const LocalJob &J = local_job(p, split, blk, nblk);
  state_local<1024, 8>(J.a, J.lists + 4 * (u64)J.nq, J.list_len + 4, blk, nblk);
}

// part_base and row: exclusive sums of the parts and segments per state,
// with the totals at [nq]; workgroup 2 i + c scans column c of job i.
constexpr int kLocScanNT = 1024;
__global__ __launch_bounds__(kLocScanNT) void k_loc_scan(LocalPair p) {
  constexpr u32 kWaves = kLocScanNT / kWave, kBatch = 8;
  __shared__ u32 s_tot[kWaves];
  const LocalJob &J = p.j[blockIdx.x >> 1];
  const bool segs = blockIdx.x & 1u;
  const u32 *in = segs ? J.a.scnt : J.a.pcnt;
  u32 *out = segs ? J.row : J.part_base;
  const u32 n = J.nq;
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  // wave w sums, then scans, the entries [w S, w S + S), S a multiple of 64
  const u32 seg = (n + kWaves * kWave - 1) / (kWaves * kWave) * kWave;
  const u32 b = min(n, w * seg), e = min(n, b + seg);
  u32 sum = 0;
  for (u32 c = b; c < e; c += kBatch * kWave) {
    u32 v[kBatch];
#pragma unroll
    for (u32 q = 0; q < kBatch; ++q) {
      const u32 i = c + q * kWave + lane;
      v[q] = i < e ? in[i] : 0u;
    }
#pragma unroll
    for (u32 q = 0; q < kBatch; ++q) sum += v[q];
  }
  sum = wave_total(sum);
  if (lane == 0) s_tot[w] = sum;
  __syncthreads();
  u32 carry = 0;
  for (u32 k = 0; k < w; ++k) carry += s_tot[k];
  if (w == kWaves - 1 && lane == 0) out[n] = carry + sum;
  for (u32 c = b; c < e; c += kBatch * kWave) {  // wave-uniform bounds
    u32 v[kBatch];
#pragma unroll
    for (u32 q = 0; q < kBatch; ++q) {
      const u32 i = c + q * kWave + lane;
      v[q] = i < e ? in[i] : 0u;
    }
#pragma unroll
    for (u32 q = 0; q < kBatch; ++q) {
      const u32 i = c + q * kWave + lane;
      const u32 incl = wave_inclusive_total(v[q]);
      if (i < e) out[i] = carry + incl - v[q];
      carry += (u32)__builtin_amdgcn_readlane((int)incl, kWave - 1);
    }
  }
}

// Moves each state's parts and segments from its arc offset to their final
// places; the totals go to counts[0] (segments) and counts[1] (parts).
__global__ void k_loc_place(LocalPair p, u32 split) {
  u32 blk, nblk;
  const LocalJob &J = local_job(p, split, blk, nblk);
  const u32 nq = J.nq;
  for (u64 i = (u64)blk * blockDim.x + threadIdx.x; i < J.n; i += (u64)nblk * blockDim.x) {
    const u32 q = (u32)J.skey[i];
    const u32 j = (u32)i - J.a.abase[q];
    if (j < J.a.pcnt[q]) J.parts[J.part_base[q] + j] = J.a.ptmp[i];
    if (j < J.a.scnt[q]) {
      J.seg_sym[J.row[q] + j] = J.a.ssym[i];
      J.seg_off[J.row[q] + j] = J.a.soff[i];
    }
    if (i == 0) {
      J.seg_off[J.row[nq]] = (u32)J.n;
      J.counts[0] = J.row[nq];
      J.counts[1] = J.part_base[nq];
    }
  }
}

__global__ void k_loc_flags(LocalPair p, u32 split) {
  u32 blk, nblk;
  const LocalJob &J = local_job(p, split, blk, nblk);
  cell_flags_body(J.row, J.seg_sym, J.seg_off, J.a.arcs, J.part_base, J.nq, J.cell_flag, J.n,
                  J.wts, J.gw, blk, nblk);
}

}  // namespace

void build_cell_flags(const Csr &c, u32 *cell_flag, hipStream_t s) {
  const u64 nw = c.num_arcs + kArcTail;
  const unsigned gw = (unsigned)std::min<u64>(ceil_div(nw, kNT), 4096);
  const unsigned g = (unsigned)std::min<u64>(ceil_div(c.num_states, kNT / kWave), 1u << 16);
  hipLaunchKernelGGL(k_cell_flags, dim3(gw + g), dim3(kNT), 0, s, c.row, c.seg_sym, c.seg_off,
                     c.arcs, c.part_base, c.num_states, cell_flag, c.num_arcs, c.wts, gw);
}

void check_csr_ranges(const fstc_fst &m, bool by_output) {
  if (m.num_arcs >= (1ull << 32))
    throw Error(FSTC_ERR_RANGE, "num_arcs must be below 2^32");
  const int bq = (int)bits_for(m.num_states - 1);
  const u32 ninner = by_output ? m.num_osyms : m.num_isyms;
  const u32 nouter = by_output ? m.num_isyms : m.num_osyms;
  const int bi = (int)bits_for(ninner ? ninner - 1 : 0);
  const int bo = (int)bits_for(nouter ? nouter - 1 : 0);
  if (2 * bq + bo > 64 || bq + bi > 64)
    throw Error(FSTC_ERR_RANGE, "state and symbol ids do not fit the 64-bit CSR sort keys");
}

void alloc_csr(const fstc_fst &m, Buf &b, Csr &c) {
  const u64 n = m.num_arcs, nq = m.num_states;
  const u64 n1 = std::max<u64>(n, 1);
  const size_t sz[8] = {(nq + 1) * 4, n1 * 4, (n + 1) * 4, (n + kArcTail) * 8, (nq + 1) * 4,
                        n1 * 8, std::max<u64>(nq, 1) * 4, (n + kArcTail) * 4};
  size_t off[8], total = 0;
  for (int i = 0; i < 8; ++i) {
    off[i] = total;
    total += (sz[i] + 255) & ~(size_t)255;
  }
  char *p = static_cast<char *>(b.ensure(total));
  c.num_states = m.num_states;
  c.num_arcs = n;
  c.row = (u32 *)(p + off[0]);
  c.seg_sym = (u32 *)(p + off[1]);
  c.seg_off = (u32 *)(p + off[2]);
  c.arcs = (uint2 *)(p + off[3]);
  c.part_base = (u32 *)(p + off[4]);
  c.parts = (uint2 *)(p + off[5]);
  c.cell_flag = (u32 *)(p + off[6]);
  c.wts = (u32 *)(p + off[7]);
}

namespace {

// The per-state build (see state_local) for transducers of at most
// kLocMaxStates states whose arcs per state stay moderate on average; one
// state with a very large share of the arcs goes through the global sorts.
constexpr u32 kLocMaxStates = 1u << 17;
constexpr u64 kLocMaxAvg = 1024;
constexpr u64 kLocAnyArcs = 1u << 16;

bool use_local_build(u64 n, u32 nq) {
  return nq <= kLocMaxStates && (n <= kLocMaxAvg * nq || n <= kLocAnyArcs);
}

size_t arena_bytes(std::initializer_list<size_t> sizes) {
  size_t t = 0;
  for (size_t b : sizes) t += std::max<size_t>(256, (b + 255) & ~(size_t)255);
  return t;
}

// One input of build_csr_local.
struct LocalIn {
  const fstc_fst *m;
  bool by_output;
  Arena *T;         // its temporaries
  const Csr *c;
  u64 *counts;      // [3] device counters (segments, parts, largest part count)
};

// The per-state build of one or two inputs, every step one launch for both;
// with `flags` the cell flags and weight words too (build_cell_flags).
void build_csr_local(const LocalIn *in, int nj, bool flags, u32 *d_err, hipStream_t s) {
  LocalPair p{};
  SortJob sj[2];
  for (int i = 0; i < nj; ++i) {
    const fstc_fst &m = *in[i].m;
    const Csr &c = *in[i].c;
    Arena &T = *in[i].T;
    const u64 n = m.num_arcs;
    const u32 nq = m.num_states;
    const int bq = (int)bits_for(nq - 1);
    const u32 ninner = in[i].by_output ? m.num_osyms : m.num_isyms;
    const u32 nouter = in[i].by_output ? m.num_isyms : m.num_osyms;
    const int bi = (int)bits_for(ninner ? ninner - 1 : 0);
    const int bo = (int)bits_for(nouter ? nouter - 1 : 0);
    Tmp skey(&T), order(&T), kalt(&T), valt(&T), kb(&T), ib(&T), part_of(&T), ptmp(&T), ssym(&T),
        soff(&T), pcnt(&T), scnt(&T), abase(&T), lists(&T), ctl(&T), rtmp(&T);
    skey.ensure(n * 8); order.ensure(n * 4); kalt.ensure(n * 8); valt.ensure(n * 4);
    kb.ensure(n * 8); ib.ensure(n * 4); part_of.ensure(n * 4); ptmp.ensure(n * 8);
    ssym.ensure(n * 4); soff.ensure(n * 4);
    pcnt.ensure((u64)nq * 4); scnt.ensure((u64)nq * 4); abase.ensure(((u64)nq + 1) * 4);
    lists.ensure(kLocClasses * (u64)nq * 4);
    rtmp.ensure(radix_temp_bytes(n));
    ctl.ensure(256);  // list lengths, then the unsorted word
    LocalJob &J = p.j[i];
    static std::atomic<u32> epochs{0};
    J.unsorted = ctl.as<u32>() + 16;
    J.epoch = epochs.fetch_add(1, std::memory_order_relaxed) + 1;
    LocalArgs &a = J.a;
    a.skey = skey.as<u64>();
    a.order = order.as<u32>();
    a.abase = abase.as<u32>();
    a.dst = m.dst;
    a.inner = in[i].by_output ? m.olabel : m.ilabel;
    a.outer = in[i].by_output ? m.ilabel : m.olabel;
    a.w = m.weight;
    a.bo = bo;
    a.bp = bq + bo;
    a.bi = bi;
    a.ka = kalt.as<u64>();
    a.kb = kb.as<u64>();
    a.ia = valt.as<u32>();
    a.ib = ib.as<u32>();
    a.part_of = part_of.as<u32>();
    a.ptmp = ptmp.as<uint2>();
    a.ssym = ssym.as<u32>();
    a.soff = soff.as<u32>();
    a.arcs = c.arcs;
    a.pcnt = pcnt.as<u32>();
    a.scnt = scnt.as<u32>();
    a.maxp = in[i].counts + 2;
    J.skey = skey.as<u64>();
    J.order = order.as<u32>();
    J.abase = abase.as<u32>();
    J.src = m.src;
    J.il = m.ilabel;
    J.ol = m.olabel;
    J.n = n;
    J.nq = nq;
    J.nis = m.num_isyms;
    J.nos = m.num_osyms;
    J.lists = lists.as<u32>();
    J.list_len = ctl.as<u32>();
    J.counts = in[i].counts;
    J.row = c.row;
    J.part_base = c.part_base;
    J.seg_sym = c.seg_sym;
    J.seg_off = c.seg_off;
    J.parts = c.parts;
    // grids: at most one lane group (workgroup) per state of the list
    J.gs = make_uint4((unsigned)std::min<u64>(ceil_div(nq, 16), 4096),
                      (unsigned)std::min<u64>(ceil_div(nq, 4), 4096),
                      (unsigned)std::min<u64>(nq, 4096), (unsigned)std::min<u64>(nq, 2048));
    J.cell_flag = c.cell_flag;
    J.wts = c.wts;
    J.gw = (unsigned)std::min<u64>(ceil_div(n + kArcTail, kNT), 4096);
    // stable: arcs of a state keep their input order
    sj[i] = SortJob{skey.as<u64>(), kalt.as<u64>(), order.as<u32>(), valt.as<u32>(), n, 0, bq,
                    rtmp.p, J.unsorted, J.epoch};
  }
  // workgroups of each job for one step: the launch's grid and split
  auto launch = [&](auto kern, auto blocks, unsigned nt) {
    const unsigned g0 = blocks(p.j[0]), g1 = nj > 1 ? blocks(p.j[1]) : 0u;
    hipLaunchKernelGGL(kern, dim3(g0 + g1), dim3(nt), 0, s, p, g0);
  };
  auto per_arc = [](const LocalJob &J) { return grid_for(J.n); };
  {
    const unsigned g0 = per_arc(p.j[0]), g1 = nj > 1 ? per_arc(p.j[1]) : 0u;
    hipLaunchKernelGGL(k_loc_keys, dim3(g0 + g1), dim3(kNT), 0, s, p, g0, d_err);
  }
  radix_sort_pairs_batch(sj, nj, s);
  launch(k_loc_lists, [](const LocalJob &J) { return (unsigned)ceil_div((u64)J.nq + 1, kNT); },
         kNT);
  launch(k_loc_small, [](const LocalJob &J) { return J.gs.x + J.gs.y + J.gs.z + J.gs.w; }, 256);
  launch(k_loc_large, [](const LocalJob &J) { return (unsigned)std::min<u32>(J.nq, 512); }, 1024);
  hipLaunchKernelGGL(k_loc_scan, dim3(2 * nj), dim3(kLocScanNT), 0, s, p);
  launch(k_loc_place, per_arc, kNT);
  if (flags)
    launch(k_loc_flags, [](const LocalJob &J) {
      return J.gw + (unsigned)std::min<u64>(ceil_div(J.nq, kNT / kWave), 1u << 16);
    }, kNT);
}

}  // namespace

size_t csr_temp_bytes(const fstc_fst &m) {
  const u64 n = m.num_arcs, nq = m.num_states;
  if (n == 0) return 0;
  if (use_local_build(n, m.num_states))
    return arena_bytes({n * 8, n * 4, n * 8, n * 4, n * 8, n * 4, n * 4, n * 8, n * 4, n * 4,
                        nq * 4, nq * 4, (nq + 1) * 4, kLocClasses * nq * 4, radix_temp_bytes(n),
                        256});
  return arena_bytes({n * 8, n * 8, n * 4, n * 4, n * 8, n * 4, n * 4, (n + 1) * 4, n * 4, n * 4,
                      n * 4, std::max(radix_temp_bytes(n), scan_temp_bytes(n))});
}

void build_csr(const fstc_fst &m, bool by_output, Arena &T, const Csr &c, u64 *d_counts,
               u32 *d_err, hipStream_t s) {
  check_csr_ranges(m, by_output);
  const u64 n = m.num_arcs;
  const u32 nq = m.num_states;
  if (n == 0) {
    fill_u64(d_counts, 0, 3, s);
    fill_u32(c.row, 0, (u64)nq + 1, s);
    fill_u32(c.part_base, 0, (u64)nq + 1, s);
    fill_u32(c.seg_off, 0, 1, s);
    return;
  }
  if (use_local_build(n, nq)) {  // its first kernel clears the counters
    const LocalIn in{&m, by_output, &T, &c, d_counts};
    build_csr_local(&in, 1, false, d_err, s);
    return;
  }
  fill_u64(d_counts, 0, 3, s);
  const int bq = (int)bits_for(nq - 1);
  const u32 ninner = by_output ? m.num_osyms : m.num_isyms;
  const u32 nouter = by_output ? m.num_isyms : m.num_osyms;
  const int bi = (int)bits_for(ninner ? ninner - 1 : 0);
  const int bo = (int)bits_for(nouter ? nouter - 1 : 0);

  Tmp kp(&T), kc(&T), v1(&T), v2(&T), kalt(&T), valt(&T), flags(&T), ex(&T), apg(&T),
      pstate(&T), sstate(&T), tmp(&T);
  kp.ensure(n * 8); kc.ensure(n * 8); v1.ensure(n * 4); v2.ensure(n * 4);
  kalt.ensure(n * 8); valt.ensure(n * 4);
  flags.ensure(n * 4); ex.ensure((n + 1) * 4); apg.ensure(n * 4);
  pstate.ensure(n * 4); sstate.ensure(n * 4);
  tmp.ensure(std::max(radix_temp_bytes(n), scan_temp_bytes(n)));

  const unsigned g = grid_for(n);
  hipLaunchKernelGGL(k_csr_pack, dim3(g), dim3(kNT), 0, s, m.src, m.dst, m.ilabel, m.olabel, n,
                     nq, m.num_isyms, m.num_osyms, by_output ? 1 : 0, bq, bo, bi, kp.as<u64>(),
                     kc.as<u64>(), v1.as<u32>(), v2.as<u32>(), d_err);

  // parts: distinct (state, target, outer) in sorted order
  radix_sort_pairs(kp.as<u64>(), v1.as<u32>(), kalt.as<u64>(), valt.as<u32>(), n, 0,
                   2 * bq + bo, tmp.p, s);
  hipLaunchKernelGGL(k_head_flags, dim3(g), dim3(kNT), 0, s, kp.as<u64>(), n, flags.as<u32>());
  exclusive_scan(flags.as<u32>(), ex.as<u32>(), n, tmp.p, s);
  hipLaunchKernelGGL(k_parts, dim3(g), dim3(kNT), 0, s, kp.as<u64>(), v1.as<u32>(),
                     flags.as<u32>(), ex.as<u32>(), n, bq, bo, c.parts, pstate.as<u32>(),
                     apg.as<u32>());
  hipLaunchKernelGGL(k_copy_count, dim3(1), dim3(1), 0, s, ex.as<u32>() + n, d_counts + 1);
  // P = ex[n] parts; entries [P, n) of the part-state array are unused: set
  // them above every state so that searching all n entries is exact.
  hipLaunchKernelGGL(k_fill_tail, dim3(g), dim3(kNT), 0, s, pstate.as<u32>(),
                     (const u32 *)(ex.as<u32>() + n), n, 0xffffffffu);
  hipLaunchKernelGGL(k_state_offsets, dim3(grid_for((u64)nq + 1)), dim3(kNT), 0, s,
                     pstate.as<u32>(), n, nq, c.part_base);
  hipLaunchKernelGGL(k_max_gap, dim3(grid_for(nq)), dim3(kNT), 0, s, c.part_base, nq,
                     d_counts + 2);

  // segments: distinct (state, inner symbol) in sorted order, the arcs of a
  // segment ordered by part (the stable sort starts from the part order)
  hipLaunchKernelGGL(k_gather_keys, dim3(g), dim3(kNT), 0, s, kc.as<u64>(), v1.as<u32>(), n,
                     kalt.as<u64>(), valt.as<u32>());
  radix_sort_pairs(kalt.as<u64>(), valt.as<u32>(), kc.as<u64>(), v2.as<u32>(), n, 0, bq + bi,
                   tmp.p, s);
  hipLaunchKernelGGL(k_head_flags, dim3(g), dim3(kNT), 0, s, kalt.as<u64>(), n, flags.as<u32>());
  exclusive_scan(flags.as<u32>(), ex.as<u32>(), n, tmp.p, s);
  hipLaunchKernelGGL(k_segments, dim3(g), dim3(kNT), 0, s, kalt.as<u64>(), valt.as<u32>(),
                     flags.as<u32>(), ex.as<u32>(), n, bi, apg.as<u32>(), c.part_base,
                     m.weight, c.seg_sym, c.seg_off, sstate.as<u32>(), c.arcs);
  hipLaunchKernelGGL(k_copy_count, dim3(1), dim3(1), 0, s, ex.as<u32>() + n, d_counts + 0);
  hipLaunchKernelGGL(k_fill_tail, dim3(g), dim3(kNT), 0, s, sstate.as<u32>(),
                     (const u32 *)(ex.as<u32>() + n), n, 0xffffffffu);
  hipLaunchKernelGGL(k_state_offsets, dim3(grid_for((u64)nq + 1)), dim3(kNT), 0, s,
                     sstate.as<u32>(), n, nq, c.row);
}

bool build_csr_pair(const fstc_fst &m1, bool by_output1, Arena &T1, const Csr &c1,
                    u64 *d_counts1, const fstc_fst &m2, bool by_output2, Arena &T2,
                    const Csr &c2, u64 *d_counts2, bool flags, u32 *d_err, hipStream_t s) {
  if (m1.num_arcs == 0 || m2.num_arcs == 0 || !use_local_build(m1.num_arcs, m1.num_states) ||
      !use_local_build(m2.num_arcs, m2.num_states))
    return false;
  check_csr_ranges(m1, by_output1);
  check_csr_ranges(m2, by_output2);
  const LocalIn in[2] = {{&m1, by_output1, &T1, &c1, d_counts1},
                         {&m2, by_output2, &T2, &c2, d_counts2}};
  build_csr_local(in, 2, flags, d_err, s);
  return true;
}

}  // namespace fstc
