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
// (a 64-bit mask of the parts), flags the state.
__global__ void k_cell_flags(const u32 *row, const u32 *seg_off, const uint2 *arcs,
                             const u32 *part_base, u32 nq, u32 *flag) {
  const u32 lane = lane_id();
  const u64 nw = (u64)gridDim.x * blockDim.x / kWave;
  for (u64 q = ((u64)blockIdx.x * blockDim.x + threadIdx.x) / kWave; q < nq; q += nw) {
    bool bad = part_base[q + 1] - part_base[q] > kProdParts;
    if (!bad) {
      for (u32 sg = row[q] + lane; sg < row[q + 1]; sg += kWave) {
        const u32 a0 = seg_off[sg], n = seg_off[sg + 1] - a0;
        if (n > kProdParts) {
          bad = true;
          continue;
        }
        u64 m = 0;
        for (u32 i = 0; i < n; ++i) m |= 1ull << (arcs[a0 + i].x & 63u);
        bad |= (u32)__popcll(m) != n;
      }
    }
    const bool any = __ballot(bad) != 0;
    if (lane == 0) flag[q] = any ? 1u : 0u;
  }
}

// a[i] = v for i in [*count, n).
__global__ void k_fill_tail(u32 *a, const u32 *count, u64 n, u32 v) {
  const u64 c = *count;
  for (u64 i = c + (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x)
    a[i] = v;
}

}  // namespace

void build_cell_flags(const Csr &c, u32 *cell_flag, hipStream_t s) {
  if (!c.num_states) return;
  const unsigned g = (unsigned)std::min<u64>(ceil_div(c.num_states, kNT / kWave), 1u << 16);
  hipLaunchKernelGGL(k_cell_flags, dim3(g), dim3(kNT), 0, s, c.row, c.seg_off, c.arcs,
                     c.part_base, c.num_states, cell_flag);
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

void alloc_csr(const fstc_fst &m, Allocator &A, Buf *b, Csr &c) {
  const u64 n = m.num_arcs, nq = m.num_states;
  for (int i = 0; i < 7; ++i) b[i].A = &A;
  c.num_states = m.num_states;
  c.num_arcs = n;
  c.row = (u32 *)b[0].ensure((nq + 1) * sizeof(u32));
  c.seg_sym = (u32 *)b[1].ensure(std::max<u64>(n, 1) * sizeof(u32));
  c.seg_off = (u32 *)b[2].ensure((n + 1) * sizeof(u32));
  c.arcs = (uint2 *)b[3].ensure(std::max<u64>(n, 1) * sizeof(uint2));
  c.part_base = (u32 *)b[4].ensure((nq + 1) * sizeof(u32));
  c.parts = (uint2 *)b[5].ensure(std::max<u64>(n, 1) * sizeof(uint2));
}

void build_csr(const fstc_fst &m, bool by_output, Arena &T, const Csr &c, u64 *d_counts,
               u32 *d_err, hipStream_t s) {
  check_csr_ranges(m, by_output);
  const u64 n = m.num_arcs;
  const u32 nq = m.num_states;
  fill_u64(d_counts, 0, 3, s);
  if (n == 0) {
    fill_u32(c.row, 0, (u64)nq + 1, s);
    fill_u32(c.part_base, 0, (u64)nq + 1, s);
    fill_u32(c.seg_off, 0, 1, s);
    return;
  }
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

  // segments: distinct (state, inner symbol) in sorted order
  radix_sort_pairs(kc.as<u64>(), v2.as<u32>(), kalt.as<u64>(), valt.as<u32>(), n, 0, bq + bi,
                   tmp.p, s);
  hipLaunchKernelGGL(k_head_flags, dim3(g), dim3(kNT), 0, s, kc.as<u64>(), n, flags.as<u32>());
  exclusive_scan(flags.as<u32>(), ex.as<u32>(), n, tmp.p, s);
  hipLaunchKernelGGL(k_segments, dim3(g), dim3(kNT), 0, s, kc.as<u64>(), v2.as<u32>(),
                     flags.as<u32>(), ex.as<u32>(), n, bi, apg.as<u32>(), c.part_base,
                     m.weight, c.seg_sym, c.seg_off, sstate.as<u32>(), c.arcs);
  hipLaunchKernelGGL(k_copy_count, dim3(1), dim3(1), 0, s, ex.as<u32>() + n, d_counts + 0);
  hipLaunchKernelGGL(k_fill_tail, dim3(g), dim3(kNT), 0, s, sstate.as<u32>(),
                     (const u32 *)(ex.as<u32>() + n), n, 0xffffffffu);
  hipLaunchKernelGGL(k_state_offsets, dim3(grid_for((u64)nq + 1)), dim3(kNT), 0, s,
                     sstate.as<u32>(), n, nq, c.row);
}

}  // namespace fstc
