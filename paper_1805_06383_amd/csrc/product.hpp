// Product-merge selection of a level's sources (section 3.4 merges arcs
// with equal (source, target, input, output) keys by summing their weights;
// a source whose two states have single-arc cells merges them as a small
// matrix product, level.hpp), shared by the count kernels and the
// one-workgroup product level (merge.hip).
#pragma once

#include "level.hpp"

namespace fstc {

// A source's inner-symbol lists: segments [b1, e1) of M1's state and
// [b2, e2) of M2's.
struct Ranges {
  u32 b1, e1, b2, e2;
};

// True when every product of a weight of the state summarised by f1 with
// one of the state summarised by f2 (build_cell_flags) is a normal float32
// number after rounding: no infinity or NaN, no subnormal operand,
// |w1 w2| < 2^127 (biased exponents sum to at most 379) and
// |w1 w2| >= 2^-126 for nonzero operands (they sum to at least 128).  Such
// a product rounded to float32 is within 2^-24 of itself, relatively.
__device__ __forceinline__ bool products_normal(u32 f1, u32 f2) {
  if ((f1 | f2) & kCellSpecial) return false;
  const u32 emax = ((f1 >> kCellEmaxShift) & 0xffu) + ((f2 >> kCellEmaxShift) & 0xffu);
  const u32 emin = ((f1 >> kCellEminShift) & 0xffu) + ((f2 >> kCellEminShift) & 0xffu);
  return emax <= 379u && emin >= 128u;
}

// Product-merge selection of source u (level.hpp) from what the count
// already loaded: table entries P1 P2 and the source header written to
// phdr, or 0 (record path).  The header's last word holds the matrix-core
// form (bit 0: at most kProdMfmaParts parts per state, products_normal) and
// the aligned form (bit 1; both states kCellDense with symbol lists of one
// length n, at bit 8): the second header word is then (M1 segment begin, its
// first arc, M2 segment begin, its first arc).  Bit 2: aligned, both states
// kCellIdent and their symbol lists identical (kCellContig with one first
// symbol): the strided form, merged four sources per wave with the dense
// visited array (no symbol check there).  The cells are single-arc
// only for states of at most kProdParts parts.
__device__ __forceinline__ u32 select_product(const LevelArgs &a, u32 u, u32 q1, u32 q2,
                                              const Ranges &r, bool &mfma,
                                              bool *strided_out = nullptr) {
  const u32 f1 = a.c1.cell_flag[q1], f2 = a.c2.cell_flag[q2];
  if ((f1 | f2) & kCellBad) return 0;
  const u32 pb1 = a.c1.part_base[q1], p1 = a.c1.part_base[q1 + 1] - pb1;
  const u32 pb2 = a.c2.part_base[q2], p2 = a.c2.part_base[q2 + 1] - pb2;
  if (p1 == 0 || p2 == 0 || p1 + p2 > kProdRowSum) return 0;
  mfma = p1 <= kProdMfmaParts && p2 <= kProdMfmaParts && products_normal(f1, f2);
  const u32 n = r.e1 - r.b1;
  const bool aligned = mfma && (f1 & f2 & kCellDense) && n == r.e2 - r.b2;
  // strided: segments ordered by part on both sides and the two symbol
  // lists identical (consecutive, same first symbol, same length)
  const bool strided = aligned && (f1 & f2 & kCellIdent) && (f1 & f2 & kCellContig) &&
                       a.c1.seg_sym[r.b1] == a.c2.seg_sym[r.b2];
  if (strided_out) *strided_out = strided;
  a.phdr[2 * u] = make_uint4(pb1, pb2, p1 | (p2 << 16),
                             (mfma ? 1u : 0u) | (aligned ? 2u | (n << 8) : 0u) |
                                 (strided ? 4u : 0u));
  a.phdr[2 * u + 1] = aligned ? make_uint4(r.b1, a.c1.seg_off[r.b1], r.b2, a.c2.seg_off[r.b2])
                              : make_uint4(r.b1, r.e1, r.b2, r.e2);
  return p1 * p2;
}

}  // namespace fstc
