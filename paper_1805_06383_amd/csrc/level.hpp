// Per-level kernels of the breadth-first composition: shared arguments and
// launchers (expand.hip: join count, match emission, arc-pair write;
// merge.hip: segmented sort + reduce, visited-table insert, id assignment,
// result append).
#pragma once

#include "internal.hpp"

namespace fstc {

// Read-only view of a Csr on the device.
struct CsrView {
  const u32 *row, *seg_sym, *seg_off;
  const uint2 *arcs;
  const u32 *part_base;
  const uint2 *parts;
  u64 num_arcs;
  const u32 *cell_flag;  // [num_states] build_cell_flags; kCellBad: no product merge
};

inline CsrView view(const Csr &c) {
  return CsrView{c.row, c.seg_sym, c.seg_off, c.arcs, c.part_base, c.parts, c.num_arcs,
                 c.cell_flag};
}

// Host-visible per-level counters (one D2H copy per synchronisation).
struct Status {
  u64 R;        // unmerged composed arcs of the level
  u64 M;        // matched (source, inner symbol) segment pairs of the level
  u64 merged;   // merged arcs of the level
  u64 RB;       // records of sources merged by the multi-block path
  u32 nwide, nheavy, nbig, nnew;
  u32 err;      // kErr* bits, sticky for the whole call
  u32 max_small;  // largest record count of a source merged by the tiles
  u64 dense_records;  // records of the tiles merged through a dense table
  u64 dense_runs;     // merged arcs those tiles produced
  u64 sort_runs;      // merged arcs of the tiles merged by sorting
  u32 nsort;          // tiles k_merge_dense left to the sort kernel
  u32 scan_ctr;       // tile counter of the single-pass scans (0 between scans)
  u32 seq;            // host copy only: number of the last publication, written last
  u32 unfit;          // sources of the level of a shape the one-workgroup
                      // small-level kernel declines (kSmallShape)
  u32 nprod;          // sources of the product merge       } one u64, the total of
  u32 nprod_mfma;     // of those, summed on the matrix cores } the level's flag words
  u64 prod_records;   // their joined arc pairs (not written as records)
  u64 prod_entries;   // their (p1, p2) table entries: temp slots after the records
  u32 ngen;           // product-merge sources listed for the one-per-wave kernel
  u32 ngrp;           // sources listed for the 16-lane joins
  u32 declined;       // nonzero: the one-workgroup product level did not take the level
  u32 pad1;
};
static_assert(offsetof(Status, nprod) % 8 == 0 &&
                  offsetof(Status, nprod_mfma) == offsetof(Status, nprod) + 4,
              "the flag total is stored as one u64 over nprod, nprod_mfma");

// Product merge (merge.hip, k_prod_sources).  A source (q1, q2) is merged
// by one wavefront from its staged arc matrices instead of through records
// when its states have P1 + P2 <= kProdRowSum parts in all, the shorter of
// its two inner-symbol lists has kProdMinSymbols to 64 symbols, and neither
// state has two arcs in one (part, inner symbol) cell.  The count kernel
// selects it from the list lengths and part counts alone; the product
// kernel counts its joined pairs.
constexpr u32 kProdRowSum = 16;
constexpr u32 kProdMinSymbols = 8;
// Sources whose states have at most kProdMfmaParts parts each and whose
// weight products are normal float32 numbers (expand.hip, products_normal)
// are summed on the matrix cores (merge.hip).
constexpr u32 kProdMfmaParts = 4;

// Joins: a source whose serial join takes at most kThreadSteps binary-search
// steps (shorter length x bits of the longer length) is joined by one
// thread; one whose shorter list has at most kGroupMax symbols and whose
// longer one at most kGroupLong, by a group of kGroupLanes lanes; one whose
// shorter list is longer than kHeavyMin, by a workgroup; the others by a
// wavefront.
constexpr u32 kThreadSteps = 12;
constexpr u32 kGroupLanes = 16;
constexpr u32 kGroupMax = 32;
constexpr u32 kGroupLong = 512;
constexpr u32 kHeavyMin = 2048;

// Merge tiles: 512 threads x 8 items = 4096 records of LDS capacity.  Sources
// of more than kMergeSmall records take the multi-block path.  A tile takes
// the sources whose first record falls in a window of W records; with m the
// largest small-source count, every such source ends within the tile's
// capacity when W <= kMergeCap - m + 1 (and, when multi-block sources exist,
// W <= kMergeSmall keeps them last in their window).
constexpr int kMergeNT = 512;
constexpr int kMergeIT = 8;
constexpr int kMergeCap = kMergeNT * kMergeIT;
constexpr u64 kMergeSmall = kMergeCap / 2;
constexpr int kIdxBits = 12;  // log2(kMergeCap)
constexpr int kMaxKeyBits = 64 - 2 * kIdxBits;  // 40: part-rank bits of both sides

// A tile whose sources and keys span at most kDenseCap (source, key) pairs
// ((s1 - s0) << key_bits <= kDenseCap) is merged through a table indexed by
// that pair instead of a sort; this needs key_bits <= kDenseKeyBits.
constexpr u32 kDenseCap = 2048;
constexpr int kDenseKeyBits = 11;  // log2(kDenseCap)

// Arc-pair write pass: 512 threads x 8 records per workgroup, which covers
// kExpandGroup write tiles of kExpandTile records (the LDS staging capacity
// for match descriptors).
constexpr int kExpandNT = 512;
constexpr int kExpandIT = 8;
constexpr u64 kExpandTile = 2048;
constexpr u64 kExpandGroup = kExpandNT * kExpandIT / kExpandTile;

// Write tile t holds records [t kExpandTile, (t + 1) kExpandTile): k0 = the
// match holding its first record, base0 = that match's first record.  The
// emit kernels write the entries of the tiles whose first record falls in a
// match they emit; the matches of tile t are k0(t) .. kend(t) - 1, kend(t)
// following from entry t + 1 (k0(t + 1), plus one unless that match starts
// exactly at the tile boundary; M for the last tile).
struct ExpandTile {
  u64 k0, base0;
};

struct LevelArgs {
  CsrView c1, c2;
  const u32 *sq1, *sq2;  // state id -> q1, q2
  u32 lo, nsrc;          // sources are state ids lo .. lo + nsrc - 1
  u64 *cnt;              // [nsrc] unmerged arcs per source
  u32 *mc;               // [nsrc] matched segment pairs per source
  const u64 *roff;       // [nsrc + 1] exclusive scan of cnt
  const u64 *moff;       // [nsrc + 1] exclusive scan of mc
  u32 *wide, *heavy;     // source lists for wavefront / workgroup joins
  uint4 *wrange;         // [nsrc] segment ranges (b1, e1, b2, e2) of wide[i] at i, of
                         // grp[i] at nsrc - 1 - i (the two lists hold at most nsrc)
  Status *st;
  uint4 *match;          // [M] (M1 arc start, M2 arc start, n1, n2)
  u64 *mrbase;           // [M] first record of each match
  ExpandTile *tiles;     // [ceil(R / kExpandTile)] write-tile entries
  u32 *big;              // [nsrc] sources for the multi-block merge (st->nbig)
  u32 *pk;               // [nsrc] table entries of a product-merge source, else 0
  uint4 *phdr;           // [2 nsrc] product-merge source header (see ProdHeader)
  u32 prod;              // nonzero: sources may take the product merge
  u64 *tstart, *mend;    // [nsrc] the merge's first / end temp slot per source:
                         // zeroed by the count kernel
  u32 *newc;             // [nsrc] new pairs claimed per source: zeroed by the count
                         // kernel, written by the product merge
  u64 *pflag;            // [nsrc] 1 for a product-merge source, plus 2^32 when it
                         // takes the matrix-core form (summed by the level scan)
  u32 quad;              // nonzero: strided product sources go to the four-source
                         // kernel (dense visited array), the others to glist
  u32 *glist;            // [nsrc] product sources for the one-per-wave kernel (st->ngen)
  u32 *grp;              // [nsrc] sources for the 16-lane joins (st->ngrp)
  u32 unred;             // composition without reduction: only strided sources with
                         // the four-source kernel take the product form
};

// Target column marks of a direct product level (MergeArgs::out_src), and
// the source of an entry without a term.
constexpr u32 kDstSlot = 0x80000000u, kDstClaim = 0x40000000u, kDstSlotMask = 0x3fffffffu;
constexpr u32 kHoleSrc = 0xffffffffu;

// Written by the count kernel for a product-merge source u at phdr[2u], [2u+1]:
// (M1 part base, M2 part base, P1 | P2 << 16, matrix-core form), (M1 segment
// range begin, end, M2 segment range begin, end).

// lean: grids for lists expected empty (the previous level had none); the
// list kernels loop over their lists, so a longer list is still counted,
// by fewer workgroups.
void launch_count(const LevelArgs &a, hipStream_t s, bool lean = false);
// nwide / nheavy / ngrp: the list lengths the count kernels produced
// (st->nwide, nheavy, ngrp).
void launch_emit(const LevelArgs &a, u32 nwide, u32 nheavy, u32 ngrp, hipStream_t s);
// Writes R records: key = (part1 << b2) | part2 (u32 when key_bits <= 32,
// else u64), weight = p1 * p2.
// tiles: the ceil(R / kExpandTile) write-tile entries written by launch_emit.
void launch_expand(const uint4 *match, const u64 *mrbase, u64 M, u64 R, const CsrView &c1,
                   const CsrView &c2, int b2, bool wide_keys, void *rec_key, float *rec_w,
                   ExpandTile *tiles, u32 *err, hipStream_t s);

struct MergeArgs {
  const void *rec_key;
  const float *rec_w;
  u64 R;
  const u64 *roff;
  u32 nsrc, lo;
  const u32 *sq1, *sq2;
  const u32 *pbase1, *pbase2;
  const uint2 *parts1, *parts2;
  int key_bits, b2;
  // visited set: a hash table of pair keys (hkeys, hmask; ids by slot in
  // vis) or, when vn2 != 0, a dense array vis[r1 vn2 + r2] (slot = pair
  // index) holding kUnvisited, kClaimed or the pair's id
  u64 *hkeys;
  u64 hmask;
  u32 *vis;
  u32 vn2;
  u32 *newlist;
  u64 newcap;
  uint4 *temp;     // [R] merged runs: (source, key lo, key hi, weight bits) from the
                   // merge, then (slot, a, c, weight bits) after launch_emit_runs
  u32 *runsrc;     // [R] level-local source of the merged run at each temp slot
                   // (written with the visited-table insert)
  u64 *tstart;     // [nsrc] first temp slot of each source's merged arcs (0 if none)
  u64 *mend;       // [nsrc] one past its last slot (0 if none)
  u64 window;      // W: tile t takes the sources starting in [t W, (t + 1) W)
  uint4 *tiles;    // [ntiles = ceil(R / W)] scratch: tile descriptors
  u32 *sortlist;   // [ntiles] scratch: tiles left to the sort kernel
  u32 *tile_runs;  // [ntiles] merged runs each tile wrote (zero-filled before the merge)
  u64 ntiles;
  Status *st;
  // multi-block path
  u32 *big;        // [nbig] level-local source indices
  // fused expand + merge: the level's matches instead of its records
  const uint4 *match;   // [M] (M1 arc start, M2 arc start, n1, n2)
  const u64 *mrbase;    // [M] first record of each match
  const u64 *moff;      // [nsrc + 1] first match of each source
  const uint2 *arcs1, *arcs2;  // CSR arcs (part rank, weight bits)
  const u32 *wts1, *wts2;      // their weight words alone (Csr::wts)
  // product merge: the sources with pk[u] != 0 own temp slots
  // R + poff[u] .. R + poff[u] + pk[u] - 1 (prodpos slots in all)
  const u32 *pk;
  const uint4 *phdr;
  const u64 *poff;
  u64 prodpos;
  u64 *pcnt;  // [nsrc] joined arc pairs of each product-merge source (written by it)
  u32 *newc;  // [nsrc] new pairs each product-merge source claimed (written by it)
  const u64 *R_dev;  // product merge launched before the host knew R: the level's
                     // record count on the device (the kernel merges only if 0)
  u32 quad;          // the strided product sources are merged four per wave
  const u32 *glist;  // the other product sources (st->ngen of them)
  // direct product level (out_src != NULL; dense visited array only): the
  // product kernel writes source u's merged arcs straight to the result
  // columns at out_base + poff[u] + r instead of to temp, with the target
  // column holding the id when the target had one, else its slot with
  // kDstSlot (and kDstClaim when this entry claimed it); entries past the
  // source's merged count get src = kHoleSrc
  u32 *out_src, *out_dst, *out_il, *out_ol;
  float *out_w;
  u64 out_base;
  const u32 *row1, *seg_sym1, *seg_off1, *row2, *seg_sym2, *seg_off2;
  // composition without reduction, a level of strided product sources
  // (utab != NULL): the four-source kernel resolves only the targets, entry
  // r of source u at utab[poff[u] + r] marked like the target column of a
  // direct level; launch_unreduced_product then writes every joined pair
  u32 *utab;
};

// Small levels in one workgroup (merge.hip, k_small_levels): while a level
// has at most kSmallSources sources and kSmallRecords joined pairs, one
// workgroup joins, sorts and merges its records in LDS, inserts the targets,
// numbers the new pairs in (q1, q2) order and appends the merged arcs, then
// goes on with the next level; it stops at the first level it cannot take
// (too large, or a capacity below), at the depth cap, or when the search
// ends, and leaves the loop state in *ss for the host.
constexpr u32 kSmallSources = 512;
constexpr u32 kSmallRecords = 1024;
// Joins it takes: the shorter list at most kSmallShortList symbols, the
// longer at most kSmallLongList, at most kSmallPerSource joined pairs per
// source (one thread joins and emits a source: longer joins and larger
// sources are the per-level kernels' work, done by many lanes).
constexpr u32 kSmallShortList = 32, kSmallLongList = 4096, kSmallPerSource = 64;
// Why it stopped: a level too large (sources, joined pairs), a capacity, the
// end of the search, or a source of a shape it does not take (a long list
// or many joined pairs: a property of the inputs' states more than of the
// level).
enum : u32 { kSmallTooLarge = 1, kSmallCapacity = 2, kSmallDone = 3, kSmallShape = 4 };
struct SmallState {
  u64 lo, hi, n_states, arcs, premerge;
  u64 max_frontier, max_level_pre;
  u32 depth, levels, new_levels, reason;
};
struct SmallArgs {
  const u32 *row1, *seg_sym1, *seg_off1, *part_base1;
  const uint2 *arcs1, *parts1;
  const u32 *row2, *seg_sym2, *seg_off2, *part_base2;
  const uint2 *arcs2, *parts2;
  int b2, key_bits;
  MergeArgs va;  // visited set: vis, vn2, hkeys, hmask, st
  u32 *sq1, *sq2;
  u64 state_cap;  // at most this many states after a level (arrays, hash load, caps)
  u64 arc_cap;    // at most this many result arcs after a level
  u32 *out_src, *out_dst, *out_il, *out_ol;
  float *out_w;
  u32 max_levels;
  SmallState *ss;
};
void launch_small_levels(const SmallArgs &a, hipStream_t s);

// Composition without reduction, a level whose sources all took the
// four-source form and whose targets utab holds as ids: source u's joined
// pairs as arcs at out_base + off[u] .. (off: exclusive scan of the joined
// pairs per source), entry (p1, p2) times symbol g at
// (p1 P2 + p2) na + g, weight the float32 product of the two arc weights.
void launch_unreduced_product(const MergeArgs &a, const u64 *off, hipStream_t s);

// Tile descriptors of the level (a.tiles), then the two tile merges: the
// dense-table kernel (only when a.key_bits <= kDenseKeyBits) and the sort
// kernel, which takes every tile the dense kernel did not merge.
void launch_tile_sources(const MergeArgs &a, hipStream_t s);
void launch_merge_dense(const MergeArgs &a, hipStream_t s);
void launch_merge_sort(const MergeArgs &a, bool wide_keys, hipStream_t s);
// Fused expand + merge of every tile (in place of launch_expand and
// launch_merge_dense; needs key_bits <= kDenseKeyBits, no multi-block
// sources, 32-bit record keys).  narrow: both arc arrays below 2^29 arcs.
void launch_fuse_merge(const MergeArgs &a, bool narrow, hipStream_t s);
// Product merge of the sources with a.pk[u] != 0: their merged arcs, with
// visited-table inserts, at temp[R + poff[u] ...) (or the result, on a
// direct level) and tstart / mend: with a.quad, the strided sources four per
// wave and the listed ones (a.glist) one per wave; else every one of them
// one per wave from the list.  narrow: both arc arrays below 2^29 arcs.
// lean: a grid for a listed-source list expected empty (the previous level
// had none; the waves loop over the list).
void launch_prod_sources(const MergeArgs &a, bool narrow, hipStream_t s, bool lean = false);
// Multi-block merge of the nbig sources listed in a.big; bigoff has nbig + 1
// entries (exclusive scan of their record counts, total RB).
void launch_big_counts(const u64 *roff, const u32 *big, u32 nbig, u64 *bigcnt, hipStream_t s);
void merge_big(const MergeArgs &a, bool wide_keys, u32 nbig, const u64 *bigoff, u64 RB,
               Arena &T, hipStream_t s);

// vn2 != 0: dense visited array (MergeArgs), hkeys unused.
void launch_insert_start(u64 *hkeys, u64 hmask, u32 *hvals, u32 vn2, u32 s1, u32 s2, u32 *sq1,
                         u32 *sq2, u32 *err, hipStream_t s);
void launch_rehash(const u64 *okeys, const u32 *ovals, u64 ocap, u64 *nkeys, u32 *nvals,
                   u64 nmask, u32 *err, hipStream_t s);
// Dense visited array vis (|Q1| |Q2| entries, already kUnvisited) from the
// state arrays: vis[sq1[i] vn2 + sq2[i]] = i for every state id i < n.
void launch_states_to_dense(const u32 *sq1, const u32 *sq2, u64 n, u32 *vis, u32 vn2,
                            hipStream_t s);
// ids base .. base + nnew - 1 in new-list order (or the order in `order`).
void launch_assign(const u32 *slots, u32 nnew, u32 base, const u64 *hkeys, u32 *hvals, u32 vn2,
                   u32 *sq1, u32 *sq2, hipStream_t s);
// The same for min(*count, cap) new pairs, the count read on the device
// (the host need not know it yet); nothing when count is NULL.
void launch_assign_counted(const u32 *slots, const u64 *count, u32 cap, u32 base,
                           const u64 *hkeys, u32 *hvals, u32 vn2, u32 *sq1, u32 *sq2,
                           hipStream_t s);
void launch_newkeys(const u32 *newlist, u32 nnew, const u64 *hkeys, u32 vn2, int bq2, u64 *keys,
                    u32 *vals, hipStream_t s);
// Result append of the level's merged arcs: the runs of merge tile t go to
// output positions aoff[first source of t] + r, those of multi-block source u
// to aoff[u] + r (aoff: exclusive scan of merged arcs per source), so the
// output stays grouped by source id.  dst ids come from hvals.
// M: merged arcs of the level (the output arrays' length from osrc on).
void launch_compact(const MergeArgs &a, const u64 *aoff, u32 nbig, u64 M, const u32 *hvals,
                    u32 *osrc, u32 *odst, u32 *oil, u32 *ool, float *ow, hipStream_t s);
// Result append source by source (tstart[u] .. mend[u] - 1 to aoff[u] ...):
// the form used when product-merge sources sit between tile-merged ones.
void launch_compact_sources(const MergeArgs &a, const u64 *aoff, u64 M, const u32 *hvals,
                            u32 *osrc, u32 *odst, u32 *oil, u32 *ool, float *ow, hipStream_t s);
// Visited-table inserts and label lookups for every merged arc of the
// tile-merged sources (merge_big does its own).
void launch_emit_tiles(const MergeArgs &a, hipStream_t s);
// New-state list of the level from the claimed-slot flags of the tile runs,
// the multi-block runs and the product-merge slots.  Returns the device
// address of its length (for launch_merged_total), or NULL when there is
// nothing to list.
// wcnt: newlist_waves(a, RB) u32; woff: that + 1 u64.
// scan_state: scan_lb_state_bytes(newlist_waves(a, RB)) bytes of single-pass
// scan state (see exclusive_scan_lb).
u64 newlist_waves(const MergeArgs &a, u64 RB);
// The same list for a level whose sources all took the product merge (no
// records): newoff, the exclusive scan of a.newc, gives each source's first
// list entry; 16 lanes per source with claims write its claimed slots in
// temp order.
void launch_newlist_sources(const MergeArgs &a, const u64 *newoff, hipStream_t s);
// Direct product level (see MergeArgs::out_src): ids base + newoff[u] + i for
// the claimed entries of source u in entry order (visited array, state
// arrays and the entries' target column).  The other targets the level
// marked with a slot keep the mark until launch_fix_marked.
void launch_assign_direct(const MergeArgs &a, const u64 *newoff, u32 base, u32 *sq1, u32 *sq2,
                          hipStream_t s);
// The n target entries from a.out_dst + a.out_base: every one still marked
// with a visited-array slot replaced by that slot's id (once every level
// that marked them has assigned its ids; several levels in one pass).
void launch_fix_marked(const MergeArgs &a, u64 n, hipStream_t s);
// Removes the entries without a term (src = kHoleSrc) from the n result rows
// at out_base: source u's merged arcs move from out_base + poff[u] to
// out_base + aoff[u] (aoff: exclusive scan of merged arcs per source), through
// `tmp` (20 n bytes).
void launch_close_holes(const MergeArgs &a, const u64 *aoff, u64 n, void *tmp, hipStream_t s);
const u64 *launch_newlist(const MergeArgs &a, const u64 *bigoff, u32 nbig, u64 RB, u32 *wcnt,
                          u64 *woff, void *scan_state, hipStream_t s);
// Composition without reduction: every record of the level becomes an arc
// (osrc.. at [0, R)), its target pair claimed in the visited table and each
// new claim flagged in `newbits` (one bit per table slot, cleared by the
// caller); odst receives table slots until launch_fix_dst maps them to ids.
void launch_unreduced(const MergeArgs &a, bool wide_keys, u32 *newbits, u32 *osrc, u32 *odst,
                      u32 *oil, u32 *ool, float *ow, hipStream_t s);
// New-state list from the claim bitmap, in slot order (st->nnew = its
// length).  wcnt: bitlist_waves(nwords) u32; woff: that + 1 u64; scan_tmp:
// scan_temp_bytes(bitlist_waves(nwords)) bytes.
u64 bitlist_waves(u64 nwords);
void launch_bitlist(const u32 *bits, u64 nwords, u32 *list, u64 cap, u32 *wcnt, u64 *woff,
                    void *scan_tmp, Status *st, hipStream_t s);
// dst[k] = hvals[dst[k]] for k < n.
void launch_fix_dst(u32 *dst, u64 n, const u32 *hvals, hipStream_t s);
void launch_finals(const u32 *sq1, const u32 *sq2, u64 n, const uint8_t *f1, const uint8_t *f2,
                   uint8_t *fin, hipStream_t s);
// It also copies *st to `host` (pinned, coherent host memory the device can
// write) and then sets host->seq = seq, so that the host can wait for the
// copy by watching that word (the count scan's last tile does the same
// after the level's first phase, ScanPublish).
// Level total of merged arcs, new pairs (*new_total, when not NULL), the
// product merge's joined pairs (*pair_total: the sum of a.pcnt over the
// level's sources, records included, less st->R) and the dense / sort tile
// statistics of st; after publishing it clears the level counters of *st
// for the next level (what launch_reset_level does).
void launch_merged_total(const u64 *a_total, const u64 *new_total, const u64 *pair_total,
                         const MergeArgs &a, Status *host, u32 seq, hipStream_t s);
void launch_reset_level(Status *st, hipStream_t s);
// The 32-bit words of Status that the level-counter clearing zeroes (bit i:
// word i), for a publication that clears them itself (ScanPublish).
u64 level_clear_mask();

// One-workgroup product level (merge.hip, k_product_level): a level of at
// most kTinySources sources, every one a strided product source (the four-
// source matrix-core form) with the dense visited array, taken whole by one
// workgroup: selection, entry offsets, the product merge, id assignment,
// the level totals and their publication (as `seq`, with the counters
// cleared after), one launch instead of the per-level kernels (the targets
// another source claimed stay marked until launch_fix_marked).
// It changes nothing but the sources' headers when a source is of another
// form: then it publishes the counters with `declined` set (and clears
// nothing) and the level takes the per-level kernels.  The result columns
// must hold out_base + nsrc * 64 rows and the state arrays base + nsrc * 64
// entries; la's pk, phdr, tstart, mend, newc and cnt arrays and poff (also
// ma.poff, written here) nsrc + 1.
constexpr u32 kTinySources = 64;
void launch_product_level(const LevelArgs &la, const MergeArgs &ma, u64 *poff, u64 *newoff,
                          u32 base, u32 *sq1, u32 *sq2, Status *host, u32 seq, hipStream_t s);

}  // namespace fstc
