/*
 * fstc -- reachable-state weighted FST composition on AMD MI355X (gfx950).
 *
 * C ABI of the library libfstc.so.  Every step of the composition runs in
 * HIP kernels of this library; the caller supplies device buffers, a stream
 * and (optionally) an allocator.
 *
 * Method: Argueta & Chiang, "Composing Finite State Transducers on GPUs".
 *   - Transducer M = (Q, Sigma, Gamma, s, F, delta) and the composition
 *     M1 o M2 over state pairs: section 2.
 *   - Pair (q1 q2) -a:c/p1*p2-> (r1 r2) for every M1 arc q1 -a:b/p1-> r1 and
 *     M2 arc q2 -b:c/p2-> r2 sharing the inner symbol b; identical
 *     (source, target, input, output) arcs are merged by adding their
 *     weights: section 2 (arc rule and the sentence after it).
 *   - Only pairs reachable from the start pair are built, by a breadth-first
 *     search over pairs: section 3.1, section 3.2 (Algorithm 1) and
 *     section 3.4 (Algorithm 2; the device-resident frontier and visited set
 *     follow the future-work direction of section 5).
 *   - Transducer storage by (state, inner symbol): section 3.3.
 *
 * Semantics fixed by this library where the paper is silent:
 *   - Labels are ordinary symbols 0..n-1; there is no epsilon (section 2).
 *   - Input arcs are a multiset: listed duplicates each join separately.
 *   - Weights are float32 in the (+, x) semiring.  Each product p1*p2 is
 *     rounded to float32; merged sums are accumulated in float64 and rounded
 *     to float32 once.  Arcs exist regardless of weight (zero weights kept).
 *   - State ids of the result are dense, 0 is the start pair, ids grow with
 *     breadth-first depth.  Within one depth the numbering is unspecified
 *     unless opts->deterministic_ids is set (then ordered by (q1, q2)).
 *   - Result arcs are grouped by source id in increasing id order; within a
 *     source they are ordered by (target q1, input, target q2, output) ranks.
 */
#ifndef FSTC_H
#define FSTC_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes.  No exception crosses the ABI. */
enum {
  FSTC_OK = 0,
  FSTC_ERR_INVALID_ARG = 1, /* null pointer, start >= num_states, an arc's
                               state or label out of range (checked on the
                               device), num_states == 0, bad bit range */
  FSTC_ERR_ALPHABET = 2,    /* m1->num_osyms != m2->num_isyms (Gamma is
                               shared, section 2) */
  FSTC_ERR_RANGE = 3,       /* a size exceeds a packing limit: num_arcs or
                               num_states >= 2^32, or a per-state key does not
                               fit the 64-bit sort keys (see fstc_compose) */
  FSTC_ERR_CAPACITY = 4,    /* result would exceed opts->max_states /
                               opts->max_arcs, or 2^32-1 states */
  FSTC_ERR_OOM = 5,         /* an allocation failed */
  FSTC_ERR_HIP = 6,         /* a HIP runtime call failed */
  FSTC_ERR_INTERNAL = 7     /* a device-side consistency check failed */
};

/* A weighted transducer as a coordinate list of arcs, all arrays in device
 * memory, owned by the caller and only read during a call.  Arc k is
 * src[k] -ilabel[k]:olabel[k]/weight[k]-> dst[k]. */
typedef struct fstc_fst {
  uint32_t num_states;   /* |Q| >= 1                                    */
  uint32_t start;        /* s, < num_states                             */
  uint32_t num_isyms;    /* input alphabet size (labels < num_isyms)    */
  uint32_t num_osyms;    /* output alphabet size (labels < num_osyms)   */
  uint64_t num_arcs;     /* < 2^32; may be 0                            */
  const uint32_t *src;   /* [num_arcs] source state                     */
  const uint32_t *dst;   /* [num_arcs] target state                     */
  const uint32_t *ilabel;/* [num_arcs] input symbol                     */
  const uint32_t *olabel;/* [num_arcs] output symbol                    */
  const float *weight;   /* [num_arcs] weight                           */
  const uint8_t *final;  /* [num_states] nonzero = accept state (F)     */
} fstc_fst;

/* Optional allocator.  alloc returns device memory of at least `bytes`
 * usable on `stream` (NULL on failure); free returns it.  Both are called
 * from the calling thread only.  With alloc == NULL the library uses
 * hipMallocAsync / hipFreeAsync on the stream. */
typedef void *(*fstc_alloc_fn)(size_t bytes, void *ctx, hipStream_t stream);
typedef void (*fstc_free_fn)(void *ptr, size_t bytes, void *ctx, hipStream_t stream);

typedef struct fstc_opts {
  uint32_t max_levels;        /* 0: no cap.  L > 0: expand only pairs at
                                 breadth-first depth < L; depth-L pairs are
                                 states without out-arcs                  */
  uint32_t deterministic_ids; /* nonzero: ids within each depth ordered by
                                 (q1, q2)                                  */
  uint64_t max_states;        /* 0: no cap beyond 2^32-1                   */
  uint64_t max_arcs;          /* 0: no cap                                 */
  fstc_alloc_fn alloc;        /* NULL: hipMallocAsync                      */
  fstc_free_fn free;
  void *alloc_ctx;
  uint32_t no_reduction;      /* nonzero: no merging of identical arcs --
                                 every joined arc pair is an arc of the
                                 result with weight p1 * p2 (the setting the
                                 paper compares against in section 4, Table 2);
                                 the states are the same, num_arcs equals
                                 num_premerge_arcs and arcs keep no order
                                 within a source                          */
  uint32_t fused_merge;       /* nonzero: on levels whose sources all fit a
                                 merge tile and whose keys fit the dense
                                 table, generate each tile's composed arcs
                                 inside the merge (section 5's direction of
                                 keeping intermediate data on chip) instead
                                 of writing and re-reading them; same
                                 result                                   */
  uint32_t no_product_merge;  /* nonzero: every source goes through written
                                 records (count, write, sort/table merge) as
                                 the paper describes.  0: a source whose two
                                 states have few (target, outer symbol)
                                 pairs, whose arcs fill their (pair, inner
                                 symbol) cells densely and at most once
                                 each, is merged by one wavefront from its
                                 two arc matrices (sum over matched symbols
                                 of float32 products, added in float64),
                                 without records.  Same states and arcs;
                                 weights agree to float64 rounding        */
  uint32_t hash_visited;      /* nonzero: the visited set is always the hash
                                 table of pair keys.  0: it is a dense array
                                 indexed by q1 |Q2| + q2 (the paper's
                                 |Q1||Q2| table, section 3.4), 4 bytes a
                                 pair, when |Q1| |Q2| is at most 2^26, and
                                 the hash table otherwise, moved into such
                                 an array between two levels once the table
                                 would need as many bytes as the array and
                                 |Q1| |Q2| is at most 2^30; same result    */
  uint32_t phase_timing;      /* with stats: nonzero times every phase
                                 (ms_csr .. ms_assign) with HIP events at
                                 each phase boundary.  0: only the kernels
                                 behind ms_write_kernel, ms_merge_kernel,
                                 ms_sort_kernel and ms_product_kernel are
                                 timed, one event before and one after each
                                 launch, and the phase times are 0 (every
                                 event costs the stream a few microseconds) */
  uint32_t hash_min_log2;     /* 0: the hash table of pair keys is sized by
                                 the reachable pairs (load at most 1/2).
                                 1..31: it has at least 2^hash_min_log2 slots
                                 from the start (2^31 slots take 24 GiB);
                                 for tests of large slot numbers.  Values
                                 above 31 give FSTC_ERR_INVALID_ARG       */
  uint32_t no_small_levels;   /* nonzero: every level takes the per-level
                                 kernels.  0: while a level has at most 512
                                 pairs and 1,024 joined arc pairs (at most
                                 64 per pair, symbol lists of at most 32
                                 and 4,096), one workgroup joins, merges,
                                 numbers the new
                                 pairs (in (q1, q2) order) and appends the
                                 arcs of it and of the levels after it in
                                 one launch (composition with reduction only;
                                 the result is the same composition)        */
} fstc_opts;

/* Composition result.  All arrays are device memory obtained from the
 * allocator of the call; release them with fstc_result_release. */
typedef struct fstc_result {
  uint64_t num_states;        /* reachable pairs (within the level cap)     */
  uint64_t num_arcs;          /* merged composed arcs                       */
  uint64_t num_premerge_arcs; /* arc pairs joined (before merging)          */
  uint32_t num_levels;        /* breadth-first depths present (max depth+1) */
  uint32_t reserved0;
  uint32_t *state_q1;         /* [num_states] q1 of each state id           */
  uint32_t *state_q2;         /* [num_states] q2 of each state id           */
  uint8_t *final;             /* [num_states] 1 iff q1 in F1 and q2 in F2   */
  uint32_t *src;              /* [num_arcs] source state id                 */
  uint32_t *dst;              /* [num_arcs] target state id                 */
  uint32_t *ilabel;           /* [num_arcs] input symbol (from Sigma)       */
  uint32_t *olabel;           /* [num_arcs] output symbol (from Delta)      */
  float *weight;              /* [num_arcs] merged weight                   */
  void *alloc_ptr[8];         /* allocation records, for release only (the
                                 arrays may share allocations: the five arc
                                 arrays are columns of one)               */
  size_t alloc_bytes[8];
} fstc_result;

/* Per-call statistics (all optional to read). Times from HIP events on the
 * call's stream, in milliseconds; the phase times need opts->phase_timing. */
typedef struct fstc_stats {
  uint32_t num_levels;        /* breadth-first levels expanded              */
  uint32_t num_host_syncs;
  uint64_t max_frontier;      /* largest number of pairs expanded at once   */
  uint64_t max_level_premerge;/* largest per-level unmerged arc count       */
  uint64_t big_sources;       /* sources merged by the multi-block path     */
  uint64_t hash_capacity;     /* final visited-table capacity (slots)       */
  double ms_total;            /* whole call, host wall clock                */
  double ms_csr;              /* both (state, inner symbol) CSR builds      */
  double ms_count;            /* join counting + scans                      */
  double ms_expand;           /* match emission + arc-pair write pass       */
  double ms_merge;            /* segmented sort + reduce + visited inserts  */
  double ms_assign;           /* id assignment + result append              */
  double ms_write_kernel;     /* arc-pair write kernel alone, all levels    */
  double ms_merge_kernel;     /* dense-table merge kernel alone, all levels */
  uint32_t write_launches;    /* launches of the arc-pair write kernel      */
  uint32_t merge_launches;    /* launches of the dense-table merge kernel   */
  uint64_t total_matches;     /* matched (source, inner symbol) pairs       */
  uint64_t total_big_records; /* records merged by the multi-block path     */
  uint32_t record_key_bytes;  /* 4 or 8: key width of an unmerged record    */
  uint32_t key_bits;          /* part-rank bits of a record key             */
  double ms_sort_kernel;      /* sorting merge-tile kernel alone            */
  uint32_t sort_launches;     /* launches of the sorting merge-tile kernel  */
  uint32_t fused_levels;      /* levels merged by the fused kernel         */
  uint64_t total_dense_records; /* records merged through the dense table   */
  uint64_t total_dense_runs;  /* merged arcs the dense table produced        */
  uint64_t total_sort_runs;   /* merged arcs the sorting tiles produced      */
  uint64_t total_product_records; /* joined arc pairs merged by the product
                                     merge (never written as records)         */
  uint64_t total_product_sources; /* sources merged by the product merge      */
  double ms_product_kernel;   /* product-merge kernel alone, all levels      */
  uint32_t product_launches;  /* launches of the product-merge kernel        */
  uint32_t visited_form;      /* 0: hash table of pair keys throughout; 1:
                                 dense |Q1||Q2| array from the start; 2: the
                                 hash table moved into the dense array
                                 between two levels                        */
  uint64_t total_product_mfma_sources; /* of those, sources whose sums ran on
                                          the matrix cores (float64 MFMA)     */
  uint32_t direct_product_levels; /* levels of product-merge sources alone whose
                                     merged arcs the product kernel wrote
                                     straight into the result              */
  uint32_t small_levels;      /* levels done by the one-workgroup kernel
                                 (opts.no_small_levels)                     */
  uint64_t peak_device_bytes; /* largest amount of device memory the call held
                                 from its allocator at one time (result
                                 arrays and temporaries)                    */
  uint32_t group_product_levels; /* direct product levels of at most 64
                                    pairs that one workgroup took whole
                                    (counted in direct_product_levels too;
                                    off with opts.no_small_levels)          */
  uint32_t reserved2;
} fstc_stats;

/*
 * fstc_compose: the reachable part of m1 o m2 (Algorithm 1 / Algorithm 2).
 *
 *   m1, m2   transducers; m1->num_osyms must equal m2->num_isyms.
 *   opts     may be NULL (defaults: no caps, hipMallocAsync).
 *   stream   all work is ordered on this stream.  The call blocks the host
 *            a few times per breadth-first level to read sizes, and returns
 *            when every result size is known; result buffers are valid once
 *            `stream` has completed.
 *   out      receives the result (zeroed on error; nothing to release then).
 *   stats    may be NULL.
 *
 * Limits: num_arcs < 2^32 per input; state ids < 2^32 - 1; with
 * P1 / P2 the largest number of distinct (target, outer symbol) pairs among
 * the arcs leaving one state of m1 / m2, bits(P1-1) + bits(P2-1) <= 40
 * (else FSTC_ERR_RANGE).
 *
 * Threads: calls made from different host threads, each on a stream of its
 * own, may overlap on one GPU (the host-visible staging block, side streams
 * and event pool are per thread, temporaries per call).  The same holds for
 * fstc_compose_eps.
 */
int fstc_compose(const fstc_fst *m1, const fstc_fst *m2, const fstc_opts *opts,
                 hipStream_t stream, fstc_result *out, fstc_stats *stats);

/*
 * fstc_compose_eps: M1∘M2 with epsilon transitions.  The paper admits no
 * epsilon transitions (§2) and names composition filters as what admitting
 * them takes; this entry point takes the three-state epsilon filter (Mohri,
 * Pereira and Riley; Allauzen, Riley and Schalkwyk 2009), under which every
 * pair of paths of M1 and M2 with matching middle strings is aligned exactly
 * once, so that the result's weight on an (input, output) string pair is the
 * sum over middle strings y of M1's weight on (input, y) times M2's on
 * (y, output), the empty string removed.
 *
 *   eps            the label value that stands for the empty string on every
 *                  tape; it must be a symbol of all four alphabets
 *                  (eps < m1->num_isyms, m1->num_osyms = m2->num_isyms,
 *                  m2->num_osyms; else FSTC_ERR_INVALID_ARG).
 *   state_filter   may be NULL; receives a device array [num_states] of the
 *                  filter state of each state, owned by the result (freed by
 *                  fstc_result_release).
 *   other arguments as for fstc_compose; opts->max_levels caps the depth in
 *   moves of the composed search, the caps apply to the result.
 *
 * The result's states are triples (q1, q2, f): state_q1 / state_q2 hold q1 and
 * q2, state_filter f, id 0 = (start1, start2, 0).  Its arcs (the moves the
 * filter allows out of a triple, merged as fstc_compose merges unless
 * opts->no_reduction):
 *   - an M1 arc with output b != eps and an M2 arc with input b, from any f,
 *     to f = 0: input and output labels of the two arcs, weight p1 * p2;
 *   - an M1 arc with output eps and an M2 arc with input eps, from f = 0, to
 *     f = 0, likewise;
 *   - an M1 arc with output eps alone (M2 stays), from f = 0 or 2, to f = 2:
 *     labels (M1 input, eps), weight p1;
 *   - an M2 arc with input eps alone (M1 stays), from f = 0 or 1, to f = 1:
 *     labels (eps, M2 output), weight p2.
 * Accept states: q1 in F1 and q2 in F2, whatever f.  num_premerge_arcs counts
 * the moves.  Triples from which no accepting state is reachable are kept
 * (reachable states only, as fstc_compose).
 *
 * It runs as two epsilon-free compositions, (M1' ∘ F) ∘ M2', with the filter
 * F a three-state transducer and M1', M2' relabelled copies of the inputs
 * (output / input eps renamed, a weight-one loop per state); the first has
 * at most 3 |Q1| states.  Needs num_arcs + num_states < 2^32 per input.
 */
int fstc_compose_eps(const fstc_fst *m1, const fstc_fst *m2, uint32_t eps,
                     const fstc_opts *opts, hipStream_t stream, fstc_result *out,
                     uint8_t **state_filter, fstc_stats *stats);

/* Frees every buffer of a result obtained from fstc_compose (or
 * fstc_compose_eps) with the same opts (allocator) and zeroes *r.  Safe on a
 * zeroed result. */
void fstc_result_release(fstc_result *r, const fstc_opts *opts, hipStream_t stream);

/*
 * fstc_build_csr: the transducer layout of section 3.3 as the composition
 * uses it, built on the device (the paper sorts on the host).
 *
 * Arcs are grouped by source state, then by inner symbol (output symbol when
 * by_output != 0, as for M1; input symbol otherwise, as for M2), then by
 * part (below), then by input position.  Instead of
 * the dense offset array R[|Q| m + 1] of section 3.3, the layout is two-level:
 *   row[q] .. row[q+1]       segments of state q            [num_states+1]
 *   seg_sym[k]               inner symbol of segment k      [num_segments]
 *   seg_off[k] .. seg_off[k+1]  arcs of segment k           [num_segments+1]
 *   arc_part[j], arc_weight[j]  arc j in that order          [num_arcs]
 *   part_base[q]             first part of state q           [num_states+1]
 *   part_target[i], part_outer[i]  distinct (target, outer symbol) of the
 *                            arcs of a state, ordered       [num_parts]
 * arc_part[j] is the rank of arc j's (target, outer symbol) among its
 * state's distinct pairs, so its pair is part_*[part_base[q] + arc_part[j]].
 * All output arrays are device memory of the caller, sized by
 * num_states + 1 and num_arcs (segments and parts never exceed num_arcs).
 * counts[0..2] (host) receive num_segments, num_parts and the largest number
 * of parts of one state.
 */
int fstc_build_csr(const fstc_fst *m, int by_output, hipStream_t stream, uint32_t *row,
                   uint32_t *seg_sym, uint32_t *seg_off, uint32_t *arc_part,
                   float *arc_weight, uint32_t *part_base, uint32_t *part_target,
                   uint32_t *part_outer, uint64_t *counts);

/*
 * fstc_sort_pairs: stable LSD radix sort of (key, value) pairs on key bits
 * [bit_lo, bit_hi) (0 <= bit_lo <= bit_hi <= 64), in place on the device.
 * This is the sort the library uses for the CSR build, for merging large
 * sources and for deterministic ids (section 3.4 "Reduction" sorts packed
 * 64-bit keys).  keys, values: device [n]; n < 2^32.  Temporaries come from
 * hipMallocAsync on the stream.
 */
int fstc_sort_pairs(uint64_t *keys, uint32_t *values, uint64_t n, int bit_lo, int bit_hi,
                    hipStream_t stream);

/* Exclusive prefix sum out[i] = sum_{j<i} in[j] for i in [0, n]
 * (n + 1 outputs; out[n] is the total).  Device arrays. */
int fstc_exclusive_scan_u64(const uint64_t *in, uint64_t *out, uint64_t n, hipStream_t stream);

/*
 * fstc_exclusive_scan_u64_noalloc: the same scan as fstc_exclusive_scan_u64
 * (same arguments, results and return codes), for callers that cannot
 * allocate device memory (code that must not call hipMalloc or hipFree:
 * tight serving loops, harnesses that forbid allocation).  It allocates
 * nothing: the scan's temporaries (tile counter, error word, look-back state
 * of every 2048-element tile) live in a file-scope device array of the
 * library, about 17.8 MB, that each GPU it runs on holds until the process
 * ends.  The first call on a device looks the array up and clears it
 * (synchronising `stream`).  n is at most 2^28 (larger n: FSTC_ERR_RANGE,
 * nothing launched).  Every call on one GPU shares that GPU's array: calls
 * that overlap in time on one GPU, from any stream or thread, race and must
 * not be made.  Synchronises `stream` before returning.
 */
int fstc_exclusive_scan_u64_noalloc(const uint64_t *in, uint64_t *out, uint64_t n,
                                    hipStream_t stream);

/* Text for a return code, and thread-local detail of the last failure. */
const char *fstc_strerror(int code);
const char *fstc_last_error_detail(void);

/* Library version, e.g. "0.1.0". */
const char *fstc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FSTC_H */
