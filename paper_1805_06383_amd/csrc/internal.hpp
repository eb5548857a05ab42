// Internal interfaces between the translation units of libfstc.
#pragma once

#include <vector>

#include "common.hpp"

namespace fstc {

// ---------------------------------------------------------------------------
// Device memory from the caller's allocator (or hipMallocAsync), stream
// ordered on the call's stream.
struct Allocator {
  fstc_alloc_fn fa = nullptr;
  fstc_free_fn ff = nullptr;
  void *ctx = nullptr;
  hipStream_t stream = nullptr;
  u64 live_bytes = 0, peak_bytes = 0;

  void *alloc(size_t bytes);
  void free(void *p, size_t bytes);
};

// Smallest capacity (in 4-byte entries) of a buffer grown with grow_keep.
constexpr size_t kMinGrow = (size_t)1 << 18;
// State arrays start with room for every state pair when there are at most
// this many (16 MB per array).
constexpr size_t kStatePresize = (size_t)1 << 22;

// Grow-only device buffer owned by a compose call.
struct Buf {
  Allocator *A = nullptr;
  void *p = nullptr;
  size_t cap = 0;

  Buf() = default;
  explicit Buf(Allocator *a) : A(a) {}
  Buf(const Buf &) = delete;
  Buf &operator=(const Buf &) = delete;
  ~Buf() { release(); }

  void release() {
    if (p) A->free(p, cap);
    p = nullptr;
    cap = 0;
  }
  // At least `bytes`; previous contents are not kept.
  void *ensure(size_t bytes);
  // At least `bytes`, keeping the first `used` bytes.
  void *grow_keep(size_t bytes, size_t used);
  template <class T>
  T *as() const { return static_cast<T *>(p); }
  // Hands the allocation to the caller (no free on destruction).
  void *detach(size_t *bytes) {
    void *q = p;
    *bytes = cap;
    p = nullptr;
    cap = 0;
    return q;
  }
};

// Bump allocator for temporaries that die together (one breadth-first level,
// one CSR build): takes from its last chunk and, when that is full, adds one
// as large as the round's takes so far plus the request; reset() frees every
// chunk and, when there were several, keeps one of 1.5 times the largest
// round's takes, so that after the first rounds a round costs no allocator
// call and the arena holds what the rounds use.  Frees are stream ordered
// (like Buf), so a reset while kernels still read the old chunks is safe.
struct Arena {
  Allocator *A = nullptr;
  struct Chunk {
    char *p;
    size_t cap;
  };
  std::vector<Chunk> chunks;
  size_t used = 0;        // bytes taken from the last chunk
  size_t round_bytes = 0;  // bytes taken in this round, all chunks
  size_t high = 0;         // largest round_bytes of any round so far
  u64 epoch = 0;  // incremented by reset(): handles from older rounds are stale
  // When set, a take that needs a new chunk throws instead (an arena whose
  // memory another stream uses must not allocate on the owning stream then).
  bool fixed = false;

  explicit Arena(Allocator *a) : A(a) {}
  Arena(const Arena &) = delete;
  Arena &operator=(const Arena &) = delete;
  ~Arena() { release(); }
  void *take(size_t bytes);
  // Makes the next round's takes of up to `bytes` in all come from one
  // allocation (call right after construction or reset()).
  void reserve(size_t bytes);
  void reset();
  void release();
};

// A buffer of the current round of an Arena, with Buf's interface.
struct Tmp {
  Arena *T = nullptr;
  void *p = nullptr;
  u64 epoch = 0;

  explicit Tmp(Arena *t) : T(t) {}
  void *ensure(size_t bytes) {
    p = T->take(bytes);
    epoch = T->epoch;
    return p;
  }
  template <class X>
  X *as() const {
    if (p && epoch != T->epoch) throw Error(FSTC_ERR_INTERNAL, "stale arena buffer");
    return static_cast<X *>(p);
  }
};

// ---------------------------------------------------------------------------
// Two-level (state, inner symbol) layout of one input transducer.
struct Csr {
  u32 num_states = 0;
  u64 num_arcs = 0;
  u32 *row = nullptr;        // [num_states + 1] -> segment index
  u32 *seg_sym = nullptr;    // [num_arcs] inner symbol of segment
  u32 *seg_off = nullptr;    // [num_arcs + 1] -> arc index
  uint2 *arcs = nullptr;     // [num_arcs + kArcTail] (part rank within state, weight bits)
  u32 *part_base = nullptr;  // [num_states + 1]
  uint2 *parts = nullptr;    // [num_arcs] (target, outer symbol)
  u32 *cell_flag = nullptr;  // [num_states] see build_cell_flags (compose only)
  u32 *wts = nullptr;        // [num_arcs + kArcTail] arcs[j].y alone, zeros after the
                             // last arc (compose only, build_cell_flags)
};

// The arc array of a CSR built for composition (alloc_csr) has kArcTail
// spare entries after its last arc, so that kArcTail consecutive arcs may be
// loaded from any arc index (the values past the end are garbage).
constexpr u32 kArcTail = 4;

// Device counters written by the CSR build: [0] segments, [1] parts,
// [2] max parts of one state.
void build_csr(const fstc_fst &m, bool by_output, Arena &T, const Csr &out, u64 *d_counts,
               u32 *d_err, hipStream_t s);

// Both inputs' layouts on stream s, the steps of the two builds sharing
// their launches (with `flags` the cell flags and weight words too, see
// build_cell_flags), when both inputs take the per-state build; otherwise
// enqueues nothing and returns false.
bool build_csr_pair(const fstc_fst &m1, bool by_output1, Arena &T1, const Csr &c1,
                    u64 *d_counts1, const fstc_fst &m2, bool by_output2, Arena &T2,
                    const Csr &c2, u64 *d_counts2, bool flags, u32 *d_err, hipStream_t s);

// Largest part count of a state the product merge takes (level.hpp).
constexpr u32 kProdParts = 64;

// cell_flag[q] has bit kCellBad when state q has more than kProdParts parts
// or two arcs with the same part and inner symbol (parallel arcs with equal
// labels and target).  Otherwise it summarises the state's arc weights: bit
// kCellSpecial when one is infinite, NaN or subnormal, and the largest and
// smallest biased float32 exponents of its nonzero weights (0 and 255 in
// those fields when it has none), and bit kCellDense when every one of its
// segments holds exactly one arc per part (segment i's arcs are then the P
// consecutive arcs from the state's first plus P i), and kCellIdent besides
// when, in every segment, arc j has part j (the per-state builds order a
// segment's arcs by part).
// kCellContig: the state's inner symbols are consecutive.
constexpr u32 kCellBad = 1u, kCellSpecial = 2u, kCellDense = 4u, kCellIdent = 8u,
              kCellContig = 16u;
constexpr int kCellEmaxShift = 8, kCellEminShift = 16;
// Also fills c.wts.
void build_cell_flags(const Csr &c, u32 *cell_flag, hipStream_t s);

// Checks the packing limits of build_csr for one transducer; throws
// Error(FSTC_ERR_RANGE) when a key does not fit 64 bits.
void check_csr_ranges(const fstc_fst &m, bool by_output);

// Allocates the arrays of a Csr (cell flags included) as parts of one
// buffer and fills `out`.
void alloc_csr(const fstc_fst &m, Buf &buf, Csr &out);
// Arena bytes build_csr takes for m (either direction).
size_t csr_temp_bytes(const fstc_fst &m);

// Exclusive scan of n u64 values (out has n + 1 entries) using the device's
// file-scope scratch array instead of allocated temporaries (noalloc.hip);
// n at most noalloc_scan_max_n().  Synchronises the stream.
// Composition with epsilon transitions (eps.hip): the relabelled inputs and
// the filter transducer of the filter composition (M1' ∘ F) ∘ M2', and the
// map of its states back to (q1, q2, filter state).
// M1' (by_output: output eps -> e_rename, loops eps:e_loop) or M2' (input
// eps -> e_rename, loops e_loop:eps): num_arcs + num_states arcs.
void build_eps_side(const fstc_fst &m, bool by_output, u32 eps, u32 e_rename, u32 e_loop,
                    u32 *src, u32 *dst, u32 *il, u32 *ol, float *w, hipStream_t s);
// F over nsym inner symbols (E1 = nsym, E2 = nsym + 1): 3 (nsym - 1) + 5 arcs,
// 3 states, all accepting.
void build_eps_filter(u32 nsym, u32 eps, u32 *src, u32 *dst, u32 *il, u32 *ol, float *w,
                      uint8_t *final, hipStream_t s);
// q1[i] (a state of M1' ∘ F) -> aq1[q1[i]]; filt[i] = af[q1[i]].
void map_eps_states(u32 *q1, const u32 *aq1, const u32 *af, u64 n, uint8_t *filt,
                    hipStream_t s);

u64 noalloc_scan_max_n();
void noalloc_scan(const u64 *in, u64 *out, u64 n, hipStream_t s);

}  // namespace fstc
