// Internal interfaces between the translation units of libfstc.
#pragma once

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

// ---------------------------------------------------------------------------
// Two-level (state, inner symbol) layout of one input transducer.
struct Csr {
  u32 num_states = 0;
  u64 num_arcs = 0;
  u32 *row = nullptr;        // [num_states + 1] -> segment index
  u32 *seg_sym = nullptr;    // [num_arcs] inner symbol of segment
  u32 *seg_off = nullptr;    // [num_arcs + 1] -> arc index
  uint2 *arcs = nullptr;     // [num_arcs] (part rank within state, weight bits)
  u32 *part_base = nullptr;  // [num_states + 1]
  uint2 *parts = nullptr;    // [num_arcs] (target, outer symbol)
};

// Device counters written by the CSR build: [0] segments, [1] parts,
// [2] max parts of one state.
void build_csr(const fstc_fst &m, bool by_output, Allocator &A, const Csr &out, u64 *d_counts,
               u32 *d_err, hipStream_t s);

// Checks the packing limits of build_csr for one transducer; throws
// Error(FSTC_ERR_RANGE) when a key does not fit 64 bits.
void check_csr_ranges(const fstc_fst &m, bool by_output);

// Allocates the arrays of a Csr in `bufs` (7 buffers) and fills `out`.
void alloc_csr(const fstc_fst &m, Allocator &A, Buf *bufs, Csr &out);

}  // namespace fstc
