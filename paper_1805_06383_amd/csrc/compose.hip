// Host driver of the composition and the C ABI (include/fstc.h).
//
// Algorithm 2 of the paper keeps the frontier queue on the host and
// launches work per popped pair, which the authors name as the largest
// bottleneck (section 5).  Here the frontier and the visited set live on the
// device and a whole breadth-first level is expanded per step:
//
//   per level (sources = the state ids found at the previous level):
//     count + scan          -> records and matches per source      (sync 1)
//     emit + write          -> unmerged composed arcs (records)
//     merge                 -> merged arcs, new pairs claimed in the hash
//     scan                  -> merged arcs per source              (sync 2)
//     assign + append       -> ids for new pairs, arcs to the result
//
// The host reads a few counters twice per level; everything else stays in
// HBM.  Buffers are grow-only and come from the caller's allocator (PyTorch's
// caching allocator in the Python binding) or hipMallocAsync.
#include <array>
#include <chrono>
#include <cstring>
#include <functional>
#include <mutex>
#include <vector>

#include "level.hpp"

namespace fstc {

// ---------------------------------------------------------------------------
void *Allocator::alloc(size_t bytes) {
  bytes = std::max<size_t>(256, (bytes + 255) & ~(size_t)255);
  void *p = nullptr;
  if (fa) {
    p = fa(bytes, ctx, stream);
  } else {
    if (hipMallocAsync(&p, bytes, stream) != hipSuccess) p = nullptr;
    if (!p) (void)hipGetLastError();
  }
  if (!p) throw Error(FSTC_ERR_OOM, "device allocation of " + std::to_string(bytes) + " bytes failed");
  live_bytes += bytes;
  peak_bytes = std::max(peak_bytes, live_bytes);
  return p;
}

void Allocator::free(void *p, size_t bytes) {
  if (!p) return;
  bytes = std::max<size_t>(256, (bytes + 255) & ~(size_t)255);
  if (ff) ff(p, bytes, ctx, stream);
  else (void)hipFreeAsync(p, stream);
  live_bytes -= std::min<u64>(live_bytes, bytes);
}

void *Buf::ensure(size_t bytes) {
  if (bytes <= cap && p) return p;
  release();
  const size_t c = std::max<size_t>(256, (bytes + 255) & ~(size_t)255);
  p = A->alloc(c);
  cap = c;
  return p;
}

// Growth factor of the grow-only arrays: 4 while they are small (fewer and
// smaller copies of what they hold), 2 from kFastGrowBytes on.
constexpr size_t kFastGrowBytes = size_t(1) << 28;
// Largest inner alphabet for which a composition without reduction counts
// the arcs per inner symbol to bound its result (two 16 MB histograms).
constexpr u64 kJoinBoundSyms = u64(1) << 22;
// Largest state or result arrays sized from the level's bounds (see the
// early append in the level loop).
constexpr u64 kEarlyBytes = u64(1) << 30;
// Largest temp (entries x 20 bytes) reserved for a speculative product merge.
constexpr u64 kSpecBytes = u64(1) << 30;
inline size_t grown(size_t cap_bytes) { return cap_bytes * (cap_bytes < kFastGrowBytes ? 4 : 2); }

void *Buf::grow_keep(size_t bytes, size_t used) {
  if (bytes <= cap && p) return p;
  const size_t c = std::max<size_t>(std::max<size_t>(kMinGrow * 4, (bytes + 255) & ~(size_t)255),
                                    grown(cap));
  void *q = A->alloc(c);
  if (used && p) FSTC_HIP(hipMemcpyAsync(q, p, used, hipMemcpyDeviceToDevice, A->stream));
  release();
  p = q;
  cap = c;
  return p;
}

// A round that outgrows the arena adds a chunk as large as everything the
// round has taken so far plus the request (so a round needs a logarithmic
// number of chunks), and the next reset() folds the chunks into one
// allocation of 1.5 times the largest round seen: the arena tracks what the
// rounds use, not the sum of its chunks.
void *Arena::take(size_t bytes) {
  bytes = std::max<size_t>(256, (bytes + 255) & ~(size_t)255);
  if (chunks.empty() || used + bytes > chunks.back().cap) {
    if (fixed) throw Error(FSTC_ERR_INTERNAL, "fixed arena exhausted");
    const size_t c = std::max<size_t>((size_t)1 << 20, round_bytes + bytes);
    chunks.push_back({static_cast<char *>(A->alloc(c)), c});
    used = 0;
  }
  void *p = chunks.back().p + used;
  used += bytes;
  round_bytes += bytes;
  high = std::max(high, round_bytes);
  return p;
}

void Arena::reserve(size_t bytes) {
  if (used || bytes == 0) return;
  size_t total = 0;
  for (auto &c : chunks) total += c.cap;
  if (total >= bytes) return;
  release();
  chunks.push_back({static_cast<char *>(A->alloc(bytes)), bytes});
}

void Arena::reset() {
  ++epoch;
  if (chunks.size() > 1) {
    const size_t c = ((high + high / 2) + 255) & ~(size_t)255;
    release();
    chunks.push_back({static_cast<char *>(A->alloc(c)), c});
  }
  used = 0;
  round_bytes = 0;
}

void Arena::release() {
  for (auto &c : chunks) A->free(c.p, c.cap);
  chunks.clear();
  used = 0;
  round_bytes = 0;
}

namespace {

thread_local std::string g_detail;

// Per-thread page-locked staging for the few counters the host reads.
struct Staging {
  Status st;
  u64 words[16];
};

// Coherent (fine-grained) pinned memory: the publishing kernels' stores
// reach the host while they run, so the host can watch st.seq.
Staging *staging() {
  thread_local Staging *p = nullptr;
  if (!p) {
    FSTC_HIP(hipHostMalloc((void **)&p, sizeof(Staging), hipHostMallocCoherent));
    std::memset(p, 0, sizeof(Staging));
  }
  return p;
}

// A second stream of this thread on the current device (default priority,
// not blocking on the null stream), created at first use and kept for the
// thread's lifetime, with one event for forking work onto it and one for
// joining it back.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
SideStream &side_stream() {
  thread_local std::array<SideStream, 64> ss{};
  int dev = 0;
  FSTC_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) throw Error(FSTC_ERR_INVALID_ARG, "device index too large");
  SideStream &x = ss[dev];
  if (!x.s) {
    FSTC_HIP(hipStreamCreateWithFlags(&x.s, hipStreamNonBlocking));
    FSTC_HIP(hipEventCreateWithFlags(&x.fork, hipEventDisableTiming));
    FSTC_HIP(hipEventCreateWithFlags(&x.join, hipEventDisableTiming));
  }
  return x;
}

// Makes `main` wait for everything queued on the side stream when it goes
// out of scope, on every path (an exception included), so that frees
// ordered on `main` come after the side stream's kernels.
struct SideJoin {
  hipStream_t main;
  SideStream &side;
  ~SideJoin() {
    (void)hipEventRecord(side.join, side.s);
    (void)hipStreamWaitEvent(main, side.join, 0);
  }
};

// Publication numbers of this thread's staging block, never reused.
u32 next_publication() {
  thread_local u32 n = 0;
  return ++n;
}

// Keep freed blocks of the default stream-ordered pool instead of returning
// them to the driver at every synchronisation.
void tune_default_pool() {
  static std::once_flag once;
  std::call_once(once, [] {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return;
    hipMemPool_t pool;
    if (hipDeviceGetDefaultMemPool(&pool, dev) != hipSuccess) return;
    uint64_t thr = ~0ull;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
    (void)hipGetLastError();
  });
}

u64 next_pow2(u64 x) {
  u64 p = 1;
  while (p < x) p <<= 1;
  return p;
}

const char *device_error_text(u32 e) {
  if (e & kErrBadArc) return "an arc's state or label is out of range";
  if (e & kErrHashFull) return "visited table full";
  if (e & kErrNewList) return "new-state list overflow";
  if (e & kErrTileSize) return "merge tile exceeded its capacity";
  if (e & kErrScan) return "a single-pass scan timed out waiting for a predecessor tile";
  return "device index check failed";
}

enum Phase {
  kCsr, kCount, kExpand, kMerge, kAssign, kWriteKernel, kMergeKernel, kSortKernel,
  kProductKernel, kNumPhases, kNone = -1
};

inline bool kernel_phase(int p) { return p >= kWriteKernel && p < kNumPhases; }

// Timing with HIP events on the call's stream (only with stats).  T.at(p)
// marks a boundary: the current span ends there and a span of phase p (or
// none, kNone) begins.  With all phases on, every boundary records one event
// shared by the two spans; otherwise only boundaries of the single-kernel
// phases record one, so that a timed kernel costs two events.  Events are
// created once per thread and device and reused by later calls.
struct Timer {
  hipStream_t s = nullptr;
  bool on = false;   // stats wanted
  bool all = false;  // every phase, not just the kernel phases
  std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> spans;
  hipEvent_t open = nullptr;
  int cur = kNone;
  size_t used = 0;

  int device = -1;
  // events belong to the device current at their creation: one pool per device
  static std::vector<hipEvent_t> &pool(int dev) {
    static thread_local std::vector<std::vector<hipEvent_t>> p;
    if ((int)p.size() <= dev) p.resize(dev + 1);
    return p[dev];
  }
  hipEvent_t get() {
    if (device < 0) FSTC_HIP(hipGetDevice(&device));
    auto &p = pool(device);
    if (used == p.size()) {
      hipEvent_t e;
      FSTC_HIP(hipEventCreate(&e));
      p.push_back(e);
    }
    return p[used++];
  }
  bool want(int p) const { return p != kNone && (all || kernel_phase(p)); }
  void at(int next) {
    if (!on) return;
    if (want(cur) || want(next)) {
      hipEvent_t e = get();
      FSTC_HIP(hipEventRecord(e, s));
      if (want(cur) && open) spans.push_back({cur, {open, e}});
      open = want(next) ? e : nullptr;
    } else {
      open = nullptr;
    }
    cur = next;
  }
  void totals(double *ms) {
    for (auto &sp : spans) {
      float t = 0.f;
      if (hipEventElapsedTime(&t, sp.second.first, sp.second.second) == hipSuccess) ms[sp.first] += t;
    }
  }
};

// One wave publishes to the host's staging block (coherent pinned memory):
// nwords words (the CSR counts, then, with `lists`, the inner-symbol list
// lengths of the two start states as words 6 and 7), the status words but
// its sequence word, a system-scope fence, then the sequence word: the host
// waits for it (wait_published) instead of a copy and a stream
// synchronisation.
__global__ __launch_bounds__(kWave) void k_publish_counts(const u32 *row1, u32 s1, const u32 *row2,
                                                          u32 s2, int lists, const u64 *counts,
                                                          u32 nwords, const Status *st,
                                                          Status *host, u64 *host_words, u32 seq) {
  const u32 lane = threadIdx.x;
  u64 l1 = 0, l2 = 0;
  if (lists) {  // uniform
    l1 = row1[s1 + 1] - row1[s1];
    l2 = row2[s2 + 1] - row2[s2];
  }
  if (lane < nwords) host_words[lane] = lists && lane == 6 ? l1 : lists && lane == 7 ? l2 : counts[lane];
  const u32 *src = reinterpret_cast<const u32 *>(st);
  u32 *dst = reinterpret_cast<u32 *>(host);
  constexpr u32 kSeqWord = offsetof(Status, seq) / 4;
  for (u32 i = lane; i < sizeof(Status) / 4; i += kWave)
    if (i != kSeqWord) dst[i] = src[i];
  __threadfence_system();
  __builtin_amdgcn_wave_barrier();
  if (lane == 0) __hip_atomic_store(&host->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Histogram of the labels lab[0, n) below nsym into h (added to it); per
// workgroup in LDS first when the alphabet fits kHistLds entries.
constexpr u32 kHistLds = 8192;
__global__ __launch_bounds__(256) void k_label_hist(const u32 *lab, u64 n, u32 *h, u32 nsym) {
  __shared__ u32 sh[kHistLds];
  const bool lds = nsym <= kHistLds;  // uniform
  if (lds) {
    for (u32 i = threadIdx.x; i < nsym; i += blockDim.x) sh[i] = 0;
    __syncthreads();
  }
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x) {
    const u32 v = lab[i];
    if (v < nsym) atomicAdd(lds ? &sh[v] : &h[v], 1u);
  }
  if (lds) {
    __syncthreads();
    for (u32 i = threadIdx.x; i < nsym; i += blockDim.x)
      if (sh[i]) atomicAdd(&h[i], sh[i]);
  }
}

// *out = sum over i < nsym of h1[i] h2[i] (one workgroup of 1024 threads).
// With h1 / h2 the arc counts per inner symbol of the two inputs this is the
// number of joined arc pairs over all pairs of states, which bounds the arcs
// of a composition without reduction; it is below 2^64 because each input
// has fewer than 2^32 arcs.
__global__ __launch_bounds__(1024) void k_join_bound(const u32 *h1, const u32 *h2, u64 nsym,
                                                     u64 *out) {
  __shared__ u64 part[1024];
  u64 acc = 0;
  for (u64 i = threadIdx.x; i < nsym; i += 1024) acc += (u64)h1[i] * h2[i];
  part[threadIdx.x] = acc;
  __syncthreads();
  for (u32 w = 512; w; w >>= 1) {
    if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = part[0];
}

// Copies rows [0, used) of ncols columns of 4-byte entries, column i at
// src + i * sstride (entries) to dst + i * dstride; 16-byte accesses (four
// entries) when both strides are multiples of four and both bases 16-byte
// aligned, single entries otherwise.
__global__ void k_copy_columns(const u32 *src, u64 sstride, u32 *dst, u64 dstride, u64 used,
                               u32 ncols, u32 vec) {
  const u64 per = vec ? used / 4 : used;  // units per column
  const u64 n = per * ncols;
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x) {
    const u64 c = i / per, k = i - c * per;
    if (vec) {
      *reinterpret_cast<uint4 *>(dst + c * dstride + 4 * k) =
          *reinterpret_cast<const uint4 *>(src + c * sstride + 4 * k);
    } else {
      dst[c * dstride + k] = src[c * sstride + k];
    }
  }
  // the last used % 4 entries of each column in the vector form
  if (vec && blockIdx.x == 0 && threadIdx.x < ncols * 4u) {
    const u32 c = threadIdx.x / 4, j = threadIdx.x % 4;
    const u64 k = per * 4 + j;
    if (k < used) dst[c * dstride + k] = src[c * sstride + k];
  }
}

void copy_columns(const void *src, u64 sstride, void *dst, u64 dstride, u64 used, u32 ncols,
                  hipStream_t s) {
  if (!used) return;
  const bool vec = sstride % 4 == 0 && dstride % 4 == 0 &&
                   reinterpret_cast<uintptr_t>(src) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(dst) % 16 == 0;
  const u64 units = (vec ? used / 4 : used) * ncols;
  const unsigned g = (unsigned)std::max<u64>(1, std::min<u64>(ceil_div(units, 256), 8192));
  hipLaunchKernelGGL(k_copy_columns, dim3(g), dim3(256), 0, s, static_cast<const u32 *>(src),
                     sstride, static_cast<u32 *>(dst), dstride, used, ncols, vec ? 1u : 0u);
}

// The five result columns (src, dst, ilabel, olabel, weight; 4 bytes each)
// in one grow-only buffer: column i at byte i * cap * 4.  Growth is one
// allocation and one copy kernel over the rows kept, by at least 4x at every
// size: the result grows fastest in the levels where the search widens, and
// a smaller factor copies large results several times over (without
// reduction at config 4, 2x growth copied 25 GB for a 19.7 GB result).
// When a growth would come within a factor of 4 of `limit` (every row the
// search can produce, 0: unknown) it takes the limit at once, so that the
// largest rows are never copied again.
struct ArcCols {
  Buf b;
  u64 cap = 0;  // entries per column
  u64 limit = 0;
  hipStream_t s = nullptr;

  explicit ArcCols(Allocator *A, hipStream_t st) : b(A), s(st) {}
  void grow(u64 need, u64 used) {
    if (need <= cap && b.p) return;
    u64 nc = std::max<u64>(std::max<u64>(kMinGrow, need), 4 * cap);
    if (limit >= need && limit / 4 <= need) nc = std::max<u64>(nc, limit);
    nc = (nc + 63) & ~63ull;  // columns 256-byte aligned
    Buf nb(b.A);
    nb.ensure(5 * nc * 4);
    if (used && b.p) copy_columns(b.p, cap, nb.p, nc, used, 5, s);
    std::swap(b.p, nb.p);
    std::swap(b.cap, nb.cap);
    cap = nc;
  }
  u32 *col(int i) { return reinterpret_cast<u32 *>(static_cast<char *>(b.p) + (size_t)i * cap * 4); }
};

struct Composer {
  const fstc_fst &m1, &m2;
  fstc_opts o{};
  hipStream_t s;
  fstc_stats *stats;
  Allocator A;
  Timer T;
  Staging *hs = nullptr;
  Status *hs_dev = nullptr;  // hs->st as the device sees it
  Status *dst = nullptr;
  u32 nsyncs = 0;

  Composer(const fstc_fst &a, const fstc_fst &b, const fstc_opts *opts, hipStream_t st,
           fstc_stats *sp)
      : m1(a), m2(b), s(st), stats(sp) {
    if (opts) o = *opts;
    A.fa = o.alloc;
    A.ff = o.free;
    A.ctx = o.alloc_ctx;
    A.stream = s;
    T.s = s;
    T.on = stats != nullptr;
    T.all = o.phase_timing != 0;
  }

  void sync_status() {
    FSTC_HIP(hipGetLastError());
    FSTC_HIP(hipMemcpyAsync(&hs->st, dst, sizeof(Status), hipMemcpyDeviceToHost, s));
    FSTC_HIP(hipStreamSynchronize(s));
    ++nsyncs;
    if (hs->st.err) {
      throw Error((hs->st.err & kErrBadArc) ? FSTC_ERR_INVALID_ARG : FSTC_ERR_INTERNAL,
                  device_error_text(hs->st.err));
    }
  }

  // Waits until a kernel has copied the counters to hs->st and then written
  // publication number `seq` (the count scan's ScanPublish, launch_merged_total): a
  // spin on that word, with a stream query every few thousand reads so that
  // a failed or drained stream ends the wait.
  void wait_published(u32 seq) {
    FSTC_HIP(hipGetLastError());
    for (u32 i = 1;; ++i) {
      if (__atomic_load_n(&hs->st.seq, __ATOMIC_ACQUIRE) == seq) break;
      if ((i & 4095u) == 0) {
        const hipError_t q = hipStreamQuery(s);
        if (q == hipErrorNotReady) continue;
        FSTC_HIP(q);
        if (__atomic_load_n(&hs->st.seq, __ATOMIC_ACQUIRE) == seq) break;
        throw Error(FSTC_ERR_INTERNAL, "level counters were not published");
      }
      __builtin_ia32_pause();
    }
    ++nsyncs;
    if (hs->st.err) {
      throw Error((hs->st.err & kErrBadArc) ? FSTC_ERR_INVALID_ARG : FSTC_ERR_INTERNAL,
                  device_error_text(hs->st.err));
    }
  }

  void read_words(const u64 *d, int n) {
    FSTC_HIP(hipGetLastError());
    FSTC_HIP(hipMemcpyAsync(hs->words, d, n * sizeof(u64), hipMemcpyDeviceToHost, s));
    FSTC_HIP(hipStreamSynchronize(s));
    ++nsyncs;
  }

  void run(fstc_result *out);
};

void Composer::run(fstc_result *out) {
  const auto t0 = std::chrono::steady_clock::now();
  if (!o.alloc) tune_default_pool();
  hs = staging();
  FSTC_HIP(hipHostGetDevicePointer((void **)&hs_dev, hs, 0));

  static_assert(sizeof(Status) <= 256, "Status and the CSR counts share one allocation");
  Buf stb(&A);
  dst = (Status *)stb.ensure(256 + 16 * sizeof(u64));
  u64 *dcounts = reinterpret_cast<u64 *>(reinterpret_cast<char *>(dst) + 256);
  fill_u32((u32 *)dst, 0, sizeof(Status) / 4, s);

  // (a0) device layout of both inputs
  Buf cb1(&A), cb2(&A);
  Csr c1, c2;
  alloc_csr(m1, cb1, c1);
  alloc_csr(m2, cb2, c2);
  const bool product = !o.no_reduction && !o.no_product_merge;
  // without reduction, levels whose sources are all strided four-source
  // product sources resolve each source's targets once and write its joined
  // pairs from the two weight matrices (no records, no per-record probe)
  const bool unred_prod = o.no_reduction && !o.no_product_merge && !o.deterministic_ids &&
                          !o.max_arcs;
  T.at(kCsr);
  {
    // the two layouts are independent: when both take the per-state build
    // each of its steps is one launch for both inputs; otherwise M2's is
    // built on a side stream while M1's is built on the call's stream (the
    // side stream's temporaries are allocated up front, in stream order on
    // `s` before the fork)
    check_csr_ranges(m1, true);
    check_csr_ranges(m2, false);
    Arena csr_tmp(&A), csr_tmp2(&A);
    csr_tmp.reserve(csr_temp_bytes(m1));
    csr_tmp2.reserve(csr_temp_bytes(m2));
    const bool flags = product || unred_prod;
    if (!build_csr_pair(m1, true, csr_tmp, c1, dcounts + 0, m2, false, csr_tmp2, c2,
                        dcounts + 3, flags, &dst->err, s)) {
      csr_tmp2.fixed = true;
      SideStream &side = side_stream();
      FSTC_HIP(hipEventRecord(side.fork, s));
      FSTC_HIP(hipStreamWaitEvent(side.s, side.fork, 0));
      SideJoin join{s, side};
      build_csr(m2, false, csr_tmp2, c2, dcounts + 3, &dst->err, side.s);
      if (flags) build_cell_flags(c2, c2.cell_flag, side.s);
      build_csr(m1, true, csr_tmp, c1, dcounts + 0, &dst->err, s);
      if (flags) build_cell_flags(c1, c1.cell_flag, s);
    }
  }
  T.at(kNone);
  // (a1) states, visited table, start pair (before the host reads the CSR
  // counts: none of it depends on them)
  const u64 pairspace = (u64)m1.num_states * (u64)m2.num_states;
  u64 state_limit = std::min<u64>(pairspace, 0xffffffffull);
  if (o.max_states) state_limit = std::min<u64>(state_limit, o.max_states);
  Buf sq1b(&A), sq2b(&A), hkb(&A), hvb(&A);
  // state and result arrays start at kMinGrow entries, so that small
  // compositions never grow them; when there are at most kStatePresize state
  // pairs, the state arrays take them all (their growth copies are launches
  // on the level loop's critical path)
  const u64 state_start = state_limit <= kStatePresize ? std::max<u64>(kMinGrow, state_limit)
                                                       : (u64)kMinGrow;
  sq1b.ensure(state_start * 4);
  sq2b.ensure(state_start * 4);
  // single-pass scan state: zero-filled when (re)allocated, then written
  // only by the scans; sized for levels of up to state_start sources here,
  // while the CSR build runs
  Buf lbstate(&A);
  auto lb = [&](u64 n) {
    const size_t b = scan_lb_state_bytes(n);
    if (b > lbstate.cap) {
      lbstate.ensure(std::max<size_t>(b, 2 * lbstate.cap));
      fill_u32(lbstate.as<u32>(), 0, lbstate.cap / 4, s);
    }
    return lbstate.p;
  };
  (void)lb(state_start);
  // visited set: a dense array over all pairs when there are at most
  // kDensePairs of them (slot = q1 |Q2| + q2, no probing), else a hash table
  // (moved into a dense array later when that is no larger, see below)
  bool dense_vis = pairspace <= kDensePairs && !o.hash_visited;
  u32 vn2 = dense_vis ? m2.num_states : 0u;
  u64 hcap = dense_vis ? pairspace
                       : std::min<u64>(kMaxHashCap, next_pow2(std::max<u64>(
                             4096, 2 * std::min<u64>(pairspace, m1.num_arcs + m2.num_arcs + 1))));
  if (!dense_vis && o.hash_min_log2)
    hcap = std::max<u64>(hcap, std::min<u64>(kMaxHashCap, 1ull << o.hash_min_log2));
  if (dense_vis) {
    hvb.ensure(hcap * 4);
    fill_u32(hvb.as<u32>(), kUnvisited, hcap, s);
  } else {
    hkb.ensure(hcap * 8);
    hvb.ensure(hcap * 4);
    fill_u64(hkb.as<u64>(), kEmptyKey, hcap, s);
  }
  launch_insert_start(hkb.as<u64>(), hcap - 1, hvb.as<u32>(), vn2, m1.start, m2.start,
                      sq1b.as<u32>(), sq2b.as<u32>(), &dst->err, s);

  u64 *hs_words_dev = reinterpret_cast<u64 *>(reinterpret_cast<char *>(hs_dev) +
                                              offsetof(Staging, words));
  // Without reduction every joined arc pair is an arc of the result, so the
  // result has at most sum over inner symbols b of (arcs of m1 with output b)
  // (arcs of m2 with input b) arcs, the count when every pair of states is
  // reached; published in word 8 (see out_arcs.limit below).
  const u64 nsym = m1.num_osyms;
  const bool join_bound = o.no_reduction && nsym && nsym <= kJoinBoundSyms && m1.num_arcs &&
                          m2.num_arcs;
  Buf hb(&A);
  if (join_bound) {
    u32 *h = static_cast<u32 *>(hb.ensure(2 * nsym * 4));
    fill_u32(h, 0, 2 * nsym, s);
    auto hist = [&](const u32 *lab, u64 n, u32 *hh) {
      const unsigned g = (unsigned)std::min<u64>((u64)compute_units() * 2, ceil_div(n, 256 * 16));
      hipLaunchKernelGGL(k_label_hist, dim3(g), dim3(256), 0, s, lab, n, hh, (u32)nsym);
    };
    hist(m1.olabel, m1.num_arcs, h);
    hist(m2.ilabel, m2.num_arcs, h + nsym);
    hipLaunchKernelGGL(k_join_bound, dim3(1), dim3(1024), 0, s, h, h + nsym, nsym, dcounts + 8);
  }
  {
    const u32 seq0 = next_publication();
    static_assert(sizeof(Staging::words) >= 9 * sizeof(u64), "the CSR counts fit the staging words");
    hipLaunchKernelGGL(k_publish_counts, dim3(1), dim3(kWave), 0, s, c1.row, m1.start, c2.row,
                       m2.start, (m1.num_states && m2.num_states) ? 1 : 0, dcounts,
                       join_bound ? 9u : 8u, dst, hs_dev, hs_words_dev, seq0);
    wait_published(seq0);
    hb.release();
  }
  const u64 maxp1 = hs->words[2], maxp2 = hs->words[5];
  const u64 start_list1 = m1.num_states && m2.num_states ? hs->words[6] : 0,
            start_list2 = m1.num_states && m2.num_states ? hs->words[7] : 0;
  const int b1 = (int)bits_for(maxp1 ? maxp1 - 1 : 0);
  const int b2 = (int)bits_for(maxp2 ? maxp2 - 1 : 0);
  const int key_bits = b1 + b2;
  if (key_bits > kMaxKeyBits)
    throw Error(FSTC_ERR_RANGE, "per-state (target, outer symbol) ranks need " +
                                    std::to_string(key_bits) + " > 40 key bits");
  const bool wide_keys = key_bits > 32;
  const size_t rec_bytes = wide_keys ? 8 : 4;

  u64 n_states = 1, arcs = 0, premerge = 0;
  u32 lo = 0, hi = 1, depth = 0, new_levels = 0, expanded_levels = 0;
  u64 max_frontier = 0, max_level_pre = 0, big_total = 0, total_matches = 0, big_records = 0;
  u32 write_launches = 0, merge_launches = 0, sort_launches = 0, fused_levels = 0;
  u64 dense_records = 0, dense_runs = 0, sort_runs = 0, product_records = 0, product_sources = 0;
  u32 product_launches = 0;
  u64 product_mfma_sources = 0;
  u32 vis_moves = 0, direct_levels = 0;
  // the previous level was a direct product level (or none has run): the
  // next one is enqueued whole before the host reads its counts
  bool last_direct = true;
  // the previous per-level level had no listed sources: the list kernels
  // get lean grids (see launch_count, launch_prod_sources)
  bool lists_empty = false, listed_empty = false;

  ArcCols out_arcs(&A, s);
  // with reduction a state pair has at most maxp1 maxp2 merged arcs (one per
  // pair of parts)
  if (!o.no_reduction && maxp1 && maxp2 &&
      maxp1 * maxp2 <= (~0ull >> 1) / std::max<u64>(pairspace, 1))
    out_arcs.limit = std::min<u64>(pairspace, state_limit) * maxp1 * maxp2;
  if (join_bound) out_arcs.limit = hs->words[8];
  // per-level temporaries, carved from one arena reset at every level
  Arena level_tmp(&A);
  Tmp cnt(&level_tmp), mc(&level_tmp), roff(&level_tmp), moff(&level_tmp), ptot(&level_tmp),
      aoff(&level_tmp), pk(&level_tmp), pflag(&level_tmp), ftot(&level_tmp), newc(&level_tmp),
      newoff(&level_tmp), phdr(&level_tmp), poff(&level_tmp), wrange(&level_tmp), glist(&level_tmp), grp(&level_tmp), wide(&level_tmp), heavy(&level_tmp), big(&level_tmp),
      bigcnt(&level_tmp), bigoff(&level_tmp), match(&level_tmp), mrbase(&level_tmp),
      rkey(&level_tmp), rw(&level_tmp), temp(&level_tmp), newlist(&level_tmp), stmp(&level_tmp),
      dk(&level_tmp), dv(&level_tmp), dka(&level_tmp), dva(&level_tmp), dtmp(&level_tmp),
      tiles_e(&level_tmp), tiles_m(&level_tmp), tstart(&level_tmp), mend(&level_tmp),
      sortlist(&level_tmp), tile_runs(&level_tmp), wcnt(&level_tmp), woff(&level_tmp),
      wtmp(&level_tmp), runsrc(&level_tmp), newbits(&level_tmp);

  bool status_clear = true;  // level counters of *dst all zero
  // small levels (level.hpp, k_small_levels): one workgroup runs them, and
  // the levels after them, in one launch; a level it declines (too large,
  // or a capacity it must not exceed) takes the per-level kernels
  const bool small_ok = !o.no_reduction && !o.no_small_levels;
  u32 small_skip_depth = ~0u;  // the depth the one-workgroup kernel declined last
  // set when it declined a source's shape: not tried again until a level
  // taken by the per-level kernels has few sources of shapes it declines
  // (the count kernels count them)
  // (known at once when the start pair's own lists have such a shape)
  bool small_shape_off = std::min(start_list1, start_list2) > kSmallShortList ||
                         std::max(start_list1, start_list2) > kSmallLongList;
  // one-workgroup product levels (launch_product_level): off with the small
  // levels, and for the rest of the search once one declines
  const bool tiny_ok = small_ok;
  bool tiny_off = false;
  u32 tiny_levels = 0;
  u32 small_levels = 0;
  Buf ssb(&A);
  SmallState *ss_dev = small_ok ? static_cast<SmallState *>(ssb.ensure(sizeof(SmallState)))
                                : nullptr;
  static_assert(sizeof(SmallState) <= sizeof(Staging::words), "SmallState fits the staging words");
  while (true) {
    if (o.max_levels && depth >= o.max_levels) break;
    if (hi == lo) break;
    if (small_ok && !small_shape_off && hi - lo <= kSmallSources && depth != small_skip_depth) {
      constexpr u64 kSmallGrow = 1u << 16;  // room for this many states and arcs past the current
      sq1b.grow_keep((n_states + kSmallGrow) * 4, n_states * 4);
      sq2b.grow_keep((n_states + kSmallGrow) * 4, n_states * 4);
      out_arcs.grow(arcs + kSmallGrow, arcs);
      SmallArgs sa{};
      sa.row1 = c1.row; sa.seg_sym1 = c1.seg_sym; sa.seg_off1 = c1.seg_off;
      sa.part_base1 = c1.part_base; sa.arcs1 = c1.arcs; sa.parts1 = c1.parts;
      sa.row2 = c2.row; sa.seg_sym2 = c2.seg_sym; sa.seg_off2 = c2.seg_off;
      sa.part_base2 = c2.part_base; sa.arcs2 = c2.arcs; sa.parts2 = c2.parts;
      sa.b2 = b2;
      sa.key_bits = key_bits;
      sa.va.vis = hvb.as<u32>();
      sa.va.vn2 = vn2;
      sa.va.hkeys = hkb.as<u64>();
      sa.va.hmask = hcap - 1;
      sa.va.st = dst;
      sa.sq1 = sq1b.as<u32>();
      sa.sq2 = sq2b.as<u32>();
      sa.state_cap = std::min<u64>(state_limit, std::min(sq1b.cap, sq2b.cap) / 4);
      if (!dense_vis) sa.state_cap = std::min<u64>(sa.state_cap, hcap / 2);  // load at most 1/2
      sa.arc_cap = out_arcs.cap;
      if (o.max_arcs) sa.arc_cap = std::min<u64>(sa.arc_cap, o.max_arcs);
      sa.out_src = out_arcs.col(0);
      sa.out_dst = out_arcs.col(1);
      sa.out_il = out_arcs.col(2);
      sa.out_ol = out_arcs.col(3);
      sa.out_w = reinterpret_cast<float *>(out_arcs.col(4));
      sa.max_levels = o.max_levels;
      sa.ss = ss_dev;
      SmallState init{};
      init.lo = lo;
      init.hi = hi;
      init.n_states = n_states;
      init.arcs = arcs;
      init.premerge = premerge;
      init.depth = depth;
      std::memcpy(hs->words, &init, sizeof init);
      FSTC_HIP(hipMemcpyAsync(ss_dev, hs->words, sizeof init, hipMemcpyHostToDevice, s));
      if (!status_clear) {
        launch_reset_level(dst, s);
        status_clear = true;
      }
      T.at(kCount);
      launch_small_levels(sa, s);
      T.at(kNone);
      FSTC_HIP(hipMemcpyAsync(hs->words, ss_dev, sizeof(SmallState), hipMemcpyDeviceToHost, s));
      sync_status();
      SmallState out_st;
      std::memcpy(&out_st, hs->words, sizeof out_st);
      lo = (u32)out_st.lo;
      hi = (u32)out_st.hi;
      n_states = out_st.n_states;
      arcs = out_st.arcs;
      premerge = out_st.premerge;
      depth = out_st.depth;
      expanded_levels += out_st.levels;
      new_levels += out_st.new_levels;
      small_levels += out_st.levels;
      max_frontier = std::max<u64>(max_frontier, out_st.max_frontier);
      max_level_pre = std::max<u64>(max_level_pre, out_st.max_level_pre);
      if (out_st.reason == kSmallDone) break;
      if (out_st.reason == kSmallShape) small_shape_off = true;
      if (out_st.reason == kSmallTooLarge || out_st.reason == kSmallShape || out_st.levels == 0)
        small_skip_depth = depth;
      continue;  // larger capacities (a capacity stop after progress) or the per-level path
    }
    const u32 nsrc = hi - lo;
    level_tmp.reset();
    ++expanded_levels;
    max_frontier = std::max<u64>(max_frontier, nsrc);
    const u64 np1 = (u64)nsrc + 1;
    cnt.ensure(np1 * 8); mc.ensure(np1 * 4); roff.ensure(np1 * 8); moff.ensure(np1 * 8);
    ptot.ensure(np1 * 8); aoff.ensure(np1 * 8); tstart.ensure(np1 * 8); mend.ensure(np1 * 8);
    wide.ensure(np1 * 4); heavy.ensure(np1 * 4); big.ensure(np1 * 4); glist.ensure(np1 * 4);
    grp.ensure(np1 * 4);
    pk.ensure(np1 * 4); poff.ensure(np1 * 8); pflag.ensure(np1 * 8); ftot.ensure(np1 * 8);
    newc.ensure(np1 * 4); newoff.ensure(np1 * 8); phdr.ensure(np1 * 2 * sizeof(uint4));
    wrange.ensure(np1 * sizeof(uint4));
    stmp.ensure(scan_temp_bytes(np1));

    // (a2, a3) join counts and offsets
    if (!status_clear) launch_reset_level(dst, s);
    status_clear = false;
    LevelArgs la{view(c1), view(c2), sq1b.as<u32>(), sq2b.as<u32>(), lo, nsrc, cnt.as<u64>(),
                 mc.as<u32>(), roff.as<u64>(), moff.as<u64>(), wide.as<u32>(), heavy.as<u32>(),
                 wrange.as<uint4>(),
                 dst, nullptr, nullptr, nullptr, big.as<u32>(), pk.as<u32>(), phdr.as<uint4>(),
                 product ? 1u : 0u, tstart.as<u64>(), mend.as<u64>()};
    la.pflag = pflag.as<u64>();
    la.newc = newc.as<u32>();
    // strided product sources four per wave (dense visited array as of the
    // count; a move to the dense array later in the level keeps them listed)
    const bool uprod = unred_prod && dense_vis;
    const bool quad = (product || uprod) && dense_vis;
    la.prod = (product || uprod) ? 1u : 0u;
    la.unred = uprod ? 1u : 0u;
    la.quad = quad ? 1u : 0u;
    la.glist = glist.as<u32>();
    la.grp = grp.as<u32>();
    // A small level after a direct product level: one workgroup takes it
    // whole when all its sources are strided product sources (level.hpp,
    // launch_product_level), else it declines and the level takes the
    // per-level kernels (and so do the later levels).
    {
      const u64 maxk_t = std::min<u64>(maxp1 * maxp2, 64);
      if (tiny_ok && !tiny_off && product && dense_vis && last_direct && nsrc <= kTinySources &&
          !o.deterministic_ids && !o.max_arcs && (arcs + (u64)nsrc * maxk_t) * 20 <= kEarlyBytes) {
        out_arcs.grow(arcs + (u64)nsrc * maxk_t, arcs);
        const u64 newcap_t = std::min<u64>((u64)nsrc * maxk_t, pairspace - n_states);
        sq1b.grow_keep((n_states + newcap_t) * 4, n_states * 4);
        sq2b.grow_keep((n_states + newcap_t) * 4, n_states * 4);
        MergeArgs mt{};
        mt.nsrc = nsrc;
        mt.lo = lo;
        mt.st = dst;
        mt.pk = pk.as<u32>();
        mt.phdr = phdr.as<uint4>();
        mt.poff = poff.as<u64>();
        mt.parts1 = c1.parts;
        mt.parts2 = c2.parts;
        mt.arcs1 = c1.arcs;
        mt.arcs2 = c2.arcs;
        mt.wts1 = c1.wts;
        mt.wts2 = c2.wts;
        mt.vis = hvb.as<u32>();
        mt.vn2 = vn2;
        mt.hmask = hcap - 1;
        mt.pcnt = cnt.as<u64>();
        mt.newc = newc.as<u32>();
        mt.tstart = tstart.as<u64>();
        mt.mend = mend.as<u64>();
        mt.quad = 1u;
        mt.out_src = out_arcs.col(0);
        mt.out_dst = out_arcs.col(1);
        mt.out_il = out_arcs.col(2);
        mt.out_ol = out_arcs.col(3);
        mt.out_w = reinterpret_cast<float *>(out_arcs.col(4));
        mt.out_base = arcs;
        const u32 seqt = next_publication();
        T.at(kCount);
        launch_product_level(la, mt, poff.as<u64>(), newoff.as<u64>(), (u32)n_states,
                             sq1b.as<u32>(), sq2b.as<u32>(), hs_dev, seqt, s);
        T.at(kNone);
        wait_published(seqt);
        if (!hs->st.declined) {
          status_clear = true;  // the kernel cleared the level counters
          const u64 nnew_t = hs->st.nnew, merged_t = hs->st.merged, pairs_t = hs->st.prod_records;
          if (n_states + nnew_t > state_limit)
            throw Error(FSTC_ERR_CAPACITY, "reachable states exceed the state limit");
          premerge += pairs_t;
          product_records += pairs_t;
          max_level_pre = std::max(max_level_pre, pairs_t);
          product_sources += nsrc;
          product_mfma_sources += nsrc;
          ++direct_levels;
          ++tiny_levels;
          arcs += merged_t;
          n_states += nnew_t;
          if (nnew_t) ++new_levels;
          lo = hi;
          hi = (u32)n_states;
          ++depth;
          last_direct = true;
          continue;
        }
        tiny_off = true;
        launch_reset_level(dst, s);  // clears the decline mark
      }
    }
    // count + level scan: records, matches and product-merge entries per
    // source; the product sources' flags summed; the scan's last tile stores
    // the level totals (R, M, product entries, product sources) and
    // publishes the counters as publication `seq`
    auto count_and_scan = [&](u32 seq) {
      T.at(kCount);
      launch_count(la, s, lists_empty);
      ScanJob jobs[4] = {{cnt.p, true, roff.as<u64>()}, {mc.p, false, moff.as<u64>()},
                         {pk.p, false, poff.as<u64>()}, {pflag.p, true, ftot.as<u64>()}};
      jobs[3].total_only = true;
      jobs[0].total_to = &dst->R;
      jobs[1].total_to = &dst->M;
      jobs[2].total_to = &dst->prod_entries;
      jobs[3].total_to = reinterpret_cast<u64 *>(&dst->nprod);  // nprod, nprod_mfma
      const ScanPublish pub{dst, hs_dev, (u32)(sizeof(Status) / 4), (u32)(offsetof(Status, seq) / 4),
                            seq};
      exclusive_scan_lb(jobs, 4, nsrc, lb(nsrc), &dst->scan_ctr, &dst->err, s, &pub);
      T.at(kNone);
    };
    // Scan of a direct product level: new pairs per source (ids), joined
    // pairs per source (their total, less the level's records, is the
    // product merge's joined pairs) and merged arcs per source; its last
    // tile stores the level totals, publishes the counters as publication
    // `seq` and clears them for the next level (what k_merged_total does
    // for the other level forms).
    auto direct_totals_scan = [&](ScanJob (&jobs)[3], ScanPublish &pub, u32 seq) {
      jobs[0] = ScanJob{newc.p, false, newoff.as<u64>()};
      jobs[1] = ScanJob{cnt.p, true, ptot.as<u64>()};
      jobs[2] = ScanJob{mend.p, true, aoff.as<u64>()};
      jobs[0].total_to = reinterpret_cast<u64 *>(&dst->nnew);
      jobs[0].total_narrow = true;
      jobs[1].total_only = true;
      jobs[1].total_to = &dst->prod_records;
      jobs[1].total_minus = &dst->R;
      jobs[2].sub = tstart.as<u64>();
      jobs[2].total_to = &dst->merged;
      pub = ScanPublish{dst, hs_dev, (u32)(sizeof(Status) / 4), (u32)(offsetof(Status, seq) / 4), seq};
      pub.clear_mask = level_clear_mask();
    };
    const u32 seq1 = next_publication();
    count_and_scan(seq1);
    // Speculative product merge: with the dense visited array (no rehash
    // between the count and the merge) the product kernel is launched
    // before the host reads the level's counts, on temp slots reserved for
    // every source's largest table; it reads the record count on the device
    // and merges only when the level has no records -- the usual case where
    // the product merge applies -- so the GPU works through the host's
    // turnaround.  Otherwise it exits at once and the host launches it again
    // after the synchronisation.
    const u64 maxk = std::min<u64>(maxp1 * maxp2, 64);  // a source's table entries
    const bool spec = product && dense_vis && (u64)nsrc * maxk * 20 <= kSpecBytes;
    // Direct product level: the speculative product kernel writes its merged
    // arcs straight into the result (grown to hold every source's largest
    // table first); when the level turns out to have records it writes
    // nothing and the level takes the usual path.  Deterministic ids (a sort
    // of the new pairs) and an arc cap keep the usual path.
    const bool direct = spec && !o.deterministic_ids && !o.max_arcs &&
                        (arcs + (u64)nsrc * maxk) * 20 <= kEarlyBytes;
    if (spec) {
      temp.ensure((u64)nsrc * maxk * sizeof(uint4));
      runsrc.ensure((u64)nsrc * maxk * 4);
      MergeArgs pm{};  // the fields k_prod_sources reads
      pm.R = 0;
      pm.R_dev = roff.as<u64>() + nsrc;
      pm.nsrc = nsrc;
      pm.lo = lo;
      pm.st = dst;
      pm.pk = pk.as<u32>();
      pm.phdr = phdr.as<uint4>();
      pm.poff = poff.as<u64>();
      pm.parts1 = c1.parts;
      pm.parts2 = c2.parts;
      pm.arcs1 = c1.arcs;
      pm.arcs2 = c2.arcs;
      pm.wts1 = c1.wts;
      pm.wts2 = c2.wts;
      pm.seg_sym1 = c1.seg_sym;
      pm.seg_off1 = c1.seg_off;
      pm.seg_sym2 = c2.seg_sym;
      pm.seg_off2 = c2.seg_off;
      pm.vis = hvb.as<u32>();
      pm.vn2 = vn2;
      pm.hkeys = hkb.as<u64>();
      pm.hmask = hcap - 1;
      pm.temp = temp.as<uint4>();
      pm.runsrc = runsrc.as<u32>();
      pm.tstart = tstart.as<u64>();
      pm.mend = mend.as<u64>();
      pm.pcnt = cnt.as<u64>();
      pm.newc = newc.as<u32>();
      pm.quad = la.quad;
      pm.glist = glist.as<u32>();
      if (direct) {
        out_arcs.grow(arcs + (u64)nsrc * maxk, arcs);
        pm.out_src = out_arcs.col(0);
        pm.out_dst = out_arcs.col(1);
        pm.out_il = out_arcs.col(2);
        pm.out_ol = out_arcs.col(3);
        pm.out_w = reinterpret_cast<float *>(out_arcs.col(4));
        pm.out_base = arcs;
      }
      T.at(kProductKernel);
      launch_prod_sources(pm, std::max(c1.num_arcs, c2.num_arcs) < (1ull << 29), s,
                          listed_empty);
      T.at(kNone);
    }
    // Direct level enqueued whole: after the product kernel, the scans, id
    // assignment and totals of a direct level go to the stream too (its
    // marked targets are fixed after the last level), each reading the level's record count on the device and doing
    // nothing when it is not zero (k_merged_total then only publishes the
    // count's totals); the host waits once, at that publication, sized by
    // bounds: every source's largest table for the new pairs and arcs.
    const bool ahead = direct && last_direct;
    u32 seq_wait = seq1;
    if (ahead) {
      const u64 newcap_b = std::min<u64>((u64)nsrc * maxk, pairspace - n_states);
      sq1b.grow_keep((n_states + newcap_b) * 4, n_states * 4);
      sq2b.grow_keep((n_states + newcap_b) * 4, n_states * 4);
      T.at(kAssign);
      // the scan's last tile stores the level totals (new pairs, joined
      // pairs, merged arcs), publishes the counters and clears them for the
      // next level; skipped (a level with records) it publishes the count's
      // totals as they are
      seq_wait = next_publication();
      ScanJob jobs[3];
      ScanPublish pub;
      direct_totals_scan(jobs, pub, seq_wait);
      pub.when_skipped = true;
      exclusive_scan_lb(jobs, 3, nsrc, lb(nsrc), &dst->scan_ctr, &dst->err, s, &pub,
                        roff.as<u64>() + nsrc);
      MergeArgs md{};  // the fields the direct-level kernels read
      md.R_dev = roff.as<u64>() + nsrc;
      md.nsrc = nsrc;
      md.lo = lo;
      md.st = dst;
      md.newc = newc.as<u32>();
      md.poff = poff.as<u64>();
      md.tstart = tstart.as<u64>();
      md.mend = mend.as<u64>();
      md.vis = hvb.as<u32>();
      md.vn2 = vn2;
      md.hmask = hcap - 1;
      md.out_src = out_arcs.col(0);
      md.out_dst = out_arcs.col(1);
      md.out_il = out_arcs.col(2);
      md.out_ol = out_arcs.col(3);
      md.out_w = reinterpret_cast<float *>(out_arcs.col(4));
      md.out_base = arcs;
      launch_assign_direct(md, newoff.as<u64>(), (u32)n_states, sq1b.as<u32>(), sq2b.as<u32>(), s);
      T.at(kNone);
    }
    wait_published(seq_wait);
    if (uprod && hs->st.nprod && hs->st.R) {
      // without reduction a level takes the product form only whole: this
      // one has other sources too, so every source goes through records
      launch_reset_level(dst, s);
      la.prod = la.unred = la.quad = 0u;
      const u32 seq1b = next_publication();
      count_and_scan(seq1b);
      wait_published(seq1b);
    }
    const u64 R = hs->st.R, M = hs->st.M;
    const u32 nbig = hs->st.nbig, nprod = hs->st.nprod;
    lists_empty = hs->st.nwide == 0 && hs->st.nheavy == 0 && hs->st.ngrp == 0;
    listed_empty = hs->st.ngen == 0;
    // tried again once at most one source in eight of a level is of such a
    // shape (then the next, smaller levels usually have none)
    if (small_shape_off && (u64)hs->st.unfit * 8 < nsrc) small_shape_off = false;
    const u64 prodpos = nprod ? hs->st.prod_entries : 0;  // product-merge temp slots
    if (R == 0 && nprod == 0) break;  // no arc leaves this level: no new states either
    premerge += R;
    max_level_pre = std::max(max_level_pre, R);
    product_sources += nprod;
    product_mfma_sources += hs->st.nprod_mfma;
    big_total += nbig;

    match.ensure(M * sizeof(uint4));
    mrbase.ensure(M * 8);
    rkey.ensure(R * rec_bytes);
    rw.ensure(R * 4);
    // (every ensure takes new arena space: a speculative product merge that
    // ran keeps the temp and runsrc it wrote)
    if (!o.no_reduction && !(spec && R == 0)) {
      temp.ensure((R + prodpos) * sizeof(uint4));
      runsrc.ensure((R + prodpos) * 4);
    }
    tiles_e.ensure(ceil_div(R, kExpandTile) * sizeof(ExpandTile));
    // merge window: as wide as the largest small source allows (see level.hpp)
    const u64 max_small = std::max<u32>(1, hs->st.max_small);
    const u64 window = nbig ? kMergeSmall : (u64)kMergeCap - max_small + 1;
    const u64 ntiles = ceil_div(R, window);
    tiles_m.ensure(ntiles * sizeof(uint4));
    sortlist.ensure(ntiles * 4);
    tile_runs.ensure(ntiles * 4);
    const u64 newcap = std::min<u64>(R + prodpos, pairspace - n_states);
    newlist.ensure(std::max<u64>(newcap, 1) * 4);

    // visited table: keep the load factor at most 1/2 for every pair this
    // level could add
    // (at most kMaxHashCap slots: an insert into a full table reports it)
    const u64 need = std::min<u64>(2 * (n_states + newcap), kMaxHashCap);
    if (!dense_vis && need > hcap && !o.hash_visited && pairspace <= kDenseMaxPairs &&
        next_pow2(need) * 12 >= pairspace * 4) {
      // the grown table (8-byte keys, 4-byte ids) would be at least as large
      // as the dense array over all pairs: move the visited set there (the
      // level's inserts have not started; every state so far has its id)
      Buf nv(&A);
      nv.ensure(pairspace * 4);
      fill_u32(nv.as<u32>(), kUnvisited, pairspace, s);
      launch_states_to_dense(sq1b.as<u32>(), sq2b.as<u32>(), n_states, nv.as<u32>(),
                             m2.num_states, s);
      hkb.release();
      std::swap(hvb.p, nv.p); std::swap(hvb.cap, nv.cap);
      hcap = pairspace;
      dense_vis = true;
      vn2 = m2.num_states;
      ++vis_moves;
    } else if (!dense_vis && need > hcap) {
      const u64 ncap = next_pow2(need);
      Buf nk(&A), nv(&A);
      nk.ensure(ncap * 8);
      nv.ensure(ncap * 4);
      fill_u64(nk.as<u64>(), kEmptyKey, ncap, s);
      launch_rehash(hkb.as<u64>(), hvb.as<u32>(), hcap, nk.as<u64>(), nv.as<u32>(), ncap - 1,
                    &dst->err, s);
      std::swap(hkb.p, nk.p); std::swap(hkb.cap, nk.cap);
      std::swap(hvb.p, nv.p); std::swap(hvb.cap, nv.cap);
      hcap = ncap;
    }

    // (a4) match descriptors and the arc-pair write pass
    la.match = match.as<uint4>();
    la.mrbase = mrbase.as<u64>();
    la.tiles = tiles_e.as<ExpandTile>();
    T.at(kExpand);
    if (M) launch_emit(la, hs->st.nwide, hs->st.nheavy, hs->st.ngrp, s);
    // fused levels generate each tile's records inside the merge instead
    const bool fuse = o.fused_merge && !o.no_reduction && key_bits <= kDenseKeyBits && nbig == 0;
    if (!fuse && R) {
      T.at(kWriteKernel);
      launch_expand(match.as<uint4>(), mrbase.as<u64>(), M, R, view(c1), view(c2), b2, wide_keys,
                    rkey.p, rw.as<float>(), tiles_e.as<ExpandTile>(), &dst->err, s);
      ++write_launches;
    }
    T.at(kNone);
    total_matches += M;

    // (a6) merge identical arcs, claim new pairs (or, without reduction,
    // keep every record as an arc)
    MergeArgs ma{};
    ma.rec_key = rkey.p;
    ma.rec_w = rw.as<float>();
    ma.R = R;
    ma.roff = roff.as<u64>();
    ma.nsrc = nsrc;
    ma.lo = lo;
    ma.sq1 = sq1b.as<u32>();
    ma.sq2 = sq2b.as<u32>();
    ma.pbase1 = c1.part_base;
    ma.pbase2 = c2.part_base;
    ma.parts1 = c1.parts;
    ma.parts2 = c2.parts;
    ma.key_bits = key_bits;
    ma.b2 = b2;
    ma.hkeys = hkb.as<u64>();
    ma.hmask = hcap - 1;
    ma.vis = hvb.as<u32>();
    ma.vn2 = vn2;
    ma.newlist = newlist.as<u32>();
    ma.newcap = newcap;
    ma.temp = temp.as<uint4>();
    ma.runsrc = runsrc.as<u32>();
    ma.tiles = tiles_m.as<uint4>();
    ma.sortlist = sortlist.as<u32>();
    ma.tile_runs = tile_runs.as<u32>();
    ma.ntiles = ntiles;
    ma.window = window;
    ma.tstart = tstart.as<u64>();
    ma.mend = mend.as<u64>();
    ma.st = dst;
    ma.big = big.as<u32>();
    ma.match = match.as<uint4>();
    ma.mrbase = mrbase.as<u64>();
    ma.moff = moff.as<u64>();
    ma.arcs1 = c1.arcs;
    ma.arcs2 = c2.arcs;
    ma.wts1 = c1.wts;
    ma.wts2 = c2.wts;
    ma.pk = pk.as<u32>();
    ma.phdr = phdr.as<uint4>();
    ma.pcnt = cnt.as<u64>();  // product-merge sources have no records: their slots are free
    ma.newc = newc.as<u32>();
    ma.poff = poff.as<u64>();
    ma.quad = la.quad;
    ma.glist = glist.as<u32>();
    ma.prodpos = prodpos;
    ma.row1 = c1.row;
    ma.seg_sym1 = c1.seg_sym;
    ma.seg_off1 = c1.seg_off;
    ma.row2 = c2.row;
    ma.seg_sym2 = c2.seg_sym;
    ma.seg_off2 = c2.seg_off;
    u64 RB = 0;
    u32 nnew = 0;
    u64 merged = 0;
    // (a7) the level's merged arcs appended to the result: at most M of them
    auto append = [&](u64 M) {
      if (!M) return;
      out_arcs.grow(arcs + M, arcs);
      u32 *osrc = out_arcs.col(0) + arcs, *odst = out_arcs.col(1) + arcs,
          *oil = out_arcs.col(2) + arcs, *ool = out_arcs.col(3) + arcs;
      float *ow = reinterpret_cast<float *>(out_arcs.col(4)) + arcs;
      if (nprod)  // product-merge sources interleave with the tiles' sources
        launch_compact_sources(ma, aoff.as<u64>(), M, hvb.as<u32>(), osrc, odst, oil, ool, ow, s);
      else
        launch_compact(ma, aoff.as<u64>(), nbig, M, hvb.as<u32>(), osrc, odst, oil, ool, ow, s);
    };
    // Early append: when the capacities they need, bounded since the first
    // synchronisation, are small, id assignment and the result append go to
    // the stream before the host reads the level's totals, and the GPU runs
    // them while the host waits (deterministic ids and an arc cap need the
    // exact counts first).
    const bool direct_level = direct && R == 0;  // the speculative launch wrote the result
    bool assigned = false;                        // ids and arcs of the level are in place
    const bool early = !direct_level && !o.no_reduction && !o.deterministic_ids && !o.max_arcs &&
                       (n_states + newcap) * 8 <= kEarlyBytes &&
                       (arcs + R + prodpos) * 20 <= kEarlyBytes;
    last_direct = direct_level;
    if (direct_level && ahead) {
      // everything ran before the wait: read the totals
      ++product_launches;
      status_clear = true;  // the totals scan cleared the level counters
      nnew = hs->st.nnew;
      merged = hs->st.merged;
      premerge += hs->st.prod_records;
      product_records += hs->st.prod_records;
      max_level_pre = std::max(max_level_pre, hs->st.prod_records);
      if (merged < prodpos) {  // entries without a term leave holes: close them
        ma.out_src = out_arcs.col(0);
        ma.out_dst = out_arcs.col(1);
        ma.out_il = out_arcs.col(2);
        ma.out_ol = out_arcs.col(3);
        ma.out_w = reinterpret_cast<float *>(out_arcs.col(4));
        ma.out_base = arcs;
        Tmp rows(&level_tmp);
        rows.ensure(prodpos * 20);
        launch_close_holes(ma, aoff.as<u64>(), prodpos, rows.p, s);
      }
      assigned = true;
      ++direct_levels;
    } else if (direct_level) {
      // the level's merged arcs are in the result at arcs + poff[u]: new
      // pairs per source scanned into id offsets, joined pairs and merged
      // arcs per source summed (the latter scanned too, for entries without
      // a term), ids of the claimed entries, then the other new targets
      ++product_launches;
      T.at(kAssign);
      const u32 seq2 = next_publication();
      {
        ScanJob jobs[3];
        ScanPublish pub;
        direct_totals_scan(jobs, pub, seq2);
        exclusive_scan_lb(jobs, 3, nsrc, lb(nsrc), &dst->scan_ctr, &dst->err, s, &pub);
      }
      ma.out_src = out_arcs.col(0);
      ma.out_dst = out_arcs.col(1);
      ma.out_il = out_arcs.col(2);
      ma.out_ol = out_arcs.col(3);
      ma.out_w = reinterpret_cast<float *>(out_arcs.col(4));
      ma.out_base = arcs;
      sq1b.grow_keep((n_states + newcap) * 4, n_states * 4);
      sq2b.grow_keep((n_states + newcap) * 4, n_states * 4);
      launch_assign_direct(ma, newoff.as<u64>(), (u32)n_states, sq1b.as<u32>(), sq2b.as<u32>(), s);
      T.at(kNone);
      wait_published(seq2);
      status_clear = true;  // the totals scan cleared the level counters
      nnew = hs->st.nnew;
      merged = hs->st.merged;
      premerge += hs->st.prod_records;
      product_records += hs->st.prod_records;
      max_level_pre = std::max(max_level_pre, hs->st.prod_records);
      if (merged < prodpos) {  // entries without a term leave holes: close them
        Tmp rows(&level_tmp);
        rows.ensure(prodpos * 20);
        launch_close_holes(ma, aoff.as<u64>(), prodpos, rows.p, s);
      }
      assigned = true;
      ++direct_levels;
    } else if (!o.no_reduction) {
      T.at(kMerge);
      if (R) {
        fill_u32(tile_runs.as<u32>(), 0, ntiles, s);
        launch_tile_sources(ma, s);
        if (fuse) {
          T.at(kMergeKernel);
          launch_fuse_merge(ma, std::max(c1.num_arcs, c2.num_arcs) < (1ull << 29), s);
          ++merge_launches;
          ++fused_levels;
        } else if (key_bits <= kDenseKeyBits) {
          T.at(kMergeKernel);
          launch_merge_dense(ma, s);
          ++merge_launches;
        }
        T.at(kSortKernel);
        launch_merge_sort(ma, wide_keys, s);
        ++sort_launches;
        T.at(kMerge);
      }
      if (nbig) {
        bigcnt.ensure((u64)nbig * 8);
        bigoff.ensure(((u64)nbig + 1) * 8);
        launch_big_counts(roff.as<u64>(), big.as<u32>(), nbig, bigcnt.as<u64>(), s);
        exclusive_scan(bigcnt.as<u64>(), bigoff.as<u64>(), nbig, stmp.p, s);
        read_words(bigoff.as<u64>() + nbig, 1);
        RB = hs->words[0];
        big_records += RB;
        merge_big(ma, wide_keys, nbig, bigoff.as<u64>(), RB, level_tmp, s);
      }
      if (nprod) {
        if (!(spec && R == 0)) {  // (else the speculative launch merged them)
          T.at(kProductKernel);
          launch_prod_sources(ma, std::max(c1.num_arcs, c2.num_arcs) < (1ull << 29), s);
          T.at(kMerge);
        }
        ++product_launches;
      }
      // merged arcs per source (mend - tstart) scanned into result offsets;
      // the per-source joined pairs (records, or the product merge's terms)
      // summed for the level's product-merge pairs
      // (on a level of product-merge sources alone, also the new pairs
      // each source claimed, for the new-pair list)
      const bool prod_only = R == 0;
      {
        ScanJob jobs[3] = {{mend.p, true, aoff.as<u64>()}, {cnt.p, true, ptot.as<u64>()},
                           {newc.p, false, newoff.as<u64>()}};
        jobs[0].sub = tstart.as<u64>();
        jobs[1].total_only = true;
        exclusive_scan_lb(jobs, prod_only ? 3 : 2, nsrc, lb(nsrc), &dst->scan_ctr, &dst->err, s);
      }
      launch_emit_tiles(ma, s);
      const u64 *new_total = nullptr;
      if (prod_only) {
        launch_newlist_sources(ma, newoff.as<u64>(), s);
        new_total = newoff.as<u64>() + nsrc;
      } else {
        const u64 nw = newlist_waves(ma, RB);
        wcnt.ensure(nw * 4);
        woff.ensure((nw + 1) * 8);
        new_total = launch_newlist(ma, nbig ? bigoff.as<u64>() : nullptr, nbig, RB,
                                   wcnt.as<u32>(), woff.as<u64>(), lb(nw), s);
      }
      const u32 seq2 = next_publication();
      launch_merged_total(aoff.as<u64>() + nsrc, new_total, ptot.as<u64>() + nsrc, ma, hs_dev,
                          seq2, s);
      if (early) {
        T.at(kAssign);
        sq1b.grow_keep((n_states + newcap) * 4, n_states * 4);
        sq2b.grow_keep((n_states + newcap) * 4, n_states * 4);
        launch_assign_counted(newlist.as<u32>(), new_total, (u32)newcap, (u32)n_states,
                              hkb.as<u64>(), hvb.as<u32>(), vn2, sq1b.as<u32>(), sq2b.as<u32>(),
                              s);
        append(R + prodpos);
      }
      T.at(kNone);
      wait_published(seq2);
      status_clear = true;  // k_merged_total cleared the level counters

      nnew = hs->st.nnew;
      merged = hs->st.merged;
      premerge += hs->st.prod_records;
      product_records += hs->st.prod_records;
      max_level_pre = std::max(max_level_pre, R + hs->st.prod_records);
      dense_records += hs->st.dense_records;
      dense_runs += hs->st.dense_runs;
      sort_runs += hs->st.sort_runs;
    } else if (nprod) {
      // without reduction, every source a strided product source (R == 0):
      // the four-source kernel resolves each source's targets into utab
      // (claims marked), the claims are numbered and the marks fixed as on
      // a direct level, then every joined pair is written from the two
      // weight matrices
      T.at(kMerge);
      Tmp utab(&level_tmp);
      utab.ensure(std::max<u64>(prodpos, 1) * 4);
      MergeArgs pa{};
      pa.nsrc = nsrc;
      pa.lo = lo;
      pa.st = dst;
      pa.pk = pk.as<u32>();
      pa.phdr = phdr.as<uint4>();
      pa.poff = poff.as<u64>();
      pa.parts1 = c1.parts;
      pa.parts2 = c2.parts;
      pa.arcs1 = c1.arcs;
      pa.arcs2 = c2.arcs;
      pa.wts1 = c1.wts;
      pa.wts2 = c2.wts;
      pa.seg_sym1 = c1.seg_sym;
      pa.seg_off1 = c1.seg_off;
      pa.seg_sym2 = c2.seg_sym;
      pa.seg_off2 = c2.seg_off;
      pa.vis = hvb.as<u32>();
      pa.vn2 = vn2;
      pa.hmask = hcap - 1;
      pa.tstart = tstart.as<u64>();
      pa.mend = mend.as<u64>();
      pa.pcnt = cnt.as<u64>();
      pa.newc = newc.as<u32>();
      pa.quad = 1;
      pa.glist = glist.as<u32>();
      pa.utab = utab.as<u32>();
      T.at(kProductKernel);
      launch_prod_sources(pa, std::max(c1.num_arcs, c2.num_arcs) < (1ull << 29), s);
      ++product_launches;
      T.at(kAssign);
      {
        ScanJob jobs[2] = {{newc.p, false, newoff.as<u64>()}, {cnt.p, true, ptot.as<u64>()}};
        exclusive_scan_lb(jobs, 2, nsrc, lb(nsrc), &dst->scan_ctr, &dst->err, s);
      }
      const u64 newcap_u = std::min<u64>(prodpos, pairspace - n_states);
      sq1b.grow_keep((n_states + newcap_u) * 4, n_states * 4);
      sq2b.grow_keep((n_states + newcap_u) * 4, n_states * 4);
      pa.out_dst = utab.as<u32>();
      pa.out_base = 0;
      launch_assign_direct(pa, newoff.as<u64>(), (u32)n_states, sq1b.as<u32>(), sq2b.as<u32>(), s);
      launch_fix_marked(pa, prodpos, s);
      const u32 seq2 = next_publication();
      launch_merged_total(ptot.as<u64>() + nsrc, newoff.as<u64>() + nsrc, ptot.as<u64>() + nsrc,
                          pa, hs_dev, seq2, s);
      T.at(kNone);
      wait_published(seq2);
      status_clear = true;  // the totals scan cleared the level counters
      nnew = hs->st.nnew;
      merged = hs->st.merged;  // every joined pair is an arc
      premerge += merged;
      product_records += merged;
      max_level_pre = std::max(max_level_pre, merged);
      T.at(kMerge);
      out_arcs.grow(arcs + merged, arcs);
      pa.out_src = out_arcs.col(0);
      pa.out_dst = out_arcs.col(1);
      pa.out_il = out_arcs.col(2);
      pa.out_ol = out_arcs.col(3);
      pa.out_w = reinterpret_cast<float *>(out_arcs.col(4));
      pa.out_base = arcs;
      T.at(kWriteKernel);  // the level's write pass: every joined pair to the result
      launch_unreduced_product(pa, ptot.as<u64>(), s);
      ++write_launches;
      T.at(kNone);
      assigned = true;
    } else {
      if (o.max_arcs && arcs + R > o.max_arcs)
        throw Error(FSTC_ERR_CAPACITY, "composed arcs exceed opts->max_arcs");
      out_arcs.grow(arcs + R, arcs);
      u32 *osrc = out_arcs.col(0), *odst = out_arcs.col(1), *oil = out_arcs.col(2),
          *ool = out_arcs.col(3);
      float *ow = reinterpret_cast<float *>(out_arcs.col(4));
      T.at(kMerge);
      const u64 nwords = ceil_div(hcap, 32);
      newbits.ensure(nwords * 4);
      fill_u32(newbits.as<u32>(), 0, nwords, s);
      launch_unreduced(ma, wide_keys, newbits.as<u32>(), osrc + arcs, odst + arcs, oil + arcs,
                       ool + arcs, ow + arcs, s);
      const u64 nw = bitlist_waves(nwords);
      wcnt.ensure(nw * 4);
      woff.ensure((nw + 1) * 8);
      wtmp.ensure(scan_temp_bytes(nw));
      launch_bitlist(newbits.as<u32>(), nwords, newlist.as<u32>(), newcap, wcnt.as<u32>(),
                     woff.as<u64>(), wtmp.p, dst, s);
      T.at(kNone);
      sync_status();
      nnew = hs->st.nnew;
      merged = R;
    }
    if (n_states + nnew > state_limit)
      throw Error(FSTC_ERR_CAPACITY, "reachable states exceed the state limit");
    if (!o.no_reduction && o.max_arcs && arcs + merged > o.max_arcs)
      throw Error(FSTC_ERR_CAPACITY, "composed arcs exceed opts->max_arcs");

    // (a5) ids for the new pairs; (a7) append the level's arcs (done above
    // for an early append)
    const u64 ns_new = n_states + nnew;
    if (!early && !assigned) {
      T.at(kAssign);
      sq1b.grow_keep(ns_new * 4, n_states * 4);
      sq2b.grow_keep(ns_new * 4, n_states * 4);
      const u32 *slots = newlist.as<u32>();
      if (o.deterministic_ids && nnew > 1) {
        const int bq1 = (int)bits_for(m1.num_states - 1), bq2 = (int)bits_for(m2.num_states - 1);
        dk.ensure((u64)nnew * 8); dv.ensure((u64)nnew * 4);
        dka.ensure((u64)nnew * 8); dva.ensure((u64)nnew * 4);
        dtmp.ensure(radix_temp_bytes(nnew));
        launch_newkeys(newlist.as<u32>(), nnew, hkb.as<u64>(), vn2, bq2, dk.as<u64>(), dv.as<u32>(), s);
        radix_sort_pairs(dk.as<u64>(), dv.as<u32>(), dka.as<u64>(), dva.as<u32>(), nnew, 0,
                         bq1 + bq2, dtmp.p, s);
        slots = dv.as<u32>();
      }
      launch_assign(slots, nnew, (u32)n_states, hkb.as<u64>(), hvb.as<u32>(), vn2, sq1b.as<u32>(),
                    sq2b.as<u32>(), s);
      if (o.no_reduction)
        launch_fix_dst(out_arcs.col(1) + arcs, merged, hvb.as<u32>(), s);
      else
        append(merged);
      T.at(kNone);
    }
    arcs += merged;
    n_states = ns_new;
    if (nnew) ++new_levels;
    lo = hi;
    hi = (u32)n_states;
    ++depth;
  }

  // Direct product levels leave the targets that another source of their
  // level claimed marked with their visited-array slot: every slot has its
  // id by now, so one pass over the result replaces them (the levels read
  // no target of the result meanwhile).
  if (direct_levels && arcs) {
    MergeArgs mf{};
    mf.st = dst;
    mf.vis = hvb.as<u32>();
    mf.hmask = hcap - 1;
    mf.out_dst = out_arcs.col(1);
    mf.out_base = 0;
    launch_fix_marked(mf, arcs, s);
  }
  // (a7) accept states
  Buf finb(&A);
  finb.ensure(n_states);
  launch_finals(sq1b.as<u32>(), sq2b.as<u32>(), n_states, m1.final, m2.final, finb.as<uint8_t>(), s);
  {
    const u32 seqf = next_publication();
    hipLaunchKernelGGL(k_publish_counts, dim3(1), dim3(kWave), 0, s, nullptr, 0u, nullptr, 0u, 0,
                       nullptr, 0u, dst, hs_dev, hs_words_dev, seqf);
    wait_published(seqf);
  }

  std::memset(out, 0, sizeof(*out));
  out->num_states = n_states;
  out->num_arcs = arcs;
  out->num_premerge_arcs = premerge;
  out->num_levels = new_levels + 1;
  // states: one allocation per array; arcs: the five columns of one
  // allocation (alloc_ptr[3]); alloc_ptr[4..7] stay NULL
  Buf *keep[3] = {&sq1b, &sq2b, &finb};
  void **fields[3] = {(void **)&out->state_q1, (void **)&out->state_q2, (void **)&out->final};
  for (int i = 0; i < 3; ++i) {
    size_t b = 0;
    void *p = keep[i]->detach(&b);
    out->alloc_ptr[i] = p;
    out->alloc_bytes[i] = b;
    *fields[i] = p;
  }
  if (arcs) {
    out->src = out_arcs.col(0);
    out->dst = out_arcs.col(1);
    out->ilabel = out_arcs.col(2);
    out->olabel = out_arcs.col(3);
    out->weight = reinterpret_cast<float *>(out_arcs.col(4));
    size_t b = 0;
    out->alloc_ptr[3] = out_arcs.b.detach(&b);
    out->alloc_bytes[3] = b;
  }
  if (stats) {
    double ms[kNumPhases] = {};
    T.totals(ms);
    stats->ms_write_kernel = ms[kWriteKernel];
    stats->ms_merge_kernel = ms[kMergeKernel];
    stats->write_launches = write_launches;
    stats->merge_launches = merge_launches;
    stats->ms_sort_kernel = ms[kSortKernel];
    stats->sort_launches = sort_launches;
    stats->fused_levels = fused_levels;
    stats->total_dense_records = dense_records;
    stats->total_dense_runs = dense_runs;
    stats->total_product_records = product_records;
    stats->total_product_sources = product_sources;
    stats->ms_product_kernel = ms[kProductKernel];
    stats->product_launches = product_launches;
    stats->total_product_mfma_sources = product_mfma_sources;
    stats->total_sort_runs = sort_runs;
    stats->total_matches = total_matches;
    stats->total_big_records = big_records;
    stats->record_key_bytes = (u32)rec_bytes;
    stats->key_bits = (u32)key_bits;
    stats->num_levels = expanded_levels;
    stats->num_host_syncs = nsyncs;
    stats->max_frontier = max_frontier;
    stats->max_level_premerge = max_level_pre;
    stats->big_sources = big_total;
    stats->hash_capacity = hcap;
    stats->visited_form = vis_moves ? 2u : dense_vis ? 1u : 0u;
    stats->direct_product_levels = direct_levels;
    stats->peak_device_bytes = A.peak_bytes;
    stats->group_product_levels = tiny_levels;
    stats->small_levels = small_levels;
    if (T.all) {
      stats->ms_csr = ms[kCsr];
      stats->ms_count = ms[kCount];
      stats->ms_expand = ms[kExpand] + ms[kWriteKernel];
      stats->ms_merge = ms[kMerge] + ms[kMergeKernel] + ms[kSortKernel] + ms[kProductKernel];
      stats->ms_assign = ms[kAssign];
    }
    stats->ms_total =
        std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  }
}

int fail(int code, const std::string &msg) {
  g_detail = msg;
  return code;
}

int check_fst(const fstc_fst *m, const char *name) {
  if (!m) return fail(FSTC_ERR_INVALID_ARG, std::string(name) + " is NULL");
  if (m->num_states == 0) return fail(FSTC_ERR_INVALID_ARG, std::string(name) + ": num_states is 0");
  if (m->start >= m->num_states)
    return fail(FSTC_ERR_INVALID_ARG, std::string(name) + ": start >= num_states");
  if (!m->final) return fail(FSTC_ERR_INVALID_ARG, std::string(name) + ": final is NULL");
  if (m->num_arcs && (!m->src || !m->dst || !m->ilabel || !m->olabel || !m->weight))
    return fail(FSTC_ERR_INVALID_ARG, std::string(name) + ": an arc array is NULL");
  if (m->num_arcs >= (1ull << 32))
    return fail(FSTC_ERR_RANGE, std::string(name) + ": num_arcs must be below 2^32");
  return FSTC_OK;
}

int run_guarded(const char *what, hipStream_t s, const std::function<void()> &f) {
  try {
    f();
    return FSTC_OK;
  } catch (const Error &e) {
    (void)hipStreamSynchronize(s);
    (void)hipGetLastError();
    return fail(e.code, std::string(what) + ": " + e.what());
  } catch (const std::bad_alloc &) {
    return fail(FSTC_ERR_OOM, std::string(what) + ": host allocation failed");
  } catch (const std::exception &e) {
    return fail(FSTC_ERR_INTERNAL, std::string(what) + ": " + e.what());
  }
}

__global__ void k_split_uint2(const uint2 *in, u64 n, u32 *x, u32 *y) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x) {
    const uint2 v = in[i];
    x[i] = v.x;
    y[i] = v.y;
  }
}

}  // namespace
}  // namespace fstc

using namespace fstc;

extern "C" {

int fstc_compose(const fstc_fst *m1, const fstc_fst *m2, const fstc_opts *opts,
                 hipStream_t stream, fstc_result *out, fstc_stats *stats) {
  if (out) std::memset(out, 0, sizeof(*out));
  if (stats) std::memset(stats, 0, sizeof(*stats));
  if (!out) return fail(FSTC_ERR_INVALID_ARG, "out is NULL");
  int rc = check_fst(m1, "m1");
  if (rc) return rc;
  rc = check_fst(m2, "m2");
  if (rc) return rc;
  if (m1->num_osyms != m2->num_isyms)
    return fail(FSTC_ERR_ALPHABET, "m1->num_osyms != m2->num_isyms");
  if (opts && ((opts->alloc == nullptr) != (opts->free == nullptr)))
    return fail(FSTC_ERR_INVALID_ARG, "opts->alloc and opts->free must be set together");
  if (opts && opts->hash_min_log2 > 31)
    return fail(FSTC_ERR_INVALID_ARG, "opts->hash_min_log2 must be at most 31");
  try {
    check_csr_ranges(*m1, true);
    check_csr_ranges(*m2, false);
  } catch (const Error &e) {
    return fail(e.code, e.what());
  }
  return run_guarded("fstc_compose", stream, [&] {
    Composer c(*m1, *m2, opts, stream, stats);
    c.run(out);
  });
}

int fstc_compose_eps(const fstc_fst *m1, const fstc_fst *m2, uint32_t eps, const fstc_opts *opts,
                     hipStream_t stream, fstc_result *out, uint8_t **state_filter,
                     fstc_stats *stats) {
  if (out) std::memset(out, 0, sizeof(*out));
  if (state_filter) *state_filter = nullptr;
  if (stats) std::memset(stats, 0, sizeof(*stats));
  if (!out) return fail(FSTC_ERR_INVALID_ARG, "out is NULL");
  int rc = check_fst(m1, "m1");
  if (rc) return rc;
  rc = check_fst(m2, "m2");
  if (rc) return rc;
  if (m1->num_osyms != m2->num_isyms)
    return fail(FSTC_ERR_ALPHABET, "m1->num_osyms != m2->num_isyms");
  if (eps >= m1->num_isyms || eps >= m1->num_osyms || eps >= m2->num_osyms)
    return fail(FSTC_ERR_INVALID_ARG, "eps must be a symbol of every alphabet");
  const u32 G = m1->num_osyms;  // E1 = G, E2 = G + 1 extend the inner alphabet
  if (G > 0xfffffffdu) return fail(FSTC_ERR_RANGE, "inner alphabet too large for two more symbols");
  if (m1->num_arcs + m1->num_states >= (1ull << 32) || m2->num_arcs + m2->num_states >= (1ull << 32))
    return fail(FSTC_ERR_RANGE, "num_arcs + num_states must be below 2^32");
  if (opts && ((opts->alloc == nullptr) != (opts->free == nullptr)))
    return fail(FSTC_ERR_INVALID_ARG, "opts->alloc and opts->free must be set together");
  if (opts && opts->hash_min_log2 > 31)
    return fail(FSTC_ERR_INVALID_ARG, "opts->hash_min_log2 must be at most 31");
  return run_guarded("fstc_compose_eps", stream, [&] {
    const auto t0 = std::chrono::steady_clock::now();
    Allocator A;
    if (opts) {
      A.fa = opts->alloc;
      A.ff = opts->free;
      A.ctx = opts->alloc_ctx;
    } else {
      tune_default_pool();
    }
    A.stream = stream;
    // the relabelled inputs and the filter, five arrays each (4 B per arc
    // and array) in one buffer per transducer, the filter's accept flags last
    struct Side {
      Buf b;
      fstc_fst f{};
      explicit Side(Allocator *a) : b(a) {}
      void carve(u64 n, u32 nq, u32 start, u32 nin, u32 nout, const uint8_t *final) {
        const u64 cols = (std::max<u64>(n, 1) + 63) & ~63ull;
        char *p = static_cast<char *>(b.ensure(cols * 20 + 256));
        f = fstc_fst{nq, start, nin, nout, n, (const u32 *)p, (const u32 *)(p + cols * 4),
                     (const u32 *)(p + cols * 8), (const u32 *)(p + cols * 12),
                     (const float *)(p + cols * 16), final ? final : (const uint8_t *)(p + cols * 20)};
      }
      u32 *col(int i) const { return const_cast<u32 *>(i == 0 ? f.src : i == 1 ? f.dst : i == 2 ? f.ilabel : f.olabel); }
      float *w() const { return const_cast<float *>(f.weight); }
    };
    Side s1(&A), s2(&A), sf(&A);
    s1.carve(m1->num_arcs + m1->num_states, m1->num_states, m1->start, m1->num_isyms, G + 2,
             m1->final);
    s2.carve(m2->num_arcs + m2->num_states, m2->num_states, m2->start, G + 2, m2->num_osyms,
             m2->final);
    sf.carve(3ull * (G - 1) + 5, 3, 0, G + 2, G + 2, nullptr);
    build_eps_side(*m1, true, eps, G + 1, G, s1.col(0), s1.col(1), s1.col(2), s1.col(3), s1.w(),
                   stream);
    build_eps_side(*m2, false, eps, G, G + 1, s2.col(0), s2.col(1), s2.col(2), s2.col(3), s2.w(),
                   stream);
    build_eps_filter(G, eps, sf.col(0), sf.col(1), sf.col(2), sf.col(3), sf.w(),
                     const_cast<uint8_t *>(sf.f.final), stream);
    // M1' ∘ F: every joined pair is an arc (weights w1 * 1 exactly), the
    // whole search (at most 3 |Q1| states)
    fstc_opts oa{};
    if (opts) oa = *opts;
    oa.max_levels = 0;
    oa.max_states = 0;
    oa.max_arcs = 0;
    oa.no_reduction = 1;
    oa.fused_merge = 0;
    oa.phase_timing = 0;
    check_csr_ranges(s1.f, true);
    check_csr_ranges(sf.f, false);
    fstc_result ra{};
    struct Release {
      fstc_result *r;
      Allocator *A;
      bool armed = true;
      ~Release() {
        if (!armed) return;
        for (int i = 0; i < 8; ++i)
          if (r->alloc_ptr[i]) A->free(r->alloc_ptr[i], r->alloc_bytes[i]);
        std::memset(r, 0, sizeof(*r));
      }
    };
    Release ga{&ra, &A};
    {
      Composer c(s1.f, sf.f, &oa, stream, nullptr);
      c.run(&ra);
    }
    // (M1' ∘ F) ∘ M2' with the caller's options; its start is id 0 = (s1, 0)
    if (ra.num_states >= (1ull << 32)) throw Error(FSTC_ERR_RANGE, "filter composition too large");
    const fstc_fst fa{(u32)ra.num_states, 0, m1->num_isyms, G + 2, ra.num_arcs, ra.src, ra.dst,
                      ra.ilabel, ra.olabel, ra.weight, ra.final};
    check_csr_ranges(fa, true);
    check_csr_ranges(s2.f, false);
    Release go{out, &A};
    {
      Composer c(fa, s2.f, opts, stream, stats);
      c.run(out);
    }
    Buf fb(&A);
    uint8_t *filt = static_cast<uint8_t *>(fb.ensure(std::max<u64>(out->num_states, 1)));
    map_eps_states(out->state_q1, ra.state_q1, ra.state_q2, out->num_states, filt, stream);
    FSTC_HIP(hipGetLastError());
    size_t bytes = 0;
    out->alloc_ptr[4] = fb.detach(&bytes);
    out->alloc_bytes[4] = bytes;
    if (state_filter) *state_filter = filt;
    go.armed = false;
    if (stats)
      stats->ms_total =
          std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  });
}

void fstc_result_release(fstc_result *r, const fstc_opts *opts, hipStream_t stream) {
  if (!r) return;
  Allocator A;
  if (opts) {
    A.fa = opts->alloc;
    A.ff = opts->free;
    A.ctx = opts->alloc_ctx;
  }
  A.stream = stream;
  for (int i = 0; i < 8; ++i)
    if (r->alloc_ptr[i]) A.free(r->alloc_ptr[i], r->alloc_bytes[i]);
  std::memset(r, 0, sizeof(*r));
}

int fstc_build_csr(const fstc_fst *m, int by_output, hipStream_t stream, uint32_t *row,
                   uint32_t *seg_sym, uint32_t *seg_off, uint32_t *arc_part, float *arc_weight,
                   uint32_t *part_base, uint32_t *part_target, uint32_t *part_outer,
                   uint64_t *counts) {
  int rc = check_fst(m, "m");
  if (rc) return rc;
  if (!row || !seg_off || !part_base || !counts)
    return fail(FSTC_ERR_INVALID_ARG, "an output array is NULL");
  if (m->num_arcs && (!seg_sym || !arc_part || !arc_weight || !part_target || !part_outer))
    return fail(FSTC_ERR_INVALID_ARG, "an output array is NULL");
  try {
    check_csr_ranges(*m, by_output != 0);
  } catch (const Error &e) {
    return fail(e.code, e.what());
  }
  return run_guarded("fstc_build_csr", stream, [&] {
    Allocator A;
    A.stream = stream;
    tune_default_pool();
    const u64 n = m->num_arcs;
    Buf arcs(&A), parts(&A), dc(&A), de(&A);
    Csr c;
    c.num_states = m->num_states;
    c.num_arcs = n;
    c.row = row;
    c.seg_sym = seg_sym;
    c.seg_off = seg_off;
    c.part_base = part_base;
    c.arcs = (uint2 *)arcs.ensure(std::max<u64>(n, 1) * sizeof(uint2));
    c.parts = (uint2 *)parts.ensure(std::max<u64>(n, 1) * sizeof(uint2));
    u64 *d_counts = (u64 *)dc.ensure(3 * 8);
    u32 *d_err = (u32 *)de.ensure(4);
    fill_u32(d_err, 0, 1, stream);
    {
      Arena tmp(&A);
      build_csr(*m, by_output != 0, tmp, c, d_counts, d_err, stream);
    }
    if (n) {
      const unsigned g = (unsigned)std::min<u64>(ceil_div(n, 256), 1u << 16);
      hipLaunchKernelGGL(k_split_uint2, dim3(g), dim3(256), 0, stream, c.arcs, n, arc_part,
                         (u32 *)arc_weight);
      hipLaunchKernelGGL(k_split_uint2, dim3(g), dim3(256), 0, stream, c.parts, n, part_target,
                         part_outer);
    }
    Staging *hs = staging();
    FSTC_HIP(hipGetLastError());
    FSTC_HIP(hipMemcpyAsync(hs->words, d_counts, 3 * 8, hipMemcpyDeviceToHost, stream));
    FSTC_HIP(hipMemcpyAsync(&hs->st.err, d_err, 4, hipMemcpyDeviceToHost, stream));
    FSTC_HIP(hipStreamSynchronize(stream));
    if (hs->st.err) throw Error(FSTC_ERR_INVALID_ARG, device_error_text(hs->st.err));
    counts[0] = hs->words[0];
    counts[1] = hs->words[1];
    counts[2] = hs->words[2];
  });
}

int fstc_sort_pairs(uint64_t *keys, uint32_t *values, uint64_t n, int bit_lo, int bit_hi,
                    hipStream_t stream) {
  if (n && (!keys || !values)) return fail(FSTC_ERR_INVALID_ARG, "keys or values is NULL");
  if (bit_lo < 0 || bit_hi > 64 || bit_lo > bit_hi)
    return fail(FSTC_ERR_INVALID_ARG, "bit range must satisfy 0 <= lo <= hi <= 64");
  if (n >= (1ull << 32)) return fail(FSTC_ERR_RANGE, "n must be below 2^32");
  return run_guarded("fstc_sort_pairs", stream, [&] {
    if (n <= 1 || bit_lo == bit_hi) return;
    Allocator A;
    A.stream = stream;
    tune_default_pool();
    Buf ka(&A), va(&A), tmp(&A);
    ka.ensure(n * 8);
    va.ensure(n * 4);
    tmp.ensure(radix_temp_bytes(n));
    radix_sort_pairs(keys, values, ka.as<u64>(), va.as<u32>(), n, bit_lo, bit_hi, tmp.p, stream);
    FSTC_HIP(hipGetLastError());
  });
}

int fstc_exclusive_scan_u64(const uint64_t *in, uint64_t *out, uint64_t n, hipStream_t stream) {
  if (!out || (n && !in)) return fail(FSTC_ERR_INVALID_ARG, "in or out is NULL");
  return run_guarded("fstc_exclusive_scan_u64", stream, [&] {
    Allocator A;
    A.stream = stream;
    tune_default_pool();
    // single-pass scan: zero-filled state, a counter and an error word
    Buf state(&A), words(&A);
    state.ensure(scan_lb_state_bytes(n));
    words.ensure(8);
    fill_u32(state.as<u32>(), 0, state.cap / 4, stream);
    fill_u32(words.as<u32>(), 0, 2, stream);
    const ScanJob job{in, true, out};
    exclusive_scan_lb(&job, 1, n, state.p, words.as<u32>(), words.as<u32>() + 1, stream);
    Staging *hs = staging();
    FSTC_HIP(hipGetLastError());
    FSTC_HIP(hipMemcpyAsync(&hs->st.err, words.as<u32>() + 1, 4, hipMemcpyDeviceToHost, stream));
    FSTC_HIP(hipStreamSynchronize(stream));
    if (hs->st.err) throw Error(FSTC_ERR_INTERNAL, device_error_text(hs->st.err));
  });
}

int fstc_exclusive_scan_u64_noalloc(const uint64_t *in, uint64_t *out, uint64_t n,
                                    hipStream_t stream) {
  if (!out || (n && !in)) return fail(FSTC_ERR_INVALID_ARG, "in or out is NULL");
  if (n > noalloc_scan_max_n())
    return fail(FSTC_ERR_RANGE, "n = " + std::to_string(n) + " exceeds the scratch capacity of " +
                                    std::to_string(noalloc_scan_max_n()) + " elements");
  return run_guarded("fstc_exclusive_scan_u64_noalloc", stream,
                     [&] { noalloc_scan(in, out, n, stream); });
}

const char *fstc_strerror(int code) {
  switch (code) {
    case FSTC_OK: return "success";
    case FSTC_ERR_INVALID_ARG: return "invalid argument";
    case FSTC_ERR_ALPHABET: return "alphabet mismatch: m1 output alphabet != m2 input alphabet";
    case FSTC_ERR_RANGE: return "size exceeds a packing limit";
    case FSTC_ERR_CAPACITY: return "result exceeds a capacity limit";
    case FSTC_ERR_OOM: return "device allocation failed";
    case FSTC_ERR_HIP: return "HIP runtime error";
    case FSTC_ERR_INTERNAL: return "internal consistency check failed";
    default: return "unknown error code";
  }
}

const char *fstc_last_error_detail(void) { return g_detail.c_str(); }

const char *fstc_version(void) { return "0.1.0"; }

}  // extern "C"
