// Merging of identical composed arcs, visited-set update and result append
// for one breadth-first level.
//
// The paper merges the arcs of each popped pair by sorting them on a packed
// 64-bit key (a, c, r1r2) and summing runs of equal keys (section 3.4,
// "Reduction"; Algorithm 2, the sort and reduce of delta[q1q2]), and it
// tracks visited pairs in a table of |Q1||Q2| entries updated atomically,
// assigning each new pair the next id (section 3.4, "Updating frontier and
// visited set").  Here:
//   * a record's key is (rank of its M1 (target, input) pair) : (rank of its
//     M2 (target, output) pair), which fixes (r1r2, a, c) for its source;
//     ranks are per state (csr.hip), so keys are short;
//   * a workgroup takes the whole sources whose records start in a window
//     (at most 4096 records in all), sorts them in LDS by (source, key) with
//     a stable radix sort ranked by wave ballots, and sums every run of
//     equal keys in float64; sources of more than 2048 records are merged by
//     a device-wide radix sort and a segmented reduce;
//   * the visited set is an open-addressing hash table of 64-bit pair keys
//     (r1 << 32 | r2) in HBM, filled with atomicCAS; a pair is looked up
//     once per merged arc, after merging, so repeated targets cost one probe
//     per distinct arc rather than one per joined arc pair;
//   * pairs claimed by the CAS are appended to a new-state list, and get the
//     next ids once the level is merged (launch_assign).
#include "level.hpp"
#include "product.hpp"
#include "radix_rank.hpp"

namespace fstc {
namespace {

constexpr int NT = kMergeNT;
constexpr int IT = kMergeIT;
constexpr int C = kMergeCap;
constexpr int NW = NT / kWave;

inline unsigned grid1(u64 n, int nt = 256) {
  return (unsigned)std::max<u64>(1, std::min<u64>(ceil_div(n, nt), 1u << 20));
}

// Linear-probing insert of `key` (never kEmptyKey).  Returns its slot and
// sets is_new when this call claimed the slot.  The probe loop is bounded by
// the table size.
__device__ __forceinline__ u32 hash_insert(u64 *keys, u64 mask, u64 key, bool &is_new, u32 *err) {
  u64 h = mix64(key) & mask;
  for (u64 probe = 0; probe <= mask; ++probe) {
    const u64 cur = __hip_atomic_load(&keys[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (cur == key) {
      is_new = false;
      return (u32)h;
    }
    if (cur == kEmptyKey) {
      const u64 old = atomicCAS((unsigned long long *)&keys[h], (unsigned long long)kEmptyKey,
                                (unsigned long long)key);
      if (old == kEmptyKey) {
        is_new = true;
        return (u32)h;
      }
      if (old == key) {
        is_new = false;
        return (u32)h;
      }
    }
    h = (h + 1) & mask;
  }
  set_error(err, kErrHashFull);
  is_new = false;
  return 0;
}

// Tile of workgroup b among g: workgroup b runs on XCD b % 8; XCD x gets
// tiles [x * q + min(x, r), ...) in order (q = g / 8, r = g % 8).
__device__ __forceinline__ u32 xcd_tile(u32 b, u32 g) {
  const u32 x = b % 8, i = b / 8, q = g / 8, r = g % 8;
  return x * q + min(x, r) + i;
}

// Position in the wave-striped layout (element e = w*512 + j*64 + lane) that
// lane `lane` of wave w reads as item j, for the sorted element
// p = w*512 + lane*8 + j: each thread then holds 8 consecutive elements.
__device__ __forceinline__ u32 blocked_slot(u32 p) {
  return (p & ~(u32)(kWave * IT - 1)) | ((p % IT) * kWave) | ((p / IT) % kWave);
}

// Tiles that the dense-table kernel takes (see k_merge_dense); it flags in
// the descriptor (kRerouted) a tile it leaves to the sort kernel.
constexpr u32 kRerouted = 0x80000000u;
constexpr u64 kListedGrid = 2048;  // workgroups walking the list of tiles left to sort
constexpr int kEmitBatch = 4;      // runs per lane in flight when a tile has many
constexpr u32 kDenseEPT = kDenseCap / NT;  // table entries per thread when listing runs
constexpr u32 kExactSpan = 26;  // binades of a tile summed exactly in 64-bit fixed point
static_assert(kDenseCap % NT == 0 && (1u << kDenseKeyBits) == kDenseCap, "dense table shape");

__device__ __forceinline__ bool dense_tile(const uint4 &td, int key_bits) {
  return td.x < td.y && key_bits <= kDenseKeyBits &&
         ((u64)(td.y - td.x) << key_bits) <= (u64)kDenseCap;
}

// Exclusive prefix over the waves of the block of one value per wave (taken
// from any lane); *total receives the block total.  All threads must call it.
__device__ __forceinline__ u32 block_offset(u32 wave_value, u32 *s_tmp, u32 *total) {
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  __syncthreads();
  if (lane == 0) s_tmp[w] = wave_value;
  __syncthreads();
  u32 base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const u32 t = s_tmp[i];
    if ((u32)i < w) base += t;
    tot += t;
  }
  *total = tot;
  return base;
}

// Linear-probing insert of B keys at once (lanes with act[i] unset skip
// item i).  Each round issues the probe loads of all pending items before
// testing any, so their latencies overlap.  Slots only ever change from
// kEmptyKey to a key, so a stale read of kEmptyKey is settled by the CAS and
// a plain (workgroup-scope) read is enough.  Bounded by the table size.
template <int B>
__device__ __forceinline__ void hash_insert_batch(u64 *keys, u64 mask, const u64 (&key)[B],
                                                  const bool (&act)[B], u32 (&slot)[B],
                                                  bool (&is_new)[B], u32 *err) {
  u64 h[B];
  bool pend[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    pend[i] = act[i];
    is_new[i] = false;
    slot[i] = 0;
    h[i] = mix64(key[i]) & mask;
  }
  for (u64 probe = 0; probe <= mask; ++probe) {
    u64 cur[B];
#pragma unroll
    for (int i = 0; i < B; ++i)
      cur[i] = pend[i] ? __hip_atomic_load(&keys[h[i]], __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP)
                       : 0;
    bool any = false;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      if (!pend[i]) continue;
      if (cur[i] == kEmptyKey) {
        cur[i] = atomicCAS((unsigned long long *)&keys[h[i]], (unsigned long long)kEmptyKey,
                           (unsigned long long)key[i]);
        if (cur[i] == kEmptyKey) {
          is_new[i] = true;
          slot[i] = (u32)h[i];
          pend[i] = false;
          continue;
        }
      }
      if (cur[i] == key[i]) {
        slot[i] = (u32)h[i];
        pend[i] = false;
        continue;
      }
      h[i] = (h[i] + 1) & mask;
      any = true;
    }
    if (!any) return;
  }
  set_error(err, kErrHashFull);
}

// Visited-set insert of B target pairs (key = r1 << 32 | r2): the hash
// table, or the dense array when a.vn2 != 0 (slot = r1 vn2 + r2; a claim is
// a CAS from kUnvisited to kClaimed, tried only when a plain read of the
// entry still sees kUnvisited -- entries never return to it).  known[i]:
// the pair's id when an earlier level gave it one and the dense array holds
// it, else kUnvisited.
template <int B>
__device__ __forceinline__ void visit_batch(const MergeArgs &a, const u64 (&key)[B],
                                            const bool (&act)[B], u32 (&slot)[B],
                                            bool (&is_new)[B], u32 (&known)[B]) {
  if (!a.vn2) {
    hash_insert_batch<B>(a.hkeys, a.hmask, key, act, slot, is_new, &a.st->err);
#pragma unroll
    for (int i = 0; i < B; ++i) known[i] = kUnvisited;
    return;
  }
  u32 cur[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    slot[i] = act[i] ? (u32)(key[i] >> 32) * a.vn2 + (u32)key[i] : 0u;
    is_new[i] = false;
    cur[i] = act[i] ? __hip_atomic_load(&a.vis[slot[i]], __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_WORKGROUP)
                    : 0u;
  }
#pragma unroll
  for (int i = 0; i < B; ++i) {
    known[i] = cur[i] < kClaimed ? cur[i] : kUnvisited;  // ids are below both markers
    if (act[i] && cur[i] == kUnvisited) is_new[i] = atomicCAS(&a.vis[slot[i]], kUnvisited, kClaimed) == kUnvisited;
  }
}

// The part pairs of B merged arcs -> visited-table insert of the target pair
// (r1, r2) and the run record (slot | kNewFlag if claimed, a, c, weight) at
// temp[tpos], source u at runsrc[tpos] (the new-state list is built from
// these flags by k_newlist, without a shared counter).  A target that
// already has an id in the dense array is recorded as id | kIdFlag, so the
// result append needs no visited-array lookup for it.
template <int B>
__device__ __forceinline__ void emit_parts(const MergeArgs &a, const bool (&act)[B],
                                           const u32 (&u)[B], const uint2 (&P1)[B],
                                           const uint2 (&P2)[B], const u64 (&tpos)[B],
                                           const float (&w)[B]) {
  u64 hk[B];
#pragma unroll
  for (int i = 0; i < B; ++i) hk[i] = ((u64)P1[i].x << 32) | (u64)P2[i].x;
  u32 slot[B], known[B];
  bool is_new[B];
  visit_batch<B>(a, hk, act, slot, is_new, known);
#pragma unroll
  for (int i = 0; i < B; ++i) {
    if (act[i]) {
      const u32 x = known[i] != kUnvisited ? known[i] | kIdFlag
                                           : slot[i] | (is_new[i] ? kNewFlag : 0u);
      a.temp[tpos[i]] = make_uint4(x, P1[i].y, P2[i].y, __float_as_uint(w[i]));
      a.runsrc[tpos[i]] = u[i];
    }
  }
}

template <int B>
__device__ __forceinline__ void emit_batch(const MergeArgs &a, const bool (&act)[B],
                                           const u32 (&u)[B], const u64 (&key)[B],
                                           const u64 (&tpos)[B], const float (&w)[B]) {
  u32 q1[B], q2[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    q1[i] = act[i] ? a.sq1[a.lo + u[i]] : 0;
    q2[i] = act[i] ? a.sq2[a.lo + u[i]] : 0;
  }
  u32 pb1[B], pb2[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    pb1[i] = act[i] ? a.pbase1[q1[i]] : 0;
    pb2[i] = act[i] ? a.pbase2[q2[i]] : 0;
  }
  uint2 P1[B], P2[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    P1[i] = act[i] ? a.parts1[pb1[i] + (u32)(key[i] >> a.b2)] : make_uint2(0, 0);
    P2[i] = act[i] ? a.parts2[pb2[i] + (u32)(key[i] & ((1ull << a.b2) - 1))] : make_uint2(0, 0);
  }
  emit_parts<B>(a, act, u, P1, P2, tpos, w);
}

// LDS of the sorting tile merge.
struct SortLds {
  u64 keys[C];
  float w[C];
  u32 segsrc[C];
  u32 cnt[NW * 256];
  u32 base[256];
  u32 tmp[NW];
  double wsum[NW];
  u32 wflag[NW];
};

// Sorting merge of tile `tile` by the whole block.
template <class KT>
__device__ __forceinline__ void merge_sort_tile(const MergeArgs &a, u32 tile, SortLds &L) {
  u64 *s_keys = L.keys;
  float *s_w = L.w;
  u32 *s_segsrc = L.segsrc, *s_cnt = L.cnt, *s_base = L.base, *s_tmp = L.tmp;
  double *s_wsum = L.wsum;
  u32 *s_wflag = L.wflag;
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const u64 tstart = (u64)tile * a.window;
  const uint4 td = a.tiles[tile];
  const u32 s0 = td.x, s1 = td.y;
  if (s0 >= s1) return;
  if (dense_tile(td, a.key_bits) && !(td.w & kRerouted)) return;  // merged by k_merge_dense
  const u32 n = td.w & ~kRerouted;
  const u64 rb = tstart + td.z;
  if (n > (u32)C || (u64)td.z + n > (u64)C) {
    if (threadIdx.x == 0) set_error(&a.st->err, kErrTileSize);
    return;
  }
  if (n == 0) return;
  // the tile's records, at window positions [td.z, td.z + n) of [tstart, tstart + kMergeCap)
  const KT *rk = static_cast<const KT *>(a.rec_key) + tstart;
  const float *rwin = a.rec_w + tstart;
  KT wkey[IT];
  float wwt[IT];
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const u32 wpos = w * (kWave * IT) + j * kWave + lane;
    const bool in = wpos >= td.z && wpos - td.z < n;
    wkey[j] = in ? rk[wpos] : KT(0);
    wwt[j] = in ? rwin[wpos] : 0.f;
  }
  const u32 off = td.z;  // window position of tile element 0

  // 1. mark the first record of every non-empty source with its index + 1
  u32 *s_mark = reinterpret_cast<u32 *>(s_keys);
  for (u32 i = threadIdx.x; i < n; i += NT) s_mark[i] = 0;
  __syncthreads();
  for (u32 u = s0 + threadIdx.x; u < s1; u += NT) {
    const u64 c = a.roff[u + 1] - a.roff[u];
    if (c) s_mark[a.roff[u] - rb] = u + 1;
  }
  __syncthreads();
  if (s_mark[0] == 0) {  // impossible: element 0 starts a source
    if (threadIdx.x == 0) set_error(&a.st->err, kErrBounds);
    return;
  }

  // 2. sort key = segment : record key : element index.  Items are window
  //    positions; window order is element order, which keeps the ranking
  //    stable.  The segment of an element is the number of source starts at
  //    or before it (a 0/1 prefix count: one ballot per item row).
  u64 skey[IT];
  u32 f[IT], mark[IT];
  u32 valid = 0;  // bit j: item j holds a tile element
  u32 wrun = 0;
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const u32 wpos = w * (kWave * IT) + j * kWave + lane;
    const u32 e = wpos - off;  // wraps (and fails e < n) before the tile
    const bool v = wpos >= off && e < n;
    valid |= (v ? 1u : 0u) << j;
    mark[j] = 0;
    skey[j] = 0;
    if (v) {
      skey[j] = ((u64)wkey[j] << kIdxBits) | e;
      s_w[e] = wwt[j];
      mark[j] = s_mark[e];
    }
    const u64 m = __ballot(mark[j] != 0);
    f[j] = wrun + count_below(m) + (mark[j] ? 1u : 0u);
    wrun += (u32)__popcll(m);
  }
  u32 nseg;
  {
    const u32 wbase = block_offset(wrun, s_tmp, &nseg);
#pragma unroll
    for (int j = 0; j < IT; ++j) f[j] += wbase;
  }
  const int segshift = a.key_bits + kIdxBits;
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    if (mark[j]) s_segsrc[f[j] - 1] = mark[j] - 1;
    skey[j] |= (u64)(f[j] - 1) << segshift;  // f >= 1 for every valid item
  }
  __syncthreads();  // s_mark (aliasing s_keys) fully read

  // 3. stable LSD radix sort on bits [kIdxBits, segshift + segbits).  The
  //    last pass stores sorted element p at blocked_slot(p), so that after the
  //    read-back thread (w, lane) holds the consecutive sorted elements
  //    w*512 + lane*8 + j, j = 0..7.
  const int hi_bit = segshift + bits_for_dev(nseg - 1);
  const int npass = hi_bit > kIdxBits ? (hi_bit - kIdxBits + 7) / 8 : 0;
  for (int pass = 0; pass < npass; ++pass) {
    const int shift = kIdxBits + 8 * pass;
    const int bits = min(8, hi_bit - shift);
    const u32 dmask = (1u << bits) - 1u;
    u32 dig[IT], rid[IT];
#pragma unroll
    for (int j = 0; j < IT; ++j) dig[j] = (u32)(skey[j] >> shift) & dmask;
    block_rank_digits<NT, IT>(dig, valid, bits, rid, s_cnt, s_base, s_tmp);
    const bool last_pass = pass == npass - 1;
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      if (!((valid >> j) & 1u)) continue;
      const u32 pos = s_base[dig[j]] + rid[j];
      s_keys[last_pass ? blocked_slot(pos) : pos] = skey[j];
    }
    __syncthreads();
    // read back: striped positions e < n, or after the last pass the
    // consecutive elements p = w*512 + lane*8 + j < n stored at slot e
    valid = 0;
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const u32 e = w * (kWave * IT) + j * kWave + lane;
      const u32 p = w * (kWave * IT) + lane * IT + j;
      const bool v = last_pass ? p < n : e < n;
      if (v) skey[j] = s_keys[e];
      valid |= (v ? 1u : 0u) << j;
    }
    __syncthreads();
  }
  if (npass == 0) {
    // sorted order is element order: element e (index bits of the key) goes
    // to blocked_slot(e)
#pragma unroll
    for (int j = 0; j < IT; ++j)
      if ((valid >> j) & 1u) s_keys[blocked_slot((u32)skey[j] & ((1u << kIdxBits) - 1))] = skey[j];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const u32 e = w * (kWave * IT) + j * kWave + lane;
      const u32 p = w * (kWave * IT) + lane * IT + j;
      if (p < n) skey[j] = s_keys[e];
    }
    __syncthreads();
  }

  // 4. runs of equal (segment, key) over the thread's consecutive elements
  //    p0 + j < n; run sums: serial within the thread, one segmented scan of
  //    the per-thread open run across threads (float64, fixed combining order)
  const u64 KM = ~((1ull << kIdxBits) - 1);
  const u32 IM = (1u << kIdxBits) - 1;
  const u32 p0 = w * (kWave * IT) + lane * IT;
  const u32 nv = p0 < n ? min((u32)IT, n - p0) : 0u;  // items holding elements
  u64 prevk = ~0ull, nextk = ~0ull;
  if (p0 > 0 && p0 - 1 < n) prevk = s_keys[blocked_slot(p0 - 1)] & KM;
  if (p0 + IT < n) nextk = s_keys[blocked_slot(p0 + IT)] & KM;
  u32 hmask = 0, tmask = 0, nhmask = 0;  // run head, run tail, before the thread's first head
  double part[IT];
  double acc = 0.0;
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const bool v = (u32)j < nv;
    const u64 mk = skey[j] & KM;
    const u64 before = j == 0 ? prevk : (skey[j - 1] & KM);
    const u64 after = j == IT - 1 ? nextk : ((u32)j + 1 < nv ? (skey[j + 1] & KM) : ~0ull);
    const bool hd = v && (p0 + j == 0 || before != mk);
    const bool tl = v && (p0 + j == n - 1 || after != mk);
    hmask |= (hd ? 1u : 0u) << j;
    tmask |= (tl ? 1u : 0u) << j;
    if (hd) acc = 0.0;
    if (v) acc += (double)s_w[(u32)skey[j] & IM];
    part[j] = acc;
  }
  const u32 hc = __popc(hmask);
  const u32 seen = hmask ? 1u : 0u;
  nhmask = hmask ? ((1u << (__ffs(hmask) - 1)) - 1u) : 0xffu;
  // segmented scan of (seen, acc) over lanes, then over waves
  double x = acc;
  u32 fl = seen;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const double y = __shfl_up(x, d, kWave);
    const u32 g = __shfl_up(fl, d, kWave);
    if (lane >= (u32)d) {
      if (!fl) x += y;
      fl |= g;
    }
  }
  double carry = __shfl_up(x, 1, kWave);
  u32 cflag = __shfl_up(fl, 1, kWave);
  if (lane == 0) {
    carry = 0.0;
    cflag = 0;
  }
  if (lane == kWave - 1) {
    s_wsum[w] = x;
    s_wflag[w] = fl;
  }
  // run index base: heads in earlier threads
  const u32 hinc = wave_inclusive_sum(hc);
  u32 nruns;
  const u32 hwave = block_offset(__shfl(hinc, kWave - 1, kWave), s_tmp, &nruns);  // barriers
  const u32 hbase = hwave + hinc - hc;
  if (!cflag) {
    double pre = 0.0;
    for (u32 v = 0; v < w; ++v) pre = s_wflag[v] ? s_wsum[v] : pre + s_wsum[v];
    carry += pre;
  }

  // 5. every run's last element publishes (sorted position, weight) under
  //    its run number; the block then emits the runs in parallel, run r of
  //    the tile to temp[rb + r].  The first and last run of a source record
  //    where its merged arcs start and end.
  __syncthreads();  // every s_w read done: run sums reuse s_w
  float *s_runsum = s_w;
  u16 *s_runpos = reinterpret_cast<u16 *>(s_cnt);  // sort counters are free now
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    if (!((tmask >> j) & 1u)) continue;
    // runs started at or before item j: heads in earlier threads + own heads
    const u32 r = hbase + __popc(hmask & ((2u << j) - 1u)) - 1u;
    const double sm = part[j] + (((nhmask >> j) & 1u) ? carry : 0.0);
    s_runsum[r] = (float)sm;
    s_runpos[r] = (u16)(p0 + j);
  }
  __syncthreads();
  const u64 keymask = (1ull << a.key_bits) - 1;
  for (u32 r = threadIdx.x; r < nruns; r += NT) {
    const u64 sk = s_keys[blocked_slot(s_runpos[r])];
    const u64 seg = sk >> segshift;
    const u64 key = (sk >> kIdxBits) & keymask;
    const u32 u = s_segsrc[seg];
    a.temp[rb + r] = make_uint4(u, (u32)key, (u32)(key >> 32), __float_as_uint(s_runsum[r]));
    const bool first = r == 0 || (s_keys[blocked_slot(s_runpos[r - 1])] >> segshift) != seg;
    const bool last =
        r == nruns - 1 || (s_keys[blocked_slot(s_runpos[r + 1])] >> segshift) != seg;
    if (first) a.tstart[u] = rb + r;
    if (last) a.mend[u] = rb + r + 1;
  }
  if (threadIdx.x == 0) a.tile_runs[tile] = nruns;
}

// Every tile of the level, one per workgroup.  XCD-aware tile order:
// workgroups are dealt round-robin to the 8 XCDs, so each XCD gets a
// contiguous run of tiles, whose record windows then stay in its L2.
template <class KT>
__global__ __launch_bounds__(NT, 4) void k_merge_tiles(MergeArgs a) {
  __shared__ SortLds L;
  merge_sort_tile<KT>(a, xcd_tile(blockIdx.x, gridDim.x), L);
}

// The tiles k_merge_dense listed in a.sortlist (a.st->nsort of them); a
// fixed grid walks the list.
template <class KT>
__global__ __launch_bounds__(NT, 4) void k_merge_listed(MergeArgs a) {
  __shared__ SortLds L;
  const u32 nsort = __hip_atomic_load(&a.st->nsort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (u32 i = blockIdx.x; i < nsort; i += gridDim.x) {
    merge_sort_tile<KT>(a, a.sortlist[i], L);
    __syncthreads();  // LDS reused by the next tile
  }
}

// ---------------------------------------------------------------------------
// Dense-table merge: a tile whose sources and keys span at most kDenseCap
// (source, key) pairs needs no sort.  Entry (segment, key) of an LDS table,
// segment = rank of the source among the tile's non-empty sources, collects
// the records with that key.  Sums are exact-order-independent: each entry
// adds its products as 64-bit two's-complement integers in units of
// 2^(E - 177), E the largest biased exponent among them (pass 1 takes the
// maximum, pass 2 adds).  A product of biased exponent be and significand m
// (24 bits with the hidden bit) becomes floor(+-m * 2^27 / 2^(E - be)), so
// every term is below 2^51 in magnitude, a sum of 4096 stays below 2^63, and
// the result does not depend on the order of the atomic adds; each term loses
// at most one unit, 2^-50 of the entry's largest term.  When all nonzero
// weights of the tile lie within kExactSpan binades of the smallest one
// (exponent Emin), the first pass is skipped: every term is m * 2^(be - Emin)
// exactly, in units of 2^(Emin - 150), and each sum is exact.  Entries present in
// the tile become runs in (segment, key) order, the order of the sort path.
// A tile holding an infinite or NaN weight is left to the sort kernel
// (descriptor flag kRerouted).
__device__ __forceinline__ void list_for_sort(const MergeArgs &a, u32 tile) {
  const u32 i = atomicAdd(&a.st->nsort, 1u);
  if (i < a.ntiles) a.sortlist[i] = tile;
}

// Biased exponent of a weight, denormals and zero counted as 1.
__device__ __forceinline__ u32 fx_bexp(float x) { return max((__float_as_uint(x) >> 23) & 0xffu, 1u); }

// Significand of a weight with the hidden bit, signed.
__device__ __forceinline__ int fx_sig(float x) {
  const u32 bits = __float_as_uint(x);
  const u32 mag = (bits & 0x7fffffu) | (((bits >> 23) & 0xffu) ? 0x800000u : 0u);
  return (bits >> 31) ? -(int)mag : (int)mag;
}

// LDS of the dense-table merge.
struct DenseLds {
  unsigned long long sum[kDenseCap];
  u32 exp[kDenseCap];  // 0: entry absent, else largest biased exponent + 1
  u32 segsrc[kDenseCap];
  u16 runseg[kDenseCap];
  u32 bits[C / 32];  // bit e: tile element e starts a source
  u32 pre[C / 32];   // set bits in the words before
  u32 tmp[NW];
  u32 emin, emax, nonfinite;  // over the tile's nonzero weights
};

// A tile's inputs to the dense merge: the record offsets of its first
// sources (thread t: sources s0 + t + k*NT) and its records (item j of lane
// l of wave w: tile element w*512 + j*64 + l, at min(e, n - 1)).
struct DenseRecs {
  u64 r0[kDenseEPT], r1[kDenseEPT];
  u32 key[IT];
  float wt[IT];
};

__device__ __forceinline__ void dense_load_offsets(const MergeArgs &a, const uint4 &td,
                                                   DenseRecs &in) {
#pragma unroll
  for (u32 k = 0; k < kDenseEPT; ++k) {
    in.r0[k] = in.r1[k] = 0;
    if (td.x + k * NT < td.y) {  // uniform; loads at clamped sources
      const u32 u = min(td.x + threadIdx.x + k * NT, td.y - 1);
      in.r0[k] = a.roff[u];
      in.r1[k] = a.roff[u + 1];
    }
  }
}

__device__ __forceinline__ void dense_load_records(const MergeArgs &a, u32 tile, const uint4 &td,
                                                   DenseRecs &in) {
  const u32 n = td.w;
  const u64 rb = (u64)tile * a.window + td.z;
  const u32 *rk = static_cast<const u32 *>(a.rec_key) + rb;
  const float *rw = a.rec_w + rb;
  const u32 e0 = (threadIdx.x / kWave) * (kWave * IT) + lane_id();
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const u32 e = min(e0 + j * kWave, n - 1);
    in.key[j] = __builtin_nontemporal_load(rk + e);  // read once: streaming loads
    in.wt[j] = __builtin_nontemporal_load(rw + e);
  }
}

// Present entries of the dense table (s_exp != 0) of tile `tile` -> runs
// rb + r in entry order (entry i = segment << kb | key), with the source
// ranges tstart / mend and the tile's run count.  Thread t lists entries
// t*kDenseEPT .. t*kDenseEPT + kDenseEPT - 1 of the first tsize.
__device__ __forceinline__ void dense_list_runs(const MergeArgs &a, u32 tile, u64 rb, u32 tsize,
                                                int kb, DenseLds &L) {
  unsigned long long *s_sum = L.sum;
  u32 *s_exp = L.exp, *s_segsrc = L.segsrc, *s_tmp = L.tmp;
  u16 *s_runseg = L.runseg;
  u32 pmask = 0;
#pragma unroll
  for (u32 k = 0; k < kDenseEPT; ++k) {
    const u32 i = threadIdx.x * kDenseEPT + k;
    if (i < tsize && s_exp[i] != 0) pmask |= 1u << k;
  }
  const u32 pc = __popc(pmask);
  const u32 pinc = wave_inclusive_sum(pc);
  u32 nruns;
  u32 r = block_offset(__shfl(pinc, kWave - 1, kWave), s_tmp, &nruns) + pinc - pc;
  const u32 kmask = (1u << kb) - 1u;
#pragma unroll
  for (u32 k = 0; k < kDenseEPT; ++k) {
    if (!((pmask >> k) & 1u)) continue;
    const u32 i = threadIdx.x * kDenseEPT + k;
    const int E = (int)s_exp[i] - 1;
    const double v = ldexp((double)(long long)s_sum[i], E - 177);
    const u32 seg = i >> kb;
    a.temp[rb + r] = make_uint4(s_segsrc[seg], i & kmask, 0u, __float_as_uint((float)v));
    s_runseg[r] = (u16)seg;
    ++r;
  }
  __syncthreads();
  for (u32 q = threadIdx.x; q < nruns; q += NT) {
    const u32 seg = s_runseg[q];
    const u32 u = s_segsrc[seg];
    if (q == 0 || s_runseg[q - 1] != seg) a.tstart[u] = rb + q;
    if (q == nruns - 1 || s_runseg[q + 1] != seg) a.mend[u] = rb + q + 1;
  }
  if (threadIdx.x == 0) a.tile_runs[tile] = nruns;
}

// Dense-table merge of tile `tile` (a dense tile within the tile capacity,
// as k_merge_dense checks) from its inputs `in`.
__device__ __forceinline__ void dense_merge_tile(const MergeArgs &a, u32 tile, const uint4 td,
                                                 const DenseRecs &in, DenseLds &L) {
  unsigned long long *s_sum = L.sum;
  u32 *s_exp = L.exp, *s_segsrc = L.segsrc, *s_bits = L.bits, *s_pre = L.pre;
  u32 &s_emin = L.emin, &s_emax = L.emax, &s_nonfinite = L.nonfinite;
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const u32 n = td.w, off = td.z;
  const u64 rb = (u64)tile * a.window + off;  // first record of the tile
  // 1. source starts -> bitmap -> segment of every element
  if (threadIdx.x < C / 32) s_bits[threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    s_emin = 0xffu;
    s_emax = 0;
    s_nonfinite = 0;
  }
  // a dense tile has at most kDenseCap sources: thread t takes sources
  // s0 + t + k*NT, k < kDenseEPT, and keeps their start (or kNoStart)
  constexpr u32 kNoStart = 0xffffffffu;
  u32 start[kDenseEPT];
  const u64 *r0 = in.r0, *r1 = in.r1;
  const u32 *key = in.key;
  const float *wt = in.wt;
  const u32 e0 = w * (kWave * IT) + lane;
  __syncthreads();  // s_bits cleared
#pragma unroll
  for (u32 k = 0; k < kDenseEPT; ++k)
    start[k] = (td.x + threadIdx.x + k * NT < td.y && r1[k] != r0[k]) ? (u32)(r0[k] - rb) : kNoStart;
#pragma unroll
  for (u32 k = 0; k < kDenseEPT; ++k)
    if (start[k] != kNoStart) atomicOr(&s_bits[start[k] >> 5], 1u << (start[k] & 31));
  __syncthreads();
  if (w == 0) {
    const u32 c0 = __popc(s_bits[2 * lane]), c1 = __popc(s_bits[2 * lane + 1]);
    const u32 inc = wave_inclusive_sum(c0 + c1);
    s_pre[2 * lane] = inc - c0 - c1;
    s_pre[2 * lane + 1] = inc - c1;
  }
  __syncthreads();
  if (!(s_bits[0] & 1u)) {  // impossible: element 0 starts a source
    if (threadIdx.x == 0) set_error(&a.st->err, kErrBounds);
    return;
  }
  const u32 nseg = s_pre[C / 32 - 1] + __popc(s_bits[C / 32 - 1]);
  const int kb = a.key_bits;
  const u32 tsize = nseg << kb;
  auto seg_of = [&](u32 e) {
    return s_pre[e >> 5] + __popc(s_bits[e >> 5] & ((2u << (e & 31)) - 1u)) - 1u;
  };
#pragma unroll
  for (u32 k = 0; k < kDenseEPT; ++k)
    if (start[k] != kNoStart) s_segsrc[seg_of(start[k])] = td.x + threadIdx.x + k * NT;
  for (u32 i = threadIdx.x; i < tsize; i += NT) {
    s_sum[i] = 0;
    s_exp[i] = 0;
  }
  auto bexp = fx_bexp;
  auto sig = fx_sig;
  constexpr u32 kNone = 0xffffffffu;  // table index of an absent item
  // Item j of every lane of the wave lies in the element row
  // [w*512 + j*64, +64), two bitmap words: the segment of the lane's element
  // is the row's prefix count plus the starts at or below its lane (mbcnt).
  u32 idx[IT];
  u32 nonfinite = 0, emin = 0xffu, emax = 0;
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const u32 e = e0 + j * kWave;
    const u32 wd = (w * (kWave * IT) + j * kWave) >> 5;  // uniform
    const u32 lo = __builtin_amdgcn_readfirstlane(s_bits[wd]);
    const u32 hi = __builtin_amdgcn_readfirstlane(s_bits[wd + 1]);
    const u32 pre = __builtin_amdgcn_readfirstlane(s_pre[wd]);
    const u32 below = __builtin_amdgcn_mbcnt_hi(hi, __builtin_amdgcn_mbcnt_lo(lo, 0u));
    const u32 own = (u32)((((u64)hi << 32 | lo) >> lane) & 1u);
    const u32 seg = pre + below + own - 1u;  // elements past n: never used
    idx[j] = e < n ? (seg << kb) | (key[j] & ((1u << kb) - 1u)) : kNone;
    const u32 bits = __float_as_uint(wt[j]);
    const u32 be = bexp(wt[j]);
    const bool live = e < n && (bits & 0x7fffffffu) != 0;
    nonfinite |= (e < n && be == 0xffu) ? 1u : 0u;
    emin = live ? min(emin, be) : emin;
    emax = live ? max(emax, be) : emax;
  }
  // (nonfinite, 255 - emin) packed: the lexicographic maximum is right for
  // both (emin only matters when no lane saw a non-finite weight)
  const u32 packed = wave_max((nonfinite << 8) | (0xffu - emin));
  emax = wave_max(emax);
  if (lane == 0) {
    atomicMin(&s_emin, 0xffu - (packed & 0xffu));
    atomicMax(&s_emax, emax);
    if (packed >> 8) s_nonfinite = 1;
  }
  __syncthreads();
  if (s_nonfinite) {
    if (threadIdx.x == 0) {
      a.tiles[tile].w = n | kRerouted;
      list_for_sort(a, tile);
    }
    return;
  }
  const u32 Emin = s_emin, Emax = s_emax;
  // a thread whose items all hold one entry (or none) flushes once
  bool one_run = true;
#pragma unroll
  for (int j = 1; j < IT; ++j) one_run = one_run && (idx[j] == idx[0] || idx[j] == kNone);
  if (Emax <= Emin + kExactSpan) {
    // 2'. every nonzero weight of the tile within 2^kExactSpan binades: terms
    //     m * 2^(be - Emin) are exact in 64 bits and so are their sums (all
    //     below 2^(24 + kExactSpan + 12)); entry scale 2^(Emin - 150) is
    //     recorded as s_exp = Emin + 28 (E - 177 = Emin - 150 below).
    long long term[IT];
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const u32 be = bexp(wt[j]);
      term[j] = idx[j] == kNone ? 0ll : (long long)sig(wt[j]) << (be > Emin ? be - Emin : 0u);
    }
    if (one_run) {
      long long acc = 0;
#pragma unroll
      for (int j = 0; j < IT; ++j) acc += term[j];
      if (idx[0] != kNone) {
        atomicAdd(&s_sum[idx[0]], (unsigned long long)acc);
        s_exp[idx[0]] = Emin + 28;
      }
    } else {
      long long acc = 0;
#pragma unroll
      for (int j = 0; j < IT; ++j) {
        const bool start = j == 0 || idx[j] != idx[j - 1];
        const bool end = idx[j] != kNone && (j == IT - 1 || idx[j + 1] != idx[j]);
        acc = (start ? 0ll : acc) + term[j];
        if (end) {
          atomicAdd(&s_sum[idx[j]], (unsigned long long)acc);
          s_exp[idx[j]] = Emin + 28;
        }
      }
    }
  } else {
    // 2. largest exponent per entry.  A thread's items with equal entries
    //    (64 elements apart) are combined first: one LDS atomic per run of
    //    equal consecutive items.
    {
      u32 m = 0;
#pragma unroll
      for (int j = 0; j < IT; ++j) {
        const bool start = j == 0 || idx[j] != idx[j - 1];
        const bool end = idx[j] != kNone && (j == IT - 1 || idx[j + 1] != idx[j]);
        const u32 be = bexp(wt[j]);
        m = start ? be : max(m, be);
        if (end) atomicMax(&s_exp[idx[j]], m + 1);
      }
    }
    __syncthreads();
    // 3. fixed-point sums, combined the same way
    {
      long long acc = 0;
      u32 E = 0;
#pragma unroll
      for (int j = 0; j < IT; ++j) {
        const bool start = j == 0 || idx[j] != idx[j - 1];
        const bool end = idx[j] != kNone && (j == IT - 1 || idx[j + 1] != idx[j]);
        const u32 ex = s_exp[idx[j] != kNone ? idx[j] : 0u] - 1u;
        E = start ? ex : E;
        const long long term = ((long long)sig(wt[j]) * (1ll << 27)) >> min(E - bexp(wt[j]), 63u);
        acc = (start ? 0ll : acc) + term;
        if (end) atomicAdd(&s_sum[idx[j]], (unsigned long long)acc);
      }
    }
  }
  __syncthreads();

  dense_list_runs(a, tile, rb, tsize, kb, L);
}


__global__ __launch_bounds__(NT, 8) void k_merge_dense(MergeArgs a) {
  __shared__ DenseLds L;
  const u32 tile = xcd_tile(blockIdx.x, gridDim.x);
  const uint4 td = a.tiles[tile];
  if (td.x >= td.y || td.w == 0) return;  // no small source starts in this window
  if (!dense_tile(td, a.key_bits)) {
    if (threadIdx.x == 0) list_for_sort(a, tile);
    return;
  }
  if (td.w > (u32)C || td.z > (u32)C - td.w) {
    if (threadIdx.x == 0) set_error(&a.st->err, kErrTileSize);
    return;
  }
  DenseRecs in;
  dense_load_offsets(a, td, in);
  dense_load_records(a, tile, td, in);
  dense_merge_tile(a, tile, td, in, L);
}


// ---------------------------------------------------------------------------
// Product merge, wavefront per source (level.hpp: which sources take it).
// For a source (q1, q2) every joined arc pair is a term w1(p1, g) w2(g, p2):
// the weight of q1's arc with part p1 and inner symbol g times that of q2's
// arc with symbol g and part p2, keyed (p1, p2).  With at most one arc per
// (part, symbol) cell, the merged weight of key (p1, p2) is a sum over g
// alone.  Lane g of the wave takes symbol g of the shorter list (at most 64):
//   1. it finds the symbol in the longer list (64-symbol chunks held in
//      lanes, searched by shuffles), loads both segments' arcs and writes
//      their weights to the cells (g, p1) and (g, p2) of two matrices in the
//      wave's own LDS, every cell loaded once; a ballot per part gives the
//      64-bit mask of the symbols where that part has an arc;
//   2. each table entry (p1, p2) gets q = 64 / pow2ceil(P1 P2) lanes; lane c
//      of the entry visits the symbols g = c mod q set in mask1(p1) &
//      mask2(p2) -- exactly the entry's joined arc pairs -- adding the
//      float32 product a record would carry, in float64, in increasing g;
//      the q partial sums are combined by a fixed butterfly;
//   3. every entry with a term becomes a merged arc (visited-table insert,
//      labels from the parts, see emit_parts) at temp slot R + poff[u] + r in
//      entry order; the entry's other slots are marked empty.
// Matrix-core form (the header's last word; P1, P2 <= kProdMfmaParts and
// every product a normal float32 number, expand.hip): the cells are rows of
// four (zero where a state has no arc) and step 2 is the 4 x 64 by 64 x 4
// product of the two matrices, four v_mfma_f64_4x4x4f64.  Lane l supplies
// row 16 t + l / 4, column l mod 4 of each matrix to product t; blocks
// b = (l / 4) mod 4 of the result hold the sums over g = b mod 4, row
// rotations within 16 lanes add them, and entry (p1, p2) ends in lane
// 16 p1 + p2.  Its products are exact in float64, so the merged weight
// differs from the float32-product sum by at most 2^-24 of the sum of the
// terms' magnitudes (the selection's normal-range bound) before the
// final rounding.  Entry presence and the joined pairs come from each
// lane's outer product of its two part masks, reduced by DPP.
// Aligned form (also in the header; both states dense, symbol lists of one
// length): step 1's search is replaced by loading symbol g of both lists
// with the arcs of segment g, found from the states' first arcs alone, and
// checking afterwards that the lists agree (else step 1 runs as above).
// A merged arc's temp entry holds the target's slot, with kNewFlag when
// this entry claimed it, or, with the dense visited array, the target's id
// with kIdFlag when it had one from an earlier level; the source's claims
// go to newc[u] for the new-pair list.
// No LDS is shared between waves, so no workgroup barrier is needed.
constexpr int kProdNT = 256;
constexpr int kProdWaves = kProdNT / kWave;
constexpr u32 kProdCells = kProdRowSum * kWave;  // both matrices, 64 symbols
constexpr u32 kProdRow = kProdMfmaParts;         // cells per symbol, matrix-core form
constexpr int kProdBatch = 4;                     // arcs per side loaded at once
static_assert(kProdBatch == (int)kProdRow, "one batch holds a matrix-core segment");
static_assert(2 * kProdRow * kWave <= kProdCells, "matrix-core cells fit the wave's LDS");

// x from the lane 4 or 8 places before it (cyclically) in its row of 16.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const u64 b = (u64)__double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(u32)b, CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(u32)(b >> 32), CTRL, 0xf, 0xf, false);
  return __longlong_as_double((long long)(((u64)(u32)hi << 32) | (u64)(u32)lo));
}
constexpr int kDppRowRor4 = 0x124, kDppRowRor8 = 0x128;

template <bool NARROW>
__device__ __forceinline__ uint2 prod_arc(const uint2 *arcs, u32 j) {
  if (NARROW) return *reinterpret_cast<const uint2 *>(reinterpret_cast<const char *>(arcs) + (j << 3));
  return arcs[j];
}

__device__ __forceinline__ u32 uni(u32 x) { return (u32)__builtin_amdgcn_readfirstlane((int)x); }

// One product source u (K table entries, header h0 h1) merged by the whole
// wave; val is the wave's LDS cells.
template <bool NARROW>
__device__ __forceinline__ void prod_one(const MergeArgs &a, u64 u, u32 K, uint4 h0, uint4 h1,
                                         u32 *val) {
  // everything about the source is wave-uniform: scalar registers
  const u32 lane = lane_id();
  const u32 pb1 = uni(h0.x), pb2 = uni(h0.y), P1 = uni(h0.z & 0xffffu), P2 = uni(h0.z >> 16);
  const u32 hf = uni(h0.w);
  const bool mf = (hf & 1u) != 0;       // matrix-core form
  const bool aligned = (hf & 2u) != 0;  // dense states, lists of one length na
  const bool strided = (hf & 4u) != 0;  // aligned, segments ordered by part
  const u32 na = hf >> 8;
  const u32 b1 = uni(h1.x), b2 = uni(h1.z);
  const u32 e1 = aligned ? b1 + na : uni(h1.y), e2 = aligned ? b2 + na : uni(h1.w);
  const u32 ab1 = aligned ? uni(h1.y) : 0u, ab2 = aligned ? uni(h1.w) : 0u;  // first arcs
  const bool one_short = (e1 - b1) <= (e2 - b2);
  const u32 bs = one_short ? b1 : b2, es = one_short ? e1 : e2;
  if (P1 * P2 != K || P1 + P2 > kProdRowSum || es <= bs || es - bs > (u32)kWave ||
      (mf && (P1 > kProdRow || P2 > kProdRow)) || (aligned && !mf)) {
    // impossible: the selection checked all of it
    if (lane == 0) set_error(&a.st->err, kErrBounds);
    return;
  }
  // this lane's table entry (q lanes per entry; lane 16 p1 + p2 alone in the
  // matrix-core form), its labels and the first visited-table probe of its
  // target pair, all issued before the join
  u32 q = kWave, c = 0, p1 = 0, p2 = 0;
  bool act;
  if (mf) {
    act = (lane >> 4) < P1 && (lane & 15u) < P2;
    if (act) {
      p1 = lane >> 4;
      p2 = lane & 15u;
    }
  } else {
    while (q > 1 && (kWave / q) < K) q >>= 1;  // q = 64 / pow2ceil(K)
    const u32 e = lane / q;
    c = lane % q;
    act = e < K;
    if (act) {
      p1 = e / P2;
      p2 = e - p1 * P2;
    }
  }
  const bool owner = act && c == 0;
  // loaded by every lane, without a branch (the others load part 0 and the
  // visited-table slot of that pair, in bounds); only owners use them
  const uint2 L1 = a.parts1[pb1 + p1], L2 = a.parts2[pb2 + p2];
  const u64 hk = ((u64)L1.x << 32) | (u64)L2.x;
  u64 hslot, hcur;
  if (a.vn2) {  // wave-uniform
    hslot = (u64)L1.x * a.vn2 + L2.x;
    hcur = __hip_atomic_load(&a.vis[hslot], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  } else {
    hslot = mix64(hk) & a.hmask;
    hcur = __hip_atomic_load(&a.hkeys[hslot], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }

  const u32 *ssym = one_short ? a.seg_sym1 : a.seg_sym2;
  const u32 *lsym = one_short ? a.seg_sym2 : a.seg_sym1;
  const u32 *soffs = one_short ? a.seg_off1 : a.seg_off2;
  const u32 *loffs = one_short ? a.seg_off2 : a.seg_off1;
  const u32 le = one_short ? e2 : e1;

  // Strided form (both states' segments hold one arc per part, ordered by
  // part, and the symbol lists have one length na): the matrix-core
  // operands are loaded straight from the arc arrays -- instruction t, lane l
  // takes symbol 16 t + l / 4, part l % 4, i.e. arc ab + P g + p, which for
  // P = 4 is 64 consecutive arcs per instruction -- with no staging, no part
  // masks and no entry presence test: every entry has na terms.  The lists
  // are checked to agree (else the general join below runs).
  bool has = false;
  u32 pairs = 0;
  double acc = 0.0;
  bool summed = false;
  if (strided) {
    const bool v = lane < na;
    const u32 g0 = v ? lane : 0u;
    const u32 s1 = a.seg_sym1[b1 + g0], s2 = a.seg_sym2[b2 + g0];
    const u32 pp = lane & 3u, gq = lane >> 2;
    u32 w1[4], w2[4];
    bool in1[4], in2[4];
#pragma unroll
    for (u32 t = 0; t < 4; ++t) {
      const u32 g = gq + 16u * t;
      in1[t] = g < na && pp < P1;
      in2[t] = g < na && pp < P2;
      w1[t] = a.wts1[in1[t] ? ab1 + P1 * g + pp : ab1];
      w2[t] = a.wts2[in2[t] ? ab2 + P2 * g + pp : ab2];
    }
    if (__ballot(v && s1 == s2) == __ballot(v)) {
      double d = 0.0;
#pragma unroll
      for (u32 t = 0; t < 4; ++t) {
        const double x = in1[t] ? (double)__uint_as_float(w1[t]) : 0.0;
        const double y = in2[t] ? (double)__uint_as_float(w2[t]) : 0.0;
        d = __builtin_amdgcn_mfma_f64_4x4x4f64(x, y, d, 0, 0, 0);
      }
      d += dpp_f64<kDppRowRor4>(d);
      acc = d + dpp_f64<kDppRowRor8>(d);
      has = true;
      pairs = na * P1 * P2;
      summed = true;
    }
  }
  if (!summed) {
    // 1. join, staging, part masks.  Segment offsets are loaded with the
    //    symbols (this lane's short-list segment; the long-list chunk's, handed
    //    over by the lane that found the match), so the arc loads follow the
    //    join without another round trip.  Loads are unconditional, from
    //    indexes clamped into the lists, and their values selected after.
    //    Aligned form: lane g takes symbol g of both lists, whose arcs are the
    //    P1 (P2) consecutive ones from ab1 + P1 g (ab2 + P2 g); symbols and
    //    arcs are loaded together and the arcs used once every lane's two
    //    symbols agree (else the join below runs as for other sources).
    bool found = false, staged = false;
    u32 sa = 0, sn = 0, la = 0, ln = 0;
    uint2 x1[kProdBatch], x2[kProdBatch];
    if (aligned) {
      const bool v = lane < na;
      const u32 g = v ? lane : 0u;
      const u32 s1 = a.seg_sym1[b1 + g], s2 = a.seg_sym2[b2 + g];
  #pragma unroll
      for (int k = 0; k < kProdBatch; ++k) {
        x1[k] = prod_arc<NARROW>(a.arcs1, ab1 + P1 * g + (u32)k);
        x2[k] = prod_arc<NARROW>(a.arcs2, ab2 + P2 * g + (u32)k);
      }
      staged = __ballot(v && s1 == s2) == __ballot(v);
      found = staged && v;
    }
    if (!staged) {
      const u32 idx = bs + lane;
      const bool valid = idx < es;
      const u32 ic = valid ? idx : es - 1;
      const u32 sym0 = ssym[ic], so0 = soffs[ic], so1 = soffs[ic + 1];
      const u32 sym = valid ? sym0 : 0xffffffffu;  // labels are below 2^32 - 1
      sa = valid ? so0 : 0u;
      sn = valid ? so1 - so0 : 0u;
      const u32 smax = __shfl(sym, (int)(es - bs - 1), kWave);
      const u64 vmask = __ballot(valid);
      for (u32 cb = one_short ? b2 : b1; cb < le; cb += kWave) {
        const u32 len = min(le - cb, (u32)kWave);
        const bool in = lane < len;
        const u32 lc = cb + min(lane, len - 1);
        const u32 lv0 = lsym[lc], lo00 = loffs[lc], lo10 = loffs[lc + 1];
        const u32 lv = in ? lv0 : 0xffffffffu, lo0 = in ? lo00 : 0u, lo1 = in ? lo10 : 0u;
        if (__ballot(valid && lv == sym) == vmask) {
          // the chunk starts with the short list's symbols: lane i matches lane i
          found = valid;
          la = lo0;
          ln = lo1 - lo0;
          break;
        }
        if (__shfl(lv, 0, kWave) > smax) break;  // this chunk and later ones are past every symbol
        u32 pos = 0;  // elements of the chunk below sym
    #pragma unroll
        for (u32 step = kWave / 2; step; step >>= 1) {
          const u32 v = __shfl(lv, (int)(pos + step - 1), kWave);
          pos = v < sym ? pos + step : pos;
        }
        const u32 at = __shfl(lv, (int)pos, kWave);
        const u32 pa = __shfl(lo0, (int)pos, kWave), pe = __shfl(lo1, (int)pos, kWave);
        if (valid && at == sym) {
          found = true;
          la = pa;
          ln = pe - pa;
        }
        if (__shfl(lv, (int)(len - 1), kWave) >= smax) break;  // later chunks are past every symbol
      }
    }
    u32 pm1 = 0, pm2 = 0;  // parts with an arc at this lane's symbol (parts < 16)
    bool bad = false;
    // cells per symbol row: P1 and P2, or rows of kProdRow cleared first
    const u32 S1 = mf ? kProdRow : P1, S2 = mf ? kProdRow : P2;
    if (mf) {
      *reinterpret_cast<uint4 *>(&val[lane * kProdRow]) = make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4 *>(&val[(kWave + lane) * kProdRow]) = make_uint4(0, 0, 0, 0);
    }
    const u32 a1 = one_short ? sa : la, a2 = one_short ? la : sa;
    const u32 n1 = !found ? 0u : staged ? P1 : one_short ? sn : ln;
    const u32 n2 = !found ? 0u : staged ? P2 : one_short ? ln : sn;
    // arc k of each side is present when k < h (k in the batch); a present
    // arc's part is below P (else the source is malformed); an absent one
    // writes the spare cell
    auto stage = [&](const uint2(&x1)[kProdBatch], const uint2(&x2)[kProdBatch], u32 h1, u32 h2) {
  #pragma unroll
      for (int k = 0; k < kProdBatch; ++k) {
        const bool in1 = (u32)k < h1, in2 = (u32)k < h2;
        const bool v1 = in1 & (x1[k].x < P1), v2 = in2 & (x2[k].x < P2);
        val[v1 ? lane * S1 + x1[k].x : kProdCells] = x1[k].y;
        val[v2 ? kWave * S1 + lane * S2 + x2[k].x : kProdCells] = x2[k].y;
        pm1 |= (v1 ? 1u : 0u) << x1[k].x;
        pm2 |= (v2 ? 1u : 0u) << x2[k].x;
        bad |= (in1 & !v1) | (in2 & !v2);  // bitwise: no short-circuit branches
      }
    };
    if (mf) {
      // at most kProdRow arcs per segment (single-arc cells): kProdRow
      // consecutive arcs from the segment's first (arc 0 for a lane without a
      // match; the arc arrays have kArcTail spare entries), those past the
      // segment's end replaced by padding
      static_assert(kProdBatch <= (int)kArcTail, "segment loads stay inside the arc arrays");
      if (!staged) {
        const u32 f1 = n1 ? a1 : 0u, f2 = n2 ? a2 : 0u;
  #pragma unroll
        for (int k = 0; k < kProdBatch; ++k) {
          x1[k] = prod_arc<NARROW>(a.arcs1, f1 + (u32)k);
          x2[k] = prod_arc<NARROW>(a.arcs2, f2 + (u32)k);
        }
      }
      bad |= (n1 > kProdRow) | (n2 > kProdRow);
      stage(x1, x2, n1, n2);
    } else if (found) {
      for (u32 i0 = 0; i0 < max(n1, n2); i0 += kProdBatch) {
  #pragma unroll
        for (int k = 0; k < kProdBatch; ++k) {
          const u32 i = i0 + (u32)k;
          x1[k] = i < n1 ? prod_arc<NARROW>(a.arcs1, a1 + i) : make_uint2(0, 0);
          x2[k] = i < n2 ? prod_arc<NARROW>(a.arcs2, a2 + i) : make_uint2(0, 0);
        }
        stage(x1, x2, n1 > i0 ? n1 - i0 : 0u, n2 > i0 ? n2 - i0 : 0u);
      }
    }
    if (__ballot(bad)) {  // impossible: parts are below the state's part count
      if (lane == 0) set_error(&a.st->err, kErrBounds);
      return;
    }
    // symbol masks of the parts (bit g: symbol g has an arc of the part),
    // outside the matrix-core form: lane p holds M1 part p's in ma, M2 part
    // p's in mb
    u64 ma = 0, mb = 0;
    if (!mf) {
      for (u32 p = 0; p < P1; ++p) {
        const u64 m = __ballot((pm1 >> p) & 1u);
        ma = lane == p ? m : ma;
      }
      for (u32 p = 0; p < P2; ++p) {
        const u64 m = __ballot((pm2 >> p) & 1u);
        mb = lane == p ? m : mb;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // 2. entry sums; which entries have a term (the owner's `has`) and the
    //    source's joined pairs
    if (mf) {
      // bit 4 p1 + p2 of o: parts p1 and p2 both have an arc at this lane's
      // symbol, a joined pair (the parts' bits spread 4 apart, times pm2)
      const u32 sp = (pm1 & 1u) | ((pm1 & 2u) << 3) | ((pm1 & 4u) << 6) | ((pm1 & 8u) << 9);
      const u32 o = pm2 * sp;
      has = (wave_or(o) >> ((p1 << 2) | p2)) & 1u;
      pairs = wave_total((u32)__popc(o));
      // the 4 x 64 by 64 x 4 product on the matrix cores (see above)
      double d = 0.0;
  #pragma unroll
      for (u32 t = 0; t < 4; ++t) {
        const double x = (double)__uint_as_float(val[t * kWave + lane]);
        const double y = (double)__uint_as_float(val[(kProdRow + t) * kWave + lane]);
        d = __builtin_amdgcn_mfma_f64_4x4x4f64(x, y, d, 0, 0, 0);
      }
      d += dpp_f64<kDppRowRor4>(d);
      acc = d + dpp_f64<kDppRowRor8>(d);
    } else {
      const u64 m = __shfl(ma, (int)p1, kWave) & __shfl(mb, (int)p2, kWave);  // the entry's terms
      has = m != 0;
      pairs = wave_total(owner ? (u32)__popcll(m) : 0u);
      // lane c of the entry adds the terms of g = c, c + q, ... (bit j of mm:
      // symbol c + j q is one of the entry's terms)
      u64 mm = act ? m >> c : 0;
      const u32 qs = q < (u32)kWave ? q : 0u;  // q = 64: a single symbol per lane
      u32 ia = c * P1 + p1, ib = kWave * P1 + c * P2 + p2;
      const u32 da = q * P1, db = q * P2;
      while (mm) {  // at most 64 / q steps: every step drops q bits (all, when q = 64)
        const float t = __uint_as_float(val[ia]) * __uint_as_float(val[ib]);
        acc += (mm & 1u) ? (double)t : 0.0;
        mm = qs ? mm >> qs : 0ull;
        ia += da;
        ib += db;
      }
      for (u32 d = 1; d < q; d <<= 1) acc += __shfl_xor(acc, (int)d, kWave);
    }

  }

  // 3. merged arcs in entry order: the visited-table insert resumes from
  //    the probe loaded above; the source's joined pairs (the entries' terms)
  //    go to pcnt[u]
  const bool run = owner && has;
  const u64 rm = __ballot(run);
  const u32 nr = (u32)__popcll(rm);
  const u64 pu = a.poff[u];
  const u64 base = a.R + pu;
  const bool direct = a.out_src != nullptr;  // kernel-uniform
  if (direct && !a.vn2) {  // impossible: direct levels have the dense array
    if (lane == 0) set_error(&a.st->err, kErrBounds);
    return;
  }
  bool claimed = false;  // this lane's entry claimed a new pair
  if (run && a.vn2) {
    // dense array: the entry read above, then a claim if it was unvisited
    const bool is_new = hcur == kUnvisited &&
                        atomicCAS(&a.vis[hslot], kUnvisited, kClaimed) == kUnvisited;
    claimed = is_new;
    const bool known = hcur < kClaimed;  // an id from an earlier level
    if (direct) {
      // the merged arc itself, at its place in the result
      const u64 p = a.out_base + pu + count_below(rm);
      a.out_src[p] = a.lo + (u32)u;
      a.out_dst[p] = known ? (u32)hcur : ((u32)hslot | kDstSlot | (is_new ? kDstClaim : 0u));
      a.out_il[p] = L1.y;
      a.out_ol[p] = L2.y;
      a.out_w[p] = (float)acc;
    } else {
      const u64 t = base + count_below(rm);
      a.temp[t] = make_uint4(known ? ((u32)hcur | kIdFlag) : ((u32)hslot | (is_new ? kNewFlag : 0u)),
                             L1.y, L2.y, __float_as_uint((float)acc));
      a.runsrc[t] = (u32)u;
    }
  } else if (run) {
    u32 slot = 0;
    bool is_new = false, done = false;
    for (u64 probe = 0; probe <= a.hmask && !done; ++probe) {
      if (probe) {
        hslot = (hslot + 1) & a.hmask;
        hcur = __hip_atomic_load(&a.hkeys[hslot], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
      if (hcur == kEmptyKey) {
        hcur = atomicCAS((unsigned long long *)&a.hkeys[hslot], (unsigned long long)kEmptyKey,
                         (unsigned long long)hk);
        if (hcur == kEmptyKey) {
          is_new = true;
          done = true;
          slot = (u32)hslot;
          continue;
        }
      }
      if (hcur == hk) {
        done = true;
        slot = (u32)hslot;
      }
    }
    if (!done) set_error(&a.st->err, kErrHashFull);
    const u64 t = base + count_below(rm);
    a.temp[t] = make_uint4(slot | (is_new ? kNewFlag : 0u), L1.y, L2.y, __float_as_uint((float)acc));
    a.runsrc[t] = (u32)u;
    claimed = is_new;
  }
  if (lane >= nr && lane < K) {  // an entry without a term
    if (direct) {
      a.out_src[a.out_base + pu + lane] = kHoleSrc;
      a.out_dst[a.out_base + pu + lane] = 0u;
    } else {
      a.temp[base + lane] = make_uint4(0, 0, 0, 0);  // empty slot
    }
  }
  const u32 nclaim = (u32)__popcll(__ballot(claimed));
  if (lane == 0) {
    a.tstart[u] = base;
    a.mend[u] = base + nr;
    a.pcnt[u] = pairs;
    a.newc[u] = nclaim;
  }
}

// The listed product sources (a.glist, st->ngen of them), one per wave: the
// waves of the grid take list entries wave, wave + waves, ...  Launched
// before the host knows the list length, so the grid is sized by the level.
template <bool NARROW>
__global__ __launch_bounds__(kProdNT) void k_prod_sources(MergeArgs a) {
  // M1 (g, p1), M2 (g, p2); a spare cell; rows 16-byte aligned
  __shared__ __align__(16) u32 s_val[kProdWaves][kProdCells + 4];
  // launched before the host read the level's record count: nothing to do
  // unless the level has no records (then a.R is 0)
  if (a.R_dev && *a.R_dev != 0) return;
  const u32 w = uni(threadIdx.x / kWave);
  const u32 n = uni(__hip_atomic_load(&a.st->ngen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  const u32 nw = gridDim.x * kProdWaves;
  for (u32 i = blockIdx.x * kProdWaves + w; i < n; i += nw) {
    const u64 u = uni(a.glist[i]);
    if (u >= a.nsrc) {  // impossible: the count kernel lists level sources
      if (lane_id() == 0) set_error(&a.st->err, kErrBounds);
      return;
    }
    const u32 K = uni(a.pk[u]);
    const uint4 h0 = a.phdr[2 * u], h1 = a.phdr[2 * u + 1];
    if (K == 0) continue;  // impossible: only product sources are listed
    // the previous source's LDS reads are done before this one's writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    prod_one<NARROW>(a, u, K, h0, h1, s_val[w]);
  }
}

// Strided product sources four per wave (dense visited array).  The
// v_mfma_f64_4x4x4f64 instruction works on four independent 4 x 4 blocks;
// block b = (l / 4) mod 4 takes source 4 (wave) + b.  For instruction t
// lane l supplies, for its block's source, the weights of symbol
// 4 t + l / 16, part l mod 4 of both states (zero past the source's parts
// or symbols); after sixteen instructions (64 symbols) lane l holds entry
// (l / 16, l mod 4) of its source, so every lane owns one entry and the
// claims and stores of four sources run side by side.  Sums and entry
// order are those of the one-per-wave kernel's matrix-core form.
// The four sources 4 wv .. 4 wv + 3 (one wave; the dense visited array).
__device__ __forceinline__ void quad_merge(const MergeArgs &a, u64 wv) {
  const u32 lane = lane_id();
  const u32 b = (lane >> 2) & 3u;
  const u64 u = wv * 4 + b;
  const bool in = u < a.nsrc;
  const u64 uc = in ? u : 0;
  const u32 K = in ? a.pk[uc] : 0u;
  const uint4 h0 = a.phdr[2 * uc], h1 = a.phdr[2 * uc + 1];
  bool mine = K != 0 && (h0.w & 4u) != 0;
  const u32 P1 = mine ? h0.z & 0xffffu : 0u, P2 = mine ? h0.z >> 16 : 0u;
  const u32 na = mine ? h0.w >> 8 : 0u;
  if (mine && (P1 * P2 != K || P1 > kProdRow || P2 > kProdRow || na == 0 || na > (u32)kWave)) {
    set_error(&a.st->err, kErrBounds);  // impossible: the selection checked all of it
    mine = false;
  }
  if (__ballot(mine) == 0) return;  // whole wave
  const u32 pb1 = mine ? h0.x : 0u, pb2 = mine ? h0.y : 0u;
  const u32 ab1 = mine ? h1.y : 0u, ab2 = mine ? h1.w : 0u;
  const u32 p1 = lane >> 4, p2 = lane & 3u;
  const bool own = mine && p1 < P1 && p2 < P2;
  // the owned entry's parts and visited-array entry, issued first
  const uint2 L1 = a.parts1[own ? pb1 + p1 : 0u], L2 = a.parts2[own ? pb2 + p2 : 0u];
  const u64 hslot = own ? (u64)L1.x * a.vn2 + L2.x : 0;
  const u32 hcur = __hip_atomic_load(&a.vis[hslot], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  const u64 pu = mine ? a.poff[u] : 0;
  const u32 q = lane & 3u, gk = lane >> 4;
  u32 x1[16], x2[16];
  u32 v1 = 0, v2 = 0;  // bit t: operand t present
#pragma unroll
  for (u32 t = 0; t < 16; ++t) {
    const u32 g = 4u * t + gk;
    const bool i1 = g < na && q < P1, i2 = g < na && q < P2;
    v1 |= (i1 ? 1u : 0u) << t;
    v2 |= (i2 ? 1u : 0u) << t;
    const u32 j1 = i1 ? ab1 + P1 * g + q : 0u, j2 = i2 ? ab2 + P2 * g + q : 0u;
    x1[t] = a.wts1[j1];
    x2[t] = a.wts2[j2];
  }
  double d = 0.0;
#pragma unroll
  for (u32 t = 0; t < 16; ++t) {
    const double x = ((v1 >> t) & 1u) ? (double)__uint_as_float(x1[t]) : 0.0;
    const double y = ((v2 >> t) & 1u) ? (double)__uint_as_float(x2[t]) : 0.0;
    d = __builtin_amdgcn_mfma_f64_4x4x4f64(x, y, d, 0, 0, 0);
  }
  // merged arcs in entry order within each source (lane order within a
  // block is (p1, p2) order); every entry has na terms
  const u64 bmask = 0x000f000f000f000full << (4u * b);
  const u64 rm = __ballot(own);
  const u32 rank = count_below(rm & bmask);
  bool claimed = false;
  if (own) {
    const bool is_new = hcur == kUnvisited &&
                        atomicCAS(&a.vis[hslot], kUnvisited, kClaimed) == kUnvisited;
    claimed = is_new;
    const bool known = hcur < kClaimed;  // an id from an earlier level
    if (a.utab) {
      a.utab[pu + rank] = known ? hcur : ((u32)hslot | kDstSlot | (is_new ? kDstClaim : 0u));
    } else if (a.out_src) {
      const u64 p = a.out_base + pu + rank;
      a.out_src[p] = a.lo + (u32)u;
      a.out_dst[p] = known ? hcur : ((u32)hslot | kDstSlot | (is_new ? kDstClaim : 0u));
      a.out_il[p] = L1.y;
      a.out_ol[p] = L2.y;
      a.out_w[p] = (float)d;
    } else {
      const u64 t = a.R + pu + rank;
      a.temp[t] = make_uint4(known ? (hcur | kIdFlag) : ((u32)hslot | (is_new ? kNewFlag : 0u)),
                             L1.y, L2.y, __float_as_uint((float)d));
      a.runsrc[t] = (u32)u;
    }
  }
  const u64 cm = __ballot(claimed);
  if (mine && lane == 4u * b) {  // entry (0, 0) of the source
    a.tstart[u] = a.R + pu;
    a.mend[u] = a.R + pu + K;
    a.pcnt[u] = (u64)na * K;
    a.newc[u] = (u32)__popcll(cm & bmask);
  }
}

template <bool NARROW>
__global__ __launch_bounds__(256) void k_prod_quad(MergeArgs a) {
  if (a.R_dev && *a.R_dev != 0) return;
  if (!a.vn2) {  // impossible: launched with the dense visited array only
    if (threadIdx.x == 0) set_error(&a.st->err, kErrBounds);
    return;
  }
  quad_merge(a, ((u64)blockIdx.x * blockDim.x + threadIdx.x) / kWave);
}

// Composition without reduction, a level of strided product sources whose
// targets are resolved (utab holds ids): one wave per source, lane g for
// symbol g, writes the na joined pairs of each entry (p1, p2) -- the float32
// product of the M1 arc of part p1 and the M2 arc of part p2 at symbol g
// -- with the entry's target and labels.
__global__ __launch_bounds__(256) void k_unreduced_product(MergeArgs a, const u64 *off) {
  const u32 lane = lane_id();
  const u64 u = ((u64)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  if (u >= a.nsrc) return;
  const u32 K = a.pk[u];
  if (!K) return;
  const uint4 h0 = a.phdr[2 * u], h1 = a.phdr[2 * u + 1];
  const u32 P1 = h0.z & 0xffffu, P2 = h0.z >> 16, na = h0.w >> 8;
  if (!(h0.w & 4u) || P1 * P2 != K || P1 > 4 || P2 > 4 || na > (u32)kWave) {
    if (lane == 0) set_error(&a.st->err, kErrBounds);  // impossible: the selection checked it
    return;
  }
  const u64 base = a.out_base + off[u];
  const u32 *tab = a.utab + a.poff[u];
  const u32 src = a.lo + (u32)u;
  const bool g_ok = lane < na;
  float w1[4], w2[4];
#pragma unroll
  for (u32 p = 0; p < 4; ++p) {
    w1[p] = (g_ok && p < P1) ? __uint_as_float(a.wts1[h1.y + P1 * lane + p]) : 0.f;
    w2[p] = (g_ok && p < P2) ? __uint_as_float(a.wts2[h1.w + P2 * lane + p]) : 0.f;
  }
#pragma unroll
  for (u32 p1 = 0; p1 < 4; ++p1) {
    if (p1 >= P1) break;
    const u32 il = a.parts1[h0.x + p1].y;
#pragma unroll
    for (u32 p2 = 0; p2 < 4; ++p2) {
      if (p2 >= P2) break;
      const u32 e = p1 * P2 + p2;
      const u32 t = tab[e];
      if (t & kDstSlot) {  // impossible: every target was numbered before this kernel
        if (lane == 0) set_error(&a.st->err, kErrBounds);
        return;
      }
      const u32 ol = a.parts2[h0.y + p2].y;
      if (g_ok) {
        const u64 k = base + (u64)e * na + lane;
        a.out_src[k] = src;
        a.out_dst[k] = t;
        a.out_il[k] = il;
        a.out_ol[k] = ol;
        a.out_w[k] = w1[p1] * w2[p2];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Small levels in one workgroup (level.hpp, SmallArgs).  Per level:
//   1. each source's joined pairs counted by a walk of its two symbol lists
//      (thread per source), offsets by a workgroup scan;
//   2. records (source index, part-rank key; float32 product) written to LDS;
//   3. a bitonic sort of the records by key, then each run summed in float64
//      by the thread that holds its head, merged arcs compacted in key order;
//   4. capacities checked (before anything global changes), targets inserted
//      in the visited set, the new pairs sorted by (q1, q2) and numbered
//      after the existing states, then every merged arc appended with its
//      target's id (read back from the visited set after a barrier).
constexpr int kSmallNT = 1024;

// Bitonic sort of key[0..n) (n a power of two, at most kSmallRecords) with
// a 32-bit payload, by the whole workgroup; ends with a barrier.  Up to 64
// elements the first wave sorts them in registers (shuffles, no barrier).
__device__ __forceinline__ void small_sort(u64 *key, u32 *val, u32 n) {
  if (n <= (u32)kWave) {
    if (threadIdx.x < (u32)kWave) {
      const u32 l = threadIdx.x;
      u64 x = l < n ? key[l] : ~0ull;
      u32 v = l < n ? val[l] : 0u;
      for (u32 k = 2; k <= n; k <<= 1) {
        for (u32 j = k >> 1; j > 0; j >>= 1) {
          const u64 y = __shfl_xor(x, (int)j, kWave);
          const u32 w = __shfl_xor(v, (int)j, kWave);
          // the lower lane of a pair keeps the smaller key when sorting up
          const bool up = (l & k) == 0, lower = (l & j) == 0;
          const bool take = lower == up ? y < x : y > x;
          if (take) {
            x = y;
            v = w;
          }
        }
      }
      if (l < n) {
        key[l] = x;
        val[l] = v;
      }
    }
    __syncthreads();
    return;
  }
  for (u32 k = 2; k <= n; k <<= 1) {
    for (u32 j = k >> 1; j > 0; j >>= 1) {
      for (u32 i = threadIdx.x; i < n; i += kSmallNT) {
        const u32 ixj = i ^ j;
        if (ixj > i) {
          const bool up = (i & k) == 0;
          const u64 x = key[i], y = key[ixj];
          if ((x > y) == up) {
            key[i] = y;
            key[ixj] = x;
            const u32 t = val[i];
            val[i] = val[ixj];
            val[ixj] = t;
          }
        }
      }
      __syncthreads();
    }
  }
}



// Calls f(s1, s2) for every pair of segments with one symbol: s1 in
// [b1, e1), s2 in [b2, e2), in increasing symbol order (the shorter list
// walked, the longer one binary-searched from a moving lower bound).
template <class F>
__device__ __forceinline__ void small_join(const u32 *sym1, u32 b1, u32 e1, const u32 *sym2,
                                           u32 b2, u32 e2, F &&f) {
  const u32 n1 = e1 - b1, n2 = e2 - b2;
  if (n1 <= 4 * n2 && n2 <= 4 * n1) {
    // lists of similar lengths: a linear merge (consecutive loads, no search)
    u32 i = b1, j = b2;
    while (i < e1 && j < e2) {
      const u32 x = sym1[i], y = sym2[j];
      if (x == y) {
        f(i, j);
        ++i;
        ++j;
      } else if (x < y) {
        ++i;
      } else {
        ++j;
      }
    }
    return;
  }
  const bool one = n1 <= n2;
  const u32 *ss = one ? sym1 : sym2, *ls = one ? sym2 : sym1;
  const u32 sb = one ? b1 : b2, se = one ? e1 : e2, le = one ? e2 : e1;
  u32 lo = one ? b2 : b1;
  for (u32 i = sb; i < se && lo < le; ++i) {
    const u32 sym = ss[i];
    u32 l = lo, h = le;
    while (l < h) {
      const u32 m = (l + h) >> 1;
      if (ls[m] < sym) l = m + 1; else h = m;
    }
    if (l < le && ls[l] == sym) {
      if (one) f(i, l); else f(l, i);
      lo = l + 1;
    } else {
      lo = l;
    }
  }
}

__global__ __launch_bounds__(kSmallNT) void k_small_levels(SmallArgs a) {
  __shared__ u64 s_key[kSmallRecords];
  __shared__ u32 s_val[kSmallRecords];  // record weights (bits), then claimed slots
  __shared__ u64 m_key[kSmallRecords];
  __shared__ float m_w[kSmallRecords];
  __shared__ u32 m_x[kSmallRecords];    // target slot, kNewFlag when this insert claimed it
  __shared__ u32 m_il[kSmallRecords], m_ol[kSmallRecords];  // merged arcs' labels
  __shared__ u32 m_src[kSmallRecords];                      // and source indexes
  __shared__ u32 s_pb1[kSmallSources], s_pb2[kSmallSources];  // sources' first parts
  __shared__ u64 s_scr[kSmallNT / kWave];
  const u32 t = threadIdx.x;
  SmallState st = *a.ss;
  st.levels = st.new_levels = 0;
  st.reason = 0;
  const u64 kmask = (1ull << a.key_bits) - 1, m2 = (1ull << a.b2) - 1;
  while (true) {
    const u64 nsrc = st.hi - st.lo;
    if (nsrc == 0 || (a.max_levels && st.depth >= a.max_levels)) {
      st.reason = kSmallDone;
      break;
    }
    if (nsrc > kSmallSources) {
      st.reason = kSmallTooLarge;
      break;
    }
    // 1. joined pairs per source
    u32 q1 = 0, q2 = 0, b1 = 0, e1 = 0, b2 = 0, e2 = 0;
    u64 cnt = 0;
    bool long_join = false;
    if (t < nsrc) {
      q1 = a.sq1[st.lo + t];
      q2 = a.sq2[st.lo + t];
      b1 = a.row1[q1], e1 = a.row1[q1 + 1], b2 = a.row2[q2], e2 = a.row2[q2 + 1];
      s_pb1[t] = a.part_base1[q1];
      s_pb2[t] = a.part_base2[q2];
      long_join = min(e1 - b1, e2 - b2) > kSmallShortList || max(e1 - b1, e2 - b2) > kSmallLongList;
    }
    if (__syncthreads_or(long_join)) {
      st.reason = kSmallShape;
      break;
    }
    if (t < nsrc) {
      small_join(a.seg_sym1, b1, e1, a.seg_sym2, b2, e2, [&](u32 s1, u32 s2) {
        cnt += (u64)(a.seg_off1[s1 + 1] - a.seg_off1[s1]) * (a.seg_off2[s2 + 1] - a.seg_off2[s2]);
      });
    }
    if (__syncthreads_or(cnt > kSmallPerSource)) {
      st.reason = kSmallShape;
      break;
    }
    u64 R;
    const u64 off = block_exclusive_sum<kSmallNT, u64>(cnt, s_scr, &R);
    if (R > kSmallRecords) {  // uniform: every thread has R
      st.reason = kSmallTooLarge;
      break;
    }
    if (R == 0) {  // no arc leaves this level: no new states either
      st.reason = kSmallDone;
      break;
    }
    // 2. records: key = source index, then the part-rank key
    if (t < nsrc) {
      u32 k = (u32)off;
      small_join(a.seg_sym1, b1, e1, a.seg_sym2, b2, e2, [&](u32 s1, u32 s2) {
        for (u32 i = a.seg_off1[s1]; i < a.seg_off1[s1 + 1]; ++i) {
          const uint2 x1 = a.arcs1[i];
          for (u32 j = a.seg_off2[s2]; j < a.seg_off2[s2 + 1]; ++j) {
            const uint2 x2 = a.arcs2[j];
            s_key[k] = ((u64)t << a.key_bits) | ((u64)x1.x << a.b2) | (u64)x2.x;
            s_val[k] = __float_as_uint(__uint_as_float(x1.y) * __uint_as_float(x2.y));
            ++k;
          }
        }
      });
    }
    u32 n = 1;
    while (n < R) n <<= 1;
    for (u32 i = (u32)R + t; i < n; i += kSmallNT) s_key[i] = ~0ull;
    __syncthreads();
    // 3. sort, then runs: thread t takes records 2t, 2t + 1
    small_sort(s_key, s_val, n);
    u32 heads = 0;
#pragma unroll
    for (u32 h = 0; h < 2; ++h) {
      const u32 i = 2 * t + h;
      heads += (i < R && (i == 0 || s_key[i] != s_key[i - 1])) ? 1u : 0u;
    }
    u64 M;
    u32 pos = (u32)block_exclusive_sum<kSmallNT, u64>(heads, s_scr, &M);
#pragma unroll
    for (u32 h = 0; h < 2; ++h) {
      const u32 i = 2 * t + h;
      if (i < R && (i == 0 || s_key[i] != s_key[i - 1])) {
        double sum = 0.0;
        for (u32 j = i; j < R && s_key[j] == s_key[i]; ++j) sum += (double)__uint_as_float(s_val[j]);
        m_key[pos] = s_key[i];
        m_w[pos] = (float)sum;
        ++pos;
      }
    }
    // 4. capacities first (the level is redone from the start by the host
    // or by a later call when one does not suffice)
    if (st.n_states + M > a.state_cap || st.arcs + M > a.arc_cap) {
      st.reason = kSmallCapacity;
      break;
    }
    __syncthreads();
    for (u32 i = t; i < M; i += kSmallNT) {
      const u64 key = m_key[i];
      const u32 u = (u32)(key >> a.key_bits);
      const u64 r = key & kmask;
      const uint2 P1 = a.parts1[s_pb1[u] + (u32)(r >> a.b2)];
      const uint2 P2 = a.parts2[s_pb2[u] + (u32)(r & m2)];
      m_il[i] = P1.y;
      m_ol[i] = P2.y;
      m_src[i] = u;
      const u64 hk[1] = {((u64)P1.x << 32) | (u64)P2.x};
      const bool act[1] = {true};
      u32 slot[1], known[1];
      bool is_new[1];
      visit_batch<1>(a.va, hk, act, slot, is_new, known);
      m_x[i] = slot[0] | (is_new[0] ? kNewFlag : 0u);
      m_key[i] = hk[0];  // from here on: the target pair
    }
    __syncthreads();
    // the new pairs in (q1, q2) order: claimed entries (thread t: 2t, 2t+1)
    u32 claims = 0;
#pragma unroll
    for (u32 h = 0; h < 2; ++h) {
      const u32 i = 2 * t + h;
      claims += (i < M && (m_x[i] & kNewFlag)) ? 1u : 0u;
    }
    u64 nnew;
    u32 cpos = (u32)block_exclusive_sum<kSmallNT, u64>(claims, s_scr, &nnew);
#pragma unroll
    for (u32 h = 0; h < 2; ++h) {
      const u32 i = 2 * t + h;
      if (i < M && (m_x[i] & kNewFlag)) {
        s_key[cpos] = m_key[i];  // the target pair (r1, r2)
        s_val[cpos] = m_x[i] & ~kNewFlag;
        ++cpos;
      }
    }
    u32 nc = 1;
    while (nc < nnew) nc <<= 1;
    for (u32 i = (u32)nnew + t; i < nc; i += kSmallNT) s_key[i] = ~0ull;
    __syncthreads();
    small_sort(s_key, s_val, nc);
    for (u32 i = t; i < nnew; i += kSmallNT) {
      const u32 id = (u32)(st.n_states + i);
      a.va.vis[s_val[i]] = id;
      a.sq1[id] = (u32)(s_key[i] >> 32);
      a.sq2[id] = (u32)s_key[i];
    }
    __syncthreads();
    // merged arcs with their targets' ids
    for (u32 i = t; i < M; i += kSmallNT) {
      const u64 o = st.arcs + i;
      a.out_src[o] = (u32)st.lo + m_src[i];
      a.out_dst[o] = a.va.vis[m_x[i] & ~kNewFlag];
      a.out_il[o] = m_il[i];
      a.out_ol[o] = m_ol[i];
      a.out_w[o] = m_w[i];
    }
    st.max_frontier = max<u64>(st.max_frontier, nsrc);
    st.max_level_pre = max<u64>(st.max_level_pre, R);
    st.premerge += R;
    st.arcs += M;
    st.lo = st.hi;
    st.n_states += nnew;
    st.hi = st.n_states;
    ++st.depth;
    ++st.levels;
    if (nnew) ++st.new_levels;
    __syncthreads();  // LDS reused by the next level
  }
  if (t == 0) *a.ss = st;
}

// ---------------------------------------------------------------------------
// Fused expand + merge (the records of a tile never leave the chip).  The
// matches of the tile's sources (moff[s0] .. moff[s1]) are staged in chunks
// of kFuseChunk in LDS -- first element in the tile, first M1 and M2 arc, n2,
// and a bitmap of match starts -- and thread t produces the 8 consecutive
// tile elements from 8 t of the chunk's span the way the write pass does:
// the element's match by prefix popcount, (i, j) = divmod(offset, n2) for its
// M1 and M2 arc, then stepping; all arc loads of the run before any use.
// Keys and weights go to LDS at their element positions, and the dense merge
// reads them back in its striped order.  A tile the dense table cannot take
// writes its records to the record arrays instead and is left to the sort
// kernel.
constexpr int kFuseChunk = 512;
constexpr int kFuseRun = 8;
static_assert(kFuseRun * NT == C, "one run per thread covers a tile");

struct FuseLds {
  u32 rel[kFuseChunk + 1];  // first element of each staged match; the chunk's end
  u32 a1[kFuseChunk], a2[kFuseChunk], n2[kFuseChunk];
  u32 mbits[C / 32], mpre[C / 32];  // match starts among the tile's elements
  u16 key[C];                        // dense keys fit 11 bits
  float w[C];
};

union FuseDenseLds {
  FuseLds f;
  DenseLds d;
};

template <bool NARROW>
__device__ __forceinline__ uint2 fuse_arc(const uint2 *arcs, u32 j) {
  if (NARROW) return *reinterpret_cast<const uint2 *>(reinterpret_cast<const char *>(arcs) + (j << 3));
  return arcs[j];
}

template <bool NARROW>
__global__ __launch_bounds__(NT, 6) void k_fuse_merge(MergeArgs a) {
  __shared__ FuseDenseLds U;
  FuseLds &F = U.f;
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const u32 tile = xcd_tile(blockIdx.x, gridDim.x);
  const uint4 td = a.tiles[tile];
  if (td.x >= td.y || td.w == 0) return;  // no small source starts in this window
  const u32 n = td.w;
  if (n > (u32)C || td.z > (u32)C - n) {
    if (threadIdx.x == 0) set_error(&a.st->err, kErrTileSize);
    return;
  }
  const bool dense = dense_tile(td, a.key_bits);
  const u64 rb = (u64)tile * a.window + td.z;  // first record of the tile
  DenseRecs in;
  if (dense) dense_load_offsets(a, td, in);
  const u64 ka = a.moff[td.x], kz = a.moff[td.y];
  for (u64 kc = ka; kc < kz; kc += kFuseChunk) {
    const u32 nm = (u32)min<u64>(kFuseChunk, kz - kc);
    if (kc != ka) __syncthreads();  // previous chunk's LDS fully read
    if (threadIdx.x < C / 32) F.mbits[threadIdx.x] = 0;
    __syncthreads();
    for (u32 i = threadIdx.x; i <= nm; i += NT) {
      // element of match kc + i (i == nm: where the chunk ends)
      const u64 k = kc + i;
      const u32 rel = k < kz ? (u32)(a.mrbase[k] - rb) : n;
      F.rel[i] = rel;
      if (i < nm) {
        const uint4 m = a.match[k];
        F.a1[i] = m.x;
        F.a2[i] = m.y;
        F.n2[i] = m.w;
        atomicOr(&F.mbits[rel >> 5], 1u << (rel & 31));
      }
    }
    __syncthreads();
    if (w == 0) {
      const u32 c0 = __popc(F.mbits[2 * lane]), c1 = __popc(F.mbits[2 * lane + 1]);
      const u32 inc = wave_inclusive_sum(c0 + c1);
      F.mpre[2 * lane] = inc - c0 - c1;
      F.mpre[2 * lane + 1] = inc - c1;
    }
    __syncthreads();
    const u32 cs = F.rel[0], ce = F.rel[nm];  // the chunk's elements
    const u32 p0 = cs + kFuseRun * threadIdx.x;
    if (p0 < ce && ce <= n) {
      const u32 cnt = min((u32)kFuseRun, ce - p0);
      u32 p = p0;
      const u32 wd = p >> 5;
      u32 mi = F.mpre[wd] + __popc(F.mbits[wd] & ((2u << (p & 31)) - 1u)) - 1u;
      u32 a1 = F.a1[mi], a2 = F.a2[mi], n2 = F.n2[mi], nxt = F.rel[mi + 1];
      const u32 t = p - F.rel[mi];
      u32 i1 = t / n2, i2 = t - (t / n2) * n2;
      u32 ix1[kFuseRun], ix2[kFuseRun];
      ix1[0] = a1 + i1;
      ix2[0] = a2 + i2;
#pragma unroll
      for (int j = 1; j < kFuseRun; ++j) {
        ++p;
        ++i2;
        const bool wrap = i2 == n2;
        i2 = wrap ? 0u : i2;
        i1 += wrap ? 1u : 0u;
        if (p == nxt && (u32)j < cnt) {  // element j opens the next match
          ++mi;
          a1 = F.a1[mi];
          a2 = F.a2[mi];
          n2 = F.n2[mi];
          nxt = F.rel[mi + 1];
          i1 = i2 = 0;
        }
        const bool v = (u32)j < cnt;
        ix1[j] = v ? a1 + i1 : ix1[0];
        ix2[j] = v ? a2 + i2 : ix2[0];
      }
      uint2 A1[kFuseRun], A2[kFuseRun];
#pragma unroll
      for (int j = 0; j < kFuseRun; ++j) {
        A1[j] = fuse_arc<NARROW>(a.arcs1, ix1[j]);
        A2[j] = fuse_arc<NARROW>(a.arcs2, ix2[j]);
      }
#pragma unroll
      for (int j = 0; j < kFuseRun; ++j) {
        if ((u32)j >= cnt) continue;
        const u32 key = (A1[j].x << a.b2) | A2[j].x;
        const float wt = __uint_as_float(A1[j].y) * __uint_as_float(A2[j].y);
        if (dense) {
          F.key[p0 + j] = (u16)key;
          F.w[p0 + j] = wt;
        } else {
          static_cast<u32 *>(const_cast<void *>(a.rec_key))[rb + p0 + j] = key;
          const_cast<float *>(a.rec_w)[rb + p0 + j] = wt;
        }
      }
    }
  }
  if (!dense) {
    if (threadIdx.x == 0) list_for_sort(a, tile);
    return;
  }
  __syncthreads();  // every element generated
  const u32 e0 = w * (kWave * IT) + lane;
  bool nonfinite = false;
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const u32 e = min(e0 + j * kWave, n - 1);
    in.key[j] = F.key[e];
    in.wt[j] = F.w[e];
    nonfinite |= ((__float_as_uint(in.wt[j]) >> 23) & 0xffu) == 0xffu;
  }
  // a non-finite weight sends the tile to the sort kernel, which reads the
  // records from HBM: write them there first
  if (__syncthreads_or(nonfinite)) {
    u32 *rk = static_cast<u32 *>(const_cast<void *>(a.rec_key)) + rb;
    float *rw = const_cast<float *>(a.rec_w) + rb;
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const u32 e = e0 + j * kWave;
      if (e < n) {
        rk[e] = in.key[j];
        rw[e] = in.wt[j];
      }
    }
  }
  __syncthreads();  // the merge reuses the LDS
  dense_merge_tile(a, tile, td, in, U.d);
}

// Descriptor of merge tile t: the small sources whose first record falls in
// [t W, (t + 1) W) -- (first source, one past the last, window offset of the
// first record, number of records).
__global__ void k_tile_sources(const u64 *roff, u32 nsrc, u64 R, u64 W, u64 ntiles, uint4 *tiles) {
  for (u64 t = (u64)blockIdx.x * blockDim.x + threadIdx.x; t < ntiles; t += (u64)gridDim.x * blockDim.x) {
    const u64 tstart = t * W;
    const u32 s0 = (u32)min(lower_bound_dev<u64>(roff, (u64)nsrc + 1, tstart), (u64)nsrc);
    u32 s1 = (u32)min(lower_bound_dev<u64>(roff, (u64)nsrc + 1, min(tstart + W, R)), (u64)nsrc);
    // a multi-block source can only be the last one starting in the window
    if (s1 > s0 && roff[s1] - roff[s1 - 1] > kMergeSmall) --s1;
    const u64 rb = roff[s0];
    tiles[t] = make_uint4(s0, s1, (u32)(rb - min(rb, tstart)), (u32)(roff[s1] - rb));
  }
}

// ---------------------------------------------------------------------------
// Multi-block path for sources of more than kMergeSmall records.
__global__ void k_big_counts(const u64 *roff, const u32 *big, u32 nbig, u64 *bigcnt) {
  const u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nbig) bigcnt[i] = roff[big[i] + 1] - roff[big[i]];
}

template <class KT>
__global__ void k_big_gather(const u32 *big, const u64 *bigoff, u32 nbig, u64 RB, const u64 *roff,
                             const KT *rec_key, const float *rec_w, int key_bits, u64 *skey,
                             u32 *sval) {
  const u64 g = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= RB) return;
  const u32 i = (u32)last_le<u64>(bigoff, nbig, g);
  const u64 r = roff[big[i]] + (g - bigoff[i]);
  skey[g] = ((u64)i << key_bits) | (u64)rec_key[r];
  sval[g] = __float_as_uint(rec_w[r]);
}

__global__ void k_run_heads(const u64 *keys, u64 n, u32 *flags) {
  const u64 g = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  if (g < n) flags[g] = (g == 0 || keys[g] != keys[g - 1]) ? 1u : 0u;
}

// One thread per run head of the sorted multi-block records: sums the run
// and emits the merged arc (visited-table insert included, see emit_batch).
__global__ void k_big_reduce(MergeArgs a, const u64 *bigoff, u64 RB, const u64 *skey,
                             const u32 *sval, const u32 *flags, const u32 *ridx) {
  const u64 g = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  bool act[1] = {g < RB && flags[g] != 0};
  u32 uu[1] = {0};
  u64 key[1] = {0}, tpos[1] = {0};
  float wt[1] = {0.f};
  if (act[0]) {
    const u64 mk = skey[g];
    const u32 i = (u32)(mk >> a.key_bits);
    double acc = 0.0;
    u64 q = g;
    while (q < RB && skey[q] == mk) {
      acc += (double)__uint_as_float(sval[q]);
      ++q;
    }
    const u32 u = a.big[i];
    const u64 local = ridx[g] - ridx[bigoff[i]];
    const u64 base = a.roff[u];
    if (g == bigoff[i]) a.tstart[u] = base;
    if (q == RB || (u32)(skey[q] >> a.key_bits) != i) a.mend[u] = base + local + 1;
    uu[0] = u;
    key[0] = mk & ((1ull << a.key_bits) - 1);
    tpos[0] = base + local;
    wt[0] = (float)acc;
  }
  emit_batch<1>(a, act, uu, key, tpos, wt);
}

// Wave k of the wpt waves sharing a tile: the tile's runs at temp[rb ...] in
// chunks of 64 B (chunks k, k + wpt, ...), B per lane at a time (lane l takes
// runs r0 + l + 64 i, i < B).  Wave-uniform trip count.
template <int B>
__device__ __forceinline__ void emit_tile_runs(const MergeArgs &a, u64 rb, u32 nr, u32 lane, u32 k,
                                               u32 wpt) {
  for (u32 r0 = k * B * kWave; r0 < nr; r0 += wpt * B * kWave) {
    bool act[B];
    u32 uu[B];
    u64 key[B], tpos[B];
    float wt[B];
#pragma unroll
    for (int i = 0; i < B; ++i) {
      const u32 r = r0 + i * kWave + lane;
      act[i] = r < nr;
      uu[i] = 0;
      key[i] = 0;
      tpos[i] = 0;
      wt[i] = 0.f;
      if (act[i]) {
        const u64 t = rb + r;
        const uint4 rec = a.temp[t];
        uu[i] = rec.x;
        key[i] = (u64)rec.y | ((u64)rec.z << 32);
        tpos[i] = t;
        wt[i] = __uint_as_float(rec.w);
      }
    }
    emit_batch<B>(a, act, uu, key, tpos, wt);
  }
}

// Merged arcs of the tile-merged sources, wpt waves per merge tile (the tile
// kernels left tile_runs[t] runs at temp[t W + off, ...)): each run record
// (source, part-rank key, weight) becomes (slot, a, c, weight) -- part ranks
// mapped back to (r1, a) and (r2, c), the target pair inserted in the
// visited table, kNewFlag set on claimed slots.  Separate from the merge so
// that these dependent lookups run at full occupancy.
__global__ __launch_bounds__(256) void k_emit_tiles(MergeArgs a, u32 wpt) {
  const u32 lane = lane_id();
  const u64 gw = (u64)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  const u64 tile = gw / wpt;
  const u32 k = (u32)(gw % wpt);
  if (tile >= a.ntiles) return;
  const u32 nr = a.tile_runs[tile];
  if (k * kWave >= nr) return;
  const u64 rb = tile * a.window + a.tiles[tile].z;
  if (nr <= wpt * kWave) {
    emit_tile_runs<1>(a, rb, nr, lane, k, wpt);
  } else {
    emit_tile_runs<kEmitBatch>(a, rb, nr, lane, k, wpt);  // several lookups in flight per lane
  }
}

// New-state list without a shared counter: wave w either walks the runs of
// merge tile w (w < ntiles), or 64 positions of the multi-block record space
// (runs of multi-block source i sit at temp[roff[big[i]] + p - bigoff[i]]
// while below mend), or 64 product-merge slots temp[R + p] (empty slots
// carry no flag).  Pass 0 counts the flagged (claimed) slots per wave into
// wcnt; pass 1 writes them to newlist at woff[w] (exclusive scan of wcnt) in
// wave order.
template <int PASS>
__global__ __launch_bounds__(256) void k_newlist(MergeArgs a, const u64 *bigoff, u32 nbig, u64 RB,
                                                 u64 nbigw, u32 *wcnt, const u64 *woff) {
  const u32 lane = lane_id();
  const u64 wv = ((u64)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  if (wv >= a.ntiles + nbigw + (a.prodpos + kWave - 1) / kWave) return;
  const u64 base = PASS ? woff[wv] : 0;
  u32 cnt = 0;
  auto take = [&](bool f, u32 slot) {
    const u64 m = __ballot(f);
    if (PASS && f) {
      const u64 pos = base + cnt + count_below(m);
      if (pos < a.newcap) a.newlist[pos] = slot;
      else set_error(&a.st->err, kErrNewList);
    }
    cnt += (u32)__popcll(m);
  };
  if (wv < a.ntiles) {
    const u32 nr = a.tile_runs[wv];
    if (nr == 0) {
      if (!PASS && lane == 0) wcnt[wv] = 0;
      return;
    }
    const u64 rb = wv * a.window + a.tiles[wv].z;
    for (u32 r0 = 0; r0 < nr; r0 += kWave) {
      u32 x = 0;
      if (r0 + lane < nr) x = a.temp[rb + r0 + lane].x;
      take((x & kNewFlag) != 0, x & ~kNewFlag);
    }
  } else if (wv >= a.ntiles + nbigw) {
    const u64 p = (wv - a.ntiles - nbigw) * kWave + lane;
    const u32 x = p < a.prodpos ? a.temp[a.R + p].x : 0u;
    take((x & kNewFlag) != 0, x & ~kNewFlag);
  } else {
    const u64 p = (wv - a.ntiles) * kWave + lane;
    u32 x = 0;
    if (p < RB) {
      const u32 i = (u32)last_le<u64>(bigoff, nbig, p);
      const u32 u = a.big[i];
      const u64 t = a.roff[u] + (p - bigoff[i]);
      if (t < a.mend[u]) x = a.temp[t].x;
    }
    take((x & kNewFlag) != 0, x & ~kNewFlag);
  }
  if (!PASS && lane == 0) wcnt[wv] = cnt;
}

// New-pair list of a level whose sources all took the product merge: 16
// lanes per source (a source has at most 64 entries); a source with claims
// writes the slots of its claimed entries, in temp order, from list entry
// newoff[u].
__global__ __launch_bounds__(256) void k_newlist_sources(MergeArgs a, const u64 *newoff) {
  const u64 t = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  const u64 u = t / 16;
  const u32 j = (u32)(t % 16), lane = lane_id();
  const u32 nc = u < a.nsrc ? a.newc[u] : 0u;
  if (__ballot(nc != 0) == 0) return;  // whole wave
  u64 base = 0, n = 0, o = 0;
  if (nc) {
    base = a.tstart[u];
    n = a.mend[u] - base;
    o = newoff[u];
  }
  const u64 gmask = 0xffffull << (lane & ~15u);  // this lane's group of 16
  u32 done = 0;
  for (u32 r0 = 0; r0 < (u32)kWave; r0 += 16) {
    const u64 r = r0 + j;
    const u32 x = (nc && r < n) ? a.temp[base + r].x : 0u;
    const bool f = (x & kNewFlag) != 0;
    const u64 m = __ballot(f) & gmask;
    if (f) {
      const u64 pos = o + done + count_below(m);
      if (pos < a.newcap) a.newlist[pos] = x & ~kNewFlag;
      else set_error(&a.st->err, kErrNewList);
    }
    done += (u32)__popcll(m);
  }
}

// Direct product level: four lanes per source with claims; its claimed
// entries (kDstClaim in the result's target column, entry order) get ids
// base + newoff[u], + 1, ..., written to the visited array, the state arrays
// and the target column.  Lane j of a group holds entries j, j + 4, ... (a
// source has at most 64), all loaded before any is assigned.
// Lane t of the four lanes of source t / 4 (whole waves).
__device__ __forceinline__ void assign_direct_lanes(const MergeArgs &a, const u64 *newoff, u32 base,
                                                    u32 *sq1, u32 *sq2, u64 t) {
  const u64 u = t / 4;
  const u32 j = (u32)(t % 4), lane = lane_id();
  const u32 nc = u < a.nsrc ? a.newc[u] : 0u;
  if (__ballot(nc != 0) == 0) return;  // whole wave
  u32 *d = a.out_dst;
  u32 n = 0, id = 0;
  if (nc) {
    d += a.out_base + a.poff[u];
    n = (u32)(a.mend[u] - a.tstart[u]);
    id = base + (u32)newoff[u];
  }
  u32 x[16];
#pragma unroll
  for (u32 k = 0; k < 16; ++k) {
    const u32 r = 4 * k + j;
    x[k] = (nc && r < n) ? d[r] : 0u;
  }
  const u64 gmask = 0xfull << (lane & ~3u);  // this lane's group of four
#pragma unroll
  for (u32 k = 0; k < 16; ++k) {
    const bool f = (x[k] & kDstClaim) != 0;
    const u64 m = __ballot(f) & gmask;
    if (f) {
      const u32 slot = x[k] & kDstSlotMask;
      const u32 v = id + count_below(m);
      a.vis[slot] = v;
      sq1[v] = slot / a.vn2;
      sq2[v] = slot % a.vn2;
      d[4 * k + j] = v;
    }
    id += (u32)__popcll(m);
  }
}

__global__ __launch_bounds__(256) void k_assign_direct(MergeArgs a, const u64 *newoff, u32 base,
                                                       u32 *sq1, u32 *sq2) {
  if (a.R_dev && *a.R_dev != 0) return;  // enqueued ahead: the level has records
  assign_direct_lanes(a, newoff, base, sq1, sq2, (u64)blockIdx.x * blockDim.x + threadIdx.x);
}

// After the id assignment of direct product levels: targets still marked
// kDstSlot (claimed by another source of their level) get their ids from the
// visited array.  Four entries per thread, 16-byte accesses after a head of
// at most three.
__device__ __forceinline__ u32 fixed_target(const MergeArgs &a, u32 x) {
  if (!(x & kDstSlot)) return x;
  const u64 slot = x & kDstSlotMask;
  if (slot > a.hmask) {  // impossible: slots index the visited array
    set_error(&a.st->err, kErrBounds);
    return x;
  }
  return a.vis[slot];
}

__global__ void k_fix_marked(MergeArgs a, u64 n) {
  u32 *dst = a.out_dst + a.out_base;
  const u64 head = std::min<u64>(n, (4u - ((u32)(reinterpret_cast<uintptr_t>(dst) >> 2) & 3u)) & 3u);
  const u64 nv = (n - head) / 4;
  uint4 *body = reinterpret_cast<uint4 *>(dst + head);
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += (u64)gridDim.x * blockDim.x) {
    const uint4 x = body[i];
    if (!((x.x | x.y | x.z | x.w) & kDstSlot)) continue;
    body[i] = make_uint4(fixed_target(a, x.x), fixed_target(a, x.y), fixed_target(a, x.z),
                         fixed_target(a, x.w));
  }
  // the head and the last (n - head) % 4 entries
  if (blockIdx.x == 0 && threadIdx.x < 8) {
    const u64 k = threadIdx.x < 4 ? threadIdx.x : head + nv * 4 + (threadIdx.x - 4);
    const bool mine = threadIdx.x < 4 ? k < head : k < n;
    if (mine) dst[k] = fixed_target(a, dst[k]);
  }
}

// Direct product level with entries without a term: the n rows at out_base,
// copied to tmp, go back without those entries (source u's arcs to
// out_base + aoff[u]); 16 lanes per source.
__global__ void k_copy_rows(const MergeArgs a, u64 n, u32 *tmp) {
  const u32 *cols[5] = {a.out_src, a.out_dst, a.out_il, a.out_ol,
                        reinterpret_cast<const u32 *>(a.out_w)};
  for (u64 k = (u64)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (u64)gridDim.x * blockDim.x)
#pragma unroll
    for (int c = 0; c < 5; ++c) tmp[(u64)c * n + k] = cols[c][a.out_base + k];
}

__global__ __launch_bounds__(256) void k_close_holes(MergeArgs a, const u64 *aoff, u64 n,
                                                     const u32 *tmp) {
  const u64 t = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  const u64 u = t / 16;
  const u32 j = (u32)(t % 16);
  if (u >= a.nsrc) return;
  const u64 from = a.poff[u], to = aoff[u], m = a.mend[u] - a.tstart[u];
  if (from + m > n || to + m > n) {  // impossible: counts agree with the scans
    if (j == 0) set_error(&a.st->err, kErrBounds);
    return;
  }
  u32 *cols[5] = {a.out_src, a.out_dst, a.out_il, a.out_ol, reinterpret_cast<u32 *>(a.out_w)};
  for (u64 r = j; r < m; r += 16)
#pragma unroll
    for (int c = 0; c < 5; ++c) cols[c][a.out_base + to + r] = tmp[(u64)c * n + from + r];
}

// Level total of new states (end of the exclusive scan of the per-wave counts).
__global__ void k_new_total(const u64 *total, Status *st) { st->nnew = (u32)min<u64>(*total, 0xffffffffull); }

// ---------------------------------------------------------------------------
// Composition without reduction (every joined arc pair is an arc).  Wave per
// kUnredB * 64 consecutive records, lane-striped: a record's source by a
// binary search within the sources of the wave's first and last record; its
// part ranks back to (r1, a) and (r2, c); the target pair claimed in the
// visited table (new claims set a bit of newbits, so the new-state list
// needs no shared counter); the arc written with the table slot as target.
constexpr int kUnredB = 4;

template <class KT>
__global__ __launch_bounds__(256) void k_unreduced(MergeArgs a, u32 *newbits, u32 *osrc,
                                                   u32 *odst, u32 *oil, u32 *ool, float *ow) {
  const u32 lane = lane_id();
  const u64 wv = ((u64)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const u64 wb = wv * (u64)(kWave * kUnredB);
  if (wb >= a.R) return;
  const u64 we = min(wb + (u64)(kWave * kUnredB), a.R);
  u32 ul = 0;
  if (lane < 2) ul = (u32)last_le<u64>(a.roff, a.nsrc, lane == 0 ? wb : we - 1);
  const u32 u0 = __shfl(ul, 0, kWave), u1 = __shfl(ul, 1, kWave);
  const KT *rk = static_cast<const KT *>(a.rec_key);
  bool act[kUnredB];
  u32 uu[kUnredB], slot[kUnredB];
  u64 hk[kUnredB], r[kUnredB];
  uint2 P1[kUnredB], P2[kUnredB];
  float wt[kUnredB];
  bool is_new[kUnredB];
  u32 known[kUnredB];  // unused: the result holds slots until the ids are known
#pragma unroll
  for (int i = 0; i < kUnredB; ++i) {
    r[i] = wb + (u64)i * kWave + lane;
    act[i] = r[i] < we;
    const u64 rr = act[i] ? r[i] : wb;
    uu[i] = u0 + (u32)last_le<u64>(a.roff + u0, (u64)(u1 - u0) + 1, rr);
    const u64 key = (u64)rk[rr];
    wt[i] = a.rec_w[rr];
    const u32 q1 = a.sq1[a.lo + uu[i]], q2 = a.sq2[a.lo + uu[i]];
    P1[i] = a.parts1[a.pbase1[q1] + (u32)(key >> a.b2)];
    P2[i] = a.parts2[a.pbase2[q2] + (u32)(key & ((1ull << a.b2) - 1))];
    hk[i] = ((u64)P1[i].x << 32) | (u64)P2[i].x;
  }
  visit_batch<kUnredB>(a, hk, act, slot, is_new, known);
#pragma unroll
  for (int i = 0; i < kUnredB; ++i) {
    if (!act[i]) continue;
    if (is_new[i]) atomicOr(&newbits[slot[i] >> 5], 1u << (slot[i] & 31));
    osrc[r[i]] = a.lo + uu[i];
    odst[r[i]] = slot[i];
    oil[r[i]] = P1[i].y;
    ool[r[i]] = P2[i].y;
    ow[r[i]] = wt[i];
  }
}

// Set bits of a bitmap as a list of bit indices in increasing order: wave w
// takes words [64 w, 64 w + 64); pass 0 counts, pass 1 writes at woff[w].
template <int PASS>
__global__ __launch_bounds__(256) void k_bitlist(const u32 *bits, u64 nwords, u32 *wcnt,
                                                 const u64 *woff, u32 *list, u64 cap, Status *st) {
  const u32 lane = lane_id();
  const u64 wv = ((u64)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const u64 i = wv * kWave + lane;
  if (wv * kWave >= nwords) return;
  u32 word = i < nwords ? bits[i] : 0u;
  const u32 c = __popc(word);
  const u32 incl = wave_inclusive_sum(c);
  if (!PASS) {
    if (lane == kWave - 1) wcnt[wv] = incl;
    return;
  }
  u64 pos = woff[wv] + incl - c;
  while (word) {
    const u32 b = __ffs(word) - 1;
    word &= word - 1;
    if (pos < cap) list[pos] = (u32)(i * 32 + b);
    else set_error(&st->err, kErrNewList);
    ++pos;
  }
}

__global__ void k_fix_dst(u32 *dst, u64 n, const u32 *hvals) {
  for (u64 k = (u64)blockIdx.x * blockDim.x + threadIdx.x; k < n; k += (u64)gridDim.x * blockDim.x)
    dst[k] = hvals[dst[k]];
}

// ---------------------------------------------------------------------------
__global__ void k_insert_start(u64 *hkeys, u64 hmask, u32 *hvals, u32 vn2, u32 s1, u32 s2,
                               u32 *sq1, u32 *sq2, u32 *err) {
  bool is_new;
  const u32 slot = vn2 ? s1 * vn2 + s2 : hash_insert(hkeys, hmask, ((u64)s1 << 32) | s2, is_new, err);
  hvals[slot] = 0;
  sq1[0] = s1;
  sq2[0] = s2;
}

__global__ void k_rehash(const u64 *okeys, const u32 *ovals, u64 ocap, u64 *nkeys, u32 *nvals,
                         u64 nmask, u32 *err) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < ocap; i += (u64)gridDim.x * blockDim.x) {
    const u64 k = okeys[i];
    if (k == kEmptyKey) continue;
    bool is_new;
    const u32 slot = hash_insert(nkeys, nmask, k, is_new, err);
    nvals[slot] = ovals[i];
  }
}

// The visited set moved from the hash table into the dense array vis
// (filled with kUnvisited): state id i < n is stored at its pair's entry.
__global__ void k_states_to_dense(const u32 *sq1, const u32 *sq2, u64 n, u32 *vis, u32 vn2) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x)
    vis[(u64)sq1[i] * vn2 + sq2[i]] = (u32)i;
}

// New pair i of the list gets id base + i: i < nnew, or i < min(*count,
// nnew) when count is given (nnew is then the list's capacity).
__global__ void k_assign(const u32 *slots, u32 nnew, const u64 *count, u32 base,
                         const u64 *hkeys, u32 *hvals, u32 vn2, u32 *sq1, u32 *sq2) {
  const u64 n = count ? min<u64>(*count, nnew) : nnew;
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x) {
    const u32 slot = slots[i];
    const u32 id = base + (u32)i;
    hvals[slot] = id;
    if (vn2) {
      sq1[id] = slot / vn2;
      sq2[id] = slot % vn2;
    } else {
      const u64 k = hkeys[slot];
      sq1[id] = (u32)(k >> 32);
      sq2[id] = (u32)k;
    }
  }
}

__global__ void k_newkeys(const u32 *newlist, u32 nnew, const u64 *hkeys, u32 vn2, int bq2,
                          u64 *keys, u32 *vals) {
  const u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nnew) return;
  const u32 slot = newlist[i];
  const u64 k = vn2 ? ((u64)(slot / vn2) << 32) | (slot % vn2) : hkeys[slot];
  keys[i] = ((k >> 32) << bq2) | (k & 0xffffffffull);
  vals[i] = slot;
}

// Wave per segment of merged runs: merge tile i (i < ntiles) or multi-block
// source big[i - ntiles]; lanes copy consecutive runs.
// Target id of a merged arc's record word x: the id itself when it carries
// kIdFlag (dense visited array only: its slots and ids are below 2^30, while
// hash-table slots use bit 30 themselves), else the id the visited set now
// holds at the slot.
__device__ __forceinline__ u32 target_id(const MergeArgs &a, u32 x, const u32 *hvals) {
  return (a.vn2 && (x & kIdFlag)) ? x & ~kIdFlag : hvals[x & ~kNewFlag];
}

__global__ __launch_bounds__(256) void k_compact(MergeArgs a, const u64 *aoff, u32 nbig, u64 M,
                                                 const u32 *hvals, u32 *osrc, u32 *odst,
                                                 u32 *oil, u32 *ool, float *ow) {
  const u32 lane = lane_id();
  const u64 wv = ((u64)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  if (wv >= a.ntiles + nbig) return;
  u64 tbase, obase;
  u32 cnt;
  if (wv < a.ntiles) {
    cnt = a.tile_runs[wv];
    if (cnt == 0) return;
    const uint4 td = a.tiles[wv];
    tbase = wv * a.window + td.z;
    obase = aoff[td.x];
  } else {
    const u32 u = a.big[wv - a.ntiles];
    tbase = a.tstart[u];
    cnt = (u32)(a.mend[u] - tbase);
    obase = aoff[u];
  }
  if (tbase + cnt > a.R || obase + cnt > M) {  // impossible: counts agree with aoff
    if (lane == 0) set_error(&a.st->err, kErrBounds);
    return;
  }
  for (u32 r = lane; r < cnt; r += kWave) {
    const uint4 rec = a.temp[tbase + r];
    const u64 k = obase + r;
    osrc[k] = a.lo + a.runsrc[tbase + r];
    odst[k] = target_id(a, rec.x, hvals);
    oil[k] = rec.y;
    ool[k] = rec.z;
    ow[k] = __uint_as_float(rec.w);
  }
}

// Result append, sources in consecutive groups of 64 per wave: their merged
// arcs are consecutive in the result (aoff is the exclusive scan of the
// per-source counts mend - tstart), so the wave walks the group's output
// range 64 entries at a time, each lane finding its entry's source by a
// binary search over the group's offsets held one per lane.
__global__ __launch_bounds__(256) void k_compact_sources(MergeArgs a, const u64 *aoff, u64 M,
                                                         const u32 *hvals, u32 *osrc, u32 *odst,
                                                         u32 *oil, u32 *ool, float *ow) {
  const u32 lane = lane_id();
  const u64 u0 = ((u64)blockIdx.x * blockDim.x + threadIdx.x) / kWave * kWave;
  if (u0 >= a.nsrc) return;
  const u64 u = u0 + lane;
  const bool in = u < a.nsrc;
  const u64 tb = in ? a.tstart[u] : 0, n = in ? a.mend[u] - tb : 0;
  const u64 ob = in ? aoff[u] : 0;
  const u64 incl = wave_inclusive_sum(n);
  const u64 rel = incl - n;  // this source's first entry, relative to the group's
  const u64 total = __shfl(incl, kWave - 1, kWave);
  const u64 ob0 = __shfl(ob, 0, kWave);
  // impossible: counts agree with aoff and the temp ranges lie in temp
  const bool bad = (in && (ob != ob0 + rel || tb + n > a.R + a.prodpos)) || ob0 + total > M;
  if (__ballot(bad)) {
    if (lane == 0) set_error(&a.st->err, kErrBounds);
    return;
  }
  for (u64 p0 = 0; p0 < total; p0 += kWave) {
    const u64 p = p0 + lane;
    // last lane whose source starts at or before p (sources without arcs
    // share their start with the next one; the last of them is taken)
    u32 s = 0;
#pragma unroll
    for (u32 step = kWave / 2; step; step >>= 1) {
      const u64 r = __shfl(rel, (int)(s + step), kWave);
      s = (s + step < (u32)kWave && r <= p) ? s + step : s;
    }
    const u64 rs = __shfl(rel, (int)s, kWave);
    const u64 ts = __shfl(tb, (int)s, kWave);
    if (p < total) {
      const uint4 rec = a.temp[ts + (p - rs)];
      const u64 k = ob0 + p;
      osrc[k] = a.lo + (u32)(u0 + s);
      odst[k] = target_id(a, rec.x, hvals);
      oil[k] = rec.y;
      ool[k] = rec.z;
      ow[k] = __uint_as_float(rec.w);
    }
  }
}

__global__ void k_finals(const u32 *sq1, const u32 *sq2, u64 n, const uint8_t *f1,
                         const uint8_t *f2, uint8_t *fin) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x)
    fin[i] = (f1[sq1[i]] != 0 && f2[sq2[i]] != 0) ? 1 : 0;
}

// Copies the level counters to host memory (pinned, coherent, device-
// visible), then, after a system-scope fence, the publication number: the
// host waits for that word instead of a stream synchronisation.  Threads
// t = 0 .. nt-1 of one workgroup call it together.
__device__ __forceinline__ void publish(const Status *st, Status *host, u32 seq, u32 t, u32 nt) {
  const u32 *src = reinterpret_cast<const u32 *>(st);
  u32 *dst = reinterpret_cast<u32 *>(host);
  constexpr u32 kSeqWord = offsetof(Status, seq) / 4;
  for (u32 i = t; i < sizeof(Status) / 4; i += nt)
    if (i != kSeqWord) dst[i] = src[i];
  __threadfence_system();
  if (nt > 1) __syncthreads();
  if (t == 0) __hip_atomic_store(&host->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// (level_clear_mask names the same fields, for publications that clear them)
__device__ __forceinline__ void clear_level(Status *st) {
  st->R = st->M = st->merged = st->RB = 0;
  st->nwide = st->nheavy = st->nbig = st->nnew = 0;
  st->max_small = 0;
  st->dense_records = st->dense_runs = st->sort_runs = 0;
  st->nprod = st->nprod_mfma = 0;
  st->prod_records = st->prod_entries = 0;
  st->nsort = 0;
  st->ngen = 0;
  st->ngrp = 0;
  st->unfit = 0;
  st->declined = 0;
}


// Level totals after the merge: merged arcs (end of the scan of merged arcs
// per source), new pairs (end of the scan of the new-pair lists), the
// product merge's joined pairs (sum of the per-source joined pairs less the
// level's records), and, over the merge tiles, the records and runs of the
// tiles the dense-table kernel merged and the runs of those the sort kernel
// merged.  One workgroup: it publishes the counters to host memory and then
// clears them for the next level.
__global__ __launch_bounds__(1024) void k_merged_total(const u64 *at, const u64 *nt, const u64 *pt,
                                                       Status *st, MergeArgs a, Status *host,
                                                       u32 seq) {
  __shared__ u64 s_v[3][1024 / kWave];
  if (a.R_dev && *a.R_dev != 0) {
    // enqueued ahead of a level that turned out to have records: publish the
    // level's counters as they are (the count's totals), change nothing
    __threadfence();
    publish(st, host, seq, threadIdx.x, blockDim.x);
    return;
  }
  u64 v[3] = {0, 0, 0};
  for (u64 t = threadIdx.x; t < a.ntiles; t += blockDim.x) {
    const uint4 td = a.tiles[t];
    const u32 runs = a.tile_runs[t];
    if (td.x < td.y && dense_tile(td, a.key_bits) && !(td.w & kRerouted)) {
      v[0] += td.w;
      v[1] += runs;
    } else {
      v[2] += runs;
    }
  }
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
#pragma unroll
  for (int f = 0; f < 3; ++f) {
    v[f] = wave_sum(v[f]);
    if (lane == 0) s_v[f][w] = v[f];
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    u64 t = 0;
    for (u32 i = 0; i < blockDim.x / kWave; ++i) t += s_v[threadIdx.x][i];
    u64 *dst = threadIdx.x == 0 ? &st->dense_records : threadIdx.x == 1 ? &st->dense_runs : &st->sort_runs;
    *dst = t;
  }
  if (threadIdx.x == 3) st->merged = *at;
  if (threadIdx.x == 4 && nt) st->nnew = (u32)min<u64>(*nt, 0xffffffffull);
  if (threadIdx.x == 5) st->prod_records = *pt - st->R;
  __syncthreads();
  __threadfence();
  publish(st, host, seq, threadIdx.x, blockDim.x);
  if (threadIdx.x == 0) clear_level(st);
}

// One-workgroup product level (level.hpp, launch_product_level).  Stages,
// each ended by stage_barrier (the workgroup reads back what its other
// threads wrote to global memory):
//   1. thread per source: the product selection (the count kernels' rule);
//      any source not in the strided four-source form declines the level;
//   2. entry offsets (a workgroup scan of the table sizes);
//   3. each wave merges quads of sources (the four-source kernel's code);
//   4. new pairs and joined pairs per source scanned and summed;
//   5. ids of the claimed targets, four lanes per source;
//   6. the other marked targets of the level's entries;
//   7. the level totals, their publication, the counters cleared.
constexpr int kTinyNT = 1024;
static_assert(kTinySources <= (u32)kTinyNT, "a thread per source");

// End of a stage: every thread's stores are done (the barrier's release),
// then each thread drops its CU's L1 lines (an agent-scope acquire), so its
// next loads see what the others wrote; one workgroup shares one L2, so no
// L2 write-back is needed.
__device__ __forceinline__ void stage_barrier() {
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

__global__ __launch_bounds__(kTinyNT) void k_product_level(LevelArgs la, MergeArgs ma, u64 *poff,
                                                           u64 *newoff, u32 base, u32 *sq1,
                                                           u32 *sq2, Status *host, u32 seq) {
  __shared__ u64 s_scr[kTinyNT / kWave];
  const u32 t = threadIdx.x;
  const u32 nsrc = la.nsrc;
  Status *st = ma.st;
  // 1. selection
  u32 pk = 0;
  bool ok = true;
  if (t < nsrc) {
    const u32 sid = la.lo + t;
    const u32 q1 = la.sq1[sid], q2 = la.sq2[sid];
    const Ranges r{la.c1.row[q1], la.c1.row[q1 + 1], la.c2.row[q2], la.c2.row[q2 + 1]};
    const u32 mn = min(r.e1 - r.b1, r.e2 - r.b2);
    bool mf = false, strided = false;
    if (mn >= kProdMinSymbols && mn <= (u32)kWave) pk = select_product(la, t, q1, q2, r, mf, &strided);
    ok = pk != 0 && strided;
    la.pk[t] = ok ? pk : 0u;
    la.tstart[t] = 0;
    la.mend[t] = 0;
    la.newc[t] = 0;
    la.cnt[t] = 0;  // ma.pcnt
  }
  if (__syncthreads_or(!ok)) {
    if (t == 0) st->declined = 1u;
    __threadfence();
    __syncthreads();
    publish(st, host, seq, t, kTinyNT);
    return;
  }
  // 2. entry offsets
  u64 entries;
  const u64 off = block_exclusive_sum<kTinyNT, u64>(t < nsrc ? pk : 0u, s_scr, &entries);
  if (t < nsrc) poff[t] = off;  // ma.poff
  if (t == 0) poff[nsrc] = entries;
  stage_barrier();
  // 3. the product merge, a quad of sources per wave at a time
  const u32 nq = (nsrc + 3) / 4;
  for (u32 wv = t / kWave; wv < nq; wv += kTinyNT / kWave) quad_merge(ma, wv);
  stage_barrier();
  // 4. new pairs (id offsets) and joined pairs
  u32 nc = 0;
  u64 pairs = 0;
  if (t < nsrc) {
    nc = __hip_atomic_load(&ma.newc[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    pairs = __hip_atomic_load(&ma.pcnt[t], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  u64 nnew;
  const u64 noff = block_exclusive_sum<kTinyNT, u64>(nc, s_scr, &nnew);
  __syncthreads();  // s_scr reused
  const u64 npairs = block_sum<kTinyNT, u64>(pairs, s_scr);
  if (t < nsrc) newoff[t] = noff;
  if (t == 0) newoff[nsrc] = nnew;
  stage_barrier();
  // 5. ids of the claimed targets (whole waves: the lanes past the level
  // have no new pairs)
  for (u32 t0 = 0; t0 < 4 * nsrc; t0 += kTinyNT) assign_direct_lanes(ma, newoff, base, sq1, sq2, t0 + t);
  stage_barrier();
  // 6. totals, publication, counters cleared (the targets another source
  // claimed keep their slot marks: the composition's last pass replaces them)
  if (t == 0) {
    st->merged = entries;
    st->nnew = (u32)min<u64>(nnew, 0xffffffffull);
    st->prod_records = npairs;
    st->prod_entries = entries;
    st->nprod = nsrc;
    st->nprod_mfma = nsrc;
  }
  stage_barrier();
  publish(st, host, seq, t, kTinyNT);
  __syncthreads();
  if (t == 0) clear_level(st);
}

__global__ void k_reset_level(Status *st) {
  if (threadIdx.x == 0) clear_level(st);
}

}  // namespace

static u64 merge_grid(const MergeArgs &a) {
  const u64 g = ceil_div(a.R, a.window);
  if (g >= (1ull << 31)) throw Error(FSTC_ERR_CAPACITY, "level too large for one launch");
  return g;
}

void launch_tile_sources(const MergeArgs &a, hipStream_t s) {
  if (a.R == 0) return;
  const u64 g = merge_grid(a);
  hipLaunchKernelGGL(k_tile_sources, dim3(grid1(g)), dim3(256), 0, s, a.roff, a.nsrc, a.R,
                     a.window, g, a.tiles);
}

void launch_merge_dense(const MergeArgs &a, hipStream_t s) {
  if (a.R == 0 || a.key_bits > kDenseKeyBits) return;
  hipLaunchKernelGGL(k_merge_dense, dim3((unsigned)merge_grid(a)), dim3(NT), 0, s, a);
}

void launch_fuse_merge(const MergeArgs &a, bool narrow, hipStream_t s) {
  if (a.R == 0) return;
  if (narrow)
    hipLaunchKernelGGL(k_fuse_merge<true>, dim3((unsigned)merge_grid(a)), dim3(NT), 0, s, a);
  else
    hipLaunchKernelGGL(k_fuse_merge<false>, dim3((unsigned)merge_grid(a)), dim3(NT), 0, s, a);
}

void launch_merge_sort(const MergeArgs &a, bool wide_keys, hipStream_t s) {
  if (a.R == 0) return;
  const u64 g = merge_grid(a);
  if (a.key_bits <= kDenseKeyBits) {
    // after k_merge_dense: only the tiles it listed, walked by a fixed grid
    const unsigned gl = (unsigned)std::min<u64>(g, kListedGrid);
    if (wide_keys)
      hipLaunchKernelGGL((k_merge_listed<u64>), dim3(gl), dim3(NT), 0, s, a);
    else
      hipLaunchKernelGGL((k_merge_listed<u32>), dim3(gl), dim3(NT), 0, s, a);
  } else if (wide_keys) {
    hipLaunchKernelGGL((k_merge_tiles<u64>), dim3((unsigned)g), dim3(NT), 0, s, a);
  } else {
    hipLaunchKernelGGL((k_merge_tiles<u32>), dim3((unsigned)g), dim3(NT), 0, s, a);
  }
}

void launch_big_counts(const u64 *roff, const u32 *big, u32 nbig, u64 *bigcnt, hipStream_t s) {
  hipLaunchKernelGGL(k_big_counts, dim3((unsigned)ceil_div(nbig, 256)), dim3(256), 0, s, roff,
                     big, nbig, bigcnt);
}

void merge_big(const MergeArgs &a, bool wide_keys, u32 nbig, const u64 *bigoff, u64 RB,
               Arena &T, hipStream_t s) {
  if (nbig == 0 || RB == 0) return;
  Tmp skey(&T), sval(&T), kalt(&T), valt(&T), flags(&T), ridx(&T), tmp(&T);
  skey.ensure(RB * 8); sval.ensure(RB * 4); kalt.ensure(RB * 8); valt.ensure(RB * 4);
  flags.ensure(RB * 4); ridx.ensure((RB + 1) * 4);
  tmp.ensure(std::max(radix_temp_bytes(RB), scan_temp_bytes(RB)));
  const unsigned g = (unsigned)ceil_div(RB, 256);
  if (wide_keys)
    hipLaunchKernelGGL((k_big_gather<u64>), dim3(g), dim3(256), 0, s, a.big, bigoff, nbig, RB,
                       a.roff, (const u64 *)a.rec_key, a.rec_w, a.key_bits, skey.as<u64>(),
                       sval.as<u32>());
  else
    hipLaunchKernelGGL((k_big_gather<u32>), dim3(g), dim3(256), 0, s, a.big, bigoff, nbig, RB,
                       a.roff, (const u32 *)a.rec_key, a.rec_w, a.key_bits, skey.as<u64>(),
                       sval.as<u32>());
  const int hi = a.key_bits + (int)bits_for(nbig - 1);
  radix_sort_pairs(skey.as<u64>(), sval.as<u32>(), kalt.as<u64>(), valt.as<u32>(), RB, 0, hi,
                   tmp.p, s);
  hipLaunchKernelGGL(k_run_heads, dim3(g), dim3(256), 0, s, skey.as<u64>(), RB, flags.as<u32>());
  exclusive_scan(flags.as<u32>(), ridx.as<u32>(), RB, tmp.p, s);
  hipLaunchKernelGGL(k_big_reduce, dim3(g), dim3(256), 0, s, a, bigoff, RB, skey.as<u64>(),
                     sval.as<u32>(), flags.as<u32>(), ridx.as<u32>());
}

void launch_unreduced(const MergeArgs &a, bool wide_keys, u32 *newbits, u32 *osrc, u32 *odst,
                      u32 *oil, u32 *ool, float *ow, hipStream_t s) {
  if (a.R == 0) return;
  const u64 nw = ceil_div(a.R, (u64)kWave * kUnredB);
  const unsigned g = (unsigned)ceil_div(nw, 256 / kWave);
  if (ceil_div(nw, 256 / kWave) >= (1ull << 31)) throw Error(FSTC_ERR_CAPACITY, "level too large for one launch");
  if (wide_keys)
    hipLaunchKernelGGL(k_unreduced<u64>, dim3(g), dim3(256), 0, s, a, newbits, osrc, odst, oil, ool, ow);
  else
    hipLaunchKernelGGL(k_unreduced<u32>, dim3(g), dim3(256), 0, s, a, newbits, osrc, odst, oil, ool, ow);
}

u64 bitlist_waves(u64 nwords) { return ceil_div(std::max<u64>(nwords, 1), kWave); }

void launch_bitlist(const u32 *bits, u64 nwords, u32 *list, u64 cap, u32 *wcnt, u64 *woff,
                    void *scan_tmp, Status *st, hipStream_t s) {
  const u64 nw = bitlist_waves(nwords);
  const unsigned g = (unsigned)ceil_div(nw, 256 / kWave);
  hipLaunchKernelGGL(k_bitlist<0>, dim3(g), dim3(256), 0, s, bits, nwords, wcnt, (const u64 *)nullptr,
                     list, cap, st);
  exclusive_scan(wcnt, woff, nw, scan_tmp, s);
  hipLaunchKernelGGL(k_bitlist<1>, dim3(g), dim3(256), 0, s, bits, nwords, wcnt, (const u64 *)woff,
                     list, cap, st);
  hipLaunchKernelGGL(k_new_total, dim3(1), dim3(1), 0, s, (const u64 *)(woff + nw), st);
}

void launch_prod_sources(const MergeArgs &a, bool narrow, hipStream_t s, bool lean) {
  if (!a.nsrc) return;
  if (a.quad) {
    const unsigned gq = (unsigned)ceil_div(ceil_div(a.nsrc, 4), 256 / kWave);
    if (narrow) hipLaunchKernelGGL(k_prod_quad<true>, dim3(gq), dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_prod_quad<false>, dim3(gq), dim3(256), 0, s, a);
  }
  // the listed sources: at most one wave per level source, and at most as
  // many waves as the chip holds at once (they loop over the list)
  const u64 waves = std::min<u64>(a.nsrc, (u64)compute_units() * (lean ? 1 : 32));
  const unsigned g = (unsigned)ceil_div(waves, kProdWaves);
  if (narrow)
    hipLaunchKernelGGL(k_prod_sources<true>, dim3(g), dim3(kProdNT), 0, s, a);
  else
    hipLaunchKernelGGL(k_prod_sources<false>, dim3(g), dim3(kProdNT), 0, s, a);
}

void launch_newlist_sources(const MergeArgs &a, const u64 *newoff, hipStream_t s) {
  if (!a.nsrc) return;
  hipLaunchKernelGGL(k_newlist_sources, dim3((unsigned)ceil_div((u64)a.nsrc * 16, 256)), dim3(256),
                     0, s, a, newoff);
}

void launch_assign_direct(const MergeArgs &a, const u64 *newoff, u32 base, u32 *sq1, u32 *sq2,
                          hipStream_t s) {
  if (!a.nsrc) return;
  hipLaunchKernelGGL(k_assign_direct, dim3((unsigned)ceil_div((u64)a.nsrc * 4, 256)), dim3(256), 0,
                     s, a, newoff, base, sq1, sq2);
}

void launch_small_levels(const SmallArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_small_levels, dim3(1), dim3(kSmallNT), 0, s, a);
}

void launch_unreduced_product(const MergeArgs &a, const u64 *off, hipStream_t s) {
  if (!a.nsrc) return;
  hipLaunchKernelGGL(k_unreduced_product, dim3((unsigned)ceil_div((u64)a.nsrc * kWave, 256)),
                     dim3(256), 0, s, a, off);
}

void launch_fix_marked(const MergeArgs &a, u64 n, hipStream_t s) {
  if (!n) return;
  hipLaunchKernelGGL(k_fix_marked, dim3(grid1(ceil_div(n, 4) + 1)), dim3(256), 0, s, a, n);
}

void launch_close_holes(const MergeArgs &a, const u64 *aoff, u64 n, void *tmp, hipStream_t s) {
  if (!n || !a.nsrc) return;
  hipLaunchKernelGGL(k_copy_rows, dim3(grid1(n)), dim3(256), 0, s, a, n, static_cast<u32 *>(tmp));
  hipLaunchKernelGGL(k_close_holes, dim3((unsigned)ceil_div((u64)a.nsrc * 16, 256)), dim3(256), 0,
                     s, a, aoff, n, static_cast<const u32 *>(tmp));
}

void launch_compact_sources(const MergeArgs &a, const u64 *aoff, u64 M, const u32 *hvals,
                            u32 *osrc, u32 *odst, u32 *oil, u32 *ool, float *ow, hipStream_t s) {
  if (!a.nsrc || !M) return;
  hipLaunchKernelGGL(k_compact_sources, dim3((unsigned)ceil_div((u64)a.nsrc, 256)), dim3(256),
                     0, s, a, aoff, M, hvals, osrc, odst, oil, ool, ow);
}

void launch_fix_dst(u32 *dst, u64 n, const u32 *hvals, hipStream_t s) {
  if (!n) return;
  hipLaunchKernelGGL(k_fix_dst, dim3(grid1(n)), dim3(256), 0, s, dst, n, hvals);
}

void launch_insert_start(u64 *hkeys, u64 hmask, u32 *hvals, u32 vn2, u32 s1, u32 s2, u32 *sq1,
                         u32 *sq2, u32 *err, hipStream_t s) {
  hipLaunchKernelGGL(k_insert_start, dim3(1), dim3(1), 0, s, hkeys, hmask, hvals, vn2, s1, s2, sq1,
                     sq2, err);
}

void launch_rehash(const u64 *okeys, const u32 *ovals, u64 ocap, u64 *nkeys, u32 *nvals,
                   u64 nmask, u32 *err, hipStream_t s) {
  hipLaunchKernelGGL(k_rehash, dim3(grid1(ocap)), dim3(256), 0, s, okeys, ovals, ocap, nkeys,
                     nvals, nmask, err);
}

void launch_states_to_dense(const u32 *sq1, const u32 *sq2, u64 n, u32 *vis, u32 vn2,
                            hipStream_t s) {
  if (!n) return;
  hipLaunchKernelGGL(k_states_to_dense, dim3(grid1(n)), dim3(256), 0, s, sq1, sq2, n, vis, vn2);
}

void launch_assign(const u32 *slots, u32 nnew, u32 base, const u64 *hkeys, u32 *hvals, u32 vn2,
                   u32 *sq1, u32 *sq2, hipStream_t s) {
  if (!nnew) return;
  hipLaunchKernelGGL(k_assign, dim3((unsigned)ceil_div(nnew, 256)), dim3(256), 0, s, slots, nnew,
                     (const u64 *)nullptr, base, hkeys, hvals, vn2, sq1, sq2);
}

void launch_assign_counted(const u32 *slots, const u64 *count, u32 cap, u32 base,
                           const u64 *hkeys, u32 *hvals, u32 vn2, u32 *sq1, u32 *sq2,
                           hipStream_t s) {
  if (!count || !cap) return;
  const unsigned g = (unsigned)std::min<u64>(ceil_div(cap, 256), 2048);
  hipLaunchKernelGGL(k_assign, dim3(g), dim3(256), 0, s, slots, cap, count, base, hkeys, hvals,
                     vn2, sq1, sq2);
}

void launch_newkeys(const u32 *newlist, u32 nnew, const u64 *hkeys, u32 vn2, int bq2, u64 *keys,
                    u32 *vals, hipStream_t s) {
  if (!nnew) return;
  hipLaunchKernelGGL(k_newkeys, dim3((unsigned)ceil_div(nnew, 256)), dim3(256), 0, s, newlist,
                     nnew, hkeys, vn2, bq2, keys, vals);
}

void launch_compact(const MergeArgs &a, const u64 *aoff, u32 nbig, u64 M, const u32 *hvals,
                    u32 *osrc, u32 *odst, u32 *oil, u32 *ool, float *ow, hipStream_t s) {
  const u64 nw = a.ntiles + nbig;
  if (!nw || !M) return;
  hipLaunchKernelGGL(k_compact, dim3((unsigned)ceil_div(nw, 256 / kWave)), dim3(256), 0, s, a, aoff,
                     nbig, M, hvals, osrc, odst, oil, ool, ow);
}

u64 newlist_waves(const MergeArgs &a, u64 RB) {
  return a.ntiles + ceil_div(RB, kWave) + ceil_div(a.prodpos, (u64)kWave);
}

const u64 *launch_newlist(const MergeArgs &a, const u64 *bigoff, u32 nbig, u64 RB, u32 *wcnt,
                          u64 *woff, void *scan_state, hipStream_t s) {
  const u64 nbigw = ceil_div(RB, kWave);
  const u64 nw = newlist_waves(a, RB);
  if (nw == 0) return nullptr;  // no new pairs
  const unsigned g = (unsigned)ceil_div(nw, 256 / kWave);
  hipLaunchKernelGGL(k_newlist<0>, dim3(g), dim3(256), 0, s, a, bigoff, nbig, RB, nbigw, wcnt,
                     (const u64 *)nullptr);
  const ScanJob job{wcnt, false, woff};
  exclusive_scan_lb(&job, 1, nw, scan_state, &a.st->scan_ctr, &a.st->err, s);
  hipLaunchKernelGGL(k_newlist<1>, dim3(g), dim3(256), 0, s, a, bigoff, nbig, RB, nbigw, wcnt,
                     (const u64 *)woff);
  return woff + nw;
}

void launch_emit_tiles(const MergeArgs &a, hipStream_t s) {
  if (a.R == 0) return;
  // waves per tile: enough waves in all to fill the chip even when a level
  // has few tiles (each tile holds at most kMergeCap runs)
  const u64 target = (u64)compute_units() * 128;
  const u32 wpt = (u32)std::min<u64>(kMergeCap / kWave, std::max<u64>(1, ceil_div(target, a.ntiles)));
  hipLaunchKernelGGL(k_emit_tiles, dim3((unsigned)ceil_div(a.ntiles * wpt, 256 / kWave)), dim3(256),
                     0, s, a, wpt);
}

void launch_finals(const u32 *sq1, const u32 *sq2, u64 n, const uint8_t *f1, const uint8_t *f2,
                   uint8_t *fin, hipStream_t s) {
  if (!n) return;
  hipLaunchKernelGGL(k_finals, dim3(grid1(n)), dim3(256), 0, s, sq1, sq2, n, f1, f2, fin);
}


void launch_merged_total(const u64 *a_total, const u64 *new_total, const u64 *pair_total,
                         const MergeArgs &a, Status *host, u32 seq, hipStream_t s) {
  // one wave unless there are many merge tiles to sum
  const unsigned nt = a.ntiles > 4096 ? 1024 : kWave;
  hipLaunchKernelGGL(k_merged_total, dim3(1), dim3(nt), 0, s, a_total, new_total, pair_total,
                     a.st, a, host, seq);
}

void launch_reset_level(Status *st, hipStream_t s) {
  hipLaunchKernelGGL(k_reset_level, dim3(1), dim3(1), 0, s, st);
}

void launch_product_level(const LevelArgs &la, const MergeArgs &ma, u64 *poff, u64 *newoff,
                          u32 base, u32 *sq1, u32 *sq2, Status *host, u32 seq, hipStream_t s) {
  if (la.nsrc == 0 || la.nsrc > kTinySources || !ma.vn2 || !ma.out_dst || ma.poff != poff)
    throw Error(FSTC_ERR_INTERNAL, "one-workgroup product level out of its range");
  hipLaunchKernelGGL(k_product_level, dim3(1), dim3(kTinyNT), 0, s, la, ma, poff, newoff, base, sq1,
                     sq2, host, seq);
}

u64 level_clear_mask() {
  static_assert(sizeof(Status) <= 64 * 4, "one mask bit per word");
  u64 m = 0;
  auto add = [&](size_t off, size_t bytes) {
    for (size_t w = off / 4; w < (off + bytes) / 4; ++w) m |= 1ull << w;
  };
  // the fields clear_level zeroes
  add(offsetof(Status, R), 8);
  add(offsetof(Status, M), 8);
  add(offsetof(Status, merged), 8);
  add(offsetof(Status, RB), 8);
  add(offsetof(Status, nwide), 4);
  add(offsetof(Status, nheavy), 4);
  add(offsetof(Status, nbig), 4);
  add(offsetof(Status, nnew), 4);
  add(offsetof(Status, max_small), 4);
  add(offsetof(Status, dense_records), 8);
  add(offsetof(Status, dense_runs), 8);
  add(offsetof(Status, sort_runs), 8);
  add(offsetof(Status, nprod), 4);
  add(offsetof(Status, nprod_mfma), 4);
  add(offsetof(Status, prod_records), 8);
  add(offsetof(Status, prod_entries), 8);
  add(offsetof(Status, nsort), 4);
  add(offsetof(Status, ngen), 4);
  add(offsetof(Status, ngrp), 4);
  add(offsetof(Status, unfit), 4);
  add(offsetof(Status, declined), 4);
  return m;
}

}  // namespace fstc
