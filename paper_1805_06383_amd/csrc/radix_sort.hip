// Device-wide stable LSD radix sort of (64-bit key, 32-bit value) pairs.
//
// The paper sorts packed 64-bit keys with a library sort-by-key
// (section 3.4, "Reduction").  Here the sort is written for gfx950: 8-bit
// digits, one histogram pass and one scatter pass per digit, tiles of 4096
// elements per 256-thread workgroup, and stable in-tile ranking by wave64
// ballots (radix_rank.hpp).  Only the key bits that can differ are sorted
// (the caller passes the bit range).
#include "common.hpp"
#include "radix_rank.hpp"

namespace fstc {
namespace {

constexpr int kNT = 256;
constexpr int kIT = 16;
constexpr int kTile = kNT * kIT;

// Histogram of tile `blk` of nb: hist[d nb + blk] = elements of the tile
// with digit d.
__device__ __forceinline__ void digit_hist_tile(const u64 *keys, u64 n, int shift, u32 mask,
                                                u32 *hist, u32 nb, u32 blk) {
  __shared__ u32 h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const u64 base = (u64)blk * kTile;
  // every load issued before the first is used (indices clamped into the
  // array; n >= 2): a branch around each load would wait for every one
  u64 k[kIT];
#pragma unroll
  for (int j = 0; j < kIT; ++j) k[j] = keys[min<u64>(base + (u64)j * kNT + threadIdx.x, n - 1)];
#pragma unroll
  for (int j = 0; j < kIT; ++j)
    if (base + (u64)j * kNT + threadIdx.x < n) atomicAdd(&h[(u32)(k[j] >> shift) & mask], 1u);
  __syncthreads();
  hist[(u64)threadIdx.x * nb + blk] = h[threadIdx.x];
}

__global__ __launch_bounds__(kNT) void k_digit_hist(const u64 *keys, u64 n, int shift, u32 mask,
                                                    u32 *hist, u32 nb) {
  digit_hist_tile(keys, n, shift, mask, hist, nb, blockIdx.x);
}

// Scatter of tile `blk` of nb to the offsets of the scanned histogram.
__device__ __forceinline__ void digit_scatter_tile(const u64 *keys, const u32 *vals,
                                                   u64 *keys_out, u32 *vals_out, u64 n, int shift,
                                                   int bits, const u32 *offs, u32 nb, u32 blk) {
  __shared__ u32 s_cnt[(kNT / kWave) * 256];
  __shared__ u32 s_base[256];
  __shared__ u32 s_tmp[kNT / kWave];
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const u32 mask = (1u << bits) - 1u;
  const u64 base = (u64)blk * kTile + (u64)w * (kWave * kIT);
  u64 key[kIT];
  u32 val[kIT], dig[kIT], rid[kIT];
  u32 valid = 0;
#pragma unroll
  for (int j = 0; j < kIT; ++j) {
    const u64 e = base + (u64)j * kWave + lane;
    const bool v = e < n;
    valid |= (v ? 1u : 0u) << j;
    key[j] = v ? keys[e] : 0;
    val[j] = v ? vals[e] : 0;
    dig[j] = (u32)(key[j] >> shift) & mask;
  }
  block_rank_digits<kNT, kIT>(dig, valid, bits, rid, s_cnt, s_base, s_tmp);
#pragma unroll
  for (int j = 0; j < kIT; ++j) {
    if (!((valid >> j) & 1u)) continue;
    const u64 pos = (u64)offs[(u64)dig[j] * nb + blk] + rid[j];
    keys_out[pos] = key[j];
    vals_out[pos] = val[j];
  }
}

__global__ __launch_bounds__(kNT) void k_digit_scatter(const u64 *keys, const u32 *vals,
                                                       u64 *keys_out, u32 *vals_out, u64 n,
                                                       int shift, int bits, const u32 *offs,
                                                       u32 nb) {
  digit_scatter_tile(keys, vals, keys_out, vals_out, n, shift, bits, offs, nb, blockIdx.x);
}

// Exclusive scan of a digit histogram of at most kScan1Max entries by one
// workgroup (one launch instead of a multi-level scan).  Wave w owns the
// entries [w S, w S + S), S a multiple of 64: it sums them in coalesced
// 64-entry chunks, the waves' totals are combined in LDS, and a second pass
// over the chunks writes each entry's offset from a DPP prefix sum plus the
// running carry.
constexpr int kScan1NT = 1024;
constexpr u64 kScan1Max = 1u << 16;

__device__ __forceinline__ void hist_scan_block(const u32 *hist, u32 *offs, u32 nh) {
  constexpr u32 kWaves = kScan1NT / kWave;
  __shared__ u32 s_tot[kWaves];
  const u32 lane = lane_id(), w = threadIdx.x / kWave;
  const u32 seg = (nh + kWaves * kWave - 1) / (kWaves * kWave) * kWave;
  const u32 b = min(nh, w * seg), e = min(nh, b + seg);
  // kBatch chunks' loads are issued before any of them is used
  constexpr u32 kBatch = 8;
  u32 sum = 0;
  for (u32 c = b; c < e; c += kBatch * kWave) {
    u32 v[kBatch];
#pragma unroll
    for (u32 q = 0; q < kBatch; ++q) {
      const u32 i = c + q * kWave + lane;
      v[q] = i < e ? hist[i] : 0u;
    }
#pragma unroll
    for (u32 q = 0; q < kBatch; ++q) sum += v[q];
  }
  sum = wave_total(sum);
  if (lane == 0) s_tot[w] = sum;
  __syncthreads();
  u32 carry = 0;
  for (u32 k = 0; k < w; ++k) carry += s_tot[k];
  for (u32 c = b; c < e; c += kBatch * kWave) {  // wave-uniform bounds: every lane runs every chunk
    u32 v[kBatch];
#pragma unroll
    for (u32 q = 0; q < kBatch; ++q) {
      const u32 i = c + q * kWave + lane;
      v[q] = i < e ? hist[i] : 0u;
    }
#pragma unroll
    for (u32 q = 0; q < kBatch; ++q) {
      const u32 i = c + q * kWave + lane;
      const u32 incl = wave_inclusive_total(v[q]);
      if (i < e) offs[i] = carry + incl - v[q];
      carry += (u32)__builtin_amdgcn_readlane((int)incl, kWave - 1);
    }
  }
}

__global__ __launch_bounds__(kScan1NT) void k_hist_scan1(const u32 *hist, u32 *offs, u32 nh) {
  hist_scan_block(hist, offs, nh);
}

// One pass of a batch of sorts (radix_sort_pairs_batch): the jobs still
// sorting, workgroups [0, split) for the first and the rest for the second.
struct PassJob {
  const u64 *ki;
  const u32 *vi;
  u64 *ko;
  u32 *vo;
  u64 n;
  int shift, bits;
  u32 *hist, *offs;
  u32 nb;
  const u32 *unsorted;  // see SortJob
  u32 epoch;
  u32 copy;  // an ordered job's last pass of an odd number: ki copied to ko
};

// The job is already in order (see SortJob).
__device__ __forceinline__ bool pass_in_order(const PassJob &J) {
  return J.unsorted && *J.unsorted != J.epoch;
}
struct PassPair {
  PassJob j[2];
  u32 split;
};

__device__ __forceinline__ const PassJob &pass_job(const PassPair &p, u32 &blk) {
  if (blockIdx.x < p.split) {
    blk = blockIdx.x;
    return p.j[0];
  }
  blk = blockIdx.x - p.split;
  return p.j[1];
}

__global__ __launch_bounds__(kNT) void k_digit_hist2(PassPair p) {
  u32 blk;
  const PassJob &J = pass_job(p, blk);
  if (pass_in_order(J)) return;  // uniform
  digit_hist_tile(J.ki, J.n, J.shift, (1u << J.bits) - 1u, J.hist, J.nb, blk);
}

// workgroup i scans job i's histogram
__global__ __launch_bounds__(kScan1NT) void k_hist_scan2(PassPair p) {
  const PassJob &J = p.j[blockIdx.x];
  if (pass_in_order(J)) return;  // uniform
  hist_scan_block(J.hist, J.offs, 256u * J.nb);
}

// An ordered job's data stays where it is: in the last of an odd number of
// passes it is copied to the output (the sort's result is then copied back
// from there), otherwise nothing is done.
__global__ __launch_bounds__(kNT) void k_digit_scatter2(PassPair p) {
  u32 blk;
  const PassJob &J = pass_job(p, blk);
  if (pass_in_order(J)) {  // uniform
    if (!J.copy) return;
    const u64 base = (u64)blk * kTile;
#pragma unroll
    for (int j = 0; j < kIT; ++j) {
      const u64 e = base + (u64)j * kNT + threadIdx.x;
      if (e < J.n) {
        J.ko[e] = J.ki[e];
        J.vo[e] = J.vi[e];
      }
    }
    return;
  }
  digit_scatter_tile(J.ki, J.vi, J.ko, J.vo, J.n, J.shift, J.bits, J.offs, J.nb, blk);
}

}  // namespace

size_t radix_temp_bytes(u64 n) {
  const u64 nb = std::max<u64>(1, ceil_div(n, kTile));
  const u64 nh = 256 * nb;
  return (nh + (nh + 1)) * sizeof(u32) + scan_temp_bytes(nh) + 512;
}

void radix_sort_pairs(u64 *keys, u32 *vals, u64 *keys_alt, u32 *vals_alt, u64 n, int lo, int hi,
                      void *temp, hipStream_t s) {
  if (n <= 1 || hi <= lo) return;
  const u32 nb = (u32)ceil_div(n, kTile);
  const u64 nh = 256ull * nb;
  u32 *hist = (u32 *)temp;
  u32 *offs = hist + nh;
  void *scan_tmp = (void *)(((uintptr_t)(offs + nh + 1) + 255) & ~(uintptr_t)255);
  u64 *ki = keys, *ko = keys_alt;
  u32 *vi = vals, *vo = vals_alt;
  for (int shift = lo; shift < hi; shift += 8) {
    const int bits = std::min(8, hi - shift);
    const u32 mask = (1u << bits) - 1u;
    hipLaunchKernelGGL(k_digit_hist, dim3(nb), dim3(kNT), 0, s, ki, n, shift, mask, hist, nb);
    if (nh <= kScan1Max)
      hipLaunchKernelGGL(k_hist_scan1, dim3(1), dim3(kScan1NT), 0, s, hist, offs, (u32)nh);
    else
      exclusive_scan(hist, offs, nh, scan_tmp, s);
    hipLaunchKernelGGL(k_digit_scatter, dim3(nb), dim3(kNT), 0, s, ki, vi, ko, vo, n, shift,
                       bits, offs, nb);
    std::swap(ki, ko);
    std::swap(vi, vo);
  }
  if (ki != keys) {
    FSTC_HIP(hipMemcpyAsync(keys, ki, n * sizeof(u64), hipMemcpyDeviceToDevice, s));
    FSTC_HIP(hipMemcpyAsync(vals, vi, n * sizeof(u32), hipMemcpyDeviceToDevice, s));
  }
}

void radix_sort_pairs_batch(const SortJob *jobs, int nj, hipStream_t s) {
  if (nj < 1 || nj > 2) throw Error(FSTC_ERR_INTERNAL, "radix_sort_pairs_batch takes one or two jobs");
  u64 *ki[2], *ko[2];
  u32 *vi[2], *vo[2];
  int shift[2];
  // one workgroup scans a job's histogram: larger sorts run one by one
  for (int i = 0; i < nj; ++i) {
    if (256ull * ceil_div(jobs[i].n, kTile) > kScan1Max) {
      for (int k = 0; k < nj; ++k)
        radix_sort_pairs(jobs[k].keys, jobs[k].vals, jobs[k].keys_alt, jobs[k].vals_alt,
                         jobs[k].n, jobs[k].lo, jobs[k].hi, jobs[k].temp, s);
      return;
    }
  }
  for (int i = 0; i < nj; ++i) {
    ki[i] = jobs[i].keys; ko[i] = jobs[i].keys_alt;
    vi[i] = jobs[i].vals; vo[i] = jobs[i].vals_alt;
    shift[i] = jobs[i].lo;
  }
  auto active = [&](int i) { return jobs[i].n > 1 && shift[i] < jobs[i].hi; };
  while (true) {
    PassPair p{};
    int na = 0, who[2];
    u32 grid = 0;
    for (int i = 0; i < nj; ++i) {
      if (!active(i)) continue;
      PassJob &J = p.j[na];
      J.ki = ki[i]; J.vi = vi[i]; J.ko = ko[i]; J.vo = vo[i];
      J.n = jobs[i].n;
      J.shift = shift[i];
      J.bits = std::min(8, jobs[i].hi - shift[i]);
      J.nb = (u32)ceil_div(J.n, kTile);
      J.hist = (u32 *)jobs[i].temp;
      J.offs = J.hist + 256ull * J.nb;
      J.unsorted = jobs[i].unsorted;
      J.epoch = jobs[i].epoch;
      const int passes = (jobs[i].hi - jobs[i].lo + 7) / 8;
      J.copy = (passes & 1) && shift[i] + 8 >= jobs[i].hi ? 1u : 0u;
      if (na == 0) p.split = J.nb;
      grid += J.nb;
      who[na++] = i;
    }
    if (na == 0) break;
    hipLaunchKernelGGL(k_digit_hist2, dim3(grid), dim3(kNT), 0, s, p);
    hipLaunchKernelGGL(k_hist_scan2, dim3(na), dim3(kScan1NT), 0, s, p);
    hipLaunchKernelGGL(k_digit_scatter2, dim3(grid), dim3(kNT), 0, s, p);
    for (int a = 0; a < na; ++a) {
      const int i = who[a];
      std::swap(ki[i], ko[i]);
      std::swap(vi[i], vo[i]);
      shift[i] += 8;
    }
  }
  for (int i = 0; i < nj; ++i) {
    if (ki[i] == jobs[i].keys) continue;
    FSTC_HIP(hipMemcpyAsync(jobs[i].keys, ki[i], jobs[i].n * sizeof(u64), hipMemcpyDeviceToDevice, s));
    FSTC_HIP(hipMemcpyAsync(jobs[i].vals, vi[i], jobs[i].n * sizeof(u32), hipMemcpyDeviceToDevice, s));
  }
}

}  // namespace fstc
