// Device-wide exclusive prefix sums and fills.
//
// The per-level offsets of the frontier expansion (records per source,
// matches per source, merged arcs per source) are exclusive prefix sums, as in
// the two-stage expansion the paper adopts from Merrill et al. (section 3.4,
// "Updating frontier and visited set").  Reduce-then-scan: one pass reduces
// tiles of 4096 elements, the tile sums are scanned recursively, and a second
// pass scans each tile with its offset.  A single tile is one launch.
#include <atomic>

#include "common.hpp"

namespace fstc {
namespace {

constexpr int kScanNT = 256;
constexpr int kScanIT = 16;
constexpr int kScanTile = kScanNT * kScanIT;

template <class T>
__global__ void k_fill(T *p, T v, u64 n) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x)
    p[i] = v;
}

template <class TI, class TO>
__global__ __launch_bounds__(kScanNT) void k_tile_reduce(const TI *in, u64 n, TO *tile_sums) {
  __shared__ TO scratch[kScanNT / kWave];
  const u64 base = (u64)blockIdx.x * kScanTile;
  TO s = 0;
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) {
    u64 i = base + (u64)j * kScanNT + threadIdx.x;
    if (i < n) s += (TO)in[i];
  }
  s = block_sum<kScanNT, TO>(s, scratch);
  if (threadIdx.x == 0) tile_sums[blockIdx.x] = s;
}

// Scans tile blockIdx.x of `in` into `out`, adding tile_offsets[blockIdx.x]
// (or 0).  The last tile also writes out[n] = total.
template <class TI, class TO>
__global__ __launch_bounds__(kScanNT) void k_tile_scan(const TI *in, TO *out, u64 n,
                                                       const TO *tile_offsets) {
  __shared__ TO tile[kScanTile];
  __shared__ TO scratch[kScanNT / kWave];
  const u64 base = (u64)blockIdx.x * kScanTile;
  // coalesced load, blocked re-read
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) {
    u64 i = base + (u64)j * kScanNT + threadIdx.x;
    tile[j * kScanNT + threadIdx.x] = i < n ? (TO)in[i] : TO(0);
  }
  __syncthreads();
  TO local[kScanIT];
  TO run = 0;
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) {
    local[j] = run;
    run += tile[threadIdx.x * kScanIT + j];
  }
  TO total;
  TO excl = block_exclusive_sum<kScanNT, TO>(run, scratch, &total);
  const TO off = tile_offsets ? tile_offsets[blockIdx.x] : TO(0);
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) tile[threadIdx.x * kScanIT + j] = local[j] + excl + off;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kScanIT; ++j) {
    u64 i = base + (u64)j * kScanNT + threadIdx.x;
    if (i < n) out[i] = tile[j * kScanNT + threadIdx.x];
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) out[n] = off + total;
}

// Three arrays of one length scanned together (array 0 u64, arrays 1 and 2
// u32, all into u64): the same tiles, one launch per pass for all three.
struct Scan3 {
  const u64 *in0;
  const u32 *in1, *in2;
  u64 *out0, *out1, *out2;
};

__device__ __forceinline__ u64 scan3_in(const Scan3 &p, int k, u64 i) {
  return k == 0 ? p.in0[i] : k == 1 ? (u64)p.in1[i] : (u64)p.in2[i];
}

// tile_sums[k nb + b] = sum of tile b of array k
__global__ __launch_bounds__(kScanNT) void k_tile_reduce3(Scan3 p, u64 n, u64 *tile_sums) {
  __shared__ u64 scratch[kScanNT / kWave];
  const u64 base = (u64)blockIdx.x * kScanTile;
  for (int k = 0; k < 3; ++k) {
    u64 s = 0;
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) {
      const u64 i = base + (u64)j * kScanNT + threadIdx.x;
      if (i < n) s += scan3_in(p, k, i);
    }
    s = block_sum<kScanNT, u64>(s, scratch);
    if (threadIdx.x == 0) tile_sums[(u64)k * gridDim.x + blockIdx.x] = s;
    __syncthreads();  // scratch reused
  }
}

// Tile blockIdx.x of the three arrays, each offset by tile_offsets[k nb + b]
// (or 0); the last tile writes out_k[n].
__global__ __launch_bounds__(kScanNT) void k_tile_scan3(Scan3 p, u64 n, const u64 *tile_offsets) {
  __shared__ u64 tile[kScanTile];
  __shared__ u64 scratch[kScanNT / kWave];
  const u64 base = (u64)blockIdx.x * kScanTile;
  for (int k = 0; k < 3; ++k) {
    u64 *out = k == 0 ? p.out0 : k == 1 ? p.out1 : p.out2;
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) {
      const u64 i = base + (u64)j * kScanNT + threadIdx.x;
      tile[j * kScanNT + threadIdx.x] = i < n ? scan3_in(p, k, i) : 0ull;
    }
    __syncthreads();
    u64 local[kScanIT];
    u64 run = 0;
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) {
      local[j] = run;
      run += tile[threadIdx.x * kScanIT + j];
    }
    u64 total;
    const u64 excl = block_exclusive_sum<kScanNT, u64>(run, scratch, &total);
    const u64 off = tile_offsets ? tile_offsets[(u64)k * gridDim.x + blockIdx.x] : 0ull;
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) tile[threadIdx.x * kScanIT + j] = local[j] + excl + off;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) {
      const u64 i = base + (u64)j * kScanNT + threadIdx.x;
      if (i < n) out[i] = tile[j * kScanNT + threadIdx.x];
    }
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) out[n] = off + total;
    __syncthreads();  // tile reused
  }
}

// Exclusive scan of the nb tile sums of each array (nb <= kScanTile): one
// workgroup, the three arrays in turn.
__global__ __launch_bounds__(kScanNT) void k_sums_scan3(const u64 *sums, u64 nb, u64 *offs) {
  __shared__ u64 tile[kScanTile];
  __shared__ u64 scratch[kScanNT / kWave];
  for (int k = 0; k < 3; ++k) {
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) {
      const u64 i = (u64)j * kScanNT + threadIdx.x;
      tile[j * kScanNT + threadIdx.x] = i < nb ? sums[(u64)k * nb + i] : 0ull;
    }
    __syncthreads();
    u64 local[kScanIT];
    u64 run = 0;
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) {
      local[j] = run;
      run += tile[threadIdx.x * kScanIT + j];
    }
    u64 total;
    const u64 excl = block_exclusive_sum<kScanNT, u64>(run, scratch, &total);
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) tile[threadIdx.x * kScanIT + j] = local[j] + excl;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kScanIT; ++j) {
      const u64 i = (u64)j * kScanNT + threadIdx.x;
      if (i < nb) offs[(u64)k * nb + i] = tile[j * kScanNT + threadIdx.x];
    }
    __syncthreads();
  }
}

template <class TO>
size_t temp_elems(u64 n) {
  size_t t = 0;
  u64 nb = ceil_div(n, kScanTile);
  while (nb > 1) {
    t += nb + (nb + 1);  // tile sums + their scan
    nb = ceil_div(nb, kScanTile);
  }
  return t;
}

template <class TI, class TO>
void scan_impl(const TI *in, TO *out, u64 n, TO *temp, hipStream_t s) {
  if (n == 0) {
    hipLaunchKernelGGL((k_fill<TO>), dim3(1), dim3(64), 0, s, out, TO(0), (u64)1);
    return;
  }
  const u64 nb = ceil_div(n, kScanTile);
  if (nb == 1) {
    hipLaunchKernelGGL((k_tile_scan<TI, TO>), dim3(1), dim3(kScanNT), 0, s, in, out, n,
                       (const TO *)nullptr);
    return;
  }
  TO *sums = temp;
  TO *offs = temp + nb;
  hipLaunchKernelGGL((k_tile_reduce<TI, TO>), dim3((unsigned)nb), dim3(kScanNT), 0, s, in, n,
                     sums);
  scan_impl<TO, TO>(sums, offs, nb, temp + nb + (nb + 1), s);
  hipLaunchKernelGGL((k_tile_scan<TI, TO>), dim3((unsigned)nb), dim3(kScanNT), 0, s, in, out,
                     n, (const TO *)offs);
}

}  // namespace

int compute_units() {
  static std::atomic<int> cache[64];
  int dev = 0;
  FSTC_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) dev = 0;
  int n = cache[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    FSTC_HIP(hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev));
    n = std::max(n, 1);
    cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

void fill_u32(u32 *p, u32 v, u64 n, hipStream_t s) {
  if (!n) return;
  unsigned g = (unsigned)std::min<u64>(ceil_div(n, 256), 4096);
  hipLaunchKernelGGL((k_fill<u32>), dim3(g), dim3(256), 0, s, p, v, n);
}

void fill_u64(u64 *p, u64 v, u64 n, hipStream_t s) {
  if (!n) return;
  unsigned g = (unsigned)std::min<u64>(ceil_div(n, 256), 4096);
  hipLaunchKernelGGL((k_fill<u64>), dim3(g), dim3(256), 0, s, p, v, n);
}

size_t scan_temp_bytes(u64 n) { return temp_elems<u64>(n) * sizeof(u64) + 256; }

size_t scan3_temp_bytes(u64 n) {
  return std::max<size_t>(6 * ceil_div(std::max<u64>(n, 1), kScanTile) * sizeof(u64) + 256,
                          scan_temp_bytes(n));
}

void exclusive_scan3(const u64 *in0, u64 *out0, const u32 *in1, u64 *out1, const u32 *in2,
                     u64 *out2, u64 n, void *temp, hipStream_t s) {
  const u64 nb = ceil_div(n, kScanTile);
  if (n == 0 || nb > kScanTile) {  // empty, or too many tiles for one sums pass
    exclusive_scan(in0, out0, n, temp, s);
    exclusive_scan(in1, out1, n, temp, s);
    exclusive_scan(in2, out2, n, temp, s);
    return;
  }
  const Scan3 p{in0, in1, in2, out0, out1, out2};
  if (nb == 1) {
    hipLaunchKernelGGL(k_tile_scan3, dim3(1), dim3(kScanNT), 0, s, p, n, (const u64 *)nullptr);
    return;
  }
  u64 *sums = static_cast<u64 *>(temp), *offs = sums + 3 * nb;
  hipLaunchKernelGGL(k_tile_reduce3, dim3((unsigned)nb), dim3(kScanNT), 0, s, p, n, sums);
  hipLaunchKernelGGL(k_sums_scan3, dim3(1), dim3(kScanNT), 0, s, (const u64 *)sums, nb, offs);
  hipLaunchKernelGGL(k_tile_scan3, dim3((unsigned)nb), dim3(kScanNT), 0, s, p, n, (const u64 *)offs);
}

void exclusive_scan(const u64 *in, u64 *out, u64 n, void *temp, hipStream_t s) {
  scan_impl<u64, u64>(in, out, n, (u64 *)temp, s);
}
void exclusive_scan(const u32 *in, u64 *out, u64 n, void *temp, hipStream_t s) {
  scan_impl<u32, u64>(in, out, n, (u64 *)temp, s);
}
void exclusive_scan(const u32 *in, u32 *out, u64 n, void *temp, hipStream_t s) {
  scan_impl<u32, u32>(in, out, n, (u32 *)temp, s);
}

}  // namespace fstc
