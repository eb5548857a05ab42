// Stable ranking of radix digits inside one workgroup, built on wave64
// ballots (no per-thread digit counters).
//
// Items are held in registers in a wave-striped arrangement: element e of the
// block tile belongs to wave w = e / (64*IT), item slot j = (e / 64) % IT and
// lane e % 64, so each wave owns a contiguous run of 64*IT elements and, for a
// fixed wave, element order is (j, lane).  Ranking the slots j in order and,
// inside one slot, lanes in order therefore visits the elements in their
// original order, which makes the ranking stable.
//
// For one slot the lanes sharing a digit are found from one ballot per digit
// bit: peers = ~OR_b (ballot_b XOR sext(bit_b)) restricted to valid lanes.
// The lowest such lane updates the wave's running count for the digit.  A
// wave reads the count before the lowest lane writes it within the same
// instruction stream, so no barrier is needed inside the loop.
#pragma once

#include "common.hpp"

namespace fstc {

namespace detail {

template <int IT, int BITS>
__device__ __forceinline__ void rank_rows(const u32 (&dig)[IT], u32 valid, u32 (&rank)[IT],
                                          u32 *wc) {
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const u32 d = dig[j];
    const bool vj = (valid >> j) & 1u;
    const u64 vm = __ballot(vj);
    u32 miss_lo = 0, miss_hi = 0;  // lanes whose digit differs in some bit
#pragma unroll
    for (int b = 0; b < BITS; ++b) {
      const u32 sx = (u32)(-(int)((d >> b) & 1u));  // 0 or ~0
      const u64 bal = __ballot(sx != 0);
      miss_lo |= (u32)bal ^ sx;
      miss_hi |= (u32)(bal >> 32) ^ sx;
    }
    const u64 peers = vm & ~(((u64)miss_hi << 32) | miss_lo);
    const u32 below = count_below(peers);
    const u32 base = wc[d];
    rank[j] = base + below;
    if (vj && below == 0) wc[d] = base + (u32)__popcll(peers);
  }
}

}  // namespace detail

// `valid` has bit j set when item j holds an element.  After the call:
//   rank_in_digit[j] = number of valid block elements before item j whose
//                      digit equals item j's digit (stable order)
//   s_base[d]        = number of valid block elements with a digit < d
// Digits must be < 2^digit_bits (invalid items included: they are read but
// not counted).  s_cnt needs NT/64 * 256 u32 of LDS, s_base 256 u32, s_tmp
// NT/64 u32.  Requires NT >= 256.  All threads of the block must call it.
template <int NT, int IT>
__device__ __forceinline__ void block_rank_digits(const u32 (&dig)[IT], u32 valid,
                                                  int digit_bits, u32 (&rank_in_digit)[IT],
                                                  u32 *s_cnt, u32 *s_base, u32 *s_tmp) {
  static_assert(NT >= 256 && NT % kWave == 0, "block_rank_digits: NT >= 256");
  constexpr int NW = NT / kWave;
  const u32 w = threadIdx.x / kWave;
  u32 *wc = s_cnt + w * 256;
  for (int i = threadIdx.x; i < NW * 256; i += NT) s_cnt[i] = 0;
  __syncthreads();
  switch (digit_bits) {
    case 1: detail::rank_rows<IT, 1>(dig, valid, rank_in_digit, wc); break;
    case 2: detail::rank_rows<IT, 2>(dig, valid, rank_in_digit, wc); break;
    case 3: detail::rank_rows<IT, 3>(dig, valid, rank_in_digit, wc); break;
    case 4: detail::rank_rows<IT, 4>(dig, valid, rank_in_digit, wc); break;
    case 5: detail::rank_rows<IT, 5>(dig, valid, rank_in_digit, wc); break;
    case 6: detail::rank_rows<IT, 6>(dig, valid, rank_in_digit, wc); break;
    case 7: detail::rank_rows<IT, 7>(dig, valid, rank_in_digit, wc); break;
    default: detail::rank_rows<IT, 8>(dig, valid, rank_in_digit, wc); break;
  }
  __syncthreads();
  u32 tot = 0;
  if (threadIdx.x < 256) {
    for (int v = 0; v < NW; ++v) {
      const u32 c = s_cnt[v * 256 + threadIdx.x];
      s_cnt[v * 256 + threadIdx.x] = tot;
      tot += c;
    }
  }
  u32 total;
  const u32 ex = block_exclusive_sum<NT, u32>(threadIdx.x < 256 ? tot : 0u, s_tmp, &total);
  if (threadIdx.x < 256) s_base[threadIdx.x] = ex;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IT; ++j) rank_in_digit[j] += s_cnt[w * 256 + dig[j]];
}

}  // namespace fstc
