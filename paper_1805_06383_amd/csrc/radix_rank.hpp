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
// For one slot the lanes sharing a digit are found by intersecting one ballot
// per digit bit; the lowest such lane updates the wave's running count for the
// digit.  A wave reads the count before the lowest lane writes it within the
// same instruction stream, so no barrier is needed inside the loop.
#pragma once

#include "common.hpp"

namespace fstc {

// After the call:
//   rank_in_digit[j] = number of valid block elements before item j whose
//                      digit equals item j's digit (stable order)
//   s_base[d]        = number of valid block elements with a digit < d
// s_cnt needs NT/64 * 256 u32 of LDS, s_base 256 u32, s_tmp NT/64 u32.
// Requires NT >= 256.  All threads of the block must call it.
template <int NT, int IT>
__device__ __forceinline__ void block_rank_digits(const u32 (&dig)[IT], const bool (&valid)[IT],
                                                  int digit_bits, u32 (&rank_in_digit)[IT],
                                                  u32 *s_cnt, u32 *s_base, u32 *s_tmp) {
  static_assert(NT >= 256 && NT % kWave == 0, "block_rank_digits: NT >= 256");
  constexpr int NW = NT / kWave;
  const u32 w = threadIdx.x / kWave;
  u32 *wc = s_cnt + w * 256;
  for (int i = threadIdx.x; i < NW * 256; i += NT) s_cnt[i] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    u64 peers = __ballot(valid[j]);
    const u32 d = dig[j];
    for (int b = 0; b < digit_bits; ++b) {
      const bool bit = (d >> b) & 1u;
      const u64 bal = __ballot(bit);
      peers &= bit ? bal : ~bal;
    }
    if (valid[j]) {
      const u32 below = count_below(peers);
      const u32 base = wc[d];
      rank_in_digit[j] = base + below;
      if (below == 0) wc[d] = base + (u32)__popcll(peers);
    }
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
  for (int j = 0; j < IT; ++j)
    if (valid[j]) rank_in_digit[j] += s_cnt[w * 256 + dig[j]];
}

}  // namespace fstc
