// Composition with epsilon transitions: the inputs of the filter composition.
//
// The paper admits no epsilon transitions (§2) and names composition filters
// as what admitting them takes.  Here one label value eps is the empty string
// on every tape, and the three-state epsilon filter of Mohri, Pereira and
// Riley is itself a transducer F: composing M1' ∘ F ∘ M2' with the
// epsilon-free composition gives the filtered composition, every pair of
// paths aligned exactly once.  Over the inner alphabet Γ' = Γ ∪ {E1, E2}
// (E1 = |Γ|, E2 = |Γ| + 1; label eps no longer occurs inside):
//   M1' = M1 with every output eps renamed E2, plus a loop eps:E1 of weight 1
//         at every state (M1 stays while M2 moves);
//   M2' = M2 with every input eps renamed E1, plus a loop E2:eps of weight 1
//         at every state (M2 stays while M1 moves);
//   F   = states 0, 1, 2, all accepting; x:x from each state to 0 for every
//         symbol x of Γ other than eps (both move on a symbol); E2:E1 from 0
//         to 0 (both move on eps); E1:E1 from 0 and 1 to 1 (M2 alone);
//         E2:E2 from 0 and 2 to 2 (M1 alone).
// A state of (M1' ∘ F) ∘ M2' is ((q1, f), q2); compose.hip maps it back to
// the triple (q1, q2, f).
#include "internal.hpp"

namespace fstc {
namespace {

constexpr int kNT = 256;

// M1' (by_output) or M2' (otherwise): the n arcs of m relabelled, then one
// loop per state.
__global__ void k_eps_side(const u32 *src, const u32 *dst, const u32 *il, const u32 *ol,
                           const float *w, u64 n, u32 nq, u32 eps, u32 e_rename, u32 e_loop,
                           int by_output, u32 *osrc, u32 *odst, u32 *oil, u32 *ool, float *ow) {
  const u64 total = n + nq;
  for (u64 j = (u64)blockIdx.x * blockDim.x + threadIdx.x; j < total;
       j += (u64)gridDim.x * blockDim.x) {
    if (j < n) {
      u32 a = il[j], c = ol[j];
      if (by_output) c = c == eps ? e_rename : c;
      else a = a == eps ? e_rename : a;
      osrc[j] = src[j];
      odst[j] = dst[j];
      oil[j] = a;
      ool[j] = c;
      ow[j] = w[j];
    } else {
      const u32 q = (u32)(j - n);
      osrc[j] = q;
      odst[j] = q;
      oil[j] = by_output ? eps : e_loop;
      ool[j] = by_output ? e_loop : eps;
      ow[j] = 1.0f;
    }
  }
}

// F over an inner alphabet of nsym symbols (eps among them): 3 (nsym - 1)
// symbol arcs, then the five epsilon arcs.
__global__ void k_eps_filter(u32 nsym, u32 eps, u32 E1, u32 E2, u32 *src, u32 *dst, u32 *il,
                             u32 *ol, float *w, uint8_t *final) {
  const u64 nx = 3ull * (nsym - 1);
  const u64 total = nx + 5;
  for (u64 j = (u64)blockIdx.x * blockDim.x + threadIdx.x; j < total;
       j += (u64)gridDim.x * blockDim.x) {
    u32 s, d, a, c;
    if (j < nx) {
      const u32 r = (u32)(j / 3);
      const u32 x = r + (r >= eps ? 1u : 0u);  // the symbols other than eps
      s = (u32)(j % 3);
      d = 0;
      a = c = x;
    } else {
      const u32 k = (u32)(j - nx);
      // k = 0..4: E2:E1 0->0, E1:E1 0->1, E1:E1 1->1, E2:E2 0->2, E2:E2 2->2
      s = k == 2 ? 1u : (k == 4 ? 2u : 0u);
      d = k == 0 ? 0u : (k <= 2 ? 1u : 2u);
      a = (k == 0 || k >= 3) ? E2 : E1;
      c = k >= 3 ? E2 : E1;
    }
    src[j] = s;
    dst[j] = d;
    il[j] = a;
    ol[j] = c;
    w[j] = 1.0f;
  }
  if (blockIdx.x == 0 && threadIdx.x < 3) final[threadIdx.x] = 1;
}

// State i of (M1' ∘ F) ∘ M2' is (a, q2) with a a state of M1' ∘ F, i.e.
// (q1, f): q1 replaces a in place, f goes to filt.
__global__ void k_eps_states(u32 *q1, const u32 *aq1, const u32 *af, u64 n, uint8_t *filt) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (u64)gridDim.x * blockDim.x) {
    const u32 a = q1[i];
    q1[i] = aq1[a];
    filt[i] = (uint8_t)af[a];
  }
}

unsigned grid(u64 n) { return (unsigned)std::max<u64>(1, std::min<u64>(ceil_div(n, kNT), 4096)); }

}  // namespace

void build_eps_side(const fstc_fst &m, bool by_output, u32 eps, u32 e_rename, u32 e_loop,
                    u32 *src, u32 *dst, u32 *il, u32 *ol, float *w, hipStream_t s) {
  const u64 total = m.num_arcs + m.num_states;
  hipLaunchKernelGGL(k_eps_side, dim3(grid(total)), dim3(kNT), 0, s, m.src, m.dst, m.ilabel,
                     m.olabel, m.weight, m.num_arcs, m.num_states, eps, e_rename, e_loop,
                     by_output ? 1 : 0, src, dst, il, ol, w);
}

void build_eps_filter(u32 nsym, u32 eps, u32 *src, u32 *dst, u32 *il, u32 *ol, float *w,
                      uint8_t *final, hipStream_t s) {
  const u64 total = 3ull * (nsym - 1) + 5;
  hipLaunchKernelGGL(k_eps_filter, dim3(grid(total)), dim3(kNT), 0, s, nsym, eps, nsym, nsym + 1,
                     src, dst, il, ol, w, final);
}

void map_eps_states(u32 *q1, const u32 *aq1, const u32 *af, u64 n, uint8_t *filt,
                    hipStream_t s) {
  if (!n) return;
  hipLaunchKernelGGL(k_eps_states, dim3(grid(n)), dim3(kNT), 0, s, q1, aq1, af, n, filt);
}

}  // namespace fstc
