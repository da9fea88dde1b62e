// draft.hip -- draft-side pruning and packing (SpecLA §6.1, "Tree pruning")
// and the tree-mask -> parent-array converter (§7), batched on the device so
// that a serving loop can go from the drafter's scores to the verifier's
// parent array without a host round trip.
//
// One wavefront per sequence, lane j = candidate j (n <= 64):
//   * depth by pointer walking, then the path score level by level:
//     q_j = q_parent + logp_j in fp32, so every score is summed root first;
//   * q* by a wave maximum; the window keeps q_j >= q* - tau (fp32);
//   * over the budget T, the rank of each window node in (score desc, index
//     asc) order by counting; the first T are kept.  Scores never increase
//     along a path and parents carry smaller indices, so every ancestor ranks
//     ahead of its descendants: this prefix is ancestor-closed, and it is the
//     selection "take candidates in score order with their missing
//     ancestors until T is used up" reaches;
//   * packing: a kept node's new index is the number of kept nodes before it
//     (ballot + popcount); its new parent is its parent's new index.
#include "device.hpp"
#include "layer_ops.hpp"

namespace sla {
namespace {

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__global__ __launch_bounds__(kWave) void prune_kernel(PruneArgs a) {
  const int b = blockIdx.x;
  const int l = threadIdx.x;
  const int n = a.n;
  const bool live = l < n;
  const size_t row = (size_t)b * n;
  const int p = live ? a.parent[row + l] : -1;
  const float lp = live ? a.logp[row + l] : 0.f;
  int err = SLA_OK;
  if (wave_any(live && (p < -1 || p >= l))) err = SLA_ERR_TOPOLOGY;
  else if (wave_any(live && !(lp <= 0.f))) err = SLA_ERR_SCORE;  // also NaN
  if (l == 0) {
    if (a.status) a.status[b] = err;
    a.count[b] = 0;
  }
  if (err != SLA_OK) return;
  // depth by pointer walking (parents precede children: walks end)
  int d = live ? 1 : 0, x = p;
  while (wave_any(x >= 0)) {
    const int px = __shfl(p, x >= 0 ? x : 0);
    if (x >= 0) {
      ++d;
      x = px;
    }
  }
  int maxd = d;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) maxd = max(maxd, __shfl_xor(maxd, o));
  // scores, one level at a time: a parent's score is final before its children's
  float q = lp;
  for (int lev = 2; lev <= maxd; ++lev) {
    const float qp = __shfl(q, p >= 0 ? p : 0);
    if (d == lev) q = qp + lp;
  }
  const float qstar = wave_max(live ? q : -INFINITY);
  const float thr = qstar - a.tau;
  const bool inw = live && q >= thr;
  const uint64_t wmask = __ballot(inw);
  bool keep = inw;
  if (a.budget > 0 && __popcll(wmask) > a.budget) {
    int rank = 0;
    // every lane i, unrolled (lanes past the window have no bit in wmask):
    // wave-uniform i, so each step is a register read, not a shuffle
#pragma unroll
    for (int i = 0; i < kWave; ++i) {
      const float qi = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(q), i));
      const bool wi = (wmask >> i) & 1ull;
      rank += (wi && (qi > q || (qi == q && i < l))) ? 1 : 0;
    }
    keep = inw && rank < a.budget;
  }
  const uint64_t kmask = __ballot(keep);
  const int m = __popcll(kmask);
  const int nidx = __popcll(kmask & ((1ull << l) - 1ull));
  const int pnew = __shfl(nidx, p >= 0 ? p : 0);
  if (keep) {
    a.packed_parent[row + nidx] = p >= 0 ? pnew : -1;
    a.index_map[row + nidx] = l;
  }
  if (live && l >= m) {  // rows past the kept count
    a.packed_parent[row + l] = -1;
    a.index_map[row + l] = -1;
  }
  if (live && a.scores) a.scores[row + l] = q;
  if (l == 0) a.count[b] = m;
}

// Tree mask rows (bit j of row i: j is an ancestor of i or i itself) ->
// parent array.  In topological order a node's parent is its strict
// ancestor with the highest index; the row must then equal the parent's row
// plus the node itself, which checks the whole mask by induction.
__global__ __launch_bounds__(kWave) void mask_to_parent_kernel(MaskArgs a) {
  const int b = blockIdx.x;
  const int l = threadIdx.x;
  const int n = a.n;
  const bool live = l < n;
  const uint64_t self = 1ull << l;
  const uint64_t m = live ? a.mask[(size_t)b * n + l] : 0ull;
  const uint64_t strict = m & ~self;
  const int p = strict ? 63 - __builtin_clzll(strict) : -1;
  // parent's row by two 32-bit shuffles
  const int src = p >= 0 ? p : 0;
  const uint32_t lo = __shfl((uint32_t)m, src), hi = __shfl((uint32_t)(m >> 32), src);
  const uint64_t prow = p >= 0 ? (((uint64_t)hi << 32) | lo) : 0ull;
  const uint64_t beyond = (l + 1 < 64) ? ~((self << 1) - 1ull) : 0ull;  // bits above l
  const bool bad = live && (!(m & self) || (m & beyond) || m != (prow | self));
  const int err = wave_any(bad) ? SLA_ERR_TOPOLOGY : SLA_OK;
  if (a.status && l == 0) a.status[b] = err;
  if (live && err == SLA_OK) a.parent[(size_t)b * n + l] = p;
}

}  // namespace

hipError_t launch_prune(const PruneArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(prune_kernel, dim3((unsigned)a.B), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mask_to_parent(const MaskArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(mask_to_parent_kernel, dim3((unsigned)a.B), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace sla
