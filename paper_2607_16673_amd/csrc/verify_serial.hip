// verify_serial.hip -- state-resident verification (SpecLA §4.1) and the
// chain-decomposed hybrid schedule built on it (§4.3), with the delayed state
// update of §5.2 fused in front of both.
//
// A wavefront owns one (batch b, head h, 16-column V-tile) slice of the
// transposed state H = S^T: the full d_k rows of 16 value columns (V-dimension
// tiling keeps every output column local, §4.1 "Tiling").  Lane (g, c) holds
// column c of the contiguous row block g*R .. g*R+R-1 (R = d_k / 4) in
// registers, so a reduction over d_k is a per-lane dot product followed by
// two cross-row-group shuffles.
//
// Per node j, with H_par the on-chip state of j's parent:
//     a_j = H_par^T k_j,   b_j = H_par^T q_j,   u_j = beta_j (v_j - alpha_j a_j)
//     o_j = alpha_j b_j + (k_j . q_j) u_j                     (= S_j q_j)
//     H_j = alpha_j H_par + k_j u_j^T   (only if j has children)
// which is the GDN step S_j = alpha_j S_par (I - beta_j k_j k_j^T) +
// beta_j v_j k_j^T rewritten around the corrected value u_j (the factor
// record stored for commit).  The other layer families take the same loop:
// DeltaNet with alpha = 1; the no-delta families (scalar decay, GLA) with
// u_j = v_j; GLA's per-key gates g_j scale row i by g_j[i] in place of
// alpha_j, so b_j = H_par^T (g_j * q_j) and H_j = diag(g_j) H_par + k_j u_j^T.
//
// Serial route: one wave per slice visits the nodes in DFS pre-order; a chain
// therefore advances the registers in place.  When the next node's parent is
// not the state in registers (a branch point of a tree), that state is
// rebuilt from the committed tile kept in registers by re-applying the stored
// factors of the parent's root path -- rank-one updates only, the reductions
// of shared prefixes are never repeated.
//
// Hybrid route: the draft is split by heavy-light decomposition into
// node-disjoint chains (each node continues the chain of its parent when it
// is the parent's child with the largest subtree, ties to the smaller index;
// every other node starts a chain).  The chains are verified by the same
// per-node loop, one wave per chain, several waves per slice; a chain's level
// is the number of chain starts strictly above its head, and the chains of
// one level run in parallel once every shallower level is done (a workgroup
// barrier per level).  A chain's boundary state -- the state of its head's
// parent -- is materialised on chip from the committed tile and the rank-one
// factor records of the head's ancestors, which the shallower chains left in
// LDS; no boundary state goes to memory.  Every node's state is the committed
// tile advanced by the records of its root path in root-first order, on both
// routes, so the serial and hybrid routes agree bit for bit.
#include "serial_stage.hpp"

namespace sla {
namespace {

constexpr int kCols = kSliceCols;
constexpr int kGroups = kWave / kCols;
constexpr int kXcds = 8;  // workgroup i runs on XCD i mod 8

// Slice numbering shared by both kernels: neighbouring tiles (2m, 2m + 1)
// hold the two halves of each 128-byte row segment; their workgroups are
// numbered 8 apart, so that they run on the same XCD and share its L2
// (consecutive workgroups go to different XCDs, whose L2s would each fetch
// and write back the whole lines).  Returns false for the padding of the
// numbering.
__device__ inline bool slice_of(const VerifyArgs &a, int &tile, int &b, int &h) {
  const int ntiles = a.dv / kCols;
  const int npairs = (ntiles + 1) / 2;
  const int x = blockIdx.x;
  const int qd = x / kXcds;
  const size_t pair = (size_t)(qd / 2) * kXcds + x % kXcds;
  tile = 2 * (int)(pair % npairs) + qd % 2;
  const size_t unit_id = pair / npairs;
  if (tile >= ntiles || unit_id >= (size_t)a.B * a.H) return false;
  h = (int)(unit_id % a.H);
  b = (int)(unit_id / a.H);
  return true;
}

// VG: per-key gates (GLA), staged on chip like the keys.
template <int DK, typename T, bool CHAIN, bool VG>
__global__ __launch_bounds__(kWave) void verify_serial_kernel(VerifyArgs a) {
  constexpr int R = DK / kGroups;
  const int lane = threadIdx.x;
  const int c = lane & (kCols - 1);
  const int g = lane / kCols;
  const int n = a.n;
  int tile, b, h;
  if (!slice_of(a, tile, b, h)) return;  // padding of the numbering: no barrier follows
  const int col = tile * kCols + c;
  const int row0 = g * R;
  const size_t unit = (size_t)b * a.H + h;
  // delta-rule families correct the value against the parent state
  const bool delta = a.family == SLA_FAMILY_GDN || a.family == SLA_FAMILY_DELTANET;

  // The state tile: the only state read of this call.
  float *st = a.state + unit * DK * a.dv + col;
  float H0[R];
#pragma unroll
  for (int r = 0; r < R; ++r) H0[r] = st[(size_t)(row0 + r) * a.dv];

  // Topology table of this draft and validation of the pending path.
  NodeTopo topo;
  int err = build_topology(a.parent + (size_t)b * n, n, lane, CHAIN, topo);
  int plen = 0;
  if (err == SLA_OK && a.has_pending) {
    plen = a.pend.len[b];
    err = check_path(a.pend.parent + (size_t)b * a.pend.n, a.pend.n,
                     a.pend.path + (size_t)b * a.pend.n, plen, lane);
  }
  if (tile == 0 && h == 0 && lane == 0 && a.status) a.status[b] = err;
  if (err != SLA_OK) return;

  // Stage this unit's draft in LDS.
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const SerialStage s = carve_stage<DK, VG>(lds, n);
  int *ords = s.ia, *pars = s.ib, *kids = s.ic;
  stage_draft<DK, T, VG>(a, s, b, h, tile, lane, kWave, delta, tile == 0);
  if (lane < n) {
    ords[topo.pos] = lane;
    pars[lane] = topo.parent;
    kids[lane] = topo.n_children;
    s.ancs[lane] = topo.anc;
  }
  __syncthreads();

  // Delayed state update: commit the previous round's accepted path into the
  // tile, then write the committed tile back (the only state write).
  if (a.has_pending) {
    apply_pending<DK, R, T, VG>(a, b, h, col, row0, plen, H0);
#pragma unroll
    for (int r = 0; r < R; ++r) st[(size_t)(row0 + r) * a.dv] = H0[r];
  }

  // Node loop.
  float Hc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) Hc[r] = H0[r];
  int cur = -1;  // node whose state Hc holds (-1: committed state)
  for (int t = 0; t < n; ++t) {
    const int j = CHAIN ? t : ords[t];
    const int p = CHAIN ? t - 1 : pars[j];
    if (!CHAIN && p != cur) {
#pragma unroll
      for (int r = 0; r < R; ++r) Hc[r] = H0[r];
      if (p >= 0) {
        uint64_t m = s.ancs[p];
        while (m) {
          const int x = __builtin_ctzll(m);
          m &= m - 1;
          advance<DK, R, VG>(s, Hc, x, row0, s.us[x * kCols + c]);
        }
      }
    }
    const float u = node_step<DK, R, VG>(a, s, Hc, j, b, h, c, g, row0, col, delta);
    const bool internal = CHAIN ? (t + 1 < n) : (kids[j] > 0);
    if (internal) {
      advance<DK, R, VG>(s, Hc, j, row0, u);
      cur = j;
    } else {
      cur = p;
    }
  }
}

// ---------------------------------------------------------------- hybrid
constexpr int kMaxLevels = 8;  // light edges on a root path <= log2(64) = 6

// LDS beyond the stage: heavy-child keys and heavy children [n], per-level
// chain-head lists [kMaxLevels][n], per-level counts, the error code and the
// deepest level.
__host__ __device__ inline size_t hybrid_extra_bytes(int n) {
  return sizeof(int) * (2 * n + kMaxLevels * n + kMaxLevels + 2);
}

template <int DK, typename T, bool VG, int W>
__global__ __launch_bounds__(W * kWave) void verify_hybrid_kernel(VerifyArgs a) {
  constexpr int R = DK / kGroups;
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = tid % kWave;
  const int c = lane & (kCols - 1);
  const int g = lane / kCols;
  const int n = a.n;
  int tile, b, h;
  if (!slice_of(a, tile, b, h)) return;  // the whole workgroup: no barrier follows
  const int col = tile * kCols + c;
  const int row0 = g * R;
  const size_t unit = (size_t)b * a.H + h;
  const bool delta = a.family == SLA_FAMILY_GDN || a.family == SLA_FAMILY_DELTANET;

  // every wave holds the committed tile (the pending path applied below gives
  // bitwise the same rows in each)
  float *st = a.state + unit * DK * a.dv + col;
  float H0[R];
#pragma unroll
  for (int r = 0; r < R; ++r) H0[r] = st[(size_t)(row0 + r) * a.dv];

  extern __shared__ __attribute__((aligned(16))) float lds[];
  const SerialStage s = carve_stage<DK, VG>(lds, n);
  int *hkey = s.ia;       // [n] heavy-child key: (subtree size << 7) | (127 - child)
  int *heavy = s.ib;      // [n] heavy child, -1 for a leaf
  int *lists = reinterpret_cast<int *>(lds + serial_stage_bytes(n, DK, VG) / 4);  // [kMaxLevels][n]
  int *counts = lists + kMaxLevels * n;   // [kMaxLevels]
  int *misc = counts + kMaxLevels;        // error code, deepest level

  // ---- wave 0: topology, pending-path check, heavy-light decomposition
  if (w == 0) {
    NodeTopo topo;
    int err = build_topology(a.parent + (size_t)b * n, n, lane, false, topo);
    if (err == SLA_OK && a.has_pending) {
      err = check_path(a.pend.parent + (size_t)b * a.pend.n, a.pend.n, a.pend.path + (size_t)b * a.pend.n,
                       a.pend.len[b], lane);
    }
    if (tile == 0 && h == 0 && lane == 0 && a.status) a.status[b] = err;
    if (lane == 0) misc[0] = err;
    if (err == SLA_OK) {
      const bool live = lane < n;
      // subtree size: the nodes whose root path contains this one
      int size = 0;
      for (int i = 0; i < n; ++i) size += (int)((readlane_u64(topo.anc, i) >> lane) & 1ull);
      if (live) hkey[lane] = 0;
      if (live && topo.parent >= 0) atomicMax(&hkey[topo.parent], (size << 7) | (127 - lane));
      const int key = live ? hkey[lane] : 0;  // after every atomic of this wave (LDS keeps the wave's order)
      const int hv = key ? 127 - (key & 127) : -1;
      const int ph = __shfl(hv, topo.parent >= 0 ? topo.parent : 0);
      const bool head = live && (topo.parent < 0 || ph != lane);
      const uint64_t heads = __ballot(head);
      // level: chain starts strictly above this node's chain head
      const int lvl = live ? __popcll(topo.anc & heads) - 1 : 0;
      const int hd = live ? 63 - __builtin_clzll(topo.anc & heads) : -1;  // this node's chain head
      int len = 0;  // chain length (for a head)
      for (int i = 0; i < n; ++i) len += __builtin_amdgcn_readlane(hd, i) == lane;
      // rank within the level: longer chains first, then smaller head index
      int rank = 0;
      for (int i = 0; i < n; ++i) {
        const uint64_t hi = heads >> i;
        if (!(hi & 1ull)) continue;  // wave-uniform
        const int li = __builtin_amdgcn_readlane(lvl, i);
        const int ni = __builtin_amdgcn_readlane(len, i);
        rank += (li == lvl) && (ni > len || (ni == len && i < lane));
      }
      int cnt = 0;  // lane L < kMaxLevels: chains at level L
      for (int i = 0; i < n; ++i) {
        const int li = __builtin_amdgcn_readlane(lvl, i);
        cnt += ((heads >> i) & 1ull) && li == lane;
      }
      int deepest = head ? lvl : 0;
      for (int o = 1; o < kWave; o <<= 1) deepest = max(deepest, __shfl_xor(deepest, o));
      if (live) {
        heavy[lane] = hv;
        s.ancs[lane] = topo.anc;
      }
      // (heavy-light: a chain start at least halves the subtree, so a 64-node
      // draft has at most 6 levels above level 0; the tables hold 8)
      if (head && lvl < kMaxLevels) lists[lvl * n + rank] = lane;
      if (lane < kMaxLevels) counts[lane] = cnt;
      if (lane == 0) misc[1] = min(deepest, kMaxLevels - 1);
    }
  }
  __syncthreads();
  if (misc[0] != SLA_OK) return;  // workgroup-uniform

  // ---- every wave: stage the draft, commit the pending path into its copy of
  //      the tile; wave 0 writes the committed tile back
  stage_draft<DK, T, VG>(a, s, b, h, tile, tid, W * kWave, delta, tile == 0);
  if (a.has_pending) {
    apply_pending<DK, R, T, VG>(a, b, h, col, row0, a.pend.len[b], H0);
    if (w == 0) {
#pragma unroll
      for (int r = 0; r < R; ++r) st[(size_t)(row0 + r) * a.dv] = H0[r];
    }
  }
  __syncthreads();

  // ---- the chains, level by level; wave w takes ranks w, w + W, ...
  const int deepest = misc[1];
  for (int lvl = 0; lvl <= deepest; ++lvl) {
    const int cnt = counts[lvl];
    for (int r = w; r < cnt; r += W) {
      const int head = lists[lvl * n + r];
      // boundary state: the committed tile advanced by the head's ancestors
      float Hc[R];
#pragma unroll
      for (int i = 0; i < R; ++i) Hc[i] = H0[i];
      uint64_t m = s.ancs[head] & ~(1ull << head);
      while (m) {
        const int x = __builtin_ctzll(m);
        m &= m - 1;
        advance<DK, R, VG>(s, Hc, x, row0, s.us[x * kCols + c]);
      }
      for (int j = head; j >= 0;) {
        const float u = node_step<DK, R, VG>(a, s, Hc, j, b, h, c, g, row0, col, delta);
        const int nx = heavy[j];
        if (nx >= 0) advance<DK, R, VG>(s, Hc, j, row0, u);
        j = nx;
      }
    }
    __syncthreads();  // this level's records are in LDS for the next
  }
}

// gfx950 gives one workgroup up to 160 KiB of LDS; above the default 64 KiB
// the kernel has to opt in.
constexpr size_t kMaxLds = 160 * 1024;
constexpr size_t kDefaultLds = 64 * 1024;

template <typename K>
hipError_t launch_with_lds(K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, const VerifyArgs &a) {
  if (lds > kMaxLds) return hipErrorInvalidConfiguration;
  if (lds > kDefaultLds) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kernel, grid, block, lds, s, a);
  return hipGetLastError();
}

// tile pairs numbered in groups of eight per XCD (see slice_of), padded to whole groups
dim3 slice_grid(const VerifyArgs &a) {
  const size_t pairs = (size_t)a.B * a.H * ((a.dv / kCols + 1) / 2);
  return dim3((unsigned)(((pairs + kXcds - 1) / kXcds) * 2 * kXcds));
}

template <int DK, typename T>
hipError_t launch_dk(const VerifyArgs &a, hipStream_t s) {
  const dim3 grid = slice_grid(a);
  const bool vg = a.family == SLA_FAMILY_GLA;
  const size_t lds = serial_stage_bytes(a.n, DK, vg);
  const dim3 block(kWave);
  if (vg) {
    if (a.chain) return launch_with_lds(verify_serial_kernel<DK, T, true, true>, grid, block, lds, s, a);
    return launch_with_lds(verify_serial_kernel<DK, T, false, true>, grid, block, lds, s, a);
  }
  if (a.chain) return launch_with_lds(verify_serial_kernel<DK, T, true, false>, grid, block, lds, s, a);
  return launch_with_lds(verify_serial_kernel<DK, T, false, false>, grid, block, lds, s, a);
}

template <typename T>
hipError_t launch_t(const VerifyArgs &a, hipStream_t s) {
  switch (a.dk) {
    case 64: return launch_dk<64, T>(a, s);
    case 128: return launch_dk<128, T>(a, s);
    case 256: return launch_dk<256, T>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// Waves per workgroup: four up to 16 nodes and at d_k = 256 (two copies of a
// 256-row slice take most of a wave's registers), else eight.
template <int DK, typename T, int W>
hipError_t launch_hybrid_w(const VerifyArgs &a, hipStream_t s) {
  const dim3 grid = slice_grid(a);
  const bool vg = a.family == SLA_FAMILY_GLA;
  const size_t lds = serial_stage_bytes(a.n, DK, vg) + hybrid_extra_bytes(a.n);
  const dim3 block(W * kWave);
  if (vg) return launch_with_lds(verify_hybrid_kernel<DK, T, true, W>, grid, block, lds, s, a);
  return launch_with_lds(verify_hybrid_kernel<DK, T, false, W>, grid, block, lds, s, a);
}

template <int DK, typename T>
hipError_t launch_hybrid_dk(const VerifyArgs &a, hipStream_t s) {
  if constexpr (DK == 256) return launch_hybrid_w<DK, T, 4>(a, s);
  return a.n <= 16 ? launch_hybrid_w<DK, T, 4>(a, s) : launch_hybrid_w<DK, T, 8>(a, s);
}

template <typename T>
hipError_t launch_hybrid_t(const VerifyArgs &a, hipStream_t s) {
  switch (a.dk) {
    case 64: return launch_hybrid_dk<64, T>(a, s);
    case 128: return launch_hybrid_dk<128, T>(a, s);
    case 256: return launch_hybrid_dk<256, T>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_verify_serial(const VerifyArgs &a, int dtype, hipStream_t s) {
  return dtype == SLA_DTYPE_BF16 ? launch_t<bf16>(a, s) : launch_t<float>(a, s);
}

hipError_t launch_verify_hybrid(const VerifyArgs &a, int dtype, hipStream_t s) {
  // a chain is one chain: the serial kernel is the hybrid schedule of it
  if (a.chain) return launch_verify_serial(a, dtype, s);
  return dtype == SLA_DTYPE_BF16 ? launch_hybrid_t<bf16>(a, s) : launch_hybrid_t<float>(a, s);
}

}  // namespace sla
