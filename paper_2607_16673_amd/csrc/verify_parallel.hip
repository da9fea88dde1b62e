// verify_parallel.hip -- tree-masked factorised verification (SpecLA §4.2)
// with the delayed state update of §5.2 fused in front of it.
//
// Unrolling the gated delta rule along a root path gives, for every node j
// (gamma_j = product of alpha over P(j), D_ja = gamma_j / gamma_a):
//     H_j = gamma_j H0 + sum_{a in P(j)} D_ja k_a u_a^T
//     u_j = beta_j (v_j - gamma_j H0^T k_j) - sum_{a in P(j), a != j} beta_j D_ja (k_j.k_a) u_a
//     o_j = gamma_j H0^T q_j + sum_{a in P(j)} D_ja (q_j.k_a) u_a
// i.e. the tree-masked UT form: the corrected values solve a unit lower-
// triangular system whose off-diagonal entries are masked by strict
// ancestry (the paper's T_tree = solve_tril(I - A_tree)), and the outputs
// are a masked readout of them.  Only the committed state is ever read.
//
// Mapping (one workgroup = one (batch b, head h, 64-column V-tile), four
// wavefronts of 16 columns each):
//   * every lane loads 8 consecutive state rows of one column per 32-row
//     K-step -- exactly the B-operand fragment of v_mfma_f32_16x16x32_bf16 --
//     applies the pending accepted path, writes the committed tile back, and
//     splits each fp32 value into bf16 hi + lo for the matrix cores;
//   * P = [Q; K] H0 (2n x 64) and the tree-masked Grams [Q; K] K^T run on the
//     matrix cores (q and k are exact in bf16, so the Grams are exact
//     products with fp32 accumulation; H0 enters as hi + lo);
//   * the triangular solve runs level by level over the tree in the MFMA
//     accumulator layout, the corrected values go through LDS, and the
//     masked readout follows.  Only ancestor pairs of the Gram are kept, in
//     per-node compact lists.
#include "device.hpp"
#include "kernels.hpp"

namespace sla {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kWaveCols = 16;
constexpr int kTileCols = kWaves * kWaveCols;  // 64 state columns per workgroup
constexpr int kUPitch = kTileCols + 4;         // fp32 row pitch of U in LDS

template <int DK, int NP>
struct Lds {
  static constexpr int XP = DK + 8;                 // bf16 row pitch of [Q; K]
  static constexpr int kX = 2 * NP * XP * 2;        // bytes of [Q; K]
  static constexpr int kU = NP * kUPitch * 4;       // corrected values
  static constexpr int kL = 2 * (NP * (NP + 1) / 2) * 4;  // compact masked Grams (worst case)
  static constexpr int kTopo = NP * (8 + 4 * 6) + 16;
  static constexpr int kBytes = kX + kU + kL + kTopo;
};

__device__ __forceinline__ bf16x8 pack_hi_lo(const float (&x)[8], bf16x8 &lo) {
  bf16x8 hi;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 h = static_cast<__bf16>(x[e]);
    hi[e] = h;
    lo[e] = static_cast<__bf16>(x[e] - static_cast<float>(h));
  }
  return hi;
}

template <int DK, int NP>
__global__ __launch_bounds__(kThreads) void verify_parallel_kernel(VerifyArgs a) {
  constexpr int KS = DK / 32;   // K-steps of the contraction over d_k
  constexpr int NT = NP / 16;   // 16-node tiles
  constexpr int MT = 2 * NT;    // 16-row tiles of [Q; K]
  using L = Lds<DK, NP>;

  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  __bf16 *xs = reinterpret_cast<__bf16 *>(lds);                          // [2NP][XP]
  float *us = reinterpret_cast<float *>(lds + L::kX);                    // [NP][kUPitch]
  float *lq = reinterpret_cast<float *>(lds + L::kX + L::kU);            // compact, by node
  float *lk = lq + NP * (NP + 1) / 2;
  unsigned char *tp = lds + L::kX + L::kU + L::kL;
  uint64_t *s_anc = reinterpret_cast<uint64_t *>(tp);                    // [NP]
  int *s_par = reinterpret_cast<int *>(tp + 8 * NP);                     // [NP]
  int *s_depth = s_par + NP;                                             // [NP]
  int *s_off = s_depth + NP;                                             // [NP]
  float *s_gamma = reinterpret_cast<float *>(s_off + NP);                // [NP]
  float *s_al = s_gamma + NP;                                            // [NP]
  float *s_be = s_al + NP;                                               // [NP]
  int *s_misc = reinterpret_cast<int *>(s_be + NP);                      // err, max depth

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int lc = l & 15;   // column within the wave's 16, row within a 16-row tile
  const int lg = l >> 4;   // 8-row group within a K-step / 4-row group of a C tile
  const int H = a.H, dv = a.dv, n = a.n;
  const int ntiles = (dv + kTileCols - 1) / kTileCols;
  int wid = blockIdx.x;
  const int tile = wid % ntiles;
  wid /= ntiles;
  const int h = wid % H;
  const int b = wid / H;
  const int cw = tile * kTileCols + w * kWaveCols;  // first column of this wave
  const bool cols_live = cw < dv;
  const int col = cw + lc;
  const size_t unit = (size_t)b * H + h;

  // 1. The state tile straight into B-operand order (the only state read).
  float *st = a.state + unit * DK * dv + col;
  float hf[KS][8];
  if (cols_live) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) hf[ks][e] = st[(size_t)(ks * 32 + 8 * lg + e) * dv];
  }

  // 2. Topology, decays and compact-list offsets (wave 0).
  if (w == 0) {
    NodeTopo t;
    int err = build_topology(a.parent + (size_t)b * n, n, l, a.chain, t);
    if (err == SLA_OK && a.has_pending)
      err = check_path(a.pend.parent + (size_t)b * a.pend.n, a.pend.n, a.pend.path + (size_t)b * a.pend.n,
                       a.pend.len[b], l);
    if (err == SLA_OK) {
      const bool live = l < n;
      const size_t s = ((size_t)b * n + (live ? l : 0)) * H + h;
      const float al = live ? a.alpha[s] : 1.f;
      const float be = live ? a.beta[s] : 0.f;
      float g = 1.f;
      int off = 0, md = 0;
      for (int i = 0; i < n; ++i) {
        const float ai = __shfl(al, i);
        if ((t.anc >> i) & 1ull) g *= ai;  // root first
        const int di = __builtin_amdgcn_readlane(t.depth, i);
        if (i < l) off += di;
        md = di > md ? di : md;
      }
      if (live) {
        s_anc[l] = t.anc;
        s_par[l] = t.parent;
        s_depth[l] = t.depth;
        s_off[l] = off;
        s_gamma[l] = g;
        s_al[l] = al;
        s_be[l] = be;
      }
      if (l == 0) s_misc[1] = md;
    }
    if (l == 0) s_misc[0] = err;
  }
  __syncthreads();
  const int err = s_misc[0];
  if (tile == 0 && h == 0 && tid == 0 && a.status) a.status[b] = err;
  if (err != SLA_OK) return;
  const int maxd = s_misc[1];

  // 3. Stage [Q; K] (rows 0..NP-1: q_j, rows NP..2NP-1: k_j; zero padding).
  {
    const bf16 *q = static_cast<const bf16 *>(a.q);
    const bf16 *k = static_cast<const bf16 *>(a.k);
    constexpr int CH = DK / 8;  // 16-byte chunks per row
    for (int c = tid; c < 2 * NP * CH; c += kThreads) {
      const int row = c / CH, part = c % CH;
      const int j = row % NP;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (j < n) {
        const bf16 *src = (row < NP ? q : k) + (((size_t)b * n + j) * H + h) * DK + part * 8;
        val = *reinterpret_cast<const uint4 *>(src);
      }
      *reinterpret_cast<uint4 *>(xs + row * L::XP + part * 8) = val;
    }
    if (tile == 0) {
      // factor records independent of the V-tile
      bf16 *fk = static_cast<bf16 *>(a.fk);
      for (int c = tid; c < n * CH; c += kThreads) {
        const int j = c / CH, part = c % CH;
        const size_t off = (((size_t)b * n + j) * H + h) * DK + part * 8;
        *reinterpret_cast<uint4 *>(fk + off) = *reinterpret_cast<const uint4 *>(k + off);
      }
      if (tid < n) {
        const size_t s = ((size_t)b * n + tid) * H + h;
        a.falpha[s] = a.alpha[s];
        if (h == 0) a.fparent[(size_t)b * n + tid] = a.parent[(size_t)b * n + tid];
      }
    }
  }

  // values of the nodes this lane solves for (accumulator rows 4*lg + r)
  float vreg[NT][4];
  if (cols_live) {
    const bf16 *v = static_cast<const bf16 *>(a.v);
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = mt * 16 + 4 * lg + r;
        vreg[mt][r] = j < n ? to_f32(v[(((size_t)b * n + j) * H + h) * dv + col]) : 0.f;
      }
  }

  // 4. Delayed state update on the registers, write-back, hi/lo split.
  bf16x8 bhi[KS], blo[KS];
  if (cols_live) {
    if (a.has_pending) {
      const bf16 *pk = static_cast<const bf16 *>(a.pend.k);
      const int pn = a.pend.n;
      const int plen = a.pend.len[b];
      for (int t = 0; t < plen; ++t) {
        const int node = a.pend.path[(size_t)b * pn + t];
        const size_t s = ((size_t)b * pn + node) * H + h;
        const float al = a.pend.alpha[s];
        const float u = a.pend.u[s * dv + col];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          float kr[8];
          load_f32<8>(pk + s * DK + ks * 32 + 8 * lg, kr);
#pragma unroll
          for (int e = 0; e < 8; ++e) hf[ks][e] = apply_factor(hf[ks][e], al, kr[e], u);
        }
      }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) st[(size_t)(ks * 32 + 8 * lg + e) * dv] = hf[ks][e];
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) bhi[ks] = pack_hi_lo(hf[ks], blo[ks]);
  }
  __syncthreads();  // [Q; K] staged

  // 5. Matrix cores: P = [Q; K] H0 for this wave's 16 columns.
  f32x4 pacc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) pacc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (cols_live) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if ((mt % NT) * 16 >= n) continue;  // rows of padding only
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 af = *reinterpret_cast<const bf16x8 *>(xs + (mt * 16 + lc) * L::XP + ks * 32 + 8 * lg);
        pacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bhi[ks], pacc[mt], 0, 0, 0);
        pacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, blo[ks], pacc[mt], 0, 0, 0);
      }
    }
  }

  // 6. Tree-masked Grams: tiles (row tile mr of [Q; K], node tile na) that
  //    contain an ancestor pair, spread over the waves; each lane scatters
  //    its ancestor entries into the per-node compact lists.
  {
    int tcount = 0;
    for (int mr = 0; mr < MT; ++mr) {
      const int jt = mr % NT;
      if (jt * 16 >= n) continue;
      for (int na = 0; na <= jt; ++na, ++tcount) {
        if (tcount % kWaves != w) continue;
        f32x4 g = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 af = *reinterpret_cast<const bf16x8 *>(xs + (mr * 16 + lc) * L::XP + ks * 32 + 8 * lg);
          const bf16x8 bf =
              *reinterpret_cast<const bf16x8 *>(xs + (NP + na * 16 + lc) * L::XP + ks * 32 + 8 * lg);
          g = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bf, g, 0, 0, 0);
        }
        const int an = na * 16 + lc;  // ancestor candidate (column of the tile)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = jt * 16 + 4 * lg + r;
          if (j >= n || an > j) continue;
          const uint64_t m = s_anc[j];
          if (!((m >> an) & 1ull)) continue;
          const int rank = __popcll(m & ((1ull << an) - 1ull));
          const float dja = s_gamma[j] / s_gamma[an];
          if (mr < NT) {
            lq[s_off[j] + rank] = dja * g[r];
          } else if (an < j) {
            lk[s_off[j] + rank] = s_be[j] * dja * g[r];
          }
        }
      }
    }
  }
  __syncthreads();  // compact lists complete

  // 7. Level-synchronous solve for the corrected values u (accumulator rows
  //    of the K half), written to LDS and to the factor store.
  const size_t obase = (size_t)b * n;
  const int ucol = w * kWaveCols + lc;
  for (int d = 1; d <= maxd; ++d) {
    if (cols_live) {
#pragma unroll
      for (int mt = 0; mt < NT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = mt * 16 + 4 * lg + r;
          if (j >= n || s_depth[j] != d) continue;
          const float gj = s_gamma[j], bj = s_be[j];
          float s = bj * (vreg[mt][r] - gj * pacc[NT + mt][r]);
          uint64_t m = s_anc[j] & ~(1ull << j);
          const float *lkj = lk + s_off[j];
          int idx = 0;
          while (m) {
            const int an = __builtin_ctzll(m);
            m &= m - 1ull;
            s -= lkj[idx++] * us[an * kUPitch + ucol];
          }
          us[j * kUPitch + ucol] = s;
          a.fu[((obase + j) * H + h) * dv + col] = s;
        }
    }
    __syncthreads();
  }

  // 8. Masked readout o_j = gamma_j q_j^T H0 + sum_{a in P(j)} D_ja (q_j.k_a) u_a.
  if (cols_live) {
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = mt * 16 + 4 * lg + r;
        if (j >= n) continue;
        float o = s_gamma[j] * pacc[mt][r];
        uint64_t m = s_anc[j];
        const float *lqj = lq + s_off[j];
        int idx = 0;
        while (m) {
          const int an = __builtin_ctzll(m);
          m &= m - 1ull;
          o = __builtin_fmaf(lqj[idx++], us[an * kUPitch + ucol], o);
        }
        a.out[((obase + j) * H + h) * dv + col] = o;
      }
  }
}

constexpr size_t kMaxLds = 160 * 1024;
constexpr size_t kDefaultLds = 64 * 1024;

template <int DK, int NP>
hipError_t launch_np(const VerifyArgs &a, hipStream_t s) {
  const size_t lds = Lds<DK, NP>::kBytes;
  if (lds > kMaxLds) return hipErrorInvalidConfiguration;
  auto kern = verify_parallel_kernel<DK, NP>;
  if (lds > kDefaultLds) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int ntiles = (a.dv + kTileCols - 1) / kTileCols;
  const dim3 grid((unsigned)((size_t)a.B * a.H * ntiles));
  hipLaunchKernelGGL(kern, grid, dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

template <int DK>
hipError_t launch_dk(const VerifyArgs &a, hipStream_t s) {
  if (a.n <= 16) return launch_np<DK, 16>(a, s);
  if (a.n <= 32) return launch_np<DK, 32>(a, s);
  return launch_np<DK, 64>(a, s);
}

}  // namespace

bool parallel_supported(int dk, int dv, int n, int dtype) {
  // The hi/lo split contraction relies on q and k being exact in bf16.
  return dtype == SLA_DTYPE_BF16 && (dk == 64 || dk == 128 || dk == 256) && dv % 16 == 0 && n >= 1 &&
         n <= SLA_MAX_NODES;
}

hipError_t launch_verify_parallel(const VerifyArgs &a, int dtype, hipStream_t s) {
  if (dtype != SLA_DTYPE_BF16) return hipErrorInvalidConfiguration;
  switch (a.dk) {
    case 64: return launch_dk<64>(a, s);
    case 128: return launch_dk<128>(a, s);
    case 256: return launch_dk<256>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sla
