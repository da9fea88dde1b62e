// verify_parallel.hip -- tree-masked factorised verification (SpecLA §4.2)
// with the delayed state update of §5.2 fused in front of it.
//
// Unrolling the gated delta rule along a root path gives, for every node j
// (gamma_j = product of alpha over P(j), D_ja = gamma_j / gamma_a, a in P(j)):
//     H_j = gamma_j H0 + sum_{a in P(j)} D_ja k_a u_a^T
//     (I + Lk) U = R,   R_j = beta_j (v_j - gamma_j H0^T k_j),
//                       Lk_ja = beta_j D_ja (k_j . k_a)   for a in P(j), a != j
//     O = Gamma Q H0 + Attn U,   Attn_ja = D_ja (q_j . k_a)   for a in P(j)
// which is the tree-masked UT form: T = (I + Lk)^-1 is the paper's
// T_tree = solve_tril(I - A_tree), and O = Q^ S0^T - Attn W S0^T + Attn U.
// Both per-column products run on the matrix cores:
//     U = T R,      O = Gamma P_q + Attn U,
// and the only sequential work is the small per-unit T (each lane walks its
// own node's root path).  Only the committed state is read.
//
// One workgroup = one (batch b, head h, 64-column V-tile); four wavefronts of
// 16 state columns each.
//   setup   all global reads that do not depend on another read are issued
//           first (state tile, parent row, gates, path row, [Q; K], values);
//           wave 0 builds topology, decays and offsets; wave 1 validates the
//           pending accepted path and stages its factor records in LDS (one
//           more dependent level); waves 2-3 stage [Q; K] in LDS.
//   state   each lane holds 8 consecutive rows of one column per 32-row
//           K-step (the B fragment of v_mfma_f32_16x16x32_bf16), applies the
//           pending path, writes the committed tile back, splits fp32 into
//           bf16 hi + lo.
//   P       [Q; K] H0 on the matrix cores (q, k exact in bf16).
//   Gram    [Q; K] K^T tiles that hold ancestor pairs (exact products); Attn
//           goes to a dense LDS matrix, Lk to per-node compact lists.
//   T       per node along its root path, fp32, into a dense LDS matrix.
//   U, O    v_mfma_f32_16x16x16bf16_1k, whose B fragment is exactly the
//           accumulator layout that holds R (and then U); fp32 operands enter
//           as bf16 hi + lo (three products).
// The state tile and the per-node outputs are streamed once, with
// non-temporal hints.
#include "device.hpp"
#include "kernels.hpp"

namespace sla {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kWaveCols = 16;
constexpr int kTileCols = kWaves * kWaveCols;  // 64 state columns per workgroup
constexpr int kPMax = 8;                       // pending steps staged in LDS

template <int DK, int NP>
struct Lds {
  static constexpr int XP = DK + 8;                  // bf16 row pitch of [Q; K]
  static constexpr int DP = NP + 4;                  // fp32 row pitch of dense T and Attn
  static constexpr int kList = NP * (NP + 1) / 2;    // compact Lk capacity (floats)
  static constexpr int kXBytes = 2 * NP * XP * 2;
  static constexpr int kDenseBytes = 2 * NP * DP * 4;
  static constexpr int kA = kXBytes > kDenseBytes ? kXBytes : kDenseBytes;  // [Q; K], then T and Attn
  static constexpr int kLk = kList * 4;
  static constexpr int kPk = kPMax * DK * 2;          // pending keys (bf16)
  static constexpr int kPu = kPMax * kTileCols * 4;   // pending corrected values of this tile
  static constexpr int kTopo = NP * 8 + NP * 4 * 5 + kPMax * 4 + 16;
  static constexpr int kBytes = kA + kLk + kPk + kPu + kTopo;
};

__device__ __forceinline__ bf16x8 split8(const float (&x)[8], bf16x8 &lo) {
  bf16x8 hi;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 h = static_cast<__bf16>(x[e]);
    hi[e] = h;
    lo[e] = static_cast<__bf16>(x[e] - static_cast<float>(h));
  }
  return hi;
}

__device__ __forceinline__ void split4(f32x4 x, s16x4 &hi, s16x4 &lo) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const __bf16 h = static_cast<__bf16>(x[e]);
    hi[e] = __builtin_bit_cast(short, h);
    lo[e] = __builtin_bit_cast(short, static_cast<__bf16>(x[e] - static_cast<float>(h)));
  }
}

__device__ __forceinline__ f32x4 mfma16(s16x4 a, s16x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// acc += A B with A and B fp32 given as hi + lo (the lo * lo term is below
// fp32 resolution and dropped).
__device__ __forceinline__ f32x4 mfma16_split(s16x4 ah, s16x4 al, s16x4 bh, s16x4 bl, f32x4 acc) {
  acc = mfma16(ah, bh, acc);
  acc = mfma16(ah, bl, acc);
  return mfma16(al, bh, acc);
}

template <int DK, int NP>
__global__ __launch_bounds__(kThreads) void verify_parallel_kernel(VerifyArgs a) {
  constexpr int KS = DK / 32;  // K-steps of the contraction over d_k
  constexpr int NT = NP / 16;  // 16-node tiles
  constexpr int MT = 2 * NT;   // 16-row tiles of [Q; K]
  constexpr int CH = DK / 8;   // 16-byte chunks per [Q; K] row
  constexpr int GT = (NT * (NT + 1) + kWaves - 1) / kWaves;  // Gram tiles per wave
  using L = Lds<DK, NP>;

  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  __bf16 *xs = reinterpret_cast<__bf16 *>(lds);                  // [2NP][XP] until the Grams are done
  float *tdn = reinterpret_cast<float *>(lds);                   // [NP][DP] T, afterwards
  float *adn = tdn + NP * L::DP;                                 // [NP][DP] Attn, afterwards
  float *lk = reinterpret_cast<float *>(lds + L::kA);            // compact Lk
  __bf16 *s_pk = reinterpret_cast<__bf16 *>(lds + L::kA + L::kLk);          // [kPMax][DK]
  float *s_pu = reinterpret_cast<float *>(lds + L::kA + L::kLk + L::kPk);   // [kPMax][64]
  unsigned char *tp = lds + L::kA + L::kLk + L::kPk + L::kPu;
  uint64_t *s_anc = reinterpret_cast<uint64_t *>(tp);      // [NP]
  int *s_depth = reinterpret_cast<int *>(tp + 8 * NP);     // [NP]
  int *s_off = s_depth + NP;                                // [NP]
  float *s_gamma = reinterpret_cast<float *>(s_off + NP);  // [NP]
  float *s_rgamma = s_gamma + NP;                           // [NP] 1 / gamma
  float *s_be = s_rgamma + NP;                              // [NP]
  float *s_palpha = s_be + NP;                              // [kPMax]
  int *s_misc = reinterpret_cast<int *>(s_palpha + kPMax);  // topo err, path err, path len

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int lc = l & 15;  // column within the wave's 16 / row within a 16-row tile
  const int lg = l >> 4;  // row group
  const int H = a.H, dv = a.dv, n = a.n;
  const int ntiles = (dv + kTileCols - 1) / kTileCols;
  int wid = blockIdx.x;
  const int tile = wid % ntiles;
  wid /= ntiles;
  const int h = wid % H;
  const int b = wid / H;
  const int ucol = w * kWaveCols + lc;  // column within the tile
  const int col = tile * kTileCols + ucol;
  const bool cols_live = tile * kTileCols + w * kWaveCols < dv;  // wave-uniform
  const size_t unit = (size_t)b * H + h;
  const size_t nbase = (size_t)b * n;
  const bf16 *qg = static_cast<const bf16 *>(a.q);
  const bf16 *kg = static_cast<const bf16 *>(a.k);
  const bf16 *vg = static_cast<const bf16 *>(a.v);

  // ---- reads with no dependence on other reads: the state tile (the only
  //      state read) and the values of the nodes this lane solves for
  float *st = a.state + unit * DK * dv + col;
  float hf[KS][8];
  float vreg[NT][4];
  if (cols_live) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) hf[ks][e] = __builtin_nontemporal_load(st + (size_t)(ks * 32 + 8 * lg + e) * dv);
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = mt * 16 + 4 * lg + r;
        vreg[mt][r] = j < n ? to_f32(vg[((nbase + j) * H + h) * dv + col]) : 0.f;
      }
  }

  // ---- setup, one job per wavefront
  if (w == 0) {
    // topology, decays and compact-list offsets; lane j owns node j
    const bool live = l < n;
    const size_t s = (nbase + (live ? l : 0)) * H + h;
    const int p = live ? a.parent[nbase + l] : -1;
    const float al = live ? a.alpha[s] : 1.f;
    const float be = live ? a.beta[s] : 0.f;
    bool bad = live && (p < -1 || p >= l);
    if (a.chain) bad = bad || (live && p != l - 1);
    const int err = wave_any(bad) ? SLA_ERR_TOPOLOGY : SLA_OK;
    if (err == SLA_OK) {
      uint64_t m = live ? (1ull << l) : 0ull;
      float g = al;
      int d = live ? 1 : 0;
      int x = p;
      while (wave_any(x >= 0)) {
        const int src = x >= 0 ? x : 0;
        const float ax = __shfl(al, src);
        const int px = __shfl(p, src);
        if (x >= 0) {
          m |= 1ull << x;
          g *= ax;
          ++d;
        }
        x = x >= 0 ? px : -1;
      }
      int incl = d;  // inclusive prefix sum of depths -> compact-list offsets
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (l >= o) incl += y;
      }
      if (live) {
        s_anc[l] = m;
        s_depth[l] = d;
        s_off[l] = incl - d;
        s_gamma[l] = g;
        s_rgamma[l] = 1.f / g;
        s_be[l] = be;
      }
    }
    if (l == 0) s_misc[0] = err;
  } else if (w == 1) {
    // pending accepted path: validate and stage its records in LDS.  The
    // path row and its length are read together; the records they name are
    // the one dependent level.
    int perr = SLA_OK, plen = 0;
    if (a.has_pending) {
      const int pn = a.pend.n;
      const int32_t *prow = a.pend.path + (size_t)b * pn;
      plen = a.pend.len[b];
      const int node = l < pn ? prow[l] : -1;
      const int prev = l == 0 ? -1 : (l - 1 < pn ? prow[l - 1] : -1);
      const bool step = l < plen;
      const bool inrange = node >= 0 && node < pn;
      const int ppar = (step && inrange) ? a.pend.parent[(size_t)b * pn + node] : -2;
      const bool bad = (plen < 0 || plen > pn) || (step && (!inrange || ppar != prev));
      perr = wave_any(bad) ? SLA_ERR_PATH : SLA_OK;
      if (perr == SLA_OK) {
        const int ps = plen < kPMax ? plen : kPMax;
        if (l < ps) s_palpha[l] = a.pend.alpha[((size_t)b * pn + node) * H + h];
        const bf16 *pk = static_cast<const bf16 *>(a.pend.k);
        const int iters = (ps * CH + kWave - 1) / kWave;
        for (int it = 0; it < iters; ++it) {
          const int c = l + it * kWave;
          const int t = c / CH, part = c % CH;
          const int nt = __shfl(node, t < ps ? t : 0);
          if (c < ps * CH)
            *reinterpret_cast<uint4 *>(s_pk + t * DK + part * 8) =
                *reinterpret_cast<const uint4 *>(pk + (((size_t)b * pn + nt) * H + h) * DK + part * 8);
        }
        const int cg = tile * kTileCols + l;
        for (int t = 0; t < ps; ++t) {
          const int nt = __builtin_amdgcn_readlane(node, t);
          s_pu[t * kTileCols + l] = cg < dv ? a.pend.u[(((size_t)b * pn + nt) * H + h) * dv + cg] : 0.f;
        }
      }
    }
    if (l == 0) {
      s_misc[1] = perr;
      s_misc[2] = plen;
    }
  } else {
    // [Q; K]: rows 0..NP-1 hold q_j, rows NP..2NP-1 hold k_j; zero padding
    for (int c = tid - 2 * kWave; c < 2 * NP * CH; c += 2 * kWave) {
      const int row = c / CH, part = c % CH;
      const int j = row % NP;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (j < n) val = *reinterpret_cast<const uint4 *>((row < NP ? qg : kg) + ((nbase + j) * H + h) * DK + part * 8);
      *reinterpret_cast<uint4 *>(xs + row * L::XP + part * 8) = val;
    }
  }
  __syncthreads();
  const int err = s_misc[0] != SLA_OK ? s_misc[0] : s_misc[1];
  if (tile == 0 && h == 0 && tid == 0 && a.status) a.status[b] = err;
  if (err != SLA_OK) return;
  const int plen = s_misc[2];

  // ---- factor records that do not depend on the V-tile
  if (tile == 0) {
    bf16 *fk = static_cast<bf16 *>(a.fk);
    for (int c = tid; c < n * CH; c += kThreads) {
      const int j = c / CH, part = c % CH;
      *reinterpret_cast<uint4 *>(fk + ((nbase + j) * H + h) * DK + part * 8) =
          *reinterpret_cast<const uint4 *>(xs + (NP + j) * L::XP + part * 8);
    }
    if (tid < n) {
      const size_t s = (nbase + tid) * H + h;
      a.falpha[s] = a.alpha[s];
      if (h == 0) a.fparent[nbase + tid] = a.parent[nbase + tid];
    }
  }

  // ---- delayed state update on the registers, write-back, hi/lo split
  bf16x8 bhi[KS], blo[KS];
  if (cols_live) {
    if (a.has_pending) {
      const int ps = plen < kPMax ? plen : kPMax;
      for (int t = 0; t < ps; ++t) {
        const float al = s_palpha[t];
        const float u = s_pu[t * kTileCols + ucol];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 kv = *reinterpret_cast<const bf16x8 *>(s_pk + t * DK + ks * 32 + 8 * lg);
#pragma unroll
          for (int e = 0; e < 8; ++e) hf[ks][e] = apply_factor(hf[ks][e], al, static_cast<float>(kv[e]), u);
        }
      }
      // paths longer than the LDS stage read their records directly
      const bf16 *pk = static_cast<const bf16 *>(a.pend.k);
      const int pn = a.pend.n;
      for (int t = kPMax; t < plen; ++t) {
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
        for (int e = 0; e < 8; ++e) __builtin_nontemporal_store(hf[ks][e], st + (size_t)(ks * 32 + 8 * lg + e) * dv);
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) bhi[ks] = split8(hf[ks], blo[ks]);
  }

  // ---- P = [Q; K] H0 for this wave's 16 columns (accumulator layout: lane
  //      (lg, lc) holds rows 4 lg .. 4 lg + 3 of each 16-row tile, column lc)
  f32x4 pacc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) pacc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (cols_live) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if ((mt % NT) * 16 >= n) continue;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 af = *reinterpret_cast<const bf16x8 *>(xs + (mt * 16 + lc) * L::XP + ks * 32 + 8 * lg);
        pacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bhi[ks], pacc[mt], 0, 0, 0);
        pacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, blo[ks], pacc[mt], 0, 0, 0);
      }
    }
  }

  // ---- tree-masked Grams: tile (mr, na) of [Q; K] K^T holds rows of node
  //      tile jt = mr % NT against ancestor candidates of node tile na <= jt
  f32x4 gacc[GT];
#pragma unroll
  for (int i = 0; i < GT; ++i) gacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  {
    int tc = 0;
#pragma unroll
    for (int mr = 0; mr < MT; ++mr)
#pragma unroll
      for (int na = 0; na <= mr % NT; ++na, ++tc) {
        if (tc % kWaves != w || (mr % NT) * 16 >= n) continue;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 af = *reinterpret_cast<const bf16x8 *>(xs + (mr * 16 + lc) * L::XP + ks * 32 + 8 * lg);
          const bf16x8 bf =
              *reinterpret_cast<const bf16x8 *>(xs + (NP + na * 16 + lc) * L::XP + ks * 32 + 8 * lg);
          gacc[tc / kWaves] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bf, gacc[tc / kWaves], 0, 0, 0);
        }
      }
  }
  __syncthreads();  // [Q; K] is dead from here on; its space holds T and Attn

  // ---- zero the dense T and Attn (rows of padding nodes stay zero)
  for (int c = tid; c < 2 * NP * L::DP / 4; c += kThreads)
    reinterpret_cast<float4 *>(tdn)[c] = make_float4(0.f, 0.f, 0.f, 0.f);

  // ---- R = beta (v - gamma P_k) in the accumulator layout
  f32x4 rreg[NT];
#pragma unroll
  for (int mt = 0; mt < NT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = mt * 16 + 4 * lg + r;
      rreg[mt][r] = (cols_live && j < n) ? s_be[j] * (vreg[mt][r] - s_gamma[j] * pacc[NT + mt][r]) : 0.f;
    }
  __syncthreads();

  // ---- scatter ancestor entries of the Grams: Attn into its dense matrix,
  //      Lk into the compact list of node j at off_j + depth(a) - 1
  {
    int tc = 0;
#pragma unroll
    for (int mr = 0; mr < MT; ++mr)
#pragma unroll
      for (int na = 0; na <= mr % NT; ++na, ++tc) {
        if (tc % kWaves != w || (mr % NT) * 16 >= n) continue;
        const int an = na * 16 + lc;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = (mr % NT) * 16 + 4 * lg + r;
          if (j >= n || an > j) continue;
          if (!((s_anc[j] >> an) & 1ull)) continue;
          const float dg = s_gamma[j] * s_rgamma[an] * gacc[tc / kWaves][r];
          if (mr < NT)
            adn[j * L::DP + an] = dg;
          else if (an < j)
            lk[s_off[j] + s_depth[an] - 1] = s_be[j] * dg;
        }
      }
  }
  __syncthreads();

  // ---- T = (I + Lk)^-1, row j along P(j), deepest ancestor first:
  //      T_jj = 1,  T_ja = - sum_{e in P(j), a < e} T_je Lk_ea
  if (tid < n) {
    const int j = tid;
    const uint64_t m = s_anc[j];
    float *trow = tdn + j * L::DP;
    trow[j] = 1.f;
    uint64_t rest = m & ~(1ull << j);
    while (rest) {
      const int an = 63 - __builtin_clzll(rest);
      rest &= ~(1ull << an);
      const int ta = s_depth[an] - 1;
      uint64_t below = m & ~((2ull << an) - 1ull);
      float s = 0.f;
      while (below) {
        const int e = __builtin_ctzll(below);
        below &= below - 1ull;
        s = __builtin_fmaf(-trow[e], lk[s_off[e] + ta], s);
      }
      trow[an] = s;
    }
  }
  __syncthreads();

  // ---- U = T R, then O = Gamma P_q + Attn U, on the matrix cores; A
  //      fragments are rows j = 16 mt + lc, columns 16 ks + 4 lg .. + 3
  if (!cols_live) return;
  s16x4 rhi[NT], rlo[NT];
#pragma unroll
  for (int mt = 0; mt < NT; ++mt) split4(rreg[mt], rhi[mt], rlo[mt]);
  f32x4 uacc[NT];
#pragma unroll
  for (int mt = 0; mt < NT; ++mt) {
    uacc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (mt * 16 >= n) continue;
#pragma unroll
    for (int ks = 0; ks <= mt; ++ks) {
      const f32x4 tv = *reinterpret_cast<const f32x4 *>(tdn + (mt * 16 + lc) * L::DP + ks * 16 + 4 * lg);
      s16x4 th, tlo;
      split4(tv, th, tlo);
      uacc[mt] = mfma16_split(th, tlo, rhi[ks], rlo[ks], uacc[mt]);
    }
  }
  s16x4 uhi[NT], ulo[NT];
#pragma unroll
  for (int mt = 0; mt < NT; ++mt) split4(uacc[mt], uhi[mt], ulo[mt]);
  f32x4 oacc[NT];
#pragma unroll
  for (int mt = 0; mt < NT; ++mt) {
    oacc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (mt * 16 >= n) continue;
#pragma unroll
    for (int ks = 0; ks <= mt; ++ks) {
      const f32x4 av = *reinterpret_cast<const f32x4 *>(adn + (mt * 16 + lc) * L::DP + ks * 16 + 4 * lg);
      s16x4 ah, alo;
      split4(av, ah, alo);
      oacc[mt] = mfma16_split(ah, alo, uhi[ks], ulo[ks], oacc[mt]);
    }
  }
#pragma unroll
  for (int mt = 0; mt < NT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = mt * 16 + 4 * lg + r;
      if (j >= n) continue;
      const size_t o = ((nbase + j) * H + h) * dv + col;
      __builtin_nontemporal_store(uacc[mt][r], a.fu + o);
      __builtin_nontemporal_store(__builtin_fmaf(s_gamma[j], pacc[mt][r], oacc[mt][r]), a.out + o);
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
