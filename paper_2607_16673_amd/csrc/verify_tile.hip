// verify_tile.hip -- tree-masked factorised verification (SpecLA §4.2) with
// the delayed state update of §5.2 fused in front of it.
//
// Unrolling the gated delta rule along a root path gives, for every node j
// (gamma_j = product of alpha over P(j); for a in P(j), D_ja = product of
// alpha over the nodes of P(j) strictly below a, which equals gamma_j /
// gamma_a but is formed as a product, so no reciprocal of a decay product
// is ever taken and strong decays underflow harmlessly to zero):
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
// One workgroup = one (batch b, head h) unit's V-tile of CW x 16 columns
// (CW = 4 or 8), or TPW = 2 consecutive such tiles, with CW + 1 wavefronts
// (CW = 4) or CW (CW = 8, where column wave 0 also takes the setup work):
//   waves 0 .. CW-1 own 16 state columns each.  They issue the state tile
//              reads (in the B-fragment order of v_mfma_f32_16x16x32_bf16: 8
//              consecutive rows of one column per 32-row K-step) and the
//              value reads first thing.  The state reads and the
//              committed-row writes keep the default cache policy: a wave
//              covers only half of each 128-byte line, and with a streaming
//              hint the L2 lets the line go before the neighbouring wave
//              reads or writes the other half (measured: about 15% more HBM
//              reads, 8% more writes).  Per tile: pending path applied,
//              committed rows written back, fp32 split into bf16 hi + lo,
//              P = [Q; K] H0 accumulated on the matrix cores K-step by
//              K-step.  Then R = beta (v - gamma P_k), U = T R and
//              O = Gamma P_q + Attn U on v_mfma_f32_16x16x16bf16_1k (whose B
//              fragment is exactly the accumulator layout holding R, then U),
//              and the outputs.  With two tiles, the second tile's reads go
//              out once the first tile's registers are free.
//   wave CW    (the setup wave; wave 0 at CW = 8) owns no state of its own.
//              It takes every read that depends on another read or that
//              everything else waits for: parent row and gates -> topology,
//              decays and compact-list offsets; the pending path with the
//              previous round's parent row and gates -> validation; [Q; K] by
//              direct global->LDS loads; then, while the column waves
//              compute, the factor records the path names (also straight
//              into LDS, a second stage for a second tile) and, for two
//              16-node tiles with scalar gates, the second tile's first d_k/2
//              state rows, which would otherwise queue behind the first
//              tile's work (measured at batch 64, 16 heads, d_v 128: 37.8 ->
//              36.9 us per launch).  After the Grams it solves the per-node
//              rows of T.
// The tree-masked Grams ([Q; K] K^T tiles that hold ancestor pairs, exact
// bf16 products) run on the column waves; they and T are done while the
// first tile's state is still in flight.  Strided global accesses go through
// buffer descriptors (one VGPR offset per lane).  With fp32 activations the
// same structure runs every contraction on the fp32 matrix cores (Layout).
#include <type_traits>

#include "device.hpp"
#include "kernels.hpp"

namespace sla {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kWaveCols = 16;                    // state columns per column wave
constexpr int kPMax = 8;                          // pending steps staged in LDS
constexpr int kBP = 20;                           // fp32 row pitch of a 16x16 block
constexpr int kZ = 8;                             // root paths up to this depth solve T in registers

// Layer families by the form of their step (template parameter KIND):
//   kKindDelta  scalar gates: GDN, DeltaNet (alpha = 1) and the scalar decay
//               without the delta rule (beta = 0, so Lk = 0 and T = I, with
//               R = V in place of beta (v - gamma P_k): a run-time choice,
//               so that all three share one register allocation);
//   kKindGates  GLA: one gate per key dimension, no delta rule.  The decay
//               ratios become per-dimension, D_ja[i] (the product of the
//               i-th gates of P(j) strictly below a), so the scores
//               Attn_ja = sum_i q_j[i] D_ja[i] k_a[i] are formed on the
//               vector ALUs by walking each root path, and
//               O = Q~ H0 + Attn V with Q~_j = Gamma_j * q_j (fp32, split
//               into bf16 hi + lo).
constexpr int kKindDelta = 0, kKindGates = 1;

// F32: fp32 activations.  q, k, v and the pending keys are staged and read
// as fp32, and every contraction runs on v_mfma_f32_16x16x4_f32 with exact
// fp32 products (no hi/lo splits); else bf16 activations (16x16x32 bf16 for
// the Grams and P, hi/lo-split 16x16x16 bf16 for T R and Attn U).
template <int DK, int NP, int CW, int TPW, int KIND, bool F32>
struct Layout {
  static constexpr int kTileCols = CW * kWaveCols;
  static constexpr int ES = F32 ? 4 : 2;            // bytes per activation
  static constexpr int NT = NP / 16, KS = DK / 32, CH = DK * ES / 16, MT = 2 * NT;
  static constexpr int NB = NT * (NT + 1) / 2;      // lower-triangular 16x16 blocks
  static constexpr int kList = NP * (NP + 1) / 2;   // compact Lk capacity (floats)
  static constexpr bool kDelta = KIND == kKindDelta, kGates = KIND == kKindGates;
  static constexpr int kX = 2 * NP * CH * 16;       // [Q; K], 16-byte chunks, xor-swizzled
  static constexpr int kBlk = 16 * kBP * 4;
  static constexpr int kT = kDelta ? NB * kBlk : 0;   // T blocks
  static constexpr int kAt = NB * kBlk;             // Attn blocks
  static constexpr int kLk = kDelta ? kList * 4 : 0;
  static constexpr int kPk = kPMax * DK * ES;       // pending keys (activation dtype)
  static constexpr int kPu = TPW * kPMax * kTileCols * 4;  // pending corrected values, one stage per tile
  static constexpr int kXL = (kGates && !F32) ? kX / 2 : 0;  // low halves of Q~, same chunk layout
  static constexpr int kG = kGates ? NP * DK * 4 : 0;      // the draft's per-key gates
  static constexpr int kPg = kGates ? kPMax * DK * 4 : 0;  // pending per-key gates
  // small trees, two 64-column tiles: the second tile's first DK/2 state rows
  // are staged in LDS ahead of time (16-byte chunks, swizzled: see kernel).
  // Not for GLA: its gate stages already take 37 KB at d_k 128, and 16 KB
  // more would leave three resident workgroups per CU instead of four
  // (measured 40.1 -> 43.4 us per launch at batch 64, 16 heads).
  static constexpr bool kPrefetch = TPW == 2 && NP == 16 && CW == 4 && kDelta;
  static constexpr int kPreInstr = kPrefetch ? (DK / 2) * (kTileCols / 4) / kWave : 0;  // 16-byte loads per lane
  static constexpr int kPre = kPreInstr * kWave * 16;
  static constexpr int kTopo = NP * 8 + NP * 4 * 4 + kPMax * 4 + 16;
  static constexpr int oT = kX, oAt = oT + kT, oLk = oAt + kAt, oPk = oLk + kLk, oPu = oPk + kPk;
  static constexpr int oXL = oPu + kPu, oG = oXL + kXL, oPg = oG + kG, oPre = oPg + kPg, oTopo = oPre + kPre;
  static constexpr int kBytes = oTopo + kTopo;
};

// [Q; K] chunk (row, c) lives at row * CH + (c ^ (row & 7)): the 16 rows a
// fragment read touches fall on distinct bank groups.
template <int CH>
__device__ __forceinline__ int xchunk(int row, int c) {
  return row * CH + (c ^ (row & 7));
}

// s_waitcnt immediate that waits until at most `n` vector memory operations
// of this wave are outstanding (export and LDS counters unconstrained).
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// element (row j, column a), a <= j, of a lower-triangular 16x16-blocked matrix
__device__ __forceinline__ int blk(int j, int a) {
  const int bj = j >> 4;
  return ((bj * (bj + 1)) / 2 + (a >> 4)) * (16 * kBP) + (j & 15) * kBP + (a & 15);
}

__device__ __forceinline__ void split8(const float (&x)[8], bf16x8 &hi, bf16x8 &lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 h = static_cast<__bf16>(x[e]);
    hi[e] = h;
    lo[e] = static_cast<__bf16>(x[e] - static_cast<float>(h));
  }
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

// Waves per SIMD the register allocation is held to: 6 (80 VGPRs) where the
// tile state, accumulators and LDS allow a fourth resident workgroup per CU;
// 4 (128 VGPRs) for the eight-wave form, so that two workgroups fit a CU;
// else whatever the allocation needs.
template <int DK, int NP, int CW, bool F32>
constexpr int kMinWaves = F32 ? 1 : ((DK <= 128 && NP <= 16) ? 6 : (CW == 8 ? 4 : 1));

// KIND: the family's form (see Layout).  Without the delta rule Lk = 0, so
// T = I and U = R = V: no P_k, no Lk, no T.  WT: committed rows written
// through at device scope (launches of one full round of workgroups).
// eight column waves: column wave 0 also does the setup work, so that the
// workgroup is eight waves and two fit a CU at 124 VGPRs (a ninth wave keeps
// it to one: measured on 64-node trees at batch 64, d_v 256, 459 -> 448 us per
// launch; its state reads then go out after its record gathers)
template <int CW>
constexpr int kWaves = CW == 8 ? CW : CW + 1;

template <int DK, int NP, int CW, int TPW, int KIND, bool F32, bool WT>
__global__ __launch_bounds__(kWaves<CW> * kWave) __attribute__((amdgpu_waves_per_eu(kMinWaves<DK, NP, CW, F32>)))
void verify_tile_kernel(VerifyArgs a) {
  using L = Layout<DK, NP, CW, TPW, KIND, F32>;
  using AT = std::conditional_t<F32, float, bf16>;  // activation element
  constexpr int ES = L::ES;
  constexpr int EC = 16 / ES;  // activations per 16-byte chunk
  constexpr bool DELTA = KIND == kKindDelta;
  constexpr bool GV = KIND == kKindGates;
  const bool nodelta = !DELTA || a.family == SLA_FAMILY_DECAY;  // R = V
  constexpr int kColWaves = CW;                 // waves 0 .. CW-1 own state columns
  constexpr int kSetup = kWaves<CW> == CW ? 0 : CW;  // the setup wave
  constexpr int kTileCols = L::kTileCols;       // state columns per workgroup
  constexpr int KS = L::KS, NT = L::NT, MT = L::MT, CH = L::CH;
  constexpr int NGT = NT * (NT + 1);                        // Gram tiles (both halves)
  constexpr int GT = (NGT + kColWaves - 1) / kColWaves;     // Gram tiles per column wave

  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint4 *xs = reinterpret_cast<uint4 *>(lds);                 // [Q; K] (GLA: high halves of Q~ in place of Q)
  float *tb = reinterpret_cast<float *>(lds + L::oT);         // T blocks
  float *ab = reinterpret_cast<float *>(lds + L::oAt);        // Attn blocks
  float *lk = reinterpret_cast<float *>(lds + L::oLk);        // compact Lk
  AT *s_pk = reinterpret_cast<AT *>(lds + L::oPk);            // [kPMax][DK]
  float *s_pu = reinterpret_cast<float *>(lds + L::oPu);      // [kPMax][64]
  uint4 *xl = reinterpret_cast<uint4 *>(lds + L::oXL);        // GLA: low halves of Q~
  float *s_g = reinterpret_cast<float *>(lds + L::oG);        // GLA: [NP][DK] gates
  float *s_pg = reinterpret_cast<float *>(lds + L::oPg);      // GLA: [kPMax][DK] pending gates
  float *s_pre = reinterpret_cast<float *>(lds + L::oPre);    // second tile's first DK/2 state rows
  unsigned char *tp = lds + L::oTopo;
  uint64_t *s_anc = reinterpret_cast<uint64_t *>(tp);      // [NP]
  int *s_depth = reinterpret_cast<int *>(tp + 8 * NP);     // [NP]
  int *s_off = s_depth + NP;                                // [NP]
  float *s_gamma = reinterpret_cast<float *>(s_off + NP);  // [NP]
  float *s_be = s_gamma + NP;                               // [NP]
  float *s_palpha = s_be + NP;                              // [kPMax]
  int *s_misc = reinterpret_cast<int *>(s_palpha + kPMax);  // err, path len

  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int l = tid % kWave;
  const int lc = l & 15;  // column within a wave's 16 / row within a 16-row tile
  const int lg = l >> 4;  // row group
  const int H = a.H, dv = a.dv, n = a.n;
  // this workgroup: unit (b, h), V-tiles t0 .. t0 + cnt - 1
  const int ntiles = (dv + kTileCols - 1) / kTileCols;
  const int ngroups = (ntiles + TPW - 1) / TPW;
  int wid = blockIdx.x;
  const int t0 = (wid % ngroups) * TPW;
  wid /= ngroups;
  const int cnt = TPW;  // TPW divides the tile count (the launcher checks)
  const int h = wid % H;
  const int b = wid / H;
  const int ucol = w * kWaveCols + lc;  // column within a tile
  const size_t unit = (size_t)b * H + h;
  const size_t nbase = (size_t)b * n;
  const rsrc_t sr = make_rsrc(a.state + unit * DK * dv, (uint32_t)DK * dv * 4);
  const uint32_t nstride = (uint32_t)H * dv;  // elements between consecutive nodes of a unit
  const rsrc_t vr = make_rsrc(static_cast<const AT *>(a.v) + (nbase * H + h) * dv,
                              ((uint32_t)(n - 1) * nstride + dv) * ES);
  // wave-uniform: this wave owns columns of tile t
  auto live = [&](int t) { return w < kColWaves && t * kTileCols + w * kWaveCols < dv; };
  // state rows 8 lg + e + 32 ks of column t * kTileCols + ucol, in B-fragment order
  auto load_state = [&](int t, float (&hf)[KS][8], int ks0 = 0) {
    const uint32_t sv = (uint32_t)(8 * lg * dv + t * kTileCols + ucol) * 4;
#pragma unroll
    for (int ks = ks0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) hf[ks][e] = buf_load_f32<kPolicyDefault>(sr, sv, (uint32_t)(ks * 32 + e) * dv * 4);
  };
  // values of node j = 16 mt + 4 lg + q; rows past the last node fall
  // outside the descriptor and read zero
  auto load_values = [&](int t, uint32_t (&vraw)[NT][4]) {
    const uint32_t vv = (4 * lg * nstride + t * kTileCols + ucol) * ES;
#pragma unroll
    for (int mt = 0; mt < NT; ++mt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t o = vv + (uint32_t)(mt * 16 + q) * nstride * ES;
        if constexpr (F32)
          vraw[mt][q] = __builtin_amdgcn_raw_buffer_load_b32(vr, o, 0, kPolicyDefault);
        else
          vraw[mt][q] = __builtin_amdgcn_raw_buffer_load_b16(vr, o, 0, kPolicyDefault);
      }
  };

  // fp32 activations: the eight values k = 32 ks + 8 lg + e (e = 0..7) of
  // stage row `row`, the A operand of v_mfma_f32_16x16x4_f32 number e of
  // K-step ks, whose K index lg then pairs with state row 32 ks + 8 lg + e
  // (exactly what a column wave's state registers hold as B operands)
  auto frag8 = [&](int row, int ks, float (&x)[8]) {
    const float4 u0 = *reinterpret_cast<const float4 *>(xs + xchunk<CH>(row, 8 * ks + 2 * lg));
    const float4 u1 = *reinterpret_cast<const float4 *>(xs + xchunk<CH>(row, 8 * ks + 2 * lg + 1));
    x[0] = u0.x, x[1] = u0.y, x[2] = u0.z, x[3] = u0.w, x[4] = u1.x, x[5] = u1.y, x[6] = u1.z, x[7] = u1.w;
  };

  // ---- column waves: the first tile's state and values, issued first
  float hfa[KS][8], hfb[KS][8];  // hfb: the next tile's state (prefetching form only)
  uint32_t vraw[NT][4];  // activation bit patterns, widened where they are used
  if (live(t0)) {
    // a full round of workgroups: hold the state reads back about two
    // microseconds (80 x 64 cycles), so that every workgroup's setup reads
    // and [Q; K] enter the memory queue ahead of the state (measured per
    // launch against no delay: 20 -> +1.6%, 40 -> -1.0%, 64 -> -1.7%,
    // 80 -> -2.1%, 100 -> -1.7%)
    if (a.stagger && w != kSetup) __builtin_amdgcn_s_sleep(80);
    if (!a.late_state) load_state(t0, hfa);
    load_values(t0, vraw);
  }

  // ---- setup wave: everything that depends on another read
  int p = -1;      // setup wave, lane j: parent of node j
  float al = 1.f;  // setup wave, lane j: alpha_j
  int nodec = 0;   // setup wave, lane t: node of pending step t (clamped into the store)
  int maxd = 0;    // setup wave: the deepest root path (wave-uniform)
  if (w == kSetup) {
    for (int c = l; c < (L::kT + L::kAt) / 16; c += kWave) reinterpret_cast<uint4 *>(tb)[c] = make_uint4(0, 0, 0, 0);
    const AT *qg = static_cast<const AT *>(a.q);
    const AT *kg = static_cast<const AT *>(a.k);
    const bool live = l < n;
    const size_t s = (nbase + (live ? l : 0)) * H + h;
    p = live ? a.parent[nbase + l] : -1;
    // DeltaNet: no decay; GLA: the per-key gates enter through Q~ and Attn
    al = (!GV && live && a.family != SLA_FAMILY_DELTANET) ? a.alpha[s] : 1.f;
    const float be = (DELTA && live && a.family != SLA_FAMILY_DECAY) ? a.beta[s] : 0.f;
    // pending accepted path, with the previous round's parent row and gates
    // read whole, so that validating the path waits on no further read
    int plen = 0, node = -1, prow_parent = -2;
    float prow_alpha = 0.f;
    const int pn = a.has_pending ? a.pend.n : 1;
    const size_t prow = (size_t)b * pn;
    if (a.has_pending) {
      plen = a.pend.len[b];
      node = l < pn ? a.pend.path[prow + l] : -1;
      prow_parent = l < pn ? a.pend.parent[prow + l] : -2;
      prow_alpha = (!GV && l < pn) ? a.pend.alpha[(prow + l) * H + h] : 0.f;
    }
    // [Q; K] straight into LDS (rows 0..NP-1: q_j, NP..2NP-1: k_j; padding
    // rows repeat node 0 and are never used)
#pragma unroll 1
    for (int i = 0; i < 2 * NP * CH / kWave; ++i) {
      const int P = i * kWave + l;
      const int row = P / CH, c = (P % CH) ^ (row & 7);
      const int j = row % NP;
      load_lds16((row < NP ? qg : kg) + ((nbase + (j < n ? j : 0)) * H + h) * DK + c * EC, xs + i * kWave);
    }
    if constexpr (GV) {  // the draft's per-key gates, rows 0..NP-1 (padding rows repeat node 0)
      constexpr int GC = DK / 4;  // 16-byte chunks per gate row
#pragma unroll 1
      for (int i = 0; i < NP * GC / kWave; ++i) {
        const int P = i * kWave + l;
        const int j = P / GC;
        load_lds16(a.alpha + ((nbase + (j < n ? j : 0)) * H + h) * DK + (P % GC) * 4, s_g + i * kWave * 4);
      }
    }

    // topology, decays and compact-list offsets; lane j owns node j
    bool bad = live && (p < -1 || p >= l);
    if (a.chain) bad = bad || (live && p != l - 1);
    int err = wave_any(bad) ? SLA_ERR_TOPOLOGY : SLA_OK;
    if (err == SLA_OK) {
      // Walking up from j, g holds D_jx = product of the gates of P(j)
      // strictly below x (j included) when the walk reaches ancestor x; the
      // scalar families park it in the (not yet used) T block at (j, x) for
      // the Grams.  Only products of gates: they may underflow, never
      // overflow (no reciprocal of a decay product anywhere).
      uint64_t m = live ? (1ull << l) : 0ull;
      float g = al;
      int d = live ? 1 : 0;
      int x = p;
      if (DELTA && live) tb[blk(l, l)] = 1.f;
      while (wave_any(x >= 0)) {
        const int src = x >= 0 ? x : 0;
        const float ax = __shfl(al, src);
        const int px = __shfl(p, src);
        if (x >= 0) {
          if constexpr (DELTA) tb[blk(l, x)] = g;
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
      maxd = d;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) maxd = max(maxd, __shfl_xor(maxd, o));
      if (live) {
        s_anc[l] = m;
        s_depth[l] = d;
        s_off[l] = incl - d;
        s_gamma[l] = g;
        s_be[l] = be;
      }
    }
    // the path: step t is node path[t], whose parent must be path[t - 1]
    // (-1 for t = 0)
    const bool inrange = node >= 0 && node < pn;
    nodec = inrange ? node : 0;
    if (err == SLA_OK && a.has_pending) {
      int prev = __shfl_up(node, 1);
      if (l == 0) prev = -1;
      const int ppar = __shfl(prow_parent, nodec);
      const float pal = __shfl(prow_alpha, nodec);
      const bool step = l < plen;
      const bool pbad = (plen < 0 || plen > pn) || (step && (!inrange || ppar != prev));
      err = wave_any(pbad) ? SLA_ERR_PATH : SLA_OK;
      if (l < kPMax) s_palpha[l] = l < plen ? pal : 0.f;
    }
    if (l == 0) {
      s_misc[0] = err;
      s_misc[1] = plen;
      s_misc[2] = maxd;
    }
    if (t0 == 0 && h == 0 && l == 0 && a.status) a.status[b] = err;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // [Q; K] has landed
  }
  __syncthreads();
  const int err = s_misc[0];
  if (err != SLA_OK) return;
  // many rounds of workgroups: the state goes out only now, behind the small
  // reads the setup wave waits for
  if (kSetup != 0 && a.late_state && live(t0)) load_state(t0, hfa);
  const int plen = s_misc[1];

  // ---- setup wave: records of the first kPMax path nodes, gathered straight
  //      into LDS while the column waves compute; a gather is the wave's
  //      only LDS write until the next barrier, which waits for it
  const size_t prow = (size_t)b * (a.has_pending ? a.pend.n : 1);
  // corrected values of tile t (its columns) into stage buffer `buf`
  auto gather_u = [&](int t, int buf) {
#pragma unroll
    for (int st = 0; st < kPMax; ++st) {
      const int ntt = __builtin_amdgcn_readlane(nodec, st);
#pragma unroll
      for (int c0 = 0; c0 < kTileCols; c0 += kWave) {
        const int cg = t * kTileCols + c0 + l;
        load_lds4(a.pend.u + ((prow + ntt) * H + h) * dv + (cg < dv ? cg : dv - 1),
                  s_pu + (buf * kPMax + st) * kTileCols + c0);
      }
    }
  };
  if (w == kSetup && a.has_pending) {
    const AT *pkg = static_cast<const AT *>(a.pend.k);
    constexpr int KI = kPMax * CH / kWave;
    constexpr int GC = DK / 4;                             // 16-byte chunks per gate row
    constexpr int GI = GV ? kPMax * GC / kWave : 0;
    int nt[KI], ng[GI > 0 ? GI : 1];  // node of the step whose key (gate) chunk this lane gathers
#pragma unroll
    for (int i = 0; i < KI; ++i) nt[i] = __shfl(nodec, (i * kWave + l) / CH);
#pragma unroll
    for (int i = 0; i < GI; ++i) ng[i] = __shfl(nodec, (i * kWave + l) / GC);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < KI; ++i)
      load_lds16(pkg + ((prow + nt[i]) * H + h) * DK + ((i * kWave + l) % CH) * EC, s_pk + i * kWave * EC);
#pragma unroll
    for (int i = 0; i < GI; ++i)
      load_lds16(a.pend.alpha + ((prow + ng[i]) * H + h) * DK + ((i * kWave + l) % GC) * 4, s_pg + i * kWave * 4);
    // every tile's values at once: a later tile's would otherwise be waited
    // for on the critical path
#pragma unroll
    for (int i = 0; i < TPW; ++i) gather_u(t0 + i, i);
  }
  // ---- setup wave: the second tile's first DK/2 state rows into LDS, queued
  //      behind the record gathers.  Chunk c holds row r = c / 16, column
  //      chunk (c % 16) ^ 4 ((r / 8) % 4), so that the 16 column-wave lanes of
  //      a row group and the four row groups fall on distinct banks.  Columns
  //      past d_v (a ragged last tile) re-read column 0 and are never used.
  if constexpr (L::kPrefetch) {
    if (w == kSetup) {
      const int cb = (t0 + 1) * kTileCols;
#pragma unroll
      for (int m = 0; m < L::kPreInstr; ++m) {
        const int c = m * kWave + l;
        const int r = c >> 4;
        const int col = cb + 4 * ((c & 15) ^ (((r >> 3) & 3) << 2));
        load_lds16(a.state + (unit * DK + r) * dv + (col < dv ? col : 0), s_pre + m * kWave * 4);
      }
    }
  }

  // ---- GLA: the tree-masked scores with per-key decay ratios,
  //          Attn_ja = sum_i q_j[i] D_ja[i] k_a[i],  D_ja = product of the
  //          gates of P(j) strictly below a (j included), per key dimension,
  //      on the vector ALUs: 16 lanes per node j, each holding d_k / 16 key
  //      dimensions of qc = D_ja * q_j.  Walking up P(j) from j, every step
  //      sums qc . k_a over the 16 lanes (DPP) and then multiplies in a's
  //      gates, so qc ends as Gamma_j * q_j = Q~_j, split into bf16 hi (in
  //      place of q_j) + lo for P_q = Q~ H0.  Gate products only: they may
  //      underflow, never overflow.  The records (the key as given, the
  //      gates) are written from here.
  if constexpr (GV) {
    if (w < kColWaves) {
      constexpr int E = DK / 16;  // key dimensions per lane
      const int maxd = s_misc[2];
      unsigned char *xb = reinterpret_cast<unsigned char *>(xs);
      unsigned char *xlb = reinterpret_cast<unsigned char *>(xl);
      // byte offset of the 4 (E = 4) or 8 key dimensions d0 .. of stage row r
      auto xoff = [&](int r, int d0) {
        if constexpr (F32) return xchunk<CH>(r, d0 >> 2) * 16;  // four fp32 per chunk; d0 % 4 == 0
        return xchunk<CH>(r, d0 >> 3) * 16 + ((d0 >> 2) & 1) * 8;
      };
      auto load_row = [&](int r, int d0, float (&x)[E]) {
        if constexpr (F32) {
#pragma unroll
          for (int c = 0; c < E; c += 4) {
            const float4 u = *reinterpret_cast<const float4 *>(xb + xoff(r, d0 + c));
            x[c] = u.x, x[c + 1] = u.y, x[c + 2] = u.z, x[c + 3] = u.w;
          }
          return;
        }
#pragma unroll
        for (int c = 0; c < E; c += 8 < E ? 8 : E) {
          uint32_t wv[4];
          if constexpr (E >= 8) {
            const uint4 u = *reinterpret_cast<const uint4 *>(xb + xoff(r, d0 + c));
            wv[0] = u.x, wv[1] = u.y, wv[2] = u.z, wv[3] = u.w;
          } else {
            const uint2 u = *reinterpret_cast<const uint2 *>(xb + xoff(r, d0 + c));
            wv[0] = u.x, wv[1] = u.y;
          }
#pragma unroll
          for (int e = 0; e < (E >= 8 ? 8 : E); e += 2) {
            x[c + e] = __uint_as_float(wv[e / 2] << 16);
            x[c + e + 1] = __uint_as_float(wv[e / 2] & 0xffff0000u);
          }
        }
      };
      // the sum over the 16 lanes of a DPP row, in every lane
      auto row_sum = [](float v) {
        v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
        v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
        v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));  // row_half_mirror
        v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));  // row_mirror
        return v;
      };
#pragma unroll 1
      for (int it0 = w * kWave; it0 < NP * 16; it0 += kColWaves * kWave) {  // wave-uniform
        const int j = (it0 + l) >> 4, d0 = ((it0 + l) & 15) * E;
        const bool first = (l & 15) == 0;
        float qc[E];
        load_row(j, d0, qc);  // padding rows hold node 0's query
        uint64_t rest = j < n ? s_anc[j] : 0ull;
        // every lane takes all maxd steps, so the DPP rows stay whole
#pragma unroll 1
        for (int st = 0; st < maxd; ++st) {
          const bool act = rest != 0ull;
          const int an = act ? 63 - __builtin_clzll(rest) : 0;  // deepest ancestor left: j, then up
          rest &= ~(1ull << an);
          float ka[E];
          load_row(NP + an, d0, ka);
          float sdot = 0.f;
#pragma unroll
          for (int e = 0; e < E; ++e) sdot = __builtin_fmaf(qc[e], ka[e], sdot);
          sdot = row_sum(sdot);
          if (act && first) ab[blk(j, an)] = sdot;
          if (act) {
#pragma unroll
            for (int e = 0; e < E; e += 4) {
              const float4 gx = *reinterpret_cast<const float4 *>(s_g + an * DK + d0 + e);
              qc[e] *= gx.x;
              qc[e + 1] *= gx.y;
              qc[e + 2] *= gx.z;
              qc[e + 3] *= gx.w;
            }
          }
        }
        if (j >= n) {  // padding rows: zero low halves (their products are dropped)
          if constexpr (!F32) {
#pragma unroll
            for (int c = 0; c < E; c += 4) *reinterpret_cast<uint2 *>(xlb + xoff(j, d0 + c)) = make_uint2(0, 0);
          }
          continue;
        }
        if constexpr (F32) {  // Q~ in fp32 in place of q_j; the records: the key as given, the gates
#pragma unroll
          for (int c = 0; c < E; c += 4) {
            *reinterpret_cast<float4 *>(xb + xoff(j, d0 + c)) = make_float4(qc[c], qc[c + 1], qc[c + 2], qc[c + 3]);
            if (t0 == 0) {
              const size_t r = ((nbase + j) * H + h) * DK + d0 + c;
              *reinterpret_cast<float4 *>(static_cast<float *>(a.fk) + r) =
                  *reinterpret_cast<const float4 *>(xb + xoff(NP + j, d0 + c));
              *reinterpret_cast<float4 *>(a.falpha + r) = *reinterpret_cast<const float4 *>(s_g + j * DK + d0 + c);
            }
          }
          continue;
        }
#pragma unroll
        for (int c = 0; c < E; c += 4) {
          uint32_t hw[2], lw[2];
#pragma unroll
          for (int e2 = 0; e2 < 2; ++e2) {
            uint32_t hv = 0, lv = 0;
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
              const float x = qc[c + 2 * e2 + s2];
              const __bf16 xh = static_cast<__bf16>(x);
              const __bf16 xl2 = static_cast<__bf16>(x - static_cast<float>(xh));
              hv |= (uint32_t)__builtin_bit_cast(uint16_t, xh) << (16 * s2);
              lv |= (uint32_t)__builtin_bit_cast(uint16_t, xl2) << (16 * s2);
            }
            hw[e2] = hv;
            lw[e2] = lv;
          }
          *reinterpret_cast<uint2 *>(xb + xoff(j, d0 + c)) = make_uint2(hw[0], hw[1]);
          *reinterpret_cast<uint2 *>(xlb + xoff(j, d0 + c)) = make_uint2(lw[0], lw[1]);
          if (t0 == 0) {
            const size_t r = ((nbase + j) * H + h) * DK + d0 + c;
            *reinterpret_cast<uint2 *>(static_cast<bf16 *>(a.fk) + r) =
                *reinterpret_cast<const uint2 *>(xb + xoff(NP + j, d0 + c));
            *reinterpret_cast<float4 *>(a.falpha + r) = *reinterpret_cast<const float4 *>(s_g + j * DK + d0 + c);
          }
        }
      }
    }
    __syncthreads();
  }

  // the folded setup wave's own state reads go out after its record gathers
  if (kSetup == 0 && a.late_state && live(t0)) load_state(t0, hfa);

  // ---- tree-masked Grams over the column waves (scalar gates; GLA's scores
  //      were formed above): tile (mr, na) of [Q; K] K^T holds rows of node
  //      tile mr % NT against ancestor candidates of node tile na <= mr % NT;
  //      ancestor entries go to Attn blocks and Lk lists
  if constexpr (!GV) {
    f32x4 gacc[GT];
    int tc = 0;
#pragma unroll
    for (int mr = 0; mr < MT; ++mr)
#pragma unroll
      for (int na = 0; na <= mr % NT; ++na, ++tc) {
        if (tc % kColWaves != w || (mr % NT) * 16 >= n || (!DELTA && mr >= NT)) continue;
        f32x4 g = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if constexpr (F32) {
            float av[8], bv[8];
            frag8(mr * 16 + lc, ks, av);
            frag8(NP + na * 16 + lc, ks, bv);
#pragma unroll
            for (int e = 0; e < 8; ++e) g = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], bv[e], g, 0, 0, 0);
          } else {
            const bf16x8 af = *reinterpret_cast<const bf16x8 *>(xs + xchunk<CH>(mr * 16 + lc, ks * 4 + lg));
            const bf16x8 bf = *reinterpret_cast<const bf16x8 *>(xs + xchunk<CH>(NP + na * 16 + lc, ks * 4 + lg));
            g = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bf, g, 0, 0, 0);
          }
        }
        gacc[tc / kColWaves] = g;
      }
    tc = 0;
#pragma unroll
    for (int mr = 0; mr < MT; ++mr)
#pragma unroll
      for (int na = 0; na <= mr % NT; ++na, ++tc) {
        if (tc % kColWaves != w || (mr % NT) * 16 >= n || (!DELTA && mr >= NT)) continue;
        // every LDS read of the tile's metadata is issued before its first
        // write, so they share one round trip
        const int an = na * 16 + lc;
        const int jb = (mr % NT) * 16 + 4 * lg;
        uint32_t anc[4];  // the half of row j's ancestor mask that holds column an
        float dj[4], bj[4];  // dj: decay ratio D_{j,an}, parked in the T block (j, an)
        int oj[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          anc[q] = reinterpret_cast<const uint32_t *>(s_anc)[2 * (jb + q) + (na >> 1)];
          dj[q] = tb[blk(jb + q, an)];  // an <= 16 (jb / 16) + 15: inside the block row
          if (mr >= NT) {
            bj[q] = s_be[jb + q];
            oj[q] = s_off[jb + q];
          }
        }
        const int da = mr >= NT ? s_depth[an] : 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = jb + q;
          // rows past the last node hold stale LDS words: masked by j < n
          if (j >= n || an > j || (mr >= NT && an == j) || !((anc[q] >> (an & 31)) & 1u)) continue;
          const float dg = dj[q] * gacc[tc / kColWaves][q];
          if (mr < NT)
            ab[blk(j, an)] = dg;
          else
            lk[oj[q] + da - 1] = bj[q] * dg;
        }
      }
  }
  // the gathered records have landed (the staged state rows may still be in flight)
  if (w == kSetup) __builtin_amdgcn_s_waitcnt(waitcnt_vm(L::kPreInstr));
  __syncthreads();

  if (DELTA && w == kSetup) {
    // ---- T = (I + Lk)^-1, one lane per row j.  With p_0 .. p_{d-1} = j the
    //      root path of j and x_t = T_{j p_t}:  x_{d-1} = 1,
    //      x_t = - sum_{u > t} x_u Lk_{p_u p_t}.
    if (l < n) {
      const int j = l;
      const uint64_t m = s_anc[j];
      tb[blk(j, j)] = 1.f;
      if (maxd <= kZ) {
        // push form, deepest node first: once x_u is known its terms go to
        // every shallower position; z[k] accumulates position u - 1 - k, so
        // the next unknown is always z[0] (registers, no LDS round trip per
        // term; the Lk reads of one node are independent and go out together)
        const int d = s_depth[j];
        float z[kZ];
#pragma unroll
        for (int k = 0; k < kZ; ++k) z[k] = 0.f;
        uint64_t rest = m & ~(1ull << j);
        float xu = 1.f;
        int pu = j;
        for (int u = d - 1; u >= 1; --u) {
          const float *lrow = lk + s_off[pu];
#pragma unroll
          for (int k0 = 0; k0 < kZ; k0 += 8) {  // eight reads per round trip
            float lv[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) lv[k] = (u - 1 - k0 - k >= 0) ? lrow[u - 1 - k0 - k] : 0.f;
#pragma unroll
            for (int k = 0; k < 8; ++k) z[k0 + k] = __builtin_fmaf(xu, lv[k], z[k0 + k]);
          }
          const int pn = 63 - __builtin_clzll(rest);  // p_{u-1}: deepest ancestor left
          rest &= ~(1ull << pn);
          xu = -z[0];
          tb[blk(j, pn)] = xu;
#pragma unroll
          for (int k = 0; k + 1 < kZ; ++k) z[k] = z[k + 1];
          z[kZ - 1] = 0.f;
          pu = pn;
        }
      } else {
        // pull form for deep paths, deepest ancestor first:
        //   T_ja = - sum_{e in P(j), a < e} T_je Lk_ea
        uint64_t rest = m & ~(1ull << j);
        while (rest) {
          const int an = 63 - __builtin_clzll(rest);
          rest &= ~(1ull << an);
          const int ta = s_depth[an] - 1;
          uint64_t below = m & ~((2ull << an) - 1ull);
          float sum = 0.f;
          while (below) {
            const int e = __builtin_ctzll(below);
            below &= below - 1ull;
            sum = __builtin_fmaf(-tb[blk(j, e)], lk[s_off[e] + ta], sum);
          }
          tb[blk(j, an)] = sum;
        }
      }
    }
  }

  // ---- one V-tile: [A] delayed state update, write-back, P = [Q; K] H0
  //      (bf16: state split into hi + lo; fp32: exact) and R on the column waves; barrier (T complete);
  //      [B] U = T R, O = Gamma P_q + Attn U and the stores; then the next
  //      tile's state and values go out.
  const uint32_t obytes = ((uint32_t)(n - 1) * nstride + dv) * 4;
  const rsrc_t orr = make_rsrc(a.out + (nbase * H + h) * dv, obytes);
  const rsrc_t urr = make_rsrc(a.fu + (nbase * H + h) * dv, obytes);
  auto step = [&](int i, float (&hf)[KS][8], float (&hn)[KS][8]) {
    const int t = t0 + i;
    const bool more = i + 1 < cnt;
    const bool cols_live = live(t);
    const int col = t * kTileCols + ucol;
    const uint32_t sv = (uint32_t)(8 * lg * dv + col) * 4;
    const float *pu = s_pu + i * kPMax * kTileCols;

    // accumulator layout: lane (lg, lc) holds rows 4 lg .. 4 lg + 3 of each
    // 16-row tile, column lc
    f32x4 pq[NT];  // P_q = Q H0, accumulator layout
#pragma unroll
    for (int mt = 0; mt < NT; ++mt) pq[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 rreg[NT];
    if (cols_live) {
      const int ps = plen < kPMax ? plen : kPMax;
      const AT *pkg = static_cast<const AT *>(a.pend.k);
      const int pn = a.has_pending ? a.pend.n : 1;
      if (a.has_pending) {
        // the whole tile has normally landed by now: step-major, one LDS
        // round trip per step
        for (int st = 0; st < ps; ++st) {
          const float al = s_palpha[st];
          const float uv = pu[st * kTileCols + ucol];
          constexpr int KC = KS < 2 ? KS : 2;  // K-steps per LDS round trip
#pragma unroll
          for (int k0 = 0; k0 < KS; k0 += KC) {
            float kv[KC][8];  // the key's rows 32 (k0 + c) + 8 lg + e
            float gv[KC][8];  // GLA: the gates of the same rows
#pragma unroll
            for (int c = 0; c < KC; ++c) {
              if constexpr (F32) {
                const float4 k0v = *reinterpret_cast<const float4 *>(s_pk + st * DK + (k0 + c) * 32 + 8 * lg);
                const float4 k1v = *reinterpret_cast<const float4 *>(s_pk + st * DK + (k0 + c) * 32 + 8 * lg + 4);
                kv[c][0] = k0v.x, kv[c][1] = k0v.y, kv[c][2] = k0v.z, kv[c][3] = k0v.w;
                kv[c][4] = k1v.x, kv[c][5] = k1v.y, kv[c][6] = k1v.z, kv[c][7] = k1v.w;
              } else {
                const bf16x8 kb = *reinterpret_cast<const bf16x8 *>(s_pk + st * DK + (k0 + c) * 32 + 8 * lg);
#pragma unroll
                for (int e = 0; e < 8; ++e) kv[c][e] = static_cast<float>(kb[e]);
              }
            }
            if constexpr (GV) {
#pragma unroll
              for (int c = 0; c < KC; ++c) {
                const float4 g0 = *reinterpret_cast<const float4 *>(s_pg + st * DK + (k0 + c) * 32 + 8 * lg);
                const float4 g1 = *reinterpret_cast<const float4 *>(s_pg + st * DK + (k0 + c) * 32 + 8 * lg + 4);
                gv[c][0] = g0.x, gv[c][1] = g0.y, gv[c][2] = g0.z, gv[c][3] = g0.w;
                gv[c][4] = g1.x, gv[c][5] = g1.y, gv[c][6] = g1.z, gv[c][7] = g1.w;
              }
            }
#pragma unroll
            for (int c = 0; c < KC; ++c)
#pragma unroll
              for (int e = 0; e < 8; ++e)
                hf[k0 + c][e] = apply_factor(hf[k0 + c][e], GV ? gv[c][e] : al, kv[c][e], uv);
          }
        }
        // paths longer than the LDS stage read their records directly
        for (int st = kPMax; st < plen; ++st) {
          const int node = a.pend.path[(size_t)b * pn + st];
          const size_t r = ((size_t)b * pn + node) * H + h;
          const float al = GV ? 1.f : a.pend.alpha[r];
          const float uv = a.pend.u[r * dv + col];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) {
            float kr[8], gr[8];
            load_f32<8>(pkg + r * DK + ks * 32 + 8 * lg, kr);
            if constexpr (GV) load_f32<8>(a.pend.alpha + r * DK + ks * 32 + 8 * lg, gr);
#pragma unroll
            for (int e = 0; e < 8; ++e) hf[ks][e] = apply_factor(hf[ks][e], GV ? gr[e] : al, kr[e], uv);
          }
        }
        // committed rows back.  A wave writes half of each 128-byte line and
        // the neighbouring wave the other half.  Over many rounds of
        // workgroups the default policy lets the L2 merge the halves (a plain
        // streaming hint wrote them separately: 8% more HBM writes, 4.7%
        // longer launches).  In a single round the rows are written through
        // at device scope instead: what stays dirty in the L2 is written back
        // at the end of the kernel, on its critical path (measured at batched
        // tree serving 39.2 -> 37.9 us per launch; on the 1-node decode chain,
        // eight rounds, the default policy stays 2% faster).
        // (chosen at launch: a run-time branch between the two store loops
        // cost most of the gain)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            buf_store_f32<WT ? kPolicyStreamDevice : kPolicyDefault>(hf[ks][e], sr, sv, (uint32_t)(ks * 32 + e) * dv * 4);
      }
      // P_k = K H0 first (K-step by K-step as the tile lands; bf16: the
      // state split into hi + lo, fp32: exact products), so that
      // R = beta (v - gamma P_k) takes its place before P_q is built: the two
      // halves of P are never held at once
      f32x4 pk[NT];
#pragma unroll
      for (int mt = 0; mt < NT; ++mt) pk[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (DELTA && F32) {  // exact fp32 products: the state registers are the B operands
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int mt = 0; mt < NT; ++mt) {
            float av[8];
            frag8(NP + mt * 16 + lc, ks, av);
#pragma unroll
            for (int e = 0; e < 8; ++e) pk[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], hf[ks][e], pk[mt], 0, 0, 0);
          }
      } else if constexpr (DELTA) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          bf16x8 bhi, blo;
          split8(hf[ks], bhi, blo);
#pragma unroll
          for (int mt = 0; mt < NT; ++mt) {
            const bf16x8 af = *reinterpret_cast<const bf16x8 *>(xs + xchunk<CH>(NP + mt * 16 + lc, ks * 4 + lg));
            pk[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bhi, pk[mt], 0, 0, 0);
            pk[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, blo, pk[mt], 0, 0, 0);
          }
        }
      }
      // R in the accumulator layout (the row base is rebuilt per tile:
      // hoisted out of the tile loop it only gets spilled)
      int rb = 4 * lg;
      __asm__("" : "+v"(rb));
#pragma unroll
      for (int mt = 0; mt < NT; ++mt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = mt * 16 + rb + q;
          uint32_t vb = vraw[mt][q];
          __asm__("" : "+v"(vb));  // keeps the widening here, not next to the load
          const float vf = __uint_as_float(F32 ? vb : vb << 16);
          const float rd = DELTA ? s_be[j] * (vf - s_gamma[j] * pk[mt][q]) : vf;
          rreg[mt][q] = j < n ? (nodelta ? vf : rd) : 0.f;
        }
      if constexpr (F32) {  // Q (GLA: Q~) H0, exact fp32 products
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int mt = 0; mt < NT; ++mt) {
            float av[8];
            frag8(mt * 16 + lc, ks, av);
#pragma unroll
            for (int e = 0; e < 8; ++e) pq[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], hf[ks][e], pq[mt], 0, 0, 0);
          }
      } else {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          bf16x8 bhi, blo;
          split8(hf[ks], bhi, blo);
#pragma unroll
          for (int mt = 0; mt < NT; ++mt) {
            const bf16x8 af = *reinterpret_cast<const bf16x8 *>(xs + xchunk<CH>(mt * 16 + lc, ks * 4 + lg));
            pq[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bhi, pq[mt], 0, 0, 0);
            pq[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, blo, pq[mt], 0, 0, 0);
            if constexpr (GV) {  // Q~ lo half
              const bf16x8 afl = *reinterpret_cast<const bf16x8 *>(xl + xchunk<CH>(mt * 16 + lc, ks * 4 + lg));
              pq[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afl, bhi, pq[mt], 0, 0, 0);
            }
          }
        }
      }
    }
    // the next tile's state and values go out now, while this tile's U, O
    // and stores are computed: its state registers are free since P_q, its
    // values since R
    if (TPW > 1 && more && live(t + 1)) {
      load_state(t + 1, hn, L::kPrefetch ? KS / 2 : 0);
      load_values(t + 1, vraw);
    }
    if (L::kPrefetch && w == kSetup && i == 0) __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));  // staged rows landed
    __syncthreads();  // T complete
    if (L::kPrefetch && more && live(t + 1)) {
      // the staged rows of the next tile: row 32 ks + 8 lg + e, column chunk
      // ucol / 4 swizzled by lg
#pragma unroll
      for (int ks = 0; ks < KS / 2; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int r = ks * 32 + 8 * lg + e;
          hn[ks][e] = s_pre[(r * 16 + ((ucol >> 2) ^ (lg << 2))) * 4 + (lc & 3)];
        }
    }
    // factor records independent of the V-tile -- k (from the staged rows),
    // alpha, parent -- while the column waves compute the first tile's
    // products (off the path to the barrier above)
    if (w == kSetup && i == 0 && t0 == 0) {
      if constexpr (!GV) {  // GLA's key and gate records went out with Q~
        AT *fk = static_cast<AT *>(a.fk);
        for (int c = l; c < n * CH; c += kWave) {
          const int j = c / CH, part = c % CH;
          *reinterpret_cast<uint4 *>(fk + ((nbase + j) * H + h) * DK + part * EC) = xs[xchunk<CH>(NP + j, part)];
        }
      }
      if (l < n) {
        if constexpr (!GV) a.falpha[(nbase + l) * H + h] = al;
        if (h == 0) a.fparent[nbase + l] = p;
      }
    }
    if (cols_live) {  // no early return: every wave takes every later barrier
      // ---- U = T R, then O = Gamma P_q + Attn U, on the matrix cores; A
      //      fragments are rows j = 16 mt + lc, columns 16 ks + 4 lg .. + 3
      f32x4 uacc[NT];  // same layout as R
      if constexpr (DELTA && F32) {
        // A operand i: T[16 mt + lc][16 ks + 4 lg + i], B operand i: R[16 ks + 4 lg + i][lc]
#pragma unroll
        for (int mt = 0; mt < NT; ++mt) {
          uacc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks <= mt; ++ks) {
            const f32x4 tv = *reinterpret_cast<const f32x4 *>(tb + ((mt * (mt + 1)) / 2 + ks) * (16 * kBP) + lc * kBP + 4 * lg);
#pragma unroll
            for (int i = 0; i < 4; ++i) uacc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(tv[i], rreg[ks][i], uacc[mt], 0, 0, 0);
          }
        }
      } else if constexpr (DELTA) {
        s16x4 rhi[NT], rlo[NT];
#pragma unroll
        for (int mt = 0; mt < NT; ++mt) split4(rreg[mt], rhi[mt], rlo[mt]);
#pragma unroll
        for (int mt = 0; mt < NT; ++mt) {
          uacc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks <= mt; ++ks) {
            const f32x4 tv = *reinterpret_cast<const f32x4 *>(tb + ((mt * (mt + 1)) / 2 + ks) * (16 * kBP) + lc * kBP + 4 * lg);
            s16x4 th, tlo;
            split4(tv, th, tlo);
            uacc[mt] = mfma16_split(th, tlo, rhi[ks], rlo[ks], uacc[mt]);
          }
        }
      } else {
#pragma unroll
        for (int mt = 0; mt < NT; ++mt) uacc[mt] = rreg[mt];
      }
      s16x4 uhi[NT], ulo[NT];
      if constexpr (!F32) {
#pragma unroll
        for (int mt = 0; mt < NT; ++mt) split4(uacc[mt], uhi[mt], ulo[mt]);
      }
      // outputs and corrected values of node j at ((b n + j) H + h) dv + col;
      // rows past the last node fall outside the descriptors (the whole offset
      // is carried per lane, where the range check applies) and are dropped
      const uint32_t ov = (4 * lg * nstride + col) * 4;
#pragma unroll
      for (int mt = 0; mt < NT; ++mt) {
        f32x4 oacc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks <= mt; ++ks) {
          const f32x4 av = *reinterpret_cast<const f32x4 *>(ab + ((mt * (mt + 1)) / 2 + ks) * (16 * kBP) + lc * kBP + 4 * lg);
          if constexpr (F32) {
#pragma unroll
            for (int i = 0; i < 4; ++i) oacc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], uacc[ks][i], oacc, 0, 0, 0);
          } else {
            s16x4 ah, alo;
            split4(av, ah, alo);
            oacc = mfma16_split(ah, alo, uhi[ks], ulo[ks], oacc);
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j = mt * 16 + 4 * lg + q;
          const uint32_t vo = ov + (uint32_t)(mt * 16 + q) * nstride * 4;
          buf_store_f32<kPolicyStream>(uacc[mt][q], urr, vo, 0);
          buf_store_f32<kPolicyStream>(__builtin_fmaf(s_gamma[j], pq[mt][q], oacc[q]), orr, vo, 0);
        }
      }
    }
  };
  // straight-line, the two state register sets trading roles (in a loop
  // the compiler loses track of which loads a register still waits for;
  // four tiles in a row spill)
  static_assert(TPW == 1 || TPW == 2, "tiles per workgroup");
  step(0, hfa, hfb);
  if constexpr (TPW == 2) step(1, hfb, hfa);
}

constexpr size_t kMaxLds = 160 * 1024;
constexpr size_t kDefaultLds = 64 * 1024;

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

// The state reads of a workgroup normally go out first, so that they overlap
// the setup wave's dependent reads.  When the launch holds at least
// kLateRounds rounds of workgroups (resident workgroups per CU from the
// occupancy of the kernel instantiation), they go out after the first
// barrier instead: measured 4.5% faster on the 1-node decode chain at batch
// 256, 1% slower at one round.  At one to kLateRounds rounds the column waves
// hold them back briefly instead (stagger).
constexpr int kLateRounds = 4;

template <int DK, int NP, int CW, int TPW, int KIND, bool F32>
hipError_t launch_np_fam(const VerifyArgs &a, hipStream_t s) {
  using L = Layout<DK, NP, CW, TPW, KIND, F32>;
  const size_t lds = L::kBytes;
  if (lds > kMaxLds) return hipErrorInvalidConfiguration;
  auto kern_wb = verify_tile_kernel<DK, NP, CW, TPW, KIND, F32, false>;  // committed rows written back
  auto kern_wt = verify_tile_kernel<DK, NP, CW, TPW, KIND, F32, true>;   // written through
  if (lds > kDefaultLds) {
    for (auto k : {kern_wb, kern_wt}) {
      const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
  }
  const int ntiles = (a.dv + L::kTileCols - 1) / L::kTileCols;
  const size_t groups = (size_t)a.B * a.H * ((ntiles + TPW - 1) / TPW);
  VerifyArgs b = a;
  // resident workgroups per CU for this instantiation (registers, LDS, waves)
  static const int per_cu = [&] {
    int k = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&k, kern_wb, kWaves<CW> * kWave, lds) != hipSuccess || k < 1) k = 1;
    return k;
  }();
  const size_t slots = (size_t)per_cu * device_cus();
  b.late_state = groups >= (size_t)kLateRounds * slots;
  b.stagger = !b.late_state && groups >= slots;
  // write-through only for a full round of workgroups that all stay resident:
  // below a round the launch is latency-bound and the writes' completion
  // lengthens it (batch 1, 32 workgroups: 8.6 -> 9.9 us per round)
  hipLaunchKernelGGL(b.stagger ? kern_wt : kern_wb, dim3((unsigned)groups), dim3(kWaves<CW> * kWave), lds, s, b);
  return hipGetLastError();
}

template <int DK, int NP, int CW, int TPW, bool F32>
hipError_t launch_np(const VerifyArgs &a, hipStream_t s) {
  if (a.family == SLA_FAMILY_GLA) return launch_np_fam<DK, NP, CW, TPW, kKindGates, F32>(a, s);
  return launch_np_fam<DK, NP, CW, TPW, kKindDelta, F32>(a, s);
}

template <int DK, bool F32>
hipError_t launch_dk(const VerifyArgs &a, hipStream_t s) {
  // small trees: two V-tiles of a unit per workgroup once single tiles would
  // fill every CU's four workgroup slots twice over.  The launch is then one
  // round of long-lived workgroups instead of two, and q, k, topology, Grams
  // and T serve both tiles.  Below that, single tiles keep more workgroups
  // (and CUs) busy.
  if constexpr (DK <= 128) {
    const int ntiles = (a.dv + kWaveCols * 4 - 1) / (kWaveCols * 4);
    if (a.n <= 32 && ntiles % 2 == 0 && (size_t)a.B * a.H * ntiles >= (size_t)8 * device_cus())
      return a.n <= 16 ? launch_np<DK, 16, 4, 2, F32>(a, s) : launch_np<DK, 32, 4, 2, F32>(a, s);
  }
  if (a.n <= 16) return launch_np<DK, 16, 4, 1, F32>(a, s);
  if (a.n <= 32) return launch_np<DK, 32, 4, 1, F32>(a, s);
  // large trees: two V-tiles per workgroup -- topology, Grams and T serve
  // both, and the second tile's state loads overlap the first tile's U, O
  // and stores; with d_v a multiple of 256, tiles of 128 columns (eight
  // column waves), so that one workgroup covers 256 columns
  if constexpr (DK <= 128) {
    if (a.dv % 256 == 0) return launch_np<DK, 64, 8, 2, F32>(a, s);
    if (((a.dv + kWaveCols * 4 - 1) / (kWaveCols * 4)) % 2 == 0) return launch_np<DK, 64, 4, 2, F32>(a, s);
  }
  return launch_np<DK, 64, 4, 1, F32>(a, s);
}

}  // namespace

bool parallel_supported(int dk, int dv, int n, int dtype) {
  // bf16 activations: bf16 matrix cores (q and k exact in bf16, the fp32
  // operands split hi + lo); fp32 activations: fp32 matrix cores.  A draft
  // whose stage exceeds the LDS is refused at launch
  // (hipErrorInvalidConfiguration).
  return (dtype == SLA_DTYPE_BF16 || dtype == SLA_DTYPE_F32) && (dk == 64 || dk == 128 || dk == 256) &&
         dv % 16 == 0 && n >= 1 && n <= SLA_MAX_NODES;
}

template <bool F32>
hipError_t launch_dtype(const VerifyArgs &a, hipStream_t s) {
  switch (a.dk) {
    case 64: return launch_dk<64, F32>(a, s);
    case 128: return launch_dk<128, F32>(a, s);
    case 256: return launch_dk<256, F32>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_verify_parallel(const VerifyArgs &a, int dtype, hipStream_t s) {
  if (dtype == SLA_DTYPE_BF16) return launch_dtype<false>(a, s);
  if (dtype == SLA_DTYPE_F32) return launch_dtype<true>(a, s);
  return hipErrorInvalidConfiguration;
}

}  // namespace sla
