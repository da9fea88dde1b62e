// verify_serial.hip -- state-resident serial verification (SpecLA §4.1),
// with the delayed state update of §5.2 fused in front of it.
//
// One wavefront owns one (batch b, head h, 16-column V-tile) slice of the
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
// Nodes are visited in DFS pre-order; a chain therefore advances the
// registers in place.  When the next node's parent is
// not the state in registers (a branch point of a tree), that state is
// rebuilt from the committed tile kept in registers by re-applying the
// stored factors of the parent's root path -- rank-one updates only, the
// reductions of shared prefixes are never repeated.
#include "device.hpp"
#include "kernels.hpp"

namespace sla {
namespace {

constexpr int kCols = 16;
constexpr int kGroups = kWave / kCols;
constexpr int kXcds = 8;  // workgroup i runs on XCD i mod 8

// VG: per-key gates (GLA), staged on chip like the keys.
template <int DK, typename T, bool CHAIN, bool VG>
__global__ __launch_bounds__(kWave) void verify_serial_kernel(VerifyArgs a) {
  constexpr int R = DK / kGroups;
  const int lane = threadIdx.x;
  const int c = lane & (kCols - 1);
  const int g = lane / kCols;
  const int H = a.H, dv = a.dv, n = a.n;
  const int ntiles = dv / kCols;
  // neighbouring tiles (2m, 2m + 1) hold the two halves of each 128-byte row
  // segment: their workgroups are numbered 8 apart, so that they run on the
  // same XCD and share its L2 (consecutive workgroups go to different XCDs,
  // whose L2s would each fetch and write back the whole lines)
  const int npairs = (ntiles + 1) / 2;
  const int x = blockIdx.x;
  const int qd = x / kXcds;
  const size_t pair = (size_t)(qd / 2) * kXcds + x % kXcds;
  const int tile = 2 * (int)(pair % npairs) + qd % 2;
  const size_t unit_id = pair / npairs;
  if (tile >= ntiles || unit_id >= (size_t)a.B * H) return;  // padding of the numbering: no barrier follows
  const int h = (int)(unit_id % H);
  const int b = (int)(unit_id / H);
  const int col = tile * kCols + c;
  const int row0 = g * R;
  const size_t unit = (size_t)b * H + h;
  // delta-rule families correct the value against the parent state
  const bool delta = a.family == SLA_FAMILY_GDN || a.family == SLA_FAMILY_DELTANET;

  // The state tile: the only state read of this call.
  float *st = a.state + unit * DK * dv + col;
  float H0[R];
#pragma unroll
  for (int r = 0; r < R; ++r) H0[r] = st[(size_t)(row0 + r) * dv];

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
  float *ks = lds;                   // [n][DK]
  float *qs = ks + n * DK;           // [n][DK]
  float *gs = qs + n * DK;           // [n][DK] per-key gates (VG only)
  float *vs = gs + (VG ? n * DK : 0);  // [n][kCols]
  float *us = vs + n * kCols;        // [n][kCols]
  float *als = us + n * kCols;       // [n]
  float *bes = als + n;              // [n]
  int *ords = reinterpret_cast<int *>(bes + n);  // [n] DFS pre-order
  int *pars = ords + n;              // [n]
  int *kids = pars + n;              // [n]
  uint64_t *ancs = reinterpret_cast<uint64_t *>(kids + n + (n & 1));  // [n]

  const T *q = static_cast<const T *>(a.q);
  const T *k = static_cast<const T *>(a.k);
  const T *v = static_cast<const T *>(a.v);
  // eight elements per lane and step (one 16-byte load of bf16, two of fp32)
  for (int idx = lane; idx < n * (DK / 8); idx += kWave) {
    const int j = idx / (DK / 8), i = (idx % (DK / 8)) * 8;
    const size_t src = (((size_t)b * n + j) * H + h) * DK + i;
    float kv[8], qv[8];
    load_f32<8>(k + src, kv);
    load_f32<8>(q + src, qv);
    float4 *kd = reinterpret_cast<float4 *>(ks + j * DK + i);
    float4 *qd = reinterpret_cast<float4 *>(qs + j * DK + i);
    kd[0] = make_float4(kv[0], kv[1], kv[2], kv[3]);
    kd[1] = make_float4(kv[4], kv[5], kv[6], kv[7]);
    qd[0] = make_float4(qv[0], qv[1], qv[2], qv[3]);
    qd[1] = make_float4(qv[4], qv[5], qv[6], qv[7]);
    if (VG) {
      float gv[8];
      load_f32<8>(a.alpha + src, gv);
      float4 *gd = reinterpret_cast<float4 *>(gs + j * DK + i);
      gd[0] = make_float4(gv[0], gv[1], gv[2], gv[3]);
      gd[1] = make_float4(gv[4], gv[5], gv[6], gv[7]);
    }
  }
  for (int idx = lane; idx < n * kCols; idx += kWave) {
    const int j = idx / kCols, cc = idx % kCols;
    vs[idx] = to_f32(v[(((size_t)b * n + j) * H + h) * dv + tile * kCols + cc]);
  }
  if (lane < n) {
    const size_t s = ((size_t)b * n + lane) * H + h;
    als[lane] = (VG || a.family == SLA_FAMILY_DELTANET) ? 1.f : a.alpha[s];
    bes[lane] = delta ? a.beta[s] : 0.f;
    ords[topo.pos] = lane;
    pars[lane] = topo.parent;
    kids[lane] = topo.n_children;
    ancs[lane] = topo.anc;
  }
  // Factor records that do not depend on the V-tile: written once per unit
  // (k, gate) and once per sequence (parent).
  if (tile == 0) {
    T *fk = static_cast<T *>(a.fk);
    constexpr int E = 16 / (int)sizeof(T);  // elements per 16-byte copy
    for (int idx = lane; idx < n * (DK / E); idx += kWave) {
      const int j = idx / (DK / E), i = (idx % (DK / E)) * E;
      const size_t s = (((size_t)b * n + j) * H + h) * DK + i;
      *reinterpret_cast<uint4 *>(fk + s) = *reinterpret_cast<const uint4 *>(k + s);
    }
    if (VG)
      for (int idx = lane; idx < n * (DK / 4); idx += kWave) {
        const int j = idx / (DK / 4), i = (idx % (DK / 4)) * 4;
        const size_t s = (((size_t)b * n + j) * H + h) * DK + i;
        *reinterpret_cast<float4 *>(a.falpha + s) = *reinterpret_cast<const float4 *>(a.alpha + s);
      }
    if (lane < n) {
      const size_t s = ((size_t)b * n + lane) * H + h;
      if (!VG) a.falpha[s] = a.family == SLA_FAMILY_DELTANET ? 1.f : a.alpha[s];
      if (h == 0) a.fparent[(size_t)b * n + lane] = topo.parent;
    }
  }
  __syncthreads();

  // Delayed state update: commit the previous round's accepted path into the
  // tile, then write the committed tile back (the only state write).
  if (a.has_pending) {
    const T *pk = static_cast<const T *>(a.pend.k);
    const int pn = a.pend.n;
    for (int t = 0; t < plen; ++t) {
      const int node = a.pend.path[(size_t)b * pn + t];
      const size_t s = ((size_t)b * pn + node) * H + h;
      const float u = a.pend.u[s * dv + col];
      float kr[R], gr[R];
      load_f32<R>(pk + s * DK + row0, kr);
      if (VG) {
        load_f32<R>(a.pend.alpha + s * DK + row0, gr);
      } else {
        const float al = a.pend.alpha[s];
#pragma unroll
        for (int r = 0; r < R; ++r) gr[r] = al;
      }
#pragma unroll
      for (int r = 0; r < R; ++r) H0[r] = apply_factor(H0[r], gr[r], kr[r], u);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) st[(size_t)(row0 + r) * dv] = H0[r];
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
        uint64_t m = ancs[p];
        while (m) {
          const int x = __builtin_ctzll(m);
          m &= m - 1;
          const float al = als[x];
          const float u = us[x * kCols + c];
          const float *kx = ks + x * DK + row0;
          const float *gx = gs + x * DK + row0;
#pragma unroll
          for (int r = 0; r < R; ++r) Hc[r] = apply_factor(Hc[r], VG ? gx[r] : al, kx[r], u);
        }
      }
    }
    const float *kj = ks + j * DK + row0;
    const float *qj = qs + j * DK + row0;
    const float *gj = gs + j * DK + row0;
    float sk = 0.f, sq = 0.f, kq = 0.f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float kr = kj[r], qr = qj[r];
      sk = __builtin_fmaf(Hc[r], kr, sk);
      sq = __builtin_fmaf(Hc[r], VG ? gj[r] * qr : qr, sq);
      kq = __builtin_fmaf(kr, qr, kq);
    }
    sk += __shfl_xor(sk, 16);
    sq += __shfl_xor(sq, 16);
    kq += __shfl_xor(kq, 16);
    sk += __shfl_xor(sk, 32);
    sq += __shfl_xor(sq, 32);
    kq += __shfl_xor(kq, 32);
    const float al = als[j], be = bes[j];
    const float u = delta ? be * (vs[j * kCols + c] - al * sk) : vs[j * kCols + c];
    const float o = __builtin_fmaf(kq, u, al * sq);
    if (g == 0) {
      const size_t s = ((size_t)b * n + j) * H + h;
      a.out[s * dv + col] = o;
      a.fu[s * dv + col] = u;
      us[j * kCols + c] = u;
    }
    const bool internal = CHAIN ? (t + 1 < n) : (kids[j] > 0);
    if (internal) {
#pragma unroll
      for (int r = 0; r < R; ++r) Hc[r] = apply_factor(Hc[r], VG ? gj[r] : al, kj[r], u);
      cur = j;
    } else {
      cur = p;
    }
  }
}

size_t serial_lds_bytes(int n, int dk, bool vg) {
  return sizeof(float) * ((size_t)(vg ? 3 : 2) * n * dk + 2 * n * kCols + 2 * n) + sizeof(int) * (3 * n + (n & 1)) +
         sizeof(uint64_t) * n;
}

// gfx950 gives one workgroup up to 160 KiB of LDS; above the default 64 KiB
// the kernel has to opt in.
constexpr size_t kMaxLds = 160 * 1024;
constexpr size_t kDefaultLds = 64 * 1024;

template <typename K>
hipError_t launch_with_lds(K kernel, dim3 grid, size_t lds, hipStream_t s, const VerifyArgs &a) {
  if (lds > kMaxLds) return hipErrorInvalidConfiguration;
  if (lds > kDefaultLds) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kernel, grid, dim3(kWave), lds, s, a);
  return hipGetLastError();
}

template <int DK, typename T>
hipError_t launch_dk(const VerifyArgs &a, hipStream_t s) {
  // tile pairs numbered in groups of eight per XCD (see the kernel), padded to whole groups
  const size_t pairs = (size_t)a.B * a.H * ((a.dv / kCols + 1) / 2);
  const dim3 grid((unsigned)(((pairs + kXcds - 1) / kXcds) * 2 * kXcds));
  const bool vg = a.family == SLA_FAMILY_GLA;
  const size_t lds = serial_lds_bytes(a.n, DK, vg);
  if (vg) {
    if (a.chain) return launch_with_lds(verify_serial_kernel<DK, T, true, true>, grid, lds, s, a);
    return launch_with_lds(verify_serial_kernel<DK, T, false, true>, grid, lds, s, a);
  }
  if (a.chain) return launch_with_lds(verify_serial_kernel<DK, T, true, false>, grid, lds, s, a);
  return launch_with_lds(verify_serial_kernel<DK, T, false, false>, grid, lds, s, a);
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

}  // namespace

hipError_t launch_verify_serial(const VerifyArgs &a, int dtype, hipStream_t s) {
  return dtype == SLA_DTYPE_BF16 ? launch_t<bf16>(a, s) : launch_t<float>(a, s);
}

}  // namespace sla
