// serial_stage.hpp -- the on-chip stage of one (batch b, head h) unit's draft
// used by the state-resident kernels (serial and chain-decomposed hybrid
// verification): keys, queries (and GLA's per-key gates) in fp32, this
// 16-column V-tile's values, the gates and betas, and the factor records
// that do not depend on the V-tile.
#pragma once

#include "device.hpp"
#include "kernels.hpp"

namespace sla {

constexpr int kSliceCols = 16;  // state columns per wave (one V-tile)

// Pointers into the stage.  Layout (n nodes): ks, qs [n][DK]; gs [n][DK]
// (per-key gates only); vs, us [n][16]; als, bes [n]; four int arrays [n];
// ancs [n] (8-byte aligned).
struct SerialStage {
  float *ks, *qs, *gs, *vs, *us, *als, *bes;
  int *ia, *ib, *ic, *id;
  uint64_t *ancs;
};

__host__ __device__ inline size_t serial_stage_bytes(int n, int dk, bool vg) {
  return sizeof(float) * ((size_t)(vg ? 3 : 2) * n * dk + 2 * n * kSliceCols + 2 * n) +
         sizeof(int) * (4 * n) + sizeof(uint64_t) * n;
}

template <int DK, bool VG>
__device__ inline SerialStage carve_stage(float *lds, int n) {
  SerialStage s;
  s.ks = lds;
  s.qs = s.ks + n * DK;
  s.gs = s.qs + n * DK;
  s.vs = s.gs + (VG ? n * DK : 0);
  s.us = s.vs + n * kSliceCols;
  s.als = s.us + n * kSliceCols;
  s.bes = s.als + n;
  s.ia = reinterpret_cast<int *>(s.bes + n);
  s.ib = s.ia + n;
  s.ic = s.ib + n;
  s.id = s.ic + n;
  s.ancs = reinterpret_cast<uint64_t *>(s.id + n);  // 4 n (c DK + 34) + 16 n bytes in (c = 2 or 3): 8-byte aligned
  return s;
}

// Stage the unit's draft with `nthr` threads (thread `t`): keys, queries and
// gates as fp32 rows, the values of V-tile `tile`, alpha and beta; with
// `records`, also write the factor records that do not depend on the V-tile
// (the key as given and the gate; the parent array when h == 0).
template <int DK, typename T, bool VG>
__device__ inline void stage_draft(const VerifyArgs &a, const SerialStage &s, int b, int h, int tile, int t,
                                   int nthr, bool delta, bool records) {
  const int H = a.H, dv = a.dv, n = a.n;
  const T *q = static_cast<const T *>(a.q);
  const T *k = static_cast<const T *>(a.k);
  const T *v = static_cast<const T *>(a.v);
  // eight elements per thread and step (one 16-byte load of bf16, two of fp32)
  for (int idx = t; idx < n * (DK / 8); idx += nthr) {
    const int j = idx / (DK / 8), i = (idx % (DK / 8)) * 8;
    const size_t src = (((size_t)b * n + j) * H + h) * DK + i;
    float kv[8], qv[8];
    load_f32<8>(k + src, kv);
    load_f32<8>(q + src, qv);
    float4 *kd = reinterpret_cast<float4 *>(s.ks + j * DK + i);
    float4 *qd = reinterpret_cast<float4 *>(s.qs + j * DK + i);
    kd[0] = make_float4(kv[0], kv[1], kv[2], kv[3]);
    kd[1] = make_float4(kv[4], kv[5], kv[6], kv[7]);
    qd[0] = make_float4(qv[0], qv[1], qv[2], qv[3]);
    qd[1] = make_float4(qv[4], qv[5], qv[6], qv[7]);
    if (VG) {
      float gv[8];
      load_f32<8>(a.alpha + src, gv);
      float4 *gd = reinterpret_cast<float4 *>(s.gs + j * DK + i);
      gd[0] = make_float4(gv[0], gv[1], gv[2], gv[3]);
      gd[1] = make_float4(gv[4], gv[5], gv[6], gv[7]);
    }
  }
  for (int idx = t; idx < n * kSliceCols; idx += nthr) {
    const int j = idx / kSliceCols, cc = idx % kSliceCols;
    s.vs[idx] = to_f32(v[(((size_t)b * n + j) * H + h) * dv + tile * kSliceCols + cc]);
  }
  for (int j = t; j < n; j += nthr) {
    const size_t sj = ((size_t)b * n + j) * H + h;
    s.als[j] = (VG || a.family == SLA_FAMILY_DELTANET) ? 1.f : a.alpha[sj];
    s.bes[j] = delta ? a.beta[sj] : 0.f;
  }
  if (!records) return;
  T *fk = static_cast<T *>(a.fk);
  constexpr int E = 16 / (int)sizeof(T);  // elements per 16-byte copy
  for (int idx = t; idx < n * (DK / E); idx += nthr) {
    const int j = idx / (DK / E), i = (idx % (DK / E)) * E;
    const size_t sj = (((size_t)b * n + j) * H + h) * DK + i;
    *reinterpret_cast<uint4 *>(fk + sj) = *reinterpret_cast<const uint4 *>(k + sj);
  }
  if (VG)
    for (int idx = t; idx < n * (DK / 4); idx += nthr) {
      const int j = idx / (DK / 4), i = (idx % (DK / 4)) * 4;
      const size_t sj = (((size_t)b * n + j) * H + h) * DK + i;
      *reinterpret_cast<float4 *>(a.falpha + sj) = *reinterpret_cast<const float4 *>(a.alpha + sj);
    }
  for (int j = t; j < n; j += nthr) {
    const size_t sj = ((size_t)b * n + j) * H + h;
    if (!VG) a.falpha[sj] = a.family == SLA_FAMILY_DELTANET ? 1.f : a.alpha[sj];
    if (h == 0) a.fparent[(size_t)b * n + j] = a.parent[(size_t)b * n + j];
  }
}

// The delayed state update of one lane's rows: the pending path's records
// applied to H (rows row0 .. row0 + R - 1 of column col), root first.
template <int DK, int R, typename T, bool VG>
__device__ inline void apply_pending(const VerifyArgs &a, int b, int h, int col, int row0, int plen,
                                     float (&H)[R]) {
  const T *pk = static_cast<const T *>(a.pend.k);
  const int pn = a.pend.n, Hn = a.H, dv = a.dv;
  for (int t = 0; t < plen; ++t) {
    const int node = a.pend.path[(size_t)b * pn + t];
    const size_t s = ((size_t)b * pn + node) * Hn + h;
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
    for (int r = 0; r < R; ++r) H[r] = apply_factor(H[r], gr[r], kr[r], u);
  }
}

// One node of the state-resident loop on a lane's R rows of one column:
// the two K-reductions against the parent state Hc (in-lane, then across the
// wave's four row groups), the corrected value u_j and the output o_j
// (written by the first row group, with the factor record and the staged
// u); returns u_j in every lane.
template <int DK, int R, bool VG>
__device__ inline float node_step(const VerifyArgs &a, const SerialStage &s, const float (&Hc)[R], int j, int b,
                                  int h, int c, int g, int row0, int col, bool delta) {
  const float *kj = s.ks + j * DK + row0;
  const float *qj = s.qs + j * DK + row0;
  const float *gj = s.gs + j * DK + row0;
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
  const float al = s.als[j], be = s.bes[j];
  const float u = delta ? be * (s.vs[j * kSliceCols + c] - al * sk) : s.vs[j * kSliceCols + c];
  const float o = __builtin_fmaf(kq, u, al * sq);
  if (g == 0) {
    const size_t sj = ((size_t)b * a.n + j) * a.H + h;
    a.out[sj * a.dv + col] = o;
    a.fu[sj * a.dv + col] = u;
    s.us[j * kSliceCols + c] = u;
  }
  return u;
}

// H <- diag(g_x) H + k_x u^T on a lane's rows (a scalar gate: alpha_x H + k_x u^T)
template <int DK, int R, bool VG>
__device__ inline void advance(const SerialStage &s, float (&Hs)[R], int x, int row0, float u) {
  const float al = s.als[x];
  const float *kx = s.ks + x * DK + row0;
  const float *gx = s.gs + x * DK + row0;
#pragma unroll
  for (int r = 0; r < R; ++r) Hs[r] = apply_factor(Hs[r], VG ? gx[r] : al, kx[r], u);
}

}  // namespace sla
