// decode.hip -- verification of 1-node drafts (the decode step: a chain of
// one node, §4 with n = 1), with the delayed state update of §5.2 fused in
// front of it.
//
// With one node there is no tree to mask and no state to advance past the
// node: the call is the standalone commit's stream over the state plus two
// reductions per state column,
//     a = H0^T k,  b = H0^T (g * q),  u = beta (v - alpha a),  o = alpha b + (k . q) u
// (the GDN step read at its own node; DeltaNet: alpha = 1; no delta rule:
// u = v; GLA: per-key gates g in b and in the pending records, alpha = 1).
//
// One workgroup = one (b, h) unit's 64-column slab, all d_k rows (the slabs
// of a unit numbered back to back on one XCD in full launches), laid out as in the commit
// kernel: thread t owns float4 column group t % 16 of rows
// t / 16 + 16 r, so every state access is whole 128-byte lines, and the
// committed rows are written through at device scope when the launch has a
// workgroup per CU or more (nothing left dirty in the L2 at the end of the
// kernel).  Wave 0 validates the pending path and gathers its records into
// LDS, as the commit kernel does, with the same rank-one expression, so the
// fused and standalone routes give bitwise equal states.  The column sums
// run over the thread's rows, then across the four row groups of a wave
// (lane xor 16, 32), then across the four waves through LDS.
#include "device.hpp"
#include "kernels.hpp"

namespace sla {
namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kThreads = 256;
constexpr int kCols = 64;   // state columns per workgroup
constexpr int kStage = 8;   // path records staged in LDS; longer paths read the rest directly

template <typename T, int DK, bool VG>
__global__ __launch_bounds__(kThreads) void decode_kernel(VerifyArgs a) {
  constexpr int R = DK / 16;  // rows per thread
  __shared__ int s_err, s_len;
  __shared__ float s_alpha[kStage];
  __shared__ __attribute__((aligned(16))) unsigned char s_kraw[kStage * DK * sizeof(T)];
  __shared__ __attribute__((aligned(16))) float s_u[kStage][kCols];
  __shared__ __attribute__((aligned(16))) float s_g[VG ? kStage * DK : 4];
  __shared__ __attribute__((aligned(16))) float s_red[4][2][kCols];  // per wave: a, b
  __shared__ float s_kq[4];
  const T *s_k = reinterpret_cast<const T *>(s_kraw);
  const int tid = threadIdx.x;
  const int w = tid / kWave, l = tid % kWave;
  const int H = a.H, dv = a.dv;
  const int nslab = (dv + kCols - 1) / kCols;
  size_t uid;
  int slab;
  if (!xcd_unit_slab((size_t)a.B * H, nslab, a.xcd_group, uid, slab)) return;  // padding: no barrier follows
  const int h = (int)(uid % H);
  const int b = (int)(uid / H);
  const size_t node = (size_t)b * H + h;  // record index of the draft's only node: ((b * 1 + 0) H + h)
  const bool delta = a.family == SLA_FAMILY_GDN || a.family == SLA_FAMILY_DELTANET;

  // wave 0: the draft's parent and the pending path, ahead of the slab reads
  const int pn = a.has_pending ? a.pend.n : 1;
  const size_t rowp = (size_t)b * pn;
  int len = 0, pnode = -1, ppar = -2, p0 = 0;
  float pal = 0.f;
  if (w == 0) {
    p0 = a.parent[b];
    if (a.has_pending) {
      len = a.pend.len[b];
      pnode = l < pn ? a.pend.path[rowp + l] : -1;
      ppar = l < pn ? a.pend.parent[rowp + l] : -2;
      if (!VG) pal = l < pn ? a.pend.alpha[(rowp + l) * H + h] : 0.f;
    }
  }
  // the slab, the node's key and query rows, its values and gates
  const int cg = slab * kCols + (tid % 16) * 4;  // first column of this thread's float4
  const bool cl = cg < dv;
  const int cgc = cl ? cg : dv - 4;
  float *st = a.state + node * DK * dv;
  // whole 128-byte lines, each read once: non-temporal (measured on an
  // in-place pass over 24 rotating 64 MiB states: 5.3 -> 6.2 TB/s with the
  // stores written through)
  const rsrc_t sr = make_rsrc(st, (uint32_t)DK * dv * 4);
  // (below one workgroup per CU the launch is latency-bound: default policy)
  float4 x[R];
  const uint32_t vo = (uint32_t)((tid / 16) * dv + cgc) * 4;
  if (a.write_through) {
#pragma unroll
    for (int r = 0; r < R; ++r) x[r] = buf_load_f4<kPolicyStream>(sr, vo, (uint32_t)(16 * r * dv) * 4);
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r) x[r] = buf_load_f4<kPolicyDefault>(sr, vo, (uint32_t)(16 * r * dv) * 4);
  }
  const T *kg = static_cast<const T *>(a.k) + node * DK;
  const T *qg = static_cast<const T *>(a.q) + node * DK;
  float kr[R], qr[R], qgr[R];  // qgr: the query scaled by the node's per-key gates (GLA)
#pragma unroll
  for (int r = 0; r < R; ++r) {
    kr[r] = to_f32(kg[tid / 16 + 16 * r]);
    qr[r] = to_f32(qg[tid / 16 + 16 * r]);
    qgr[r] = VG ? qr[r] * a.alpha[node * DK + tid / 16 + 16 * r] : qr[r];
  }
  float vv[4];
  {
    const T *vg = static_cast<const T *>(a.v) + node * dv + cgc;
#pragma unroll
    for (int c = 0; c < 4; ++c) vv[c] = to_f32(vg[c]);
  }
  const float al = (VG || a.family == SLA_FAMILY_DELTANET) ? 1.f : a.alpha[node];
  const float be = delta ? a.beta[node] : 0.f;

  if (w == 0) {
    int err = wave_any(p0 != -1) ? SLA_ERR_TOPOLOGY : SLA_OK;
    const bool inrange = pnode >= 0 && pnode < pn;
    const int nodec = inrange ? pnode : 0;
    if (err == SLA_OK && a.has_pending) {
      int prev = __shfl_up(pnode, 1);
      if (l == 0) prev = -1;
      const int pp = __shfl(ppar, nodec);
      const bool bad = (len < 0 || len > pn) || (l < len && (!inrange || pp != prev));
      err = wave_any(bad) ? SLA_ERR_PATH : SLA_OK;
    }
    const float pa = __shfl(pal, nodec);
    if (l == 0) {
      s_err = err;
      s_len = a.has_pending ? len : 0;
    }
    if (l < kStage) s_alpha[l] = pa;
    if (h == 0 && slab == 0 && l == 0 && a.status) a.status[b] = err;
    if (a.has_pending) {
      // records of the first steps (indices clamped into the store): key
      // rows, gate rows and this slab's corrected values, straight into LDS
      const T *pk = static_cast<const T *>(a.pend.k);
      constexpr int KC = DK * (int)sizeof(T) / 16;
      constexpr int KI = kStage * KC / kWave;
      constexpr int GC = DK * 4 / 16;
      constexpr int GI = VG ? kStage * GC / kWave : 0;
      int nt[KI], ng[GI > 0 ? GI : 1];  // shuffles first: an LDS instruction after an LDS-DMA load waits for it
#pragma unroll
      for (int i = 0; i < KI; ++i) nt[i] = __shfl(nodec, (i * kWave + l) / KC);
#pragma unroll
      for (int i = 0; i < GI; ++i) ng[i] = __shfl(nodec, (i * kWave + l) / GC);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < KI; ++i)
        load_lds16(pk + ((rowp + nt[i]) * H + h) * DK + ((i * kWave + l) % KC) * (16 / sizeof(T)), s_kraw + i * kWave * 16);
#pragma unroll
      for (int i = 0; i < GI; ++i)
        load_lds16(a.pend.alpha + ((rowp + ng[i]) * H + h) * DK + ((i * kWave + l) % GC) * 4, s_g + i * kWave * 4);
#pragma unroll
      for (int t = 0; t < kStage; ++t) {
        const int ntt = __builtin_amdgcn_readlane(nodec, t);
        const int c = slab * kCols + l;
        load_lds4(a.pend.u + ((rowp + ntt) * H + h) * dv + (c < dv ? c : dv - 1), &s_u[t][0]);
      }
      __builtin_amdgcn_s_waitcnt(0);  // the records have landed
    }
  }
  __syncthreads();
  if (s_err != SLA_OK) return;
  len = s_len;

  // delayed update: the accepted records, root first, then the write-back
  if (len > 0) {
    const int cs = (tid % 16) * 4;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int i = tid / 16 + 16 * r;
      for (int t = 0; t < len && t < kStage; ++t) {
        const float alt = VG ? s_g[t * DK + i] : s_alpha[t];
        const float ki = to_f32(s_k[t * DK + i]);
        const float4 u = *reinterpret_cast<const float4 *>(&s_u[t][cs]);
        x[r].x = apply_factor(x[r].x, alt, ki, u.x);
        x[r].y = apply_factor(x[r].y, alt, ki, u.y);
        x[r].z = apply_factor(x[r].z, alt, ki, u.z);
        x[r].w = apply_factor(x[r].w, alt, ki, u.w);
      }
      for (int t = kStage; t < len; ++t) {
        const size_t s = (rowp + a.pend.path[rowp + t]) * H + h;
        const float alt = VG ? a.pend.alpha[s * DK + i] : a.pend.alpha[s];
        const float ki = to_f32(static_cast<const T *>(a.pend.k)[s * DK + i]);
        const float4 u = *reinterpret_cast<const float4 *>(a.pend.u + s * dv + cgc);
        x[r].x = apply_factor(x[r].x, alt, ki, u.x);
        x[r].y = apply_factor(x[r].y, alt, ki, u.y);
        x[r].z = apply_factor(x[r].z, alt, ki, u.z);
        x[r].w = apply_factor(x[r].w, alt, ki, u.w);
      }
    }
    if (cl) {
      if (a.write_through) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const u32x4 v = {__float_as_uint(x[r].x), __float_as_uint(x[r].y), __float_as_uint(x[r].z),
                           __float_as_uint(x[r].w)};
          __builtin_amdgcn_raw_buffer_store_b128(v, sr, (uint32_t)(((tid / 16 + 16 * r) * dv + cg) * 4), 0,
                                                 kPolicyStreamDevice);
        }
      } else {
#pragma unroll
        for (int r = 0; r < R; ++r) *reinterpret_cast<float4 *>(st + (size_t)(tid / 16 + 16 * r) * dv + cg) = x[r];
      }
    }
  }

  // column sums over the thread's rows, the wave's row groups, then the waves
  float sa[4] = {0.f, 0.f, 0.f, 0.f}, sb[4] = {0.f, 0.f, 0.f, 0.f}, kq = 0.f;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    sa[0] = __builtin_fmaf(x[r].x, kr[r], sa[0]);
    sa[1] = __builtin_fmaf(x[r].y, kr[r], sa[1]);
    sa[2] = __builtin_fmaf(x[r].z, kr[r], sa[2]);
    sa[3] = __builtin_fmaf(x[r].w, kr[r], sa[3]);
    sb[0] = __builtin_fmaf(x[r].x, qgr[r], sb[0]);
    sb[1] = __builtin_fmaf(x[r].y, qgr[r], sb[1]);
    sb[2] = __builtin_fmaf(x[r].z, qgr[r], sb[2]);
    sb[3] = __builtin_fmaf(x[r].w, qgr[r], sb[3]);
    kq = __builtin_fmaf(kr[r], qr[r], kq);
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    sa[c] += __shfl_xor(sa[c], 16);
    sb[c] += __shfl_xor(sb[c], 16);
    sa[c] += __shfl_xor(sa[c], 32);
    sb[c] += __shfl_xor(sb[c], 32);
  }
  kq += __shfl_xor(kq, 16);
  kq += __shfl_xor(kq, 32);
  if (l < 16) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      s_red[w][0][4 * l + c] = sa[c];
      s_red[w][1][4 * l + c] = sb[c];
    }
    if (l == 0) s_kq[w] = kq;
  }
  __syncthreads();
  if (w == 0 && l < 16 && cl) {
    const float kqt = (s_kq[0] + s_kq[1]) + (s_kq[2] + s_kq[3]);
    float o[4], u[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float at = (s_red[0][0][4 * l + c] + s_red[1][0][4 * l + c]) + (s_red[2][0][4 * l + c] + s_red[3][0][4 * l + c]);
      const float bt = (s_red[0][1][4 * l + c] + s_red[1][1][4 * l + c]) + (s_red[2][1][4 * l + c] + s_red[3][1][4 * l + c]);
      u[c] = delta ? be * (vv[c] - al * at) : vv[c];
      o[c] = __builtin_fmaf(kqt, u[c], al * bt);
    }
    __builtin_nontemporal_store(f32x4{o[0], o[1], o[2], o[3]}, reinterpret_cast<f32x4 *>(a.out + node * dv + cg));
    __builtin_nontemporal_store(f32x4{u[0], u[1], u[2], u[3]}, reinterpret_cast<f32x4 *>(a.fu + node * dv + cg));
  }
  // records that do not depend on the slab: key, gate(s), parent
  if (slab == 0) {
    T *fk = static_cast<T *>(a.fk);
    for (int i = tid; i < DK; i += kThreads) {
      fk[node * DK + i] = kg[i];
      if (VG) a.falpha[node * DK + i] = a.alpha[node * DK + i];
    }
    if (tid == 0) {
      if (!VG) a.falpha[node] = al;
      if (h == 0) a.fparent[b] = -1;
    }
  }
}

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

template <typename T, int DK>
hipError_t launch_dk(const VerifyArgs &a, hipStream_t s) {
  auto kern = a.family == SLA_FAMILY_GLA ? decode_kernel<T, DK, true> : decode_kernel<T, DK, false>;
  const int nslab = (a.dv + kCols - 1) / kCols;
  const size_t groups = (size_t)a.B * a.H * nslab;
  VerifyArgs b = a;
  b.write_through = groups >= (size_t)device_cus();
  b.xcd_group = b.write_through && nslab >= kXcdGroupMin;
  hipLaunchKernelGGL(kern, dim3((unsigned)xcd_grid((size_t)a.B * a.H, nslab, b.xcd_group)), dim3(kThreads), 0, s, b);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_t(const VerifyArgs &a, hipStream_t s) {
  switch (a.dk) {
    case 64: return launch_dk<T, 64>(a, s);
    case 128: return launch_dk<T, 128>(a, s);
    case 256: return launch_dk<T, 256>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_verify_decode(const VerifyArgs &a, int dtype, hipStream_t s) {
  if (a.n != 1) return hipErrorInvalidValue;
  return dtype == SLA_DTYPE_BF16 ? launch_t<bf16>(a, s) : launch_t<float>(a, s);
}

}  // namespace sla
