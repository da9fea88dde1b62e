// commit.hip -- immediate accepted-path commit (SpecLA §5.2 "Immediate
// update") and the device topology table (§4.2 tree mask) for inspection.
//
// Commit streams each unit's fp32 state once in and once out and applies the
// accepted path's factor records in path order,
//     H[i][c] <- g_a[i] H[i][c] + k_a[i] u_a[c]     (a = path[0], path[1], ...)
// with g_a[i] = alpha_a for the scalar-gate families and the per-key gate of
// GLA, through the same rank-one expression as the fused prologue of
// verification, so the two routes produce bitwise equal states.
#include "device.hpp"
#include "kernels.hpp"

namespace sla {
namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

constexpr int kCommitThreads = 256;
constexpr int kCommitCols = 64;   // state columns per workgroup
constexpr int kCommitStage = 8;   // path records staged in LDS; longer paths read the rest directly

// One workgroup = one (b, h) unit's 64-column slab, all d_k rows (the slabs
// of a unit numbered back to back on one XCD in full launches).  Thread t
// owns float4 column group t % 16 of rows t / 16 + 16 r: 16 threads cover a
// 256-byte row segment, so every access is whole 128-byte lines.  The slab
// is read first thing, before the path is known; wave 0 reads the path, the
// parent row and the gates whole (validation takes no dependent read), then
// gathers the records the path names straight into LDS.  An invalid path
// reports its status and leaves the state untouched.
// VG: the records hold d_k gates each (GLA), staged like the key rows.
template <typename T, int DK, bool VG>
__global__ __launch_bounds__(kCommitThreads) void commit_kernel(CommitArgs a) {
  constexpr int R = DK / 16;  // float4 groups per thread
  __shared__ int s_err, s_len;
  __shared__ float s_alpha[kCommitStage];
  __shared__ __attribute__((aligned(16))) unsigned char s_kraw[kCommitStage * DK * sizeof(T)];
  __shared__ __attribute__((aligned(16))) float s_u[kCommitStage][kCommitCols];
  __shared__ __attribute__((aligned(16))) float s_g[VG ? kCommitStage * DK : 4];  // [kCommitStage][DK]
  const T *s_k = reinterpret_cast<const T *>(s_kraw);  // [kCommitStage][DK]
  const int tid = threadIdx.x;
  const int w = tid / kWave, l = tid % kWave;
  const int H = a.H, dv = a.dv, n = a.n;
  const int nslab = (dv + kCommitCols - 1) / kCommitCols;
  size_t uid;
  int slab;
  if (!xcd_unit_slab((size_t)a.B * H, nslab, a.xcd_group, uid, slab)) return;  // padding: no barrier follows
  const int h = (int)(uid % H);
  const int b = (int)(uid / H);
  const size_t rowp = (size_t)b * n;

  // wave 0: everything the path check needs, ahead of its slab reads
  int len = 0, node = -1, par = -2;
  float al = 0.f;
  if (w == 0) {
    len = a.len[b];
    node = l < n ? a.path[rowp + l] : -1;
    par = l < n ? a.parent[rowp + l] : -2;
    if (!VG) al = l < n ? a.alpha[(rowp + l) * H + h] : 0.f;
  }
  // the slab, before the path is known
  const int cg = slab * kCommitCols + (tid % 16) * 4;  // first column of this thread's float4
  const bool cl = cg < dv;
  float *st = a.state + ((size_t)b * H + h) * DK * dv;
  // whole 128-byte lines, each read once: non-temporal (measured on an
  // in-place pass over 24 rotating 64 MiB states: 5.3 -> 6.2 TB/s with the
  // stores written through)
  const rsrc_t sr = make_rsrc(st, (uint32_t)DK * dv * 4);
  // (below one workgroup per CU the launch is latency-bound and the default
  // policy measured faster: the batch-1 commit at d_v 256, 12.9 -> 12.2 us)
  float4 x[R];
  if (cl) {
    const uint32_t vo = (uint32_t)((tid / 16) * dv + cg) * 4;
    if (a.write_through) {
#pragma unroll
      for (int r = 0; r < R; ++r) x[r] = buf_load_f4<kPolicyStream>(sr, vo, (uint32_t)(16 * r * dv) * 4);
    } else {
#pragma unroll
      for (int r = 0; r < R; ++r) x[r] = buf_load_f4<kPolicyDefault>(sr, vo, (uint32_t)(16 * r * dv) * 4);
    }
  }
  if (w == 0) {
    // step t is node path[t], whose parent must be path[t - 1] (-1 for t = 0)
    const bool inrange = node >= 0 && node < n;
    const int nodec = inrange ? node : 0;
    int prev = __shfl_up(node, 1);
    if (l == 0) prev = -1;
    const int pp = __shfl(par, nodec);
    const float pa = __shfl(al, nodec);
    const bool bad = (len < 0 || len > n) || (l < len && (!inrange || pp != prev));
    const int err = wave_any(bad) ? SLA_ERR_PATH : SLA_OK;
    if (l == 0) {
      s_err = err;
      s_len = len;
    }
    if (l < kCommitStage) s_alpha[l] = pa;
    if (h == 0 && slab == 0 && l == 0 && a.status) a.status[b] = err;
    // records of the first steps (indices clamped into the store): key rows
    // and this slab's corrected values, straight into LDS
    const T *fk = static_cast<const T *>(a.k);
    constexpr int KC = DK * (int)sizeof(T) / 16;  // 16-byte chunks per key row
    constexpr int KI = kCommitStage * KC / kWave;
    constexpr int GC = DK * 4 / 16;  // 16-byte chunks per gate row
    constexpr int GI = VG ? kCommitStage * GC / kWave : 0;
    int nt[KI], ng[GI > 0 ? GI : 1];  // shuffles first: an LDS instruction after an LDS-DMA load waits for it
#pragma unroll
    for (int i = 0; i < KI; ++i) nt[i] = __shfl(nodec, (i * kWave + l) / KC);
#pragma unroll
    for (int i = 0; i < GI; ++i) ng[i] = __shfl(nodec, (i * kWave + l) / GC);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < KI; ++i)
      load_lds16(fk + ((rowp + nt[i]) * H + h) * DK + ((i * kWave + l) % KC) * (16 / sizeof(T)), s_kraw + i * kWave * 16);
#pragma unroll
    for (int i = 0; i < GI; ++i)
      load_lds16(a.alpha + ((rowp + ng[i]) * H + h) * DK + ((i * kWave + l) % GC) * 4, s_g + i * kWave * 4);
#pragma unroll
    for (int t = 0; t < kCommitStage; ++t) {
      const int ntt = __builtin_amdgcn_readlane(nodec, t);
      const int c = slab * kCommitCols + l;
      load_lds4(a.u + ((rowp + ntt) * H + h) * dv + (c < dv ? c : dv - 1), &s_u[t][0]);
    }
    __builtin_amdgcn_s_waitcnt(0);  // the records have landed
  }
  __syncthreads();
  if (s_err != SLA_OK || !cl) return;
  len = s_len;
  const int cs = (tid % 16) * 4;  // column within the slab
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int i = tid / 16 + 16 * r;
    for (int t = 0; t < len && t < kCommitStage; ++t) {
      const float alt = VG ? s_g[t * DK + i] : s_alpha[t];
      const float ki = to_f32(s_k[t * DK + i]);
      const float4 u = *reinterpret_cast<const float4 *>(&s_u[t][cs]);
      x[r].x = apply_factor(x[r].x, alt, ki, u.x);
      x[r].y = apply_factor(x[r].y, alt, ki, u.y);
      x[r].z = apply_factor(x[r].z, alt, ki, u.z);
      x[r].w = apply_factor(x[r].w, alt, ki, u.w);
    }
    // paths longer than the stage read their records directly
    for (int t = kCommitStage; t < len; ++t) {
      const size_t s = (rowp + a.path[rowp + t]) * H + h;
      const float alt = VG ? a.alpha[s * DK + i] : a.alpha[s];
      const float ki = to_f32(static_cast<const T *>(a.k)[s * DK + i]);
      const float4 u = *reinterpret_cast<const float4 *>(a.u + s * dv + cg);
      x[r].x = apply_factor(x[r].x, alt, ki, u.x);
      x[r].y = apply_factor(x[r].y, alt, ki, u.y);
      x[r].z = apply_factor(x[r].z, alt, ki, u.z);
      x[r].w = apply_factor(x[r].w, alt, ki, u.w);
    }
  }
  if (len == 0) return;
  // whole lines; with a workgroup per CU or more, written through at device
  // scope, so that nothing is left dirty in the L2 for the end of the kernel
  // (measured against plain stores: the separate route at batched tree
  // serving 55.3 -> 48.4 us per layer, the 1-node decode chain 334 -> 293 us)
  if (a.write_through) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const u32x4 v = {__float_as_uint(x[r].x), __float_as_uint(x[r].y), __float_as_uint(x[r].z), __float_as_uint(x[r].w)};
      __builtin_amdgcn_raw_buffer_store_b128(v, sr, (uint32_t)(((tid / 16 + 16 * r) * dv + cg) * 4), 0, kPolicyStreamDevice);
    }
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r) *reinterpret_cast<float4 *>(st + (size_t)(tid / 16 + 16 * r) * dv + cg) = x[r];
  }
}

__global__ __launch_bounds__(kWave) void topology_kernel(TopologyArgs a) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int n = a.n;
  NodeTopo t;
  const int err = build_topology(a.parent + (size_t)b * n, n, lane, false, t);
  if (lane == 0) a.status[b] = err;
  if (err != SLA_OK || lane >= n) return;
  const size_t r = (size_t)b * n;
  a.depth[r + lane] = t.depth;
  a.anc[r + lane] = t.anc;
  a.order[r + t.pos] = lane;
  a.n_children[r + lane] = t.n_children;
}

int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    return 256;
  return cus;
}

template <typename T, int DK>
hipError_t launch_commit_dk(const CommitArgs &a, hipStream_t s) {
  auto kern = a.gate_vec ? commit_kernel<T, DK, true> : commit_kernel<T, DK, false>;
  const int nslab = (a.dv + kCommitCols - 1) / kCommitCols;
  const size_t groups = (size_t)a.B * a.H * nslab;
  CommitArgs b = a;
  b.write_through = groups >= (size_t)device_cus();
  b.xcd_group = b.write_through && nslab >= kXcdGroupMin;
  hipLaunchKernelGGL(kern, dim3((unsigned)xcd_grid((size_t)a.B * a.H, nslab, b.xcd_group)), dim3(kCommitThreads), 0, s, b);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_commit_t(const CommitArgs &a, hipStream_t s) {
  switch (a.dk) {
    case 64: return launch_commit_dk<T, 64>(a, s);
    case 128: return launch_commit_dk<T, 128>(a, s);
    case 256: return launch_commit_dk<T, 256>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_commit(const CommitArgs &a, int dtype, hipStream_t s) {
  return dtype == SLA_DTYPE_BF16 ? launch_commit_t<bf16>(a, s) : launch_commit_t<float>(a, s);
}

hipError_t launch_topology(const TopologyArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(topology_kernel, dim3((unsigned)a.B), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace sla
