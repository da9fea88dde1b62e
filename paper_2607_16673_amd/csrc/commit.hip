// commit.hip -- immediate accepted-path commit (SpecLA §5.2 "Immediate
// update") and the device topology table (§4.2 tree mask) for inspection.
//
// Commit streams each unit's fp32 state once in and once out and applies the
// accepted path's factor records in path order,
//     H[i][c] <- alpha_a H[i][c] + k_a[i] u_a[c]     (a = path[0], path[1], ...)
// through the same rank-one expression as the fused prologue of verification,
// so the two routes produce bitwise equal states.
#include "device.hpp"
#include "kernels.hpp"

namespace sla {
namespace {

constexpr int kCommitThreads = 256;

template <typename T>
__global__ __launch_bounds__(kCommitThreads) void commit_kernel(CommitArgs a) {
  __shared__ int s_err;
  __shared__ int s_node[SLA_MAX_NODES];
  __shared__ float s_alpha[SLA_MAX_NODES];
  const int tid = threadIdx.x;
  const int H = a.H, dk = a.dk, dv = a.dv, n = a.n;
  const int b = blockIdx.x / H;
  const int h = blockIdx.x % H;
  const int32_t *path = a.path + (size_t)b * n;
  if (tid < kWave) {
    const int len = a.len[b];
    const int e = check_path(a.parent + (size_t)b * n, n, path, len, tid);
    if (tid == 0) s_err = e;
    if (e == SLA_OK && tid < len) {
      s_node[tid] = path[tid];
      s_alpha[tid] = a.alpha[((size_t)b * n + path[tid]) * H + h];
    }
  }
  __syncthreads();
  const int err = s_err;
  if (h == 0 && tid == 0 && a.status) a.status[b] = err;
  if (err != SLA_OK) return;
  const int len = a.len[b];
  if (len == 0) return;

  const T *fk = static_cast<const T *>(a.k);
  float *st = a.state + ((size_t)b * H + h) * dk * dv;
  const int cq = dv / 4;  // float4 columns per row
  const int total = dk * cq;
  for (int f = tid; f < total; f += kCommitThreads) {
    const int i = f / cq;
    const int c = (f - i * cq) * 4;
    float4 x = *reinterpret_cast<const float4 *>(st + (size_t)i * dv + c);
    for (int t = 0; t < len; ++t) {
      const size_t s = ((size_t)b * n + s_node[t]) * H + h;
      const float al = s_alpha[t];
      const float ki = to_f32(fk[s * dk + i]);
      const float4 u = *reinterpret_cast<const float4 *>(a.u + s * dv + c);
      x.x = apply_factor(x.x, al, ki, u.x);
      x.y = apply_factor(x.y, al, ki, u.y);
      x.z = apply_factor(x.z, al, ki, u.z);
      x.w = apply_factor(x.w, al, ki, u.w);
    }
    *reinterpret_cast<float4 *>(st + (size_t)i * dv + c) = x;
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

}  // namespace

hipError_t launch_commit(const CommitArgs &a, int dtype, hipStream_t s) {
  const dim3 grid((unsigned)((size_t)a.B * a.H));
  if (dtype == SLA_DTYPE_BF16)
    hipLaunchKernelGGL(commit_kernel<bf16>, grid, dim3(kCommitThreads), 0, s, a);
  else
    hipLaunchKernelGGL(commit_kernel<float>, grid, dim3(kCommitThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_topology(const TopologyArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(topology_kernel, dim3((unsigned)a.B), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace sla
