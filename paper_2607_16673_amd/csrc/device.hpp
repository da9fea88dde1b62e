// device.hpp -- device-side building blocks shared by the libsla kernels
// (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sla.h"

namespace sla {

constexpr int kWave = 64;

// ------------------------------------------------------------------ dtypes
// bf16 activations are carried as raw 16-bit patterns; widening to fp32 is
// exact (append 16 zero bits).
struct bf16 {
  uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return __uint_as_float((uint32_t)x.bits << 16); }

// Load N consecutive activations starting at p (16-byte aligned when the
// row offset is a multiple of 16 bytes) and widen them to fp32.
template <int N>
__device__ __forceinline__ void load_f32(const float *__restrict__ p, float (&out)[N]) {
  static_assert(N % 4 == 0, "vector width");
#pragma unroll
  for (int i = 0; i < N; i += 4) {
    float4 x = *reinterpret_cast<const float4 *>(p + i);
    out[i] = x.x;
    out[i + 1] = x.y;
    out[i + 2] = x.z;
    out[i + 3] = x.w;
  }
}

template <int N>
__device__ __forceinline__ void load_f32(const bf16 *__restrict__ p, float (&out)[N]) {
  static_assert(N % 8 == 0, "vector width");
#pragma unroll
  for (int i = 0; i < N; i += 8) {
    uint4 x = *reinterpret_cast<const uint4 *>(p + i);
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      out[i + 2 * e] = __uint_as_float(w[e] << 16);
      out[i + 2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  }
}

// ------------------------------------------------------ buffer resources
// Raw buffer descriptors: a 128-bit base/size descriptor in scalar
// registers, a per-lane 32-bit VGPR offset and a wave-uniform SGPR offset.
// Strided accesses then cost one VGPR per lane instead of a 64-bit address
// per access.  Reads at offsets >= the descriptor's byte count return zero
// and writes there are dropped.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kBufWord3 = 0x00020000;  // raw 32-bit dword access, no swizzle
constexpr int kPolicyDefault = 0;
constexpr int kPolicyStream = 2;  // non-temporal: data touched once
constexpr int kPolicyStreamDevice = 18;  // non-temporal, written through at device scope (nt | sc1)

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, kBufWord3);
}

template <int POLICY>
__device__ __forceinline__ float buf_load_f32(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, POLICY));
}

template <int POLICY>
__device__ __forceinline__ void buf_store_f32(float x, rsrc_t r, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x), r, voff, soff, POLICY);
}

// four consecutive fp32 values (16 bytes)
template <int POLICY>
__device__ __forceinline__ float4 buf_load_f4(rsrc_t r, uint32_t voff, uint32_t soff) {
  typedef __attribute__((ext_vector_type(4))) float f4;
  const f4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, POLICY);
  return make_float4(v[0], v[1], v[2], v[3]);
}

template <int POLICY>
__device__ __forceinline__ void buf_store_f4(float4 x, rsrc_t r, uint32_t voff, uint32_t soff) {
  typedef __attribute__((ext_vector_type(4))) float f4;
  const f4 v = {x.x, x.y, x.z, x.w};
  __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, soff, POLICY);
}

// one bf16 activation, widened to fp32
__device__ __forceinline__ float buf_load_bf16(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, kPolicyDefault) << 16);
}

// ------------------------------------------------------ direct LDS loads
// global_load_lds: each lane's bytes go straight from memory to LDS, at
// lds_wave_base + size * lane (the base is wave-uniform); no registers are
// involved.  An LDS instruction issued after one of these waits for it.
// Kernels call these helpers, never the builtin itself: a kernel template
// whose body names the builtin gets no host-side launch stub (the link then
// fails on an undefined kernel symbol).
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void load_lds16(const void *g, void *lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (lds_void *)(lds_wave_base), 16, 0, 0);
}

__device__ __forceinline__ void load_lds4(const void *g, void *lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (lds_void *)(lds_wave_base), 4, 0, 0);
}

// ------------------------------------------------ XCD-grouped numbering
// Workgroup i of a launch runs on XCD i mod 8, and each XCD takes its
// workgroups in order.  Numbering (unit, slab) pairs so that the nslab
// column slabs of one unit are consecutive on one XCD makes the slabs that
// run at the same time cover whole rows of the unit's state, so the memory
// system sees contiguous rows instead of row segments one row pitch apart
// (in-place pass over 3 x 512 MiB states with d_v 256 in 64-column slabs:
// 5.6 -> 6.1 TB/s).  With two slabs per unit (d_v 128) the plain order,
// which puts them on neighbouring XCDs, measured faster (standalone commit
// over 24 rotating 64 MiB states: 25.9 us against 27.4 us grouped), and so
// did launches of fewer workgroups than CUs (the batch-1 commit of 8 heads at
// d_v 256: 12.2 us against 13.6 us grouped), so the caller groups from four
// slabs per unit on and with at least one workgroup per CU.  The grid is
// xcd_grid(units, nslab, group) workgroups; the padding workgroups get false.
constexpr int kXcdCount = 8;
constexpr int kXcdGroupMin = 4;  // slabs per unit from which they are grouped

__host__ __device__ inline size_t xcd_grid(size_t units, int nslab, bool group) {
  if (!group) return units * (size_t)nslab;
  return (units + kXcdCount - 1) / kXcdCount * kXcdCount * (size_t)nslab;
}

__device__ inline bool xcd_unit_slab(size_t units, int nslab, bool group, size_t &unit, int &slab) {
  const size_t i = blockIdx.x;
  if (!group) {
    slab = (int)(i % nslab);
    unit = i / nslab;
    return unit < units;
  }
  const size_t k = i / kXcdCount;  // position in this XCD's sequence
  slab = (int)(k % nslab);
  unit = (k / nslab) * kXcdCount + i % kXcdCount;
  return unit < units;
}

// ------------------------------------------------------- rank-one update
// One accepted (or materialised) node a advances the transposed state
// H = S^T elementwise:  H[i][c] <- alpha_a * H[i][c] + k_a[i] * u_a[c].
// Every kernel that advances a state -- standalone commit, the pending
// prologue of verification and the in-kernel materialisation of internal
// nodes -- goes through this one expression, so the routes agree bitwise.
__device__ __forceinline__ float apply_factor(float h, float alpha, float k_i, float u_c) {
  return __builtin_fmaf(k_i, u_c, alpha * h);
}

// ------------------------------------------------------ wave primitives
__device__ __forceinline__ bool wave_any(bool p) { return __ballot(p) != 0ull; }

__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int lane) {
  uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, lane);
  uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(x >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

// ------------------------------------------------------ topology table
// Built by one wavefront, lane j owning node j (n <= 64).  The result is
// wave-uniform in `err`; the per-node fields are valid for lane < n.
struct NodeTopo {
  int32_t parent;
  int32_t depth;     // |P(j)|, roots have depth 1
  int32_t n_children;
  int32_t pos;       // position of j in the DFS pre-order
  uint64_t anc;      // inclusive ancestor mask
};

// Returns SLA_OK or SLA_ERR_TOPOLOGY (wave-uniform).
__device__ inline int build_topology(const int32_t *__restrict__ parent_row, int n, int lane,
                                     bool chain_hint, NodeTopo &t) {
  const bool live = lane < n;
  const int32_t p = live ? parent_row[lane] : -1;
  bool bad = live && (p < -1 || p >= lane);
  if (chain_hint) bad = bad || (live && p != lane - 1);
  if (wave_any(bad)) return SLA_ERR_TOPOLOGY;

  // Inclusive ancestor mask by walking parent pointers; parents have
  // smaller indices, so every walk ends within `depth` steps.
  uint64_t m = live ? (1ull << lane) : 0ull;
  int a = p;
  while (wave_any(a >= 0)) {
    const int src = a >= 0 ? a : 0;
    const int pa = __shfl(p, src);
    if (a >= 0) m |= 1ull << a;
    a = a >= 0 ? pa : -1;
  }

  // Child counts and DFS pre-order positions.  Node i precedes node j in
  // the pre-order iff i is a strict ancestor of j, or neither contains the
  // other and the branch of i below their deepest common ancestor has the
  // smaller index (children and roots are visited in ascending order; the
  // shallowest non-shared ancestor is the lowest set bit because parents
  // carry smaller indices than their children).
  int kids = 0, pos = 0;
  for (int i = 0; i < n; ++i) {
    const int pi = __builtin_amdgcn_readlane(p, i);
    const uint64_t mi = readlane_u64(m, i);
    kids += (pi == lane);
    if (i == lane) continue;
    const uint64_t common = mi & m;
    const uint64_t only_i = mi & ~common, only_j = m & ~common;
    if (only_i == 0ull) {
      pos += 1;  // i is a strict ancestor of j
    } else if (only_j != 0ull) {
      pos += (__builtin_ctzll(only_i) < __builtin_ctzll(only_j)) ? 1 : 0;
    }
  }
  t.parent = p;
  t.anc = m;
  t.depth = __popcll(m);
  t.n_children = kids;
  t.pos = pos;
  return SLA_OK;
}

// Validate an accepted path (lanes t < len check their step) against a
// parent row of length n.  Returns SLA_OK or SLA_ERR_PATH (wave-uniform).
__device__ inline int check_path(const int32_t *__restrict__ parent_row, int n,
                                 const int32_t *__restrict__ path_row, int len, int lane) {
  if (len < 0 || len > n) return SLA_ERR_PATH;
  bool bad = false;
  if (lane < len) {
    const int a = path_row[lane];
    const int prev = lane == 0 ? -1 : path_row[lane - 1];
    bad = a < 0 || a >= n || parent_row[a] != prev;
  }
  return wave_any(bad) ? SLA_ERR_PATH : SLA_OK;
}

}  // namespace sla
