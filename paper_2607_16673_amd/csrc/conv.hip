// conv.hip -- topology-aware short causal convolution and conv-state commit.
//
// The GDN layer mixes every channel of its q, k and v projections over the
// last K (= 4) tokens with a depthwise causal convolution and SiLU, and keeps
// the last K - 1 committed inputs as a second per-layer state C next to S
// (SpecLA §7).  Under speculation the tokens in front of draft node j are the
// nodes of its own root path, nearest first, and past the root the rows of C,
// newest first (tree mask of §4.2).  Commit (§5.1-5.2) shifts the accepted
// inputs into C; fused in front of a verification it is the delayed update
// of §5.2 applied to C.
//
// One workgroup = one sequence b and a chunk of 512 channels, 8 per lane,
// with up to four waves (eight above 32 nodes) that split the draft's nodes.
// Each wave first reads
// the parent row into lanes (lane j holds node j), then issues its share of
// the chunk's draft rows straight into LDS (global_load_lds_dwordx4: 16
// bytes per lane, one instruction per bf16 row, two per fp32 row), and the
// weights into registers.  Topology and path checks are wave shuffles.  The
// accepted rows are gathered (at most K - 1 of them, whatever the path
// length) and the committed rows written back.  After one barrier every
// node's window is read from LDS by ancestor index: K fused multiply-adds
// per channel, SiLU, one 16-byte store per lane.  Wave 0 alone reads the
// conv state, checks topology and path, gathers the accepted rows and writes
// the committed rows back; the others read them from LDS.
// A 1-node draft (the decode step) takes a single wave that reads its row
// and the conv state straight into registers (conv_node_kernel).
// The bound is HBM: the draft rows and outputs stream once, the conv state
// is read and written once, the weights are shared by every sequence.
#include "device.hpp"
#include "layer_ops.hpp"

namespace sla {
namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kCpl = 8;               // channels per lane
constexpr int kChunk = kWave * kCpl;  // channels per workgroup
constexpr int kConvWaves = 8;         // most waves per verify workgroup (nodes split between them)

// 16-byte pieces per lane per row
template <typename XT>
constexpr int kPieces = (int)sizeof(XT) * kCpl / 16;

__device__ __forceinline__ void widen(const u32x4 (&r)[1], float (&f)[kCpl], bf16) {
  const uint32_t w[4] = {r[0].x, r[0].y, r[0].z, r[0].w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = __uint_as_float(w[e] << 16);
    f[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
  }
}

__device__ __forceinline__ void widen(const u32x4 (&r)[2], float (&f)[kCpl], float) {
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    f[4 * q] = __uint_as_float(r[q].x);
    f[4 * q + 1] = __uint_as_float(r[q].y);
    f[4 * q + 2] = __uint_as_float(r[q].z);
    f[4 * q + 3] = __uint_as_float(r[q].w);
  }
}

// round to nearest even, the bf16 pattern in the low 16 bits
__device__ __forceinline__ uint32_t bf16_rne(float x) {
  return (uint32_t)__builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
}

__device__ __forceinline__ void store_row(bf16 *y, const float (&f)[kCpl]) {
  u32x4 o;
  o.x = bf16_rne(f[0]) | (bf16_rne(f[1]) << 16);
  o.y = bf16_rne(f[2]) | (bf16_rne(f[3]) << 16);
  o.z = bf16_rne(f[4]) | (bf16_rne(f[5]) << 16);
  o.w = bf16_rne(f[6]) | (bf16_rne(f[7]) << 16);
  __builtin_nontemporal_store(o, reinterpret_cast<u32x4 *>(y));
}

// fp32 rows: a lane's 32 bytes go out as two 16-byte stores, so each store
// instruction covers half of every line; the default policy lets the L2 merge
// the halves (a streaming hint writes them separately)
__device__ __forceinline__ void store_row(float *y, const float (&f)[kCpl]) {
  reinterpret_cast<f32x4 *>(y)[0] = f32x4{f[0], f[1], f[2], f[3]};
  reinterpret_cast<f32x4 *>(y)[1] = f32x4{f[4], f[5], f[6], f[7]};
}

template <typename XT>
__device__ __forceinline__ void load_row(const XT *p, float (&f)[kCpl]) {
  u32x4 r[kPieces<XT>];
#pragma unroll
  for (int q = 0; q < kPieces<XT>; ++q) r[q] = reinterpret_cast<const u32x4 *>(p)[q];
  widen(r, f, XT{});
}

__device__ __forceinline__ void load_f8(const float *p, float (&f)[kCpl]) {
  const f32x4 a = reinterpret_cast<const f32x4 *>(p)[0];
  const f32x4 b = reinterpret_cast<const f32x4 *>(p)[1];
  f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
  f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
}

// committed conv-state rows: a lane's 32 bytes are contiguous and a wave's
// 2 KB cover whole lines, so they stream past the L2 (measured: the 1-node
// decode chain 14.0 -> 13.65 us per launch, the others unchanged; rows left
// dirty in the L2 are written back at the end of the kernel)
__device__ __forceinline__ void store_f8(float *p, const float (&f)[kCpl]) {
  __builtin_nontemporal_store(f32x4{f[0], f[1], f[2], f[3]}, reinterpret_cast<f32x4 *>(p));
  __builtin_nontemporal_store(f32x4{f[4], f[5], f[6], f[7]}, reinterpret_cast<f32x4 *>(p) + 1);
}

// silu(a) = a / (1 + exp(-a)) with the hardware exp2 and reciprocal (each
// about 1 ulp): relative error ~1e-6, far below one bf16 rounding and below
// the fp32 bar.  a -> -inf gives -0 (exp2 overflows to inf, rcp(inf) = 0).
__device__ __forceinline__ float silu(float a) {
  return a * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(a * -1.4426950408889634f));
}

// The path of a pending (or standalone) commit, checked against the parent
// row of the draft it came from; lane t holds step t.  Returns SLA_OK or
// SLA_ERR_PATH (wave-uniform).  `node` is lane t's node id (clamped).
__device__ __forceinline__ int check_commit_path(const int32_t *parent_row, const int32_t *path_row, int n,
                                                 int len, int lane, int &node) {
  const int pv = lane < n ? parent_row[lane] : -2;
  const int a = lane < n ? path_row[lane] : -1;
  int prev = __shfl_up(a, 1);
  if (lane == 0) prev = -1;
  const bool inrange = a >= 0 && a < n;
  node = inrange ? a : 0;
  const int pa = __shfl(pv, node);
  const bool bad = (len < 0 || len > n) || (lane < len && (!inrange || pa != prev));
  return wave_any(bad) ? SLA_ERR_PATH : SLA_OK;
}

// Committed rows after accepting len nodes: with Z = [C[0..K-2], x_{a_1}..
// x_{a_len}], the new C[r] is Z[len + r].  `cs` holds this lane's channels of
// the old rows on entry and of the new rows on return; `node` is the lane
// layout of the path (lane t: node of step t).
template <typename XT, int K>
__device__ __forceinline__ void commit_rows(float (&cs)[K > 1 ? K - 1 : 1][kCpl], const XT *xrows, size_t row_stride,
                                            int len, int node, int c0) {
  if constexpr (K > 1) {
    float nw[K - 1][kCpl];
#pragma unroll
    for (int r = 0; r < K - 1; ++r) {
      const int z = len + r;  // position in Z
      if (z < K - 1) {
#pragma unroll
        for (int e = 0; e < kCpl; ++e) nw[r][e] = cs[z][e];
      } else {
        const int a = __builtin_amdgcn_readlane(node, z - (K - 1));
        load_row(xrows + (size_t)a * row_stride + c0, nw[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < K - 1; ++r)
#pragma unroll
      for (int e = 0; e < kCpl; ++e) cs[r][e] = nw[r][e];
  }
}

// Lane j's window sources: for lag s, the node id of its s-th ancestor, or
// -(r + 1) for committed row r once the path has run out.
template <int K>
__device__ __forceinline__ void window_sources(int p, int lane, int (&src)[K]) {
  int a = lane, past = 0;
#pragma unroll
  for (int s = 0; s < K; ++s) {
    src[s] = a >= 0 ? a : -(K - 1 - past) - 1;
    if (s + 1 < K) {
      const int pa = __shfl(p, a >= 0 ? a : 0);
      if (a >= 0) {
        a = pa;
        if (a < 0) past = 1;
      } else {
        ++past;
      }
    }
  }
}

template <typename XT, int K>
__global__ __launch_bounds__(kConvWaves * kWave) void conv_verify_kernel(ConvArgs a) {
  constexpr int P = kPieces<XT>;
  constexpr int KR = K > 1 ? K - 1 : 1;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  const int w = threadIdx.x / kWave;
  const int l = threadIdx.x % kWave;
  const int nw = blockDim.x / kWave;
  const int nchunks = (a.D + kChunk - 1) / kChunk;
  const int b = blockIdx.x / nchunks;
  const int c0raw = (blockIdx.x % nchunks) * kChunk + l * kCpl;
  const bool live = c0raw < a.D;
  const int c0 = live ? c0raw : a.D - kCpl;  // lanes past the last channel re-read the last 8
  const int n = a.n;
  // LDS: draft rows [n][P][64 lanes x 16 B], then the committed rows
  // [K-1][2][64 x 16 B] (fp32, 8 channels per lane), then the verdict
  f32x4 *crows = reinterpret_cast<f32x4 *>(lds + (size_t)n * P * kWave * 16);
  int *s_err = reinterpret_cast<int *>(crows + KR * 2 * kWave);
  // with several waves: [2K pieces][64 lanes], lane l's weights, 16 bytes per piece
  f32x4 *wrows = reinterpret_cast<f32x4 *>(s_err + 4);

  // every wave: the parent row (lane j: node j), then its share of the draft
  // rows (j = w, w + nw, ...) straight into LDS
  const int p = l < n ? a.parent[(size_t)b * n + l] : -1;
  int pv = -2, pa = -1, plen = 0;
  const int pn = a.has_pending ? a.pend_n : 1;
  if (w == 0 && a.has_pending) {  // wave 0 also takes the pending path
    pv = l < pn ? a.pend_parent[(size_t)b * pn + l] : -2;
    pa = l < pn ? a.path[(size_t)b * pn + l] : -1;
    plen = a.len[b];
  }
  const XT *x = static_cast<const XT *>(a.x) + (size_t)b * n * a.D;
  for (int j = w; j < n; j += nw)
#pragma unroll
    for (int q = 0; q < P; ++q)
      load_lds16(reinterpret_cast<const unsigned char *>(x + (size_t)j * a.D + c0) + 16 * q,
                 lds + (size_t)(j * P + q) * (kWave * 16));
  // with several waves, the chunk's weights once per workgroup (a lane's 8 K
  // floats are contiguous in [D][K]): piece v of every lane in one
  // instruction, laid out [v][lane] so that the reads after the barrier are
  // conflict-free.  A single wave reads its own straight into registers.
  const bool wshared = nw > 1;
  if (wshared)
    for (int v = w; v < 2 * K; v += nw) load_lds16(a.weight + (size_t)c0 * K + 4 * v, wrows + v * kWave);
  int src[K];
  window_sources<K>(p, l, src);

  // wave 0: topology, the pending path, the committed rows (at most K - 1
  // accepted rows gathered) into LDS and, with a pending path, back to HBM
  if (w == 0) {
    float cs[KR][kCpl];
    float *crow = K > 1 ? a.conv_state + (size_t)b * (K - 1) * a.D + c0 : nullptr;
    if constexpr (K > 1) {
#pragma unroll
      for (int r = 0; r < K - 1; ++r) load_f8(crow + (size_t)r * a.D, cs[r]);
    }
    int err = wave_any(l < n && (p < -1 || p >= l)) ? SLA_ERR_TOPOLOGY : SLA_OK;
    if (err == SLA_OK && a.has_pending) {
      int prev = __shfl_up(pa, 1);
      if (l == 0) prev = -1;
      const bool inrange = pa >= 0 && pa < pn;
      const int node = inrange ? pa : 0;
      const int ppar = __shfl(pv, node);
      const bool bad = (plen < 0 || plen > pn) || (l < plen && (!inrange || ppar != prev));
      err = wave_any(bad) ? SLA_ERR_PATH : SLA_OK;
      if (err == SLA_OK && plen > 0) {
        commit_rows<XT, K>(cs, static_cast<const XT *>(a.pend_x) + (size_t)b * pn * a.D, (size_t)a.D, plen, node,
                           c0);
        if constexpr (K > 1) {
          if (live) {
#pragma unroll
            for (int r = 0; r < K - 1; ++r) store_f8(crow + (size_t)r * a.D, cs[r]);
          }
        }
      }
    }
    if constexpr (K > 1) {
#pragma unroll
      for (int r = 0; r < K - 1; ++r) {
        crows[(2 * r) * kWave + l] = f32x4{cs[r][0], cs[r][1], cs[r][2], cs[r][3]};
        crows[(2 * r + 1) * kWave + l] = f32x4{cs[r][4], cs[r][5], cs[r][6], cs[r][7]};
      }
    }
    if (l == 0) *s_err = err;
    if (a.status && l == 0 && blockIdx.x % nchunks == 0) a.status[b] = err;
  }
  float bias[kCpl];
  if (a.bias) {
    load_f8(a.bias + c0, bias);
  } else {
#pragma unroll
    for (int e = 0; e < kCpl; ++e) bias[e] = 0.f;
  }
  __builtin_amdgcn_s_waitcnt(0);  // this wave's rows and weight pieces have landed
  __syncthreads();                // and every other wave's, and the committed rows
  if (*s_err != SLA_OK) return;
  float wt[K][kCpl];
  {
    float flat[K * kCpl];
    const f32x4 *wv = reinterpret_cast<const f32x4 *>(a.weight + (size_t)c0 * K);
#pragma unroll
    for (int v = 0; v < 2 * K; ++v) {
      const f32x4 t = wshared ? wrows[v * kWave + l] : wv[v];
      flat[4 * v] = t.x; flat[4 * v + 1] = t.y; flat[4 * v + 2] = t.z; flat[4 * v + 3] = t.w;
    }
#pragma unroll
    for (int e = 0; e < kCpl; ++e)
#pragma unroll
      for (int i = 0; i < K; ++i) wt[i][e] = flat[e * K + i];
  }

  XT *y = static_cast<XT *>(a.y) + (size_t)b * n * a.D + c0;
  const u32x4 *rows = reinterpret_cast<const u32x4 *>(lds) + l;
  for (int j = w; j < n; j += nw) {
    float acc[kCpl];
#pragma unroll
    for (int e = 0; e < kCpl; ++e) acc[e] = bias[e];
#pragma unroll
    for (int s = 0; s < K; ++s) {
      const int sj = __builtin_amdgcn_readlane(src[s], j);  // lag s of node j
      float z[kCpl];
      if (sj >= 0) {
        u32x4 r[P];
#pragma unroll
        for (int q = 0; q < P; ++q) r[q] = rows[(sj * P + q) * kWave];
        widen(r, z, XT{});
      } else {
        const int rr = -sj - 1;  // committed row
        const f32x4 lo = crows[(2 * rr) * kWave + l], hi = crows[(2 * rr + 1) * kWave + l];
        z[0] = lo.x; z[1] = lo.y; z[2] = lo.z; z[3] = lo.w;
        z[4] = hi.x; z[5] = hi.y; z[6] = hi.z; z[7] = hi.w;
      }
      // tap K-1-s multiplies lag s
#pragma unroll
      for (int e = 0; e < kCpl; ++e) acc[e] = __builtin_fmaf(wt[K - 1 - s][e], z[e], acc[e]);
    }
    if (a.activation == SLA_ACT_SILU) {
#pragma unroll
      for (int e = 0; e < kCpl; ++e) acc[e] = silu(acc[e]);
    }
    if (live) store_row(y + (size_t)j * a.D, acc);
  }
}

// 1-node drafts (the decode step): one wave per sequence and 512-channel
// chunk reads its node's row straight into registers -- no LDS stage, no
// barrier (measured at batch 256: 13.7 -> 13.05 us per launch).  With more
// nodes the LDS stage above wins: reading every window row from memory made
// 16-node trees 30% and 64-node trees 68% slower.
template <typename XT, int K>
__global__ __launch_bounds__(kWave) void conv_node_kernel(ConvArgs a) {
  constexpr int KR = K > 1 ? K - 1 : 1;
  const int l = threadIdx.x;
  const int nchunks = (a.D + kChunk - 1) / kChunk;
  const int b = blockIdx.x / nchunks;
  const int c0raw = (blockIdx.x % nchunks) * kChunk + l * kCpl;
  const bool live = c0raw < a.D;
  const int c0 = live ? c0raw : a.D - kCpl;  // lanes past the last channel re-read the last 8
  const int n = a.n;
  const int pn = a.has_pending ? a.pend_n : 1;

  const int p = l < n ? a.parent[(size_t)b * n + l] : -1;
  int pv = -2, pa = -1, plen = 0;
  if (a.has_pending) {
    pv = l < pn ? a.pend_parent[(size_t)b * pn + l] : -2;
    pa = l < pn ? a.path[(size_t)b * pn + l] : -1;
    plen = a.len[b];
  }
  float cs[KR][kCpl];
  float *crow = K > 1 ? a.conv_state + (size_t)b * (K - 1) * a.D + c0 : nullptr;
  if constexpr (K > 1) {
#pragma unroll
    for (int r = 0; r < K - 1; ++r) load_f8(crow + (size_t)r * a.D, cs[r]);
  }
  float wt[K][kCpl];
  {
    float flat[K * kCpl];
    const f32x4 *wv = reinterpret_cast<const f32x4 *>(a.weight + (size_t)c0 * K);
#pragma unroll
    for (int v = 0; v < 2 * K; ++v) {
      const f32x4 t = wv[v];
      flat[4 * v] = t.x; flat[4 * v + 1] = t.y; flat[4 * v + 2] = t.z; flat[4 * v + 3] = t.w;
    }
#pragma unroll
    for (int e = 0; e < kCpl; ++e)
#pragma unroll
      for (int i = 0; i < K; ++i) wt[i][e] = flat[e * K + i];
  }
  float bias[kCpl];
  if (a.bias) {
    load_f8(a.bias + c0, bias);
  } else {
#pragma unroll
    for (int e = 0; e < kCpl; ++e) bias[e] = 0.f;
  }
  int err = wave_any(l < n && (p < -1 || p >= l)) ? SLA_ERR_TOPOLOGY : SLA_OK;
  int node = 0;
  if (err == SLA_OK && a.has_pending) {
    int prev = __shfl_up(pa, 1);
    if (l == 0) prev = -1;
    const bool inrange = pa >= 0 && pa < pn;
    node = inrange ? pa : 0;
    const int ppar = __shfl(pv, node);
    const bool bad = (plen < 0 || plen > pn) || (l < plen && (!inrange || ppar != prev));
    err = wave_any(bad) ? SLA_ERR_PATH : SLA_OK;
  }
  if (a.status && l == 0 && blockIdx.x % nchunks == 0) a.status[b] = err;
  if (err != SLA_OK) return;
  if (a.has_pending && plen > 0) {
    commit_rows<XT, K>(cs, static_cast<const XT *>(a.pend_x) + (size_t)b * pn * a.D, (size_t)a.D, plen, node, c0);
    if constexpr (K > 1) {
      if (live) {
#pragma unroll
        for (int r = 0; r < K - 1; ++r) store_f8(crow + (size_t)r * a.D, cs[r]);
      }
    }
  }
  int src[K];
  window_sources<K>(p, l, src);

  const XT *x = static_cast<const XT *>(a.x) + (size_t)b * n * a.D + c0;
  XT *y = static_cast<XT *>(a.y) + (size_t)b * n * a.D + c0;
  {
    const int j = 0;
    float acc[kCpl];
#pragma unroll
    for (int e = 0; e < kCpl; ++e) acc[e] = bias[e];
#pragma unroll
    for (int s = 0; s < K; ++s) {
      const int sj = __builtin_amdgcn_readlane(src[s], j);  // lag s of node j
      float z[kCpl];
      if (sj >= 0) {
        load_row(x + (size_t)sj * a.D, z);
      } else {
        const int rr = -sj - 1;  // committed row
#pragma unroll
        for (int e = 0; e < kCpl; ++e) z[e] = cs[0][e];
#pragma unroll
        for (int r = 1; r < KR; ++r)
          if (rr == r)
#pragma unroll
            for (int e = 0; e < kCpl; ++e) z[e] = cs[r][e];
      }
#pragma unroll
      for (int e = 0; e < kCpl; ++e) acc[e] = __builtin_fmaf(wt[K - 1 - s][e], z[e], acc[e]);
    }
    if (a.activation == SLA_ACT_SILU) {
#pragma unroll
      for (int e = 0; e < kCpl; ++e) acc[e] = silu(acc[e]);
    }
    if (live) store_row(y + (size_t)j * a.D, acc);
  }
}

template <typename XT, int K>
__global__ __launch_bounds__(kWave) void conv_commit_kernel(ConvArgs a) {
  constexpr int KR = K > 1 ? K - 1 : 1;
  const int l = threadIdx.x;
  const int nchunks = (a.D + kChunk - 1) / kChunk;
  const int b = blockIdx.x / nchunks;
  const int c0raw = (blockIdx.x % nchunks) * kChunk + l * kCpl;
  const bool live = c0raw < a.D;
  const int c0 = live ? c0raw : a.D - kCpl;
  float cs[KR][kCpl];
  float *crow = K > 1 ? a.conv_state + (size_t)b * (K - 1) * a.D + c0 : nullptr;
  if constexpr (K > 1) {
#pragma unroll
    for (int r = 0; r < K - 1; ++r) load_f8(crow + (size_t)r * a.D, cs[r]);
  }
  const int n = a.n;
  const int len = a.len[b];
  int node = 0;
  const int err = check_commit_path(a.parent + (size_t)b * n, a.path + (size_t)b * n, n, len, l, node);
  if (a.status && l == 0 && blockIdx.x % nchunks == 0) a.status[b] = err;
  if (err != SLA_OK || len == 0) return;
  commit_rows<XT, K>(cs, static_cast<const XT *>(a.x) + (size_t)b * n * a.D, (size_t)a.D, len, node, c0);
  if constexpr (K > 1) {
    if (live) {
#pragma unroll
      for (int r = 0; r < K - 1; ++r) store_f8(crow + (size_t)r * a.D, cs[r]);
    }
  }
}

template <typename XT, int K>
hipError_t launch_k(const ConvArgs &a, bool commit, hipStream_t s) {
  const int nchunks = (a.D + kChunk - 1) / kChunk;
  const dim3 grid((unsigned)((size_t)a.B * nchunks));
  if (commit) {
    hipLaunchKernelGGL((conv_commit_kernel<XT, K>), grid, dim3(kWave), 0, s, a);
    return hipGetLastError();
  }
  if (a.n == 1) {
    hipLaunchKernelGGL((conv_node_kernel<XT, K>), grid, dim3(kWave), 0, s, a);
    return hipGetLastError();
  }
  const int K1 = K > 1 ? K - 1 : 1;
  // the waves split the draft's nodes: eight for drafts of more than 32 nodes,
  // else up to four (measured at batch 256, 64-node trees: 157 -> 143 us per
  // launch with eight; at batch 64, 16-node trees eight were 25% slower); with
  // several, the chunk's weights are staged in LDS once
  const int waves = a.n > 32 ? kConvWaves : (a.n < 4 ? a.n : 4);
  const size_t lds = (size_t)a.n * kPieces<XT> * kWave * 16 + (size_t)K1 * 2 * kWave * 16 + 16 +
                     (waves > 1 ? (size_t)2 * K * kWave * 16 : 0);
  auto kern = conv_verify_kernel<XT, K>;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, grid, dim3(waves * kWave), lds, s, a);
  return hipGetLastError();
}

template <typename XT>
hipError_t launch_t(const ConvArgs &a, bool commit, hipStream_t s) {
  switch (a.K) {
    case 1: return launch_k<XT, 1>(a, commit, s);
    case 2: return launch_k<XT, 2>(a, commit, s);
    case 3: return launch_k<XT, 3>(a, commit, s);
    case 4: return launch_k<XT, 4>(a, commit, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_conv(const ConvArgs &a, int dtype, bool commit, hipStream_t s) {
  return dtype == SLA_DTYPE_BF16 ? launch_t<bf16>(a, commit, s) : launch_t<float>(a, commit, s);
}

}  // namespace sla
