// api.cpp -- host side of the libsla C ABI (declared in include/sla.h):
// argument validation, alias checks, route selection and kernel launches on
// the caller's stream, plus the synchronous host topology helpers.
// Nothing here allocates device memory or keeps state between calls.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "kernels.hpp"
#include "layer_ops.hpp"
#include "sla.h"

namespace {

constexpr int kVersion = 20000;  // 2.0.0: the route moved into sla_shape

bool dk_ok(int dk) { return dk == 64 || dk == 128 || dk == 256; }

size_t act_bytes(int dtype) { return dtype == SLA_DTYPE_BF16 ? 2 : 4; }

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};

Range range_of(const void *p, size_t bytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return Range{a, a + bytes};
}

bool overlaps(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

int check_shape(const sla_shape *s) {
  if (!s) return SLA_ERR_NULL;
  if (s->batch < 1 || s->heads < 1 || s->n_nodes < 1 || s->n_nodes > SLA_MAX_NODES) return SLA_ERR_SHAPE;
  if (s->d_k < 1 || s->d_v < 16 || s->d_v > 1024 || s->d_v % 16 != 0) return SLA_ERR_SHAPE;
  if (s->qkv_dtype != SLA_DTYPE_F32 && s->qkv_dtype != SLA_DTYPE_BF16) return SLA_ERR_DTYPE;
  if (s->topology != SLA_TOPO_TREE && s->topology != SLA_TOPO_CHAIN) return SLA_ERR_SHAPE;
  if (s->family < SLA_FAMILY_GDN || s->family > SLA_FAMILY_GLA) return SLA_ERR_SHAPE;
  if (!dk_ok(s->d_k)) return SLA_ERR_UNSUPPORTED;
  // grid sizes stay far inside 2^31 workgroups
  if ((uint64_t)s->batch * (uint64_t)s->heads * (uint64_t)(s->d_v / 16) > (1ull << 30)) return SLA_ERR_SHAPE;
  // one sequence's rows of one tensor (all nodes and heads) are addressed with
  // 32-bit byte offsets from the unit's first row
  const uint64_t width = (uint64_t)(s->d_v > s->d_k ? s->d_v : s->d_k);
  if ((uint64_t)SLA_MAX_NODES * (uint64_t)s->heads * width * 4 >= (1ull << 31)) return SLA_ERR_SHAPE;
  return SLA_OK;
}

struct FactorSizes {
  size_t k, u, alpha, parent;
};

// gates per (b, j, h): one per key dimension for GLA, else one
size_t gate_width(const sla_shape *s) { return s->family == SLA_FAMILY_GLA ? (size_t)s->d_k : 1; }

FactorSizes factor_sizes(const sla_shape *s, int n) {
  const size_t bnh = (size_t)s->batch * n * s->heads;
  return FactorSizes{bnh * s->d_k * act_bytes(s->qkv_dtype), bnh * s->d_v * sizeof(float),
                     bnh * gate_width(s) * sizeof(float), (size_t)s->batch * n * sizeof(int32_t)};
}

// which inputs the family's step reads
bool reads_alpha(int family) { return family != SLA_FAMILY_DELTANET; }
bool reads_beta(int family) { return family == SLA_FAMILY_GDN || family == SLA_FAMILY_DELTANET; }

bool factors_complete(const sla_factors *f) { return f && f->k && f->u && f->alpha && f->parent; }

int hip_status(hipError_t e) { return e == hipSuccess ? SLA_OK : SLA_ERR_HIP; }

int check_conv_shape(const sla_conv_shape *s) {
  if (!s) return SLA_ERR_NULL;
  if (s->batch < 1 || s->n_nodes < 1 || s->n_nodes > SLA_MAX_NODES) return SLA_ERR_SHAPE;
  if (s->channels < 8 || s->channels % 8 != 0 || s->channels > (1 << 20)) return SLA_ERR_SHAPE;
  if (s->kernel_size < 1 || s->kernel_size > SLA_CONV_MAX_KERNEL) return SLA_ERR_SHAPE;
  if (s->x_dtype != SLA_DTYPE_F32 && s->x_dtype != SLA_DTYPE_BF16) return SLA_ERR_DTYPE;
  if (s->activation != SLA_ACT_NONE && s->activation != SLA_ACT_SILU) return SLA_ERR_SHAPE;
  if ((uint64_t)s->batch * (uint64_t)((s->channels + 511) / 512) > (1ull << 30)) return SLA_ERR_SHAPE;
  return SLA_OK;
}

}  // namespace

extern "C" {

int sla_version(void) { return kVersion; }

const char *sla_status_string(int status) {
  switch (status) {
    case SLA_OK: return "ok";
    case SLA_ERR_NULL: return "null pointer";
    case SLA_ERR_SHAPE: return "size out of range";
    case SLA_ERR_DTYPE: return "unknown activation dtype";
    case SLA_ERR_TOPOLOGY: return "parent array is not in topological order";
    case SLA_ERR_PATH: return "accepted path is not a root path";
    case SLA_ERR_ALIAS: return "pending factors overlap output factors";
    case SLA_ERR_UNSUPPORTED: return "unsupported configuration";
    case SLA_ERR_HIP: return "HIP runtime error";
    case SLA_ERR_SCORE: return "draft log-probability above 0 or NaN";
    default: return "unknown status";
  }
}

size_t sla_factors_bytes(const sla_shape *shape) {
  if (check_shape(shape) != SLA_OK) return 0;
  const FactorSizes f = factor_sizes(shape, shape->n_nodes);
  return f.k + f.u + f.alpha + f.parent;
}

int sla_verify(const sla_shape *shape, float *state, const sla_pending *pending,
               const void *q, const void *k, const void *v, const float *alpha, const float *beta,
               const int32_t *parent_idx, float *out, const sla_factors *factors, int32_t *status,
               hipStream_t stream) {
  int st = check_shape(shape);
  if (st != SLA_OK) return st;
  const int fam = shape->family;
  const int route = shape->route;
  if (!state || !q || !k || !v || (reads_alpha(fam) && !alpha) || (reads_beta(fam) && !beta) || !parent_idx ||
      !out || !factors_complete(factors))
    return SLA_ERR_NULL;
  if (route != SLA_ROUTE_AUTO && route != SLA_ROUTE_SERIAL && route != SLA_ROUTE_PARALLEL && route != SLA_ROUTE_HYBRID)
    return SLA_ERR_SHAPE;
  if (pending) {
    if (!factors_complete(&pending->f) || !pending->path || !pending->len) return SLA_ERR_NULL;
    if (pending->n_nodes < 1 || pending->n_nodes > SLA_MAX_NODES) return SLA_ERR_SHAPE;
    const FactorSizes po = factor_sizes(shape, shape->n_nodes);
    const FactorSizes pi = factor_sizes(shape, pending->n_nodes);
    const Range outs[4] = {range_of(factors->k, po.k), range_of(factors->u, po.u),
                           range_of(factors->alpha, po.alpha), range_of(factors->parent, po.parent)};
    const Range ins[4] = {range_of(pending->f.k, pi.k), range_of(pending->f.u, pi.u),
                          range_of(pending->f.alpha, pi.alpha), range_of(pending->f.parent, pi.parent)};
    for (const Range &x : outs)
      for (const Range &y : ins)
        if (overlaps(x, y)) return SLA_ERR_ALIAS;
    if (!aligned16(pending->f.k) || !aligned16(pending->f.u)) return SLA_ERR_UNSUPPORTED;
    if (fam == SLA_FAMILY_GLA && !aligned16(pending->f.alpha)) return SLA_ERR_UNSUPPORTED;
  }
  if (!aligned16(state) || !aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out) ||
      !aligned16(factors->k) || !aligned16(factors->u))
    return SLA_ERR_UNSUPPORTED;
  if (fam == SLA_FAMILY_GLA && (!aligned16(alpha) || !aligned16(factors->alpha))) return SLA_ERR_UNSUPPORTED;

  const bool chain = shape->topology == SLA_TOPO_CHAIN;
  bool use_parallel;
  const bool parallel_ok = sla::parallel_supported(shape->d_k, shape->d_v, shape->n_nodes, shape->qkv_dtype);
  if (route == SLA_ROUTE_PARALLEL) {
    if (!parallel_ok) return SLA_ERR_UNSUPPORTED;
    use_parallel = true;
  } else if (route == SLA_ROUTE_SERIAL || route == SLA_ROUTE_HYBRID) {
    use_parallel = false;
  } else {
    // drafts of either activation dtype, chains included, go to the
    // tree-masked contraction on the matrix cores: its one dense contraction
    // streams the state better than per-node reductions do (fp32 16-node
    // trees at batch 64: 47.8 us against 129 us serial; 64-node trees at
    // batch 256: 0.76 ms against 9.7 ms on the hybrid)
    use_parallel = parallel_ok;
  }

  sla::VerifyArgs a;
  memset(&a, 0, sizeof(a));
  a.B = shape->batch;
  a.H = shape->heads;
  a.dk = shape->d_k;
  a.dv = shape->d_v;
  a.n = shape->n_nodes;
  a.chain = chain;
  a.family = fam;
  a.has_pending = pending != nullptr;
  a.state = state;
  if (pending) {
    a.pend.k = pending->f.k;
    a.pend.u = pending->f.u;
    a.pend.alpha = pending->f.alpha;
    a.pend.parent = pending->f.parent;
    a.pend.n = pending->n_nodes;
    a.pend.path = pending->path;
    a.pend.len = pending->len;
  }
  a.q = q;
  a.k = k;
  a.v = v;
  a.alpha = alpha;
  a.beta = beta;
  a.parent = parent_idx;
  a.out = out;
  a.fk = factors->k;
  a.fu = factors->u;
  a.falpha = factors->alpha;
  a.fparent = factors->parent;
  a.status = status;
  // trees the contraction cannot stage on chip take, on the automatic route,
  // the chain-decomposed hybrid where its parallel chains pay (fp32 64-node
  // trees at batch 256: 9.7 ms against 11.8 ms serial; launches of few
  // workgroups, where latency decides), else the serial route (fp32 16-node
  // trees at batch 64: 129 us serial against 228 us hybrid)
  const bool few = (size_t)shape->batch * shape->heads * (shape->d_v / 16) <= 512;
  const bool hybrid_pays = !chain && shape->n_nodes > 1 && (shape->n_nodes > 32 || few);
  const bool hybrid = route == SLA_ROUTE_HYBRID || (route == SLA_ROUTE_AUTO && !use_parallel && hybrid_pays);
  hipError_t e;
  if (route == SLA_ROUTE_AUTO && shape->n_nodes == 1)  // the decode step: its own streaming kernel
    e = sla::launch_verify_decode(a, shape->qkv_dtype, stream);
  else if (hybrid)
    e = sla::launch_verify_hybrid(a, shape->qkv_dtype, stream);
  else
    e = use_parallel ? sla::launch_verify_parallel(a, shape->qkv_dtype, stream)
                     : sla::launch_verify_serial(a, shape->qkv_dtype, stream);
  // a draft whose on-chip stage does not fit the contraction's LDS (more
  // than 32 nodes at d_k = 256 with GLA's per-key gates or fp32 activations)
  // is refused before any launch; the automatic route then takes the hybrid
  // or the serial one by the rule above
  if (e == hipErrorInvalidConfiguration && use_parallel && route == SLA_ROUTE_AUTO)
    e = hybrid_pays ? sla::launch_verify_hybrid(a, shape->qkv_dtype, stream)
                    : sla::launch_verify_serial(a, shape->qkv_dtype, stream);
  if (e == hipErrorInvalidConfiguration) return SLA_ERR_UNSUPPORTED;
  return hip_status(e);
}

int sla_commit(const sla_shape *shape, float *state, const sla_factors *factors, const int32_t *path,
               const int32_t *len, int32_t *status, hipStream_t stream) {
  int st = check_shape(shape);
  if (st != SLA_OK) return st;
  if (!state || !factors_complete(factors) || !path || !len) return SLA_ERR_NULL;
  if (!aligned16(state) || !aligned16(factors->u)) return SLA_ERR_UNSUPPORTED;
  if (shape->family == SLA_FAMILY_GLA && !aligned16(factors->alpha)) return SLA_ERR_UNSUPPORTED;
  sla::CommitArgs a;
  a.B = shape->batch;
  a.H = shape->heads;
  a.dk = shape->d_k;
  a.dv = shape->d_v;
  a.n = shape->n_nodes;
  a.gate_vec = shape->family == SLA_FAMILY_GLA;
  a.state = state;
  a.k = factors->k;
  a.u = factors->u;
  a.alpha = factors->alpha;
  a.parent = factors->parent;
  a.path = path;
  a.len = len;
  a.status = status;
  return hip_status(sla::launch_commit(a, shape->qkv_dtype, stream));
}

int sla_conv_verify(const sla_conv_shape *shape, float *conv_state, const sla_conv_pending *pending,
                    const void *x, const float *weight, const float *bias, const int32_t *parent_idx, void *y,
                    int32_t *status, hipStream_t stream) {
  int st = check_conv_shape(shape);
  if (st != SLA_OK) return st;
  const int K = shape->kernel_size;
  if (!x || !weight || !parent_idx || !y || (K > 1 && !conv_state)) return SLA_ERR_NULL;
  const size_t w = act_bytes(shape->x_dtype);
  if (pending) {
    if (!pending->x || !pending->parent || !pending->path || !pending->len) return SLA_ERR_NULL;
    if (pending->n_nodes < 1 || pending->n_nodes > SLA_MAX_NODES) return SLA_ERR_SHAPE;
    const size_t out_bytes = (size_t)shape->batch * shape->n_nodes * shape->channels * w;
    const size_t in_bytes = (size_t)shape->batch * pending->n_nodes * shape->channels * w;
    if (overlaps(range_of(y, out_bytes), range_of(pending->x, in_bytes))) return SLA_ERR_ALIAS;
    if (!aligned16(pending->x)) return SLA_ERR_UNSUPPORTED;
  }
  if (!aligned16(x) || !aligned16(y) || !aligned16(weight) || (K > 1 && !aligned16(conv_state)))
    return SLA_ERR_UNSUPPORTED;
  sla::ConvArgs a;
  memset(&a, 0, sizeof(a));
  a.B = shape->batch;
  a.D = shape->channels;
  a.K = K;
  a.n = shape->n_nodes;
  a.activation = shape->activation;
  a.has_pending = pending != nullptr;
  a.conv_state = conv_state;
  a.x = x;
  a.weight = weight;
  a.bias = bias;
  a.parent = parent_idx;
  a.y = y;
  if (pending) {
    a.pend_x = pending->x;
    a.pend_parent = pending->parent;
    a.pend_n = pending->n_nodes;
    a.path = pending->path;
    a.len = pending->len;
  }
  a.status = status;
  return hip_status(sla::launch_conv(a, shape->x_dtype, false, stream));
}

int sla_conv_commit(const sla_conv_shape *shape, float *conv_state, const void *x, const int32_t *parent_idx,
                    const int32_t *path, const int32_t *len, int32_t *status, hipStream_t stream) {
  int st = check_conv_shape(shape);
  if (st != SLA_OK) return st;
  const int K = shape->kernel_size;
  if (!x || !parent_idx || !path || !len || (K > 1 && !conv_state)) return SLA_ERR_NULL;
  if (!aligned16(x) || (K > 1 && !aligned16(conv_state))) return SLA_ERR_UNSUPPORTED;
  sla::ConvArgs a;
  memset(&a, 0, sizeof(a));
  a.B = shape->batch;
  a.D = shape->channels;
  a.K = K;
  a.n = shape->n_nodes;
  a.conv_state = conv_state;
  a.x = x;
  a.parent = parent_idx;
  a.path = path;
  a.len = len;
  a.status = status;
  return hip_status(sla::launch_conv(a, shape->x_dtype, true, stream));
}

int sla_prune(const int32_t *parent, const float *logp, int32_t batch, int32_t n_nodes, float tau, int32_t budget,
              int32_t *packed_parent, int32_t *index_map, int32_t *count, float *scores, int32_t *status,
              hipStream_t stream) {
  if (!parent || !logp || !packed_parent || !index_map || !count) return SLA_ERR_NULL;
  if (batch < 1 || batch > (1 << 30) || n_nodes < 1 || n_nodes > SLA_MAX_NODES || !(tau >= 0.f)) return SLA_ERR_SHAPE;
  sla::PruneArgs a{batch, n_nodes, tau, budget, parent, logp, packed_parent, index_map, count, scores, status};
  return hip_status(sla::launch_prune(a, stream));
}

// Host pruning: scores root first (parents precede children), the window,
// the budgeted prefix in (score desc, index asc) order, then packing.
int sla_prune_host(const int32_t *parent, const float *logp, int32_t n, float tau, int32_t budget,
                   int32_t *packed_parent, int32_t *index_map, int32_t *count, float *scores) {
  if (!parent || !logp || !packed_parent || !index_map || !count) return SLA_ERR_NULL;
  if (n < 1 || n > (1 << 16) || !(tau >= 0.f)) return SLA_ERR_SHAPE;
  for (int j = 0; j < n; ++j)
    if (parent[j] < -1 || parent[j] >= j) return SLA_ERR_TOPOLOGY;
  for (int j = 0; j < n; ++j)
    if (!(logp[j] <= 0.f)) return SLA_ERR_SCORE;
  std::vector<float> q(n);
  for (int j = 0; j < n; ++j) q[j] = parent[j] >= 0 ? q[parent[j]] + logp[j] : logp[j];
  float qstar = q[0];
  for (int j = 1; j < n; ++j) qstar = std::max(qstar, q[j]);
  const float thr = qstar - tau;
  std::vector<int> window;
  for (int j = 0; j < n; ++j)
    if (q[j] >= thr) window.push_back(j);
  std::vector<char> keep(n, 0);
  if (budget > 0 && (int)window.size() > budget) {
    std::stable_sort(window.begin(), window.end(), [&](int x, int y) { return q[x] > q[y]; });
    for (int i = 0; i < budget; ++i) keep[window[i]] = 1;
  } else {
    for (int j : window) keep[j] = 1;
  }
  std::vector<int> nidx(n, -1);
  int m = 0;
  for (int j = 0; j < n; ++j)
    if (keep[j]) nidx[j] = m++;
  for (int j = 0; j < n; ++j) {
    packed_parent[j] = -1;
    index_map[j] = -1;
  }
  for (int j = 0; j < n; ++j)
    if (keep[j]) {
      packed_parent[nidx[j]] = parent[j] >= 0 ? nidx[parent[j]] : -1;
      index_map[nidx[j]] = j;
    }
  if (scores)
    for (int j = 0; j < n; ++j) scores[j] = q[j];
  *count = m;
  return SLA_OK;
}

int sla_tree_mask_to_parent(const uint64_t *mask, int32_t batch, int32_t n_nodes, int32_t *parent, int32_t *status,
                            hipStream_t stream) {
  if (!mask || !parent) return SLA_ERR_NULL;
  if (batch < 1 || batch > (1 << 30) || n_nodes < 1 || n_nodes > SLA_MAX_NODES) return SLA_ERR_SHAPE;
  sla::MaskArgs a{batch, n_nodes, mask, parent, status};
  return hip_status(sla::launch_mask_to_parent(a, stream));
}

int sla_tree_mask_to_parent_host(const uint64_t *mask, int32_t n, int32_t *parent) {
  if (!mask || !parent) return SLA_ERR_NULL;
  if (n < 1 || n > SLA_MAX_NODES) return SLA_ERR_SHAPE;
  std::vector<int32_t> p(n);
  for (int i = 0; i < n; ++i) {
    const uint64_t self = 1ull << i;
    const uint64_t row = mask[i];
    const uint64_t strict = row & ~self;
    if (!(row & self) || (i < 63 && (row >> (i + 1)))) return SLA_ERR_TOPOLOGY;
    p[i] = strict ? 63 - __builtin_clzll(strict) : -1;
    if (row != ((p[i] >= 0 ? mask[p[i]] : 0ull) | self)) return SLA_ERR_TOPOLOGY;
  }
  for (int i = 0; i < n; ++i) parent[i] = p[i];
  return SLA_OK;
}

int sla_topology(const int32_t *parent_idx, int32_t batch, int32_t n_nodes, int32_t *depth, uint64_t *anc,
                 int32_t *order, int32_t *n_children, int32_t *status, hipStream_t stream) {
  if (!parent_idx || !depth || !anc || !order || !n_children || !status) return SLA_ERR_NULL;
  if (batch < 1 || n_nodes < 1 || n_nodes > SLA_MAX_NODES) return SLA_ERR_SHAPE;
  sla::TopologyArgs a{batch, n_nodes, parent_idx, depth, anc, order, n_children, status};
  return hip_status(sla::launch_topology(a, stream));
}

// Host topology: depths and ancestor masks accumulate front to back (every
// parent precedes its child), the pre-order comes from an explicit stack.
int sla_topology_host(const int32_t *parent_idx, int32_t n, int32_t *depth, uint64_t *anc, int32_t *order,
                      int32_t *n_children, int32_t *max_depth) {
  if (!parent_idx || !depth || !anc || !order || !n_children) return SLA_ERR_NULL;
  if (n < 1 || n > SLA_MAX_NODES) return SLA_ERR_SHAPE;
  for (int j = 0; j < n; ++j)
    if (parent_idx[j] < -1 || parent_idx[j] >= j) return SLA_ERR_TOPOLOGY;
  int md = 0;
  for (int j = 0; j < n; ++j) {
    const int p = parent_idx[j];
    depth[j] = (p >= 0 ? depth[p] : 0) + 1;
    anc[j] = (p >= 0 ? anc[p] : 0ull) | (1ull << j);
    n_children[j] = 0;
    if (depth[j] > md) md = depth[j];
  }
  for (int j = 0; j < n; ++j)
    if (parent_idx[j] >= 0) ++n_children[parent_idx[j]];
  std::vector<int> stack;
  stack.reserve(n);
  for (int j = n - 1; j >= 0; --j)
    if (parent_idx[j] == -1) stack.push_back(j);
  int pos = 0;
  while (!stack.empty()) {
    const int x = stack.back();
    stack.pop_back();
    order[pos++] = x;
    for (int c = n - 1; c > x; --c)
      if (parent_idx[c] == x) stack.push_back(c);
  }
  if (max_depth) *max_depth = md;
  return SLA_OK;
}

int sla_validate_path_host(const int32_t *parent_idx, int32_t n, const int32_t *path, int32_t len) {
  if (!parent_idx || (len > 0 && !path)) return SLA_ERR_NULL;
  if (n < 1 || n > SLA_MAX_NODES) return SLA_ERR_SHAPE;
  for (int j = 0; j < n; ++j)
    if (parent_idx[j] < -1 || parent_idx[j] >= j) return SLA_ERR_TOPOLOGY;
  if (len < 0 || len > n) return SLA_ERR_PATH;
  int prev = -1;
  for (int t = 0; t < len; ++t) {
    const int a = path[t];
    if (a < 0 || a >= n || parent_idx[a] != prev) return SLA_ERR_PATH;
    prev = a;
  }
  return SLA_OK;
}

}  // extern "C"
