/*
 * oracle.c -- plain, slow, fp64 CPU reference for gated-delta-rule (GDN)
 * speculative verification of draft chains/trees and accepted-path commit.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the package smoke check and
 * the CPU-baseline leg of the benchmark may load this library.  The product
 * path (the HIP library) never links or calls it, and this file shares no
 * code, header, table or helper with it.
 *
 * What it computes (SpecLA, arXiv 2607.16673):
 *   - The GDN recurrent step with decay alpha and delta-rule strength beta,
 *         S' = alpha * S (I - beta k k^T) + beta v k^T ,   o = S' q,
 *     i.e. the gated form of the minimal update of Eq. (state-update) in
 *     §2.2, with GDN named as the target layer there.  The state is held
 *     transposed, H = S^T with shape [d_k][d_v] (v fastest), which is the
 *     K x V_tile orientation of the tiling paragraph of §4.1; the step in
 *     that orientation is
 *         H' = alpha * (H - beta k (k^T H)) + beta k v^T ,   o = H'^T q.
 *   - Verification (§4, tree mask of §4.2): every draft node j is evaluated
 *     on its own root path P(j) -- its ancestors, root first, then j -- so
 *     that updates flow only along ancestor paths and never between
 *     siblings.  The output of node j is read after node j's own update
 *     (a chain of length one is exactly one autoregressive decode step).
 *     This is written as the plain definition: for each node the committed
 *     state is copied and the steps of its root path are applied one by one.
 *     No prefix sharing, no factorisation.
 *   - Commit (§5.1 "state recovery", §5.2): the durable state after
 *     accepting the path a_1..a_A is the state after decoding those tokens
 *     one at a time, starting from the committed state.
 *   - The same definitions for the other stateful layer families whose
 *     factor records §5.1 lists (DeltaNet, scalar decay without the delta
 *     rule, GLA's per-key gates); see the section on layer families.
 *   - The short causal convolution in front of the recurrent core and its
 *     conv state (see the section at the end of this file).
 *   - Topology (§4.2 tree mask, §7 parent array): depth, inclusive
 *     ancestor bit masks, child counts and a DFS pre-order, computed by the
 *     definition (following parent pointers node by node).
 *
 * Units are (batch b, head h); they are independent and are distributed
 * over OpenMP threads when the library is built with -fopenmp.  Within a
 * unit nothing is blocked, fused or reordered.
 *
 * Layouts (all row-major, contiguous):
 *   state  [B][H][dk][dv]        q, k [B][n][H][dk]      v, out [B][n][H][dv]
 *   alpha, beta [B][n][H]        parent [B][n]           path [B][path_stride]
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_OK 0
#define OR_ERR_SHAPE (-2)
#define OR_ERR_TOPOLOGY (-4)
#define OR_ERR_PATH (-5)
#define OR_MAX_NODES 64

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads for the following parallel loops (timing only; results do not
 * depend on it: every unit is computed by one thread, in the same order). */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* One GDN step on H = S^T ([dk][dv]).  kH is caller scratch of length dv.
 *   kH[c]   = sum_i k[i] H[i][c]                       (the row k^T H)
 *   H[i][c] = alpha*(H[i][c] - beta*k[i]*kH[c]) + beta*k[i]*v[c]          */
void oracle_gdn_step(int dk, int dv, double *H, const double *k, const double *v,
                     double alpha, double beta, double *kH) {
  for (int c = 0; c < dv; ++c) {
    double s = 0.0;
    for (int i = 0; i < dk; ++i) s += k[i] * H[(size_t)i * dv + c];
    kH[c] = s;
  }
  for (int i = 0; i < dk; ++i)
    for (int c = 0; c < dv; ++c) {
      double h = H[(size_t)i * dv + c];
      H[(size_t)i * dv + c] = alpha * (h - beta * k[i] * kH[c]) + beta * k[i] * v[c];
    }
}

/* o = H^T q  (= S q). */
void oracle_readout(int dk, int dv, const double *H, const double *q, double *o) {
  for (int c = 0; c < dv; ++c) {
    double s = 0.0;
    for (int i = 0; i < dk; ++i) s += H[(size_t)i * dv + c] * q[i];
    o[c] = s;
  }
}

/* A parent array is valid when every node's parent is -1 (a child of the
 * committed state) or an earlier node: the draft is in topological order
 * (§4.2).  Returns OR_OK or OR_ERR_TOPOLOGY. */
int oracle_check_parent(const int32_t *parent, int n) {
  if (n < 1 || n > OR_MAX_NODES) return OR_ERR_SHAPE;
  for (int j = 0; j < n; ++j)
    if (parent[j] < -1 || parent[j] >= j) return OR_ERR_TOPOLOGY;
  return OR_OK;
}

/* Root path of node j, root first, j last.  Returns its length. */
int oracle_root_path(const int32_t *parent, int n, int j, int32_t *path) {
  int32_t rev[OR_MAX_NODES];
  int len = 0;
  for (int a = j; a != -1; a = parent[a]) {
    if (a < 0 || a >= n || len >= n) return -1;
    rev[len++] = a;
  }
  for (int t = 0; t < len; ++t) path[t] = rev[len - 1 - t];
  return len;
}

/* DFS pre-order: roots in ascending index, each node followed by the
 * subtrees of its children in ascending index. */
static void dfs_visit(const int32_t *parent, int n, int j, int32_t *order, int *pos) {
  order[(*pos)++] = j;
  for (int c = j + 1; c < n; ++c)
    if (parent[c] == j) dfs_visit(parent, n, c, order, pos);
}

/* Topology table of one draft (one sequence).
 *   depth[j]      = |P(j)| (a root has depth 1)
 *   anc[j]        = bit a set iff a is on P(j) (j included)
 *   n_children[j] = number of nodes whose parent is j
 *   order         = DFS pre-order (see above)
 *   *max_depth    = max_j depth[j]                                        */
int oracle_topology(const int32_t *parent, int n, int32_t *depth, uint64_t *anc,
                    int32_t *order, int32_t *n_children, int32_t *max_depth) {
  int st = oracle_check_parent(parent, n);
  if (st != OR_OK) return st;
  int md = 0;
  for (int j = 0; j < n; ++j) {
    int d = 0;
    uint64_t m = 0;
    for (int a = j; a != -1; a = parent[a]) {
      ++d;
      m |= (uint64_t)1 << a;
    }
    depth[j] = d;
    anc[j] = m;
    if (d > md) md = d;
    int c = 0;
    for (int i = 0; i < n; ++i) c += (parent[i] == j);
    n_children[j] = c;
  }
  int pos = 0;
  for (int j = 0; j < n; ++j)
    if (parent[j] == -1) dfs_visit(parent, n, j, order, &pos);
  *max_depth = md;
  return OR_OK;
}

/* An accepted path a_1..a_len is valid when it is a root path of the draft:
 * parent[a_1] = -1 and parent[a_t] = a_{t-1}.  len = 0 is the empty path. */
int oracle_validate_path(const int32_t *parent, int n, const int32_t *path, int len) {
  if (len < 0 || len > n) return OR_ERR_PATH;
  int prev = -1;
  for (int t = 0; t < len; ++t) {
    int a = path[t];
    if (a < 0 || a >= n || parent[a] != prev) return OR_ERR_PATH;
    prev = a;
  }
  return OR_OK;
}

/* ------------------------------------------------------------------------
 * Layer families.  §5.1 closes with the remark that stateful linear layers
 * keep different factor records: GLA-style layers a key, a value and a
 * gate but no delta-rule beta; DeltaNet a key, a value and beta but no
 * decay; Mamba-style selective SSMs their own decay parameters in place of
 * the delta rule.  The steps those layers take, on H = S^T ([dk][dv]):
 *   OR_FAM_GDN       H' = alpha (H - beta k (k^T H)) + beta k v^T
 *   OR_FAM_DELTANET  H' = H - beta k (k^T H) + beta k v^T     (no decay)
 *   OR_FAM_DECAY     H' = alpha H + k v^T                      (scalar decay,
 *                                                               no delta rule)
 *   OR_FAM_GLA       H'[i][c] = g[i] H[i][c] + k[i] v[c]       (one gate per
 *                                                               key dimension)
 * In the S orientation the GLA gate multiplies S from the right,
 * S' = S diag(g) + v k^T.  `gate` points at alpha (GDN, DECAY) or at the dk
 * gates (GLA) and is unused for DELTANET; beta is unused for DECAY and GLA.
 * Verification and commit are the same definitions for every family: node
 * j's output is read from the state after the steps of P(j), and a commit
 * decodes the accepted tokens one at a time. */
#define OR_FAM_GDN 0
#define OR_FAM_DELTANET 1
#define OR_FAM_DECAY 2
#define OR_FAM_GLA 3

static int family_ok(int family) { return family >= OR_FAM_GDN && family <= OR_FAM_GLA; }

/* Gates per (b, j, h) record: dk for GLA, 1 otherwise. */
static size_t gate_width(int family, int dk) { return family == OR_FAM_GLA ? (size_t)dk : 1; }

void oracle_layer_step(int family, int dk, int dv, double *H, const double *k, const double *v,
                       const double *gate, double beta, double *kH) {
  switch (family) {
    case OR_FAM_GDN:
      oracle_gdn_step(dk, dv, H, k, v, gate[0], beta, kH);
      return;
    case OR_FAM_DELTANET:
      for (int c = 0; c < dv; ++c) {
        double s = 0.0;
        for (int i = 0; i < dk; ++i) s += k[i] * H[(size_t)i * dv + c];
        kH[c] = s;
      }
      for (int i = 0; i < dk; ++i)
        for (int c = 0; c < dv; ++c) H[(size_t)i * dv + c] += beta * k[i] * (v[c] - kH[c]);
      return;
    case OR_FAM_DECAY:
      for (int i = 0; i < dk; ++i)
        for (int c = 0; c < dv; ++c) H[(size_t)i * dv + c] = gate[0] * H[(size_t)i * dv + c] + k[i] * v[c];
      return;
    case OR_FAM_GLA:
      for (int i = 0; i < dk; ++i)
        for (int c = 0; c < dv; ++c) H[(size_t)i * dv + c] = gate[i] * H[(size_t)i * dv + c] + k[i] * v[c];
      return;
  }
}

/* Verification by definition.  For every (b, h) and node j: copy the
 * committed state, apply the steps of the nodes of P(j) root first, then
 * read out o_j = H^T q_j.  status[b] (nullable) gets the per-sequence
 * topology verdict; invalid sequences produce no output.  gate is
 * [B][n][H] (or [B][n][H][dk] for GLA), NULL for DELTANET; beta [B][n][H],
 * NULL for DECAY and GLA. */
int oracle_verify_family(int family, int B, int H, int dk, int dv, int n, const double *state,
                         const double *q, const double *k, const double *v, const double *gate,
                         const double *beta, const int32_t *parent, double *out, int32_t *status) {
  if (B < 1 || H < 1 || dk < 1 || dv < 1 || n < 1 || n > OR_MAX_NODES || !family_ok(family)) return OR_ERR_SHAPE;
  const size_t gw = gate_width(family, dk);
  int bad = 0;
  for (int b = 0; b < B; ++b) {
    int st = oracle_check_parent(parent + (size_t)b * n, n);
    if (status) status[b] = st;
    if (st != OR_OK) bad = 1;
  }
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < H; ++h) {
      const int32_t *par = parent + (size_t)b * n;
      if (oracle_check_parent(par, n) != OR_OK) continue;
      double *Hw = (double *)malloc(sizeof(double) * ((size_t)dk * dv + dv));
      double *kH = Hw + (size_t)dk * dv;
      const double *H0 = state + ((size_t)b * H + h) * dk * dv;
      int32_t path[OR_MAX_NODES];
      for (int j = 0; j < n; ++j) {
        int len = oracle_root_path(par, n, j, path);
        memcpy(Hw, H0, sizeof(double) * (size_t)dk * dv);
        for (int t = 0; t < len; ++t) {
          size_t a = ((size_t)b * n + path[t]) * H + h;
          oracle_layer_step(family, dk, dv, Hw, k + a * dk, v + a * dv, gate ? gate + a * gw : NULL,
                            beta ? beta[a] : 0.0, kH);
        }
        size_t jj = ((size_t)b * n + j) * H + h;
        oracle_readout(dk, dv, Hw, q + jj * dk, out + jj * dv);
      }
      free(Hw);
    }
  return bad ? OR_ERR_TOPOLOGY : OR_OK;
}

/* The GDN case with the original argument order. */
int oracle_verify(int B, int H, int dk, int dv, int n, const double *state,
                  const double *q, const double *k, const double *v,
                  const double *alpha, const double *beta, const int32_t *parent,
                  double *out, int32_t *status) {
  return oracle_verify_family(OR_FAM_GDN, B, H, dk, dv, n, state, q, k, v, alpha, beta, parent, out, status);
}

/* Commit by definition: for every (b, h), starting from the committed
 * state, decode the accepted tokens path[b][0..len[b]) one at a time with
 * the family's step, in place.  Sequences whose path is not a root path of
 * their draft are left untouched and get OR_ERR_PATH in status[b]
 * (nullable).  gate and beta as for verification. */
int oracle_commit_family(int family, int B, int H, int dk, int dv, int n, double *state,
                         const double *k, const double *v, const double *gate,
                         const double *beta, const int32_t *parent, const int32_t *path,
                         int path_stride, const int32_t *len, int32_t *status) {
  if (B < 1 || H < 1 || dk < 1 || dv < 1 || n < 1 || n > OR_MAX_NODES || !family_ok(family)) return OR_ERR_SHAPE;
  const size_t gw = gate_width(family, dk);
  int bad = 0;
  for (int b = 0; b < B; ++b) {
    int st = oracle_check_parent(parent + (size_t)b * n, n);
    if (st == OR_OK)
      st = oracle_validate_path(parent + (size_t)b * n, n, path + (size_t)b * path_stride, len[b]);
    if (status) status[b] = st;
    if (st != OR_OK) bad = 1;
  }
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < H; ++h) {
      const int32_t *par = parent + (size_t)b * n;
      const int32_t *pth = path + (size_t)b * path_stride;
      if (oracle_check_parent(par, n) != OR_OK || oracle_validate_path(par, n, pth, len[b]) != OR_OK)
        continue;
      double *kH = (double *)malloc(sizeof(double) * dv);
      double *Hs = state + ((size_t)b * H + h) * dk * dv;
      for (int t = 0; t < len[b]; ++t) {
        size_t a = ((size_t)b * n + pth[t]) * H + h;
        oracle_layer_step(family, dk, dv, Hs, k + a * dk, v + a * dv, gate ? gate + a * gw : NULL,
                          beta ? beta[a] : 0.0, kH);
      }
      free(kH);
    }
  return bad ? OR_ERR_PATH : OR_OK;
}

int oracle_commit(int B, int H, int dk, int dv, int n, double *state,
                  const double *k, const double *v, const double *alpha,
                  const double *beta, const int32_t *parent, const int32_t *path,
                  int path_stride, const int32_t *len, int32_t *status) {
  return oracle_commit_family(OR_FAM_GDN, B, H, dk, dv, n, state, k, v, alpha, beta, parent, path,
                              path_stride, len, status);
}

/* ------------------------------------------------------------------------
 * Short causal convolution (the GDN layer's depthwise convolution of kernel
 * size K = 4 with SiLU, in front of the recurrent core; §7 and the setup of
 * §8) and its conv state C, the second per-layer state the cache holder
 * keeps next to S (§7).
 *
 * For channel c the convolution of a token sequence z_1..z_t is
 *     y_t[c] = act(bias[c] + sum_{i=0}^{K-1} w[c][i] * z_{t-K+1+i}[c]),
 * act = SiLU, silu(a) = a / (1 + exp(-a)), or the identity.  C holds the
 * last K-1 committed inputs, C[0] the oldest and C[K-2] the newest.
 *
 * Verification (§4, with the tree mask of §4.2): the tokens in front of
 * draft node j are those of its own root path P(j), and in front of those
 * the committed inputs.  By definition, per node: form the sequence
 * [C[0], .., C[K-2], x_{p_1}, .., x_{p_d}] with p_1..p_d = P(j) and take
 * the convolution at its last position.
 *
 * Commit (§5.1-5.2): accepting a_1..a_A, the new conv state is the state
 * after decoding those tokens one at a time, each step dropping the oldest
 * row of C and appending the token's input.
 *
 * Layouts: conv_state [B][K-1][D], x and y [B][n][D], w [D][K], bias [D]. */
#define OR_MAX_KERNEL 8

static double oracle_silu(double a) { return a / (1.0 + exp(-a)); }

int oracle_conv_verify(int B, int D, int K, int n, const double *conv_state, const double *x,
                       const double *w, const double *bias, int activation, const int32_t *parent,
                       double *y, int32_t *status) {
  if (B < 1 || D < 1 || K < 1 || K > OR_MAX_KERNEL || n < 1 || n > OR_MAX_NODES) return OR_ERR_SHAPE;
  int bad = 0;
  for (int b = 0; b < B; ++b) {
    int st = oracle_check_parent(parent + (size_t)b * n, n);
    if (status) status[b] = st;
    if (st != OR_OK) bad = 1;
  }
#pragma omp parallel for schedule(dynamic)
  for (int b = 0; b < B; ++b) {
    const int32_t *par = parent + (size_t)b * n;
    if (oracle_check_parent(par, n) != OR_OK) continue;
    const double *Cb = conv_state + (size_t)b * (K - 1) * D;
    int32_t path[OR_MAX_NODES];
    const double *seq[OR_MAX_KERNEL - 1 + OR_MAX_NODES];
    for (int j = 0; j < n; ++j) {
      int d = oracle_root_path(par, n, j, path);
      int L = 0;
      for (int r = 0; r < K - 1; ++r) seq[L++] = Cb + (size_t)r * D;
      for (int t = 0; t < d; ++t) seq[L++] = x + ((size_t)b * n + path[t]) * D;
      double *yj = y + ((size_t)b * n + j) * D;
      for (int c = 0; c < D; ++c) {
        double s = bias ? bias[c] : 0.0;
        for (int i = 0; i < K; ++i) s += w[(size_t)c * K + i] * seq[L - K + i][c];
        yj[c] = activation ? oracle_silu(s) : s;
      }
    }
  }
  return bad ? OR_ERR_TOPOLOGY : OR_OK;
}

int oracle_conv_commit(int B, int D, int K, int n, double *conv_state, const double *x,
                       const int32_t *parent, const int32_t *path, int path_stride, const int32_t *len,
                       int32_t *status) {
  if (B < 1 || D < 1 || K < 1 || K > OR_MAX_KERNEL || n < 1 || n > OR_MAX_NODES) return OR_ERR_SHAPE;
  int bad = 0;
  for (int b = 0; b < B; ++b) {
    const int32_t *par = parent + (size_t)b * n;
    int st = oracle_check_parent(par, n);
    if (st == OR_OK) st = oracle_validate_path(par, n, path + (size_t)b * path_stride, len[b]);
    if (status) status[b] = st;
    if (st != OR_OK) {
      bad = 1;
      continue;
    }
    double *Cb = conv_state + (size_t)b * (K - 1) * D;
    for (int t = 0; t < len[b]; ++t) {
      const double *xa = x + ((size_t)b * n + path[(size_t)b * path_stride + t]) * D;
      for (int r = 0; r + 1 < K - 1; ++r) memcpy(Cb + (size_t)r * D, Cb + (size_t)(r + 1) * D, sizeof(double) * D);
      if (K > 1) memcpy(Cb + (size_t)(K - 2) * D, xa, sizeof(double) * D);
    }
  }
  return bad ? OR_ERR_PATH : OR_OK;
}
