/*
 * sla.h -- C ABI of libsla: gated-delta-rule (GDN) speculative verification
 * of draft chains and trees against a recurrent state, with a compact
 * per-node factor store and accepted-path commit, for AMD MI355X (gfx950).
 *
 * Method: SpecLA, "Efficient Speculative Decoding for Linear-Attention
 * Models" (arXiv 2607.16673).
 *
 * Notation.  One (batch b, head h) pair is a unit.  The committed state of a
 * unit is S (d_v x d_k); it is stored transposed, H = S^T, row-major
 * [d_k][d_v] with v fastest (the K x V_tile orientation of §4.1, "Tiling").
 * A draft of n nodes is given as a parent array in topological order
 * (§4.2): parent[j] = -1 makes node j a child of the committed state,
 * otherwise parent[j] < j.  P(j) is the root path of node j, root first and
 * j last.  The GDN step of node a is
 *     S <- alpha_a S (I - beta_a k_a k_a^T) + beta_a v_a k_a^T
 * and node j outputs o_j = S_j q_j, where S_j is the state after the steps
 * of P(j) (j included) applied to the committed state.  Updates never flow
 * between siblings (tree mask of §4.2).
 *
 * Conventions for every entry point.
 *   - Pointers named as device memory must be device memory of the current
 *     HIP device; all such buffers are owned by the caller.  The library
 *     allocates nothing, keeps no state between calls, and is re-entrant.
 *   - Work is enqueued on the given stream and runs asynchronously; the
 *     call returns before the work finishes.
 *   - A negative return value is an argument error detected on the host;
 *     nothing was launched and no buffer was touched.
 *   - Data errors that only the device can see (an invalid parent array or
 *     accepted path in device memory) are reported per sequence in
 *     status[b]; such a sequence's state is left untouched and its outputs
 *     and factors are unspecified.  status may be NULL.
 *   - All tensors are dense, contiguous and row-major in the stated shapes.
 */
#ifndef SLA_H_
#define SLA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
#define SLA_OK 0
#define SLA_ERR_NULL (-1)        /* a required pointer is NULL             */
#define SLA_ERR_SHAPE (-2)       /* a size is out of range                 */
#define SLA_ERR_DTYPE (-3)       /* unknown activation dtype               */
#define SLA_ERR_TOPOLOGY (-4)    /* parent array not in topological order  */
#define SLA_ERR_PATH (-5)        /* accepted path is not a root path       */
#define SLA_ERR_ALIAS (-6)       /* pending factors overlap output factors */
#define SLA_ERR_UNSUPPORTED (-7) /* valid request the library cannot run  */
#define SLA_ERR_HIP (-8)         /* the HIP runtime reported an error      */
#define SLA_ERR_SCORE (-9)       /* a draft log-probability above 0 or NaN */

/* Activation dtypes of q, k, v (and of the stored k factor). */
#define SLA_DTYPE_F32 0
#define SLA_DTYPE_BF16 1

/* Draft topology hint.  CHAIN promises parent[j] = j - 1 for every
 * sequence (checked on the device; a violation is SLA_ERR_TOPOLOGY). */
#define SLA_TOPO_TREE 0
#define SLA_TOPO_CHAIN 1

/* Verification route (sla_shape.route).
 *   AUTO      the library chooses from the topology hint and the shape:
 *             1-node drafts (the decode step) take a streaming kernel of
 *             their own (whole-line state passes, two column sums); every
 *             other draft the parallel route.  A draft the parallel route
 *             cannot stage on chip (see sla_verify) takes the hybrid route
 *             if it is a tree of more than 32 nodes or the launch is small
 *             (batch x heads x d_v / 16 <= 512), else the serial route.
 *   SERIAL    state-resident serial verification (§4.1): each node reduces
 *             its parent state against k_j and q_j; chains advance the
 *             on-chip state in place, trees rebuild a branch point's state
 *             from the committed state and the stored factors.
 *   PARALLEL  tree-masked factorised verification (§4.2): one dense
 *             contraction of all queries and keys with the committed state
 *             on the matrix cores, then a tree-masked triangular solve for
 *             the corrected values and a tree-masked readout.  bf16
 *             activations use the bf16 matrix cores (fp32 operands split
 *             into bf16 high and low parts); fp32 activations the fp32
 *             matrix cores, with exact fp32 products.
 *   HYBRID    chain-decomposed verification (§4.3): the draft is split by
 *             heavy-light decomposition into node-disjoint chains, each
 *             verified by the serial per-node loop; chains whose boundary
 *             state (the state of the chain head's parent) is ready run in
 *             parallel, level by level.  The boundary state is rebuilt on
 *             chip from the committed state and the ancestors' factor
 *             records.  Bitwise equal to SERIAL.  A CHAIN draft is a single
 *             chain and runs as SERIAL.                                  */
#define SLA_ROUTE_AUTO 0
#define SLA_ROUTE_SERIAL 1
#define SLA_ROUTE_PARALLEL 2
#define SLA_ROUTE_HYBRID 3

#define SLA_MAX_NODES 64

/* Layer family of the recurrent core.  Stateful linear layers keep the
 * factors their own state advance consumes (the remark closing §5.1): GDN
 * a key, a value, a decay and beta; DeltaNet a key, a value and beta but no
 * decay; GLA-style layers a key, a value and a gate but no beta; selective
 * SSMs a decay in place of the delta rule.  With g the gate:
 *   GDN       S <- alpha S (I - beta k k^T) + beta v k^T   (gated delta rule)
 *   DELTANET  S <- S (I - beta k k^T) + beta v k^T         (no decay)
 *   DECAY     S <- alpha S + v k^T                          (scalar decay, no
 *                                                            delta rule: the
 *                                                            selective-SSM form)
 *   GLA       S <- S diag(g) + v k^T                        (one gate per key
 *                                                            dimension)
 * Verification, factor records and commit follow the same definitions for
 * every family (o_j = S_j q_j after the steps of P(j)). */
#define SLA_FAMILY_GDN 0
#define SLA_FAMILY_DELTANET 1
#define SLA_FAMILY_DECAY 2
#define SLA_FAMILY_GLA 3

typedef struct sla_shape {
  int32_t batch;     /* B >= 1                                              */
  int32_t heads;     /* H >= 1, with 64 H max(d_k, d_v) 4 < 2^31 (one
                        sequence's rows are addressed with 32-bit offsets) */
  int32_t d_k;       /* 64, 128 or 256                                      */
  int32_t d_v;       /* multiple of 16, 16..1024                            */
  int32_t n_nodes;   /* draft nodes per sequence, 1..SLA_MAX_NODES          */
  int32_t qkv_dtype; /* SLA_DTYPE_F32 or SLA_DTYPE_BF16                     */
  int32_t topology;  /* SLA_TOPO_TREE or SLA_TOPO_CHAIN                     */
  int32_t family;    /* SLA_FAMILY_*; 0 (GDN) when zero-initialised         */
  int32_t route;     /* SLA_ROUTE_* for sla_verify; 0 (AUTO) when
                        zero-initialised; ignored by sla_commit            */
} sla_shape;

/* Factor store (§5.1, factor buffering).  One record per node and head:
 *   k     [B][n][H][d_k]  the node's key, in the activation dtype;
 *   u     [B][n][H][d_v]  fp32 value the state advance writes: the corrected
 *                         value u_j = beta_j (v_j - alpha_j S_par k_j) of the
 *                         delta-rule families (alpha = 1 for DELTANET), with
 *                         S_par the state of node j's parent; v_j itself for
 *                         DECAY and GLA;
 *   alpha [B][n][H]       fp32 gate: alpha_j (GDN, DECAY), 1 (DELTANET);
 *         [B][n][H][d_k]  for GLA, the per-key gates g_j;
 *   parent[B][n]          int32 copy of the draft's parent array.
 * With these, node j's state is S_j = S_par diag(g_j) + u_j k_j^T (a scalar
 * gate: alpha_j S_par + u_j k_j^T), so an accepted path is committed by
 * rank-one updates alone (no reductions).  All four are device memory
 * written by sla_verify; sla_factors_bytes gives their total size. */
typedef struct sla_factors {
  void *k;
  float *u;
  float *alpha;
  int32_t *parent;
} sla_factors;

/* Pending accepted-factor buffer (§5.2, delayed state update): the factors
 * of the previous verification and the path accepted from them.
 *   f        factors written by the previous sla_verify (read only here);
 *   n_nodes  that verification's n (its parent/path row length);
 *   path     device [B][n_nodes] int32, node ids root first, -1 padded;
 *   len      device [B] int32, accepted length 0..n_nodes.
 * path[b][0..len[b]) must be a root path of f.parent[b]:
 * parent[path[0]] = -1 and parent[path[t]] = path[t-1]. */
typedef struct sla_pending {
  sla_factors f;
  int32_t n_nodes;
  const int32_t *path;
  const int32_t *len;
} sla_pending;

/* ------------------------------------------------------------ entry points */

/* sla_verify -- verify one layer's drafts for all sequences (§4), storing
 * the factor records (§5.1); optionally first commit a pending accepted
 * path into the state (fused commit-and-verify, §5.2).
 *
 *   state   device fp32 [B][H][d_k][d_v].  With pending == NULL it is only
 *           read.  Otherwise the pending path is applied and the committed
 *           state is written back in place, and verification runs from the
 *           committed state: one state read and one state write per call.
 *   pending NULL, or the previous verification's factors and accepted path.
 *           Its factor buffers must not overlap `factors` (ping-pong two
 *           factor stores), else SLA_ERR_ALIAS.
 *   q, k    device [B][n][H][d_k], shape->qkv_dtype.
 *   v       device [B][n][H][d_v], shape->qkv_dtype.
 *   alpha   device fp32 [B][n][H], the decay (GDN, DECAY); [B][n][H][d_k],
 *           the per-key gates (GLA); not read for DELTANET (may be NULL).
 *   beta    device fp32 [B][n][H], the delta-rule strength (GDN, DELTANET);
 *           not read for DECAY and GLA (may be NULL).
 *   parent_idx   device int32 [B][n]; topological order required.
 *   out     device fp32 [B][n][H][d_v]; o_j = S_j q_j.
 *   factors device factor store written for this draft (see sla_factors).
 *   status  device int32 [B] or NULL: 0, SLA_ERR_TOPOLOGY or SLA_ERR_PATH.
 * The route is shape->route (SLA_ROUTE_*; an unknown value is
 * SLA_ERR_SHAPE).  Every route stages the draft on chip.  At d_k = 256 the
 * parallel route holds drafts of up to 32 nodes with GLA's per-key gates or
 * with fp32 activations (PARALLEL: SLA_ERR_UNSUPPORTED above; AUTO then
 * takes the hybrid or serial route, as described under SLA_ROUTE_AUTO); with
 * GLA's per-key gates the serial and hybrid routes hold d_k = 256 drafts of
 * up to 50 nodes (SLA_ERR_UNSUPPORTED above).  Gates (alpha, GLA's g) lie in (0, 1]; every route only
 * multiplies them (decay ratios along a root path are products of the gates
 * between the two nodes), so any gate in that range, however small, is
 * valid: strong decays underflow towards zero as they do in exact
 * arithmetic.
 * Returns SLA_OK once the work is enqueued, or a negative error code. */
int sla_verify(const sla_shape *shape, float *state, const sla_pending *pending,
               const void *q, const void *k, const void *v, const float *alpha,
               const float *beta, const int32_t *parent_idx, float *out,
               const sla_factors *factors, int32_t *status, hipStream_t stream);

/* sla_commit -- immediate state update (§5.2): apply the accepted path's
 * factor records to the state in place, S <- S diag(g_a) + u_a k_a^T for
 * each accepted node a, root first (a scalar gate: alpha_a S + u_a k_a^T);
 * shape->family says which gate layout the factors hold.  shape->n_nodes is the n of the factors; path
 * and len are as in sla_pending.  len[b] = 0 leaves sequence b untouched.
 * The per-element arithmetic is the same as the pending prologue of
 * sla_verify, so both routes give bitwise equal states.
 *   state device fp32 [B][H][d_k][d_v]; factors: device (read only);
 *   path device int32 [B][n]; len device int32 [B]; status device int32 [B]
 *   or NULL (0 or SLA_ERR_PATH). */
int sla_commit(const sla_shape *shape, float *state, const sla_factors *factors,
               const int32_t *path, const int32_t *len, int32_t *status, hipStream_t stream);

/* sla_topology -- the per-sequence topology table the verifier builds on
 * chip (tree mask of §4.2), written out for inspection:
 *   depth      int32 [B][n]   |P(j)|, a root has depth 1;
 *   anc        uint64 [B][n]  bit a set iff node a is on P(j), j included;
 *   order      int32 [B][n]   DFS pre-order: roots ascending, children
 *                             ascending after their parent;
 *   n_children int32 [B][n];
 *   status     int32 [B]      0 or SLA_ERR_TOPOLOGY (then the row is
 *                             unspecified).
 * All pointers are device memory; none may be NULL. */
int sla_topology(const int32_t *parent_idx, int32_t batch, int32_t n_nodes, int32_t *depth,
                 uint64_t *anc, int32_t *order, int32_t *n_children, int32_t *status,
                 hipStream_t stream);

/* ------------------------------------------------- short causal convolution
 *
 * The GDN layer mixes every channel of its q, k and v projections over the
 * last K tokens with a depthwise causal convolution and SiLU before the
 * recurrent core, and keeps the last K - 1 committed inputs as a second
 * per-layer state C next to S (§7: kernel size 4, SiLU, recurrent state
 * (S, C)).  For channel c,
 *     y[c] = act(bias[c] + sum_{i=0}^{K-1} w[c][i] z_{K-1-i}[c]),
 * where z_0 is the node's own input, z_s (s >= 1) the input of its s-th
 * ancestor on P(j) while one exists, and past the root the committed rows,
 * newest first: z_s = C[K-2-(s-depth(j))] for s >= depth(j).  So every
 * node sees only its own root path (tree mask of §4.2), and a chain draft is
 * an ordinary causal sequence behind C.  act is SiLU, a / (1 + exp(-a)), or
 * the identity.  Arithmetic is fp32 (fused multiply-adds over i = 0..K-1,
 * starting from the bias); y is rounded to the activation dtype.
 *
 * Commit (§5.1-5.2): accepting a_1..a_A drops the oldest rows of C and
 * appends x_{a_1}..x_{a_A}: C keeps the last K - 1 rows of
 * [C[0], .., C[K-2], x_{a_1}, .., x_{a_A}].  The rows are copies (exact:
 * bf16 and fp32 inputs are held in fp32).  The pre-convolution inputs of
 * the draft are the conv's factor records: the caller keeps the previous
 * round's x until the next call has committed from it. */

#define SLA_ACT_NONE 0
#define SLA_ACT_SILU 1
#define SLA_CONV_MAX_KERNEL 4

typedef struct sla_conv_shape {
  int32_t batch;       /* B >= 1                                            */
  int32_t channels;    /* D, a multiple of 8, 8..(1 << 20)                  */
  int32_t kernel_size; /* K, 1..SLA_CONV_MAX_KERNEL                         */
  int32_t n_nodes;     /* draft nodes per sequence, 1..SLA_MAX_NODES        */
  int32_t x_dtype;     /* SLA_DTYPE_F32 or SLA_DTYPE_BF16 (x and y)         */
  int32_t activation;  /* SLA_ACT_NONE or SLA_ACT_SILU                      */
} sla_conv_shape;

/* Pending accepted rows for the conv state (§5.2, delayed update):
 *   x        the previous round's pre-convolution inputs, device
 *            [B][n_nodes][D] in shape->x_dtype (read only here);
 *   parent   the previous round's parent array, device int32 [B][n_nodes];
 *   n_nodes  that round's n;
 *   path,len as in sla_pending: device int32 [B][n_nodes] (-1 padded) and
 *            [B]; path[b][0..len[b]) must be a root path of parent[b]. */
typedef struct sla_conv_pending {
  const void *x;
  const int32_t *parent;
  int32_t n_nodes;
  const int32_t *path;
  const int32_t *len;
} sla_conv_pending;

/* sla_conv_verify -- the convolution of every draft node of one layer, for
 * all sequences; optionally first commit a pending accepted path into the
 * conv state (fused, as sla_verify does for S).
 *   conv_state device fp32 [B][K-1][D] (NULL allowed when K = 1).  Read only
 *              with pending == NULL; otherwise the committed rows are
 *              written back in place and the draft is convolved behind them.
 *   pending    NULL or the previous round's inputs and accepted path.  Its x
 *              must not overlap y (SLA_ERR_ALIAS).
 *   x          device [B][n][D], shape->x_dtype: the pre-convolution inputs.
 *   weight     device fp32 [D][K]: weight[c][K-1] multiplies the node's own
 *              input (the layout of a depthwise conv1d weight [D][1][K]).
 *   bias       device fp32 [D] or NULL (no bias).
 *   parent_idx device int32 [B][n]; topological order required.
 *   y          device [B][n][D], shape->x_dtype.
 *   status     device int32 [B] or NULL: 0, SLA_ERR_TOPOLOGY or
 *              SLA_ERR_PATH; such a sequence's conv state is untouched and
 *              its outputs are unspecified.
 * Returns SLA_OK once the work is enqueued, or a negative error code. */
int sla_conv_verify(const sla_conv_shape *shape, float *conv_state, const sla_conv_pending *pending,
                    const void *x, const float *weight, const float *bias, const int32_t *parent_idx,
                    void *y, int32_t *status, hipStream_t stream);

/* sla_conv_commit -- immediate conv-state update (§5.2): the accepted rows
 * of x (the draft verified last, shape->n_nodes nodes, parent array
 * parent_idx) are shifted into C in place.  path, len and status as in
 * sla_commit (status: 0 or SLA_ERR_PATH); len[b] = 0 leaves sequence b
 * untouched.  shape->activation is ignored.  Same result, bit for bit, as
 * the pending prologue of sla_conv_verify. */
int sla_conv_commit(const sla_conv_shape *shape, float *conv_state, const void *x,
                    const int32_t *parent_idx, const int32_t *path, const int32_t *len,
                    int32_t *status, hipStream_t stream);

/* ------------------------------------------ draft pruning and packing (§6.1)
 *
 * After the drafter's rollout every candidate v has a parent (-1: a child of
 * the committed state; parent[v] < v) and the log-probability logp[v] <= 0 of
 * its token given its path.  Its score is the path's joint log-probability,
 * summed root first in fp32: q(v) = q(parent(v)) + logp(v).  With q* the best
 * score and margin tau, the window keeps q(v) >= q* - tau (§6.1, "Tree
 * pruning"; the threshold q* - tau is an fp32 value).  A budget T > 0 then
 * keeps the first T window nodes in (score descending, index ascending)
 * order: since scores never increase along a path and parents carry smaller
 * indices, every ancestor ranks ahead of its descendants, so the kept set is
 * ancestor-closed -- what taking candidates in score order together with
 * their missing ancestors until T is used up selects.  Packing renumbers the
 * kept nodes 0..m-1 in their original (topological) order: packed_parent is
 * the verifier's parent array (§7), index_map[new] = old gathers the kept
 * tokens and activations.  Rows m..n-1 of both are -1. */

/* sla_prune -- batched on the device, one sequence per wavefront.
 *   parent, logp   device int32 / fp32 [B][n], n <= SLA_MAX_NODES;
 *   tau            margin (>= 0); budget T, <= 0 for none;
 *   packed_parent, index_map  device int32 [B][n] (written);
 *   count          device int32 [B]: kept nodes m (0 on a data error);
 *   scores         device fp32 [B][n] or NULL: q(v);
 *   status         device int32 [B] or NULL: 0, SLA_ERR_TOPOLOGY or
 *                  SLA_ERR_SCORE (then the rows are unspecified). */
int sla_prune(const int32_t *parent, const float *logp, int32_t batch, int32_t n_nodes, float tau,
              int32_t budget, int32_t *packed_parent, int32_t *index_map, int32_t *count, float *scores,
              int32_t *status, hipStream_t stream);

/* sla_prune_host -- the same for one host-memory sequence, synchronously on
 * the CPU, for any n in 1..65536.  Returns SLA_OK, SLA_ERR_NULL,
 * SLA_ERR_SHAPE, SLA_ERR_TOPOLOGY or SLA_ERR_SCORE; *count = m. */
int sla_prune_host(const int32_t *parent, const float *logp, int32_t n_nodes, float tau, int32_t budget,
                   int32_t *packed_parent, int32_t *index_map, int32_t *count, float *scores);

/* Tree mask -> parent array (§7, the proposal converter; the mask is M_tree
 * of §4.2).  mask[b][i] is row i as a bit set: bit j is set iff node j is an
 * ancestor of node i or i itself (n <= 64).  The parent of i is its deepest
 * strict ancestor, which in topological order is the one with the highest
 * index.  A mask that is not a tree mask in topological order (a missing
 * diagonal bit, an ancestor after its descendant, ancestors that do not form
 * one chain) is SLA_ERR_TOPOLOGY.
 *   sla_tree_mask_to_parent: device mask uint64 [B][n], parent int32 [B][n],
 *   status int32 [B] or NULL (on an error that row's parents are not written). */
int sla_tree_mask_to_parent(const uint64_t *mask, int32_t batch, int32_t n_nodes, int32_t *parent,
                            int32_t *status, hipStream_t stream);

/* Host version for one mask: returns SLA_OK, SLA_ERR_NULL, SLA_ERR_SHAPE or
 * SLA_ERR_TOPOLOGY. */
int sla_tree_mask_to_parent_host(const uint64_t *mask, int32_t n_nodes, int32_t *parent);

/* ------------------------------------------------------------ host helpers */

/* Same table as sla_topology for one host-memory parent array, computed
 * synchronously on the CPU; *max_depth may be NULL.  Returns SLA_OK,
 * SLA_ERR_NULL, SLA_ERR_SHAPE or SLA_ERR_TOPOLOGY. */
int sla_topology_host(const int32_t *parent_idx, int32_t n_nodes, int32_t *depth, uint64_t *anc,
                      int32_t *order, int32_t *n_children, int32_t *max_depth);

/* SLA_OK if path[0..len) (host memory) is a root path of the host parent
 * array, else SLA_ERR_PATH (or SLA_ERR_TOPOLOGY for a bad parent array). */
int sla_validate_path_host(const int32_t *parent_idx, int32_t n_nodes, const int32_t *path,
                           int32_t len);

/* Bytes of one factor store for this shape (k, u, alpha and parent). */
size_t sla_factors_bytes(const sla_shape *shape);

/* Static, human-readable name of a status code. */
const char *sla_status_string(int status);

/* Library ABI version (major * 10000 + minor * 100 + patch). */
int sla_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SLA_H_ */
