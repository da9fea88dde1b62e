"""Seeded synthetic inputs for GDN tree/chain verification and commit.

This module is shared by the tests, the smoke check and the benchmark to feed
*both* the HIP library and the CPU oracle.  It holds the workload recipe only
(shapes, distributions, random draft trees, accepted paths) and none of the
verification or commit arithmetic.

Workload recipe (stand-ins for the GDN-1.3B activations and recorded EAGLE
proposal trees of the paper's evaluation, §8, which are not available):
  * committed state S ~ N(0, 0.02^2), fp32, stored as H = S^T [dk][dv];
  * q, k ~ N(0, 1), L2-normalised per (layer, b, node, head) in fp64, then
    rounded (round-to-nearest-even) to the activation dtype;
  * v ~ N(0, 1), rounded to the activation dtype;
  * alpha = sigmoid(x), x ~ U(2, 5); beta = sigmoid(z), z ~ N(0, 1); fp32;
  * other layer families (the factor-record remark of §5.1): DeltaNet reads
    beta only, the scalar-decay family alpha only (both as above); GLA's
    per-key gates are g = sigmoid(z)^(1/16), z ~ N(0, 1) per (layer, b,
    node, head, key dimension), fp32 (GLA's gate with its normaliser 16);
  * strong-forgetting gates for the near-reset edge case: alpha (or each of
    GLA's per-key gates) ~ U(1e-3, 0.3), with about 3% set to 1e-6 and 2% to
    1e-20;
  * chains: parent[j] = j - 1; trees: node 0 is the root, node i > 0 picks a
    uniform parent among earlier nodes whose depth and child count are still
    below the configured limits;
  * accepted path: chains accept a uniform prefix length in [0, n]; trees
    accept the root path of a uniformly drawn node;
  * short convolution in front of the recurrent core: its channels are the
    q, k and v projections of all heads, D = H (2 d_k + d_v); pre-convolution
    inputs x ~ N(0, 1) rounded to the activation dtype; committed conv state
    (earlier inputs) drawn the same way and held in fp32; depthwise weights
    [D][K] ~ U(-1/sqrt(K), 1/sqrt(K)) in fp32 (the default initialisation of a
    depthwise conv1d), kernel size K = 4, no bias;
  * draft rollouts for pruning (§6.1): a per-level beam top-k rollout over a
    random softmax per expanded node (32-token vocabulary, logits ~ N(0, 2^2));
    each level expands the k best frontier nodes by path score, each with its
    k most likely tokens, until the candidate count is reached.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class Config:
    name: str
    index: int
    batch: int
    heads: int
    d_k: int
    d_v: int
    n_nodes: int
    chain: bool
    max_depth: int
    max_branch: int
    dtype: str
    layers: int
    description: str = ""


CONFIGS = {
    c.name: c
    for c in [
        Config("tiny_chain_f32", 0, 1, 1, 64, 64, 4, True, 4, 1, F32, 1,
               "batch 1, 1 head, dk=dv=64, chain of 4, all fp32"),
        Config("chain8_bf16", 1, 1, 16, 128, 128, 8, True, 8, 1, BF16, 1,
               "batch 1, 16 heads, dk=dv=128, chain of 8, bf16 q/k/v"),
        Config("tree32_bf16", 2, 1, 16, 128, 128, 32, False, 6, 4, BF16, 1,
               "batch 1, 16 heads, dk=dv=128, 32-node tree (depth<=6, branch<=4)"),
        Config("batched_tree_serving", 3, 64, 16, 128, 128, 16, False, 5, 3, BF16, 24,
               "batch 64, 16 heads, dk=dv=128, 16-node trees (depth<=5, branch<=3), 24 layers"),
        Config("large_batch_tree64", 4, 256, 16, 128, 256, 64, False, 8, 4, BF16, 1,
               "batch 256, 16 heads, dk=128, dv=256, 64-node trees (depth<=8, branch<=4)"),
        Config("large_batch_chain1", 5, 256, 16, 128, 256, 1, True, 1, 1, BF16, 1,
               "batch 256, 16 heads, dk=128, dv=256, 1-node chain (decode reference)"),
        Config("paper_fused_shape", 6, 1, 8, 256, 256, 4, True, 4, 1, BF16, 1,
               "batch 1, 8 heads, dk=dv=256, chain of 4 (fused commit-and-verify study shape)"),
        Config("batched_tree_serving_f32", 7, 64, 16, 128, 128, 16, False, 5, 3, F32, 24,
               "batched_tree_serving with fp32 q/k/v"),
        Config("large_batch_tree64_f32", 8, 256, 16, 128, 256, 64, False, 8, 4, F32, 1,
               "large_batch_tree64 with fp32 q/k/v"),
    ]
}


def config(name: str) -> Config:
    return CONFIGS[name]


def base_seed(cfg: Config) -> int:
    return 1000 + cfg.index


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(x) for x in key])))


# ---------------------------------------------------------------- bf16 storage
def bf16_bits(x) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); uint16 bits."""
    u = np.ascontiguousarray(np.asarray(x, dtype=np.float32)).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits) -> np.ndarray:
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16)).astype(np.uint32)
    return (b << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------- topologies
def random_tree(rng: np.random.Generator, n: int, max_depth: int, max_branch: int) -> np.ndarray:
    """Parent array of a random draft tree; node 0 is the only root."""
    parent = np.full(n, -1, np.int32)
    depth = np.zeros(n, np.int64)
    kids = np.zeros(n, np.int64)
    depth[0] = 1
    for i in range(1, n):
        eligible = [a for a in range(i) if depth[a] < max_depth and kids[a] < max_branch]
        if not eligible:
            raise ValueError("depth/branch limits too tight for %d nodes" % n)
        p = eligible[int(rng.integers(len(eligible)))]
        parent[i] = p
        depth[i] = depth[p] + 1
        kids[p] += 1
    return parent


def chain(n: int) -> np.ndarray:
    return np.arange(-1, n - 1, dtype=np.int32)


def walk_to_root(parent: np.ndarray, j: int) -> list:
    """Node ids from the root down to j (used to pick an accepted path)."""
    out = []
    a = int(j)
    while a != -1:
        out.append(a)
        a = int(parent[a])
    return out[::-1]


# ---------------------------------------------------------------- draws
def _normalised(rng: np.random.Generator, shape) -> np.ndarray:
    x = rng.standard_normal(shape)  # fp64
    x /= np.linalg.norm(x, axis=-1, keepdims=True)
    return x


def _to_dtype(x64: np.ndarray, dtype: str):
    """(storage array, exact fp32 values) for the activation dtype."""
    x32 = np.asarray(x64, dtype=np.float32)
    if dtype == BF16:
        bits = bf16_bits(x32)
        return bits, bf16_to_f32(bits)
    return x32, x32


@dataclass
class Round:
    """One speculative round of one configuration (all layers)."""
    parent: np.ndarray           # [B][n] int32
    path: np.ndarray             # [B][n] int32, -1 padded
    length: np.ndarray           # [B] int32
    q: list = field(default_factory=list)      # per layer: storage array [B][n][H][dk]
    k: list = field(default_factory=list)
    v: list = field(default_factory=list)      # [B][n][H][dv]
    q32: list = field(default_factory=list)    # exact fp32 values of the above
    k32: list = field(default_factory=list)
    v32: list = field(default_factory=list)
    alpha: list = field(default_factory=list)  # [B][n][H] fp32
    beta: list = field(default_factory=list)


def draw_topology(cfg: Config, round_index: int = 0, batch: int | None = None):
    """Parent arrays and accepted paths of one round (shared by all layers)."""
    B = cfg.batch if batch is None else batch
    n = cfg.n_nodes
    rng = _rng(base_seed(cfg), round_index, 0)
    parent = np.zeros((B, n), np.int32)
    path = np.full((B, n), -1, np.int32)
    length = np.zeros(B, np.int32)
    for b in range(B):
        if cfg.chain:
            parent[b] = chain(n)
        else:
            parent[b] = random_tree(rng, n, cfg.max_depth, cfg.max_branch)
    for b in range(B):
        if cfg.chain:
            A = 1 if n == 1 else int(rng.integers(0, n + 1))
            p = list(range(A))
        else:
            p = walk_to_root(parent[b], int(rng.integers(0, n)))
        path[b, :len(p)] = p
        length[b] = len(p)
    return parent, path, length


def draw_layer(cfg: Config, layer: int, round_index: int = 0, batch: int | None = None):
    """q, k, v, alpha, beta of one layer of one round."""
    B = cfg.batch if batch is None else batch
    n, H, dk, dv = cfg.n_nodes, cfg.heads, cfg.d_k, cfg.d_v
    rng = _rng(base_seed(cfg), round_index, 1, layer)
    q64 = _normalised(rng, (B, n, H, dk))
    k64 = _normalised(rng, (B, n, H, dk))
    v64 = rng.standard_normal((B, n, H, dv))
    alpha = (1.0 / (1.0 + np.exp(-rng.uniform(2.0, 5.0, (B, n, H))))).astype(np.float32)
    beta = (1.0 / (1.0 + np.exp(-rng.standard_normal((B, n, H))))).astype(np.float32)
    q, q32 = _to_dtype(q64, cfg.dtype)
    k, k32 = _to_dtype(k64, cfg.dtype)
    v, v32 = _to_dtype(v64, cfg.dtype)
    return dict(q=q, k=k, v=v, q32=q32, k32=k32, v32=v32, alpha=alpha, beta=beta)


FAMILIES = ("gdn", "deltanet", "decay", "gla")


def draw_gla_gates(cfg: Config, layer: int, round_index: int = 0, batch: int | None = None) -> np.ndarray:
    """GLA per-key gates of one layer of one round, [B][n][H][dk] fp32."""
    B = cfg.batch if batch is None else batch
    rng = _rng(base_seed(cfg), round_index, 5, layer)
    z = rng.standard_normal((B, cfg.n_nodes, cfg.heads, cfg.d_k))
    return ((1.0 / (1.0 + np.exp(-z))) ** (1.0 / 16.0)).astype(np.float32)


def family_gates(cfg: Config, rnd, layer_pos: int, family: str, layer: int | None = None,
                 round_index: int = 0, batch: int | None = None):
    """(alpha input, beta input) a family reads, None where it reads none."""
    if family == "gdn":
        return rnd.alpha[layer_pos], rnd.beta[layer_pos]
    if family == "deltanet":
        return None, rnd.beta[layer_pos]
    if family == "decay":
        return rnd.alpha[layer_pos], None
    if family == "gla":
        return draw_gla_gates(cfg, layer_pos if layer is None else layer, round_index, batch), None
    raise ValueError(family)


def draw_strong_gates(cfg: Config, layer: int, round_index: int = 0, batch: int | None = None,
                      family: str = "gdn") -> np.ndarray:
    """Strong-forgetting gates (the near-reset edge of a gated state):
    alpha ~ U(1e-3, 0.3), with about 3% of the gates set to 1e-6 and 2% to
    1e-20; [B][n][H] fp32, or [B][n][H][dk] per-key gates for "gla".  Along
    a root path their products leave the fp32 range within a few nodes."""
    B = cfg.batch if batch is None else batch
    shape = (B, cfg.n_nodes, cfg.heads) + ((cfg.d_k,) if family == "gla" else ())
    rng = _rng(base_seed(cfg), round_index, 7, layer)
    g = rng.uniform(1e-3, 0.3, shape)
    u = rng.uniform(0.0, 1.0, shape)
    g[u < 0.03] = 1e-6
    g[(u >= 0.03) & (u < 0.05)] = 1e-20
    return g.astype(np.float32)


def draw_state(cfg: Config, layer: int, batch: int | None = None) -> np.ndarray:
    """Committed fp32 state H = S^T of one layer, [B][H][dk][dv]."""
    B = cfg.batch if batch is None else batch
    rng = _rng(base_seed(cfg), 2, layer)
    s = rng.standard_normal((B, cfg.heads, cfg.d_k, cfg.d_v), dtype=np.float32)
    s *= np.float32(0.02)
    return s


def draw_round(cfg: Config, round_index: int = 0, layers=None, batch: int | None = None) -> Round:
    parent, path, length = draw_topology(cfg, round_index, batch)
    r = Round(parent=parent, path=path, length=length)
    for layer in (range(cfg.layers) if layers is None else layers):
        d = draw_layer(cfg, layer, round_index, batch)
        r.q.append(d["q"]); r.k.append(d["k"]); r.v.append(d["v"])
        r.q32.append(d["q32"]); r.k32.append(d["k32"]); r.v32.append(d["v32"])
        r.alpha.append(d["alpha"]); r.beta.append(d["beta"])
    return r


# ---------------------------------------------------------------- short convolution
CONV_KERNEL = 4


def conv_channels(cfg: Config) -> int:
    """Channels of the layer's short convolution: q, k and v of every head."""
    return cfg.heads * (2 * cfg.d_k + cfg.d_v)


def draw_conv_x(cfg: Config, layer: int, round_index: int = 0, batch: int | None = None,
                channels: int | None = None):
    """Pre-convolution inputs of one layer of one round, [B][n][D]:
    (storage array, exact fp32 values)."""
    B = cfg.batch if batch is None else batch
    D = conv_channels(cfg) if channels is None else channels
    rng = _rng(base_seed(cfg), round_index, 3, layer)
    return _to_dtype(rng.standard_normal((B, cfg.n_nodes, D), dtype=np.float32), cfg.dtype)


def draw_conv_weight(cfg: Config, layer: int, channels: int | None = None, kernel: int = CONV_KERNEL) -> np.ndarray:
    """Depthwise weights [D][K], fp32."""
    D = conv_channels(cfg) if channels is None else channels
    rng = _rng(base_seed(cfg), 4, layer)
    lim = 1.0 / np.sqrt(kernel)
    return rng.uniform(-lim, lim, (D, kernel)).astype(np.float32)


def draw_conv_state(cfg: Config, layer: int, batch: int | None = None, channels: int | None = None,
                    kernel: int = CONV_KERNEL) -> np.ndarray:
    """Committed conv state [B][K-1][D]: earlier inputs (activation-dtype
    values) held in fp32."""
    B = cfg.batch if batch is None else batch
    D = conv_channels(cfg) if channels is None else channels
    rng = _rng(base_seed(cfg), 5, layer)
    _, c32 = _to_dtype(rng.standard_normal((B, kernel - 1, D), dtype=np.float32), cfg.dtype)
    return np.ascontiguousarray(c32)


# ---------------------------------------------------------------- draft rollouts
def rollout(rng: np.random.Generator, n_cand: int, k: int = 4, vocab: int = 32, temp: float = 2.0,
            max_depth: int | None = None):
    """(parent [<= n_cand] int32, logp fp32) of one beam top-k rollout, nodes
    in creation (topological) order; at most max_depth levels when given."""
    parent, logp, score = [], [], []

    def children(of):
        z = rng.standard_normal(vocab) * temp
        lse = np.log(np.sum(np.exp(z - z.max()))) + z.max()
        lp = np.sort(z - lse)[::-1][:k]
        for x in lp:
            if len(parent) < n_cand:
                parent.append(of)
                logp.append(float(x))
                score.append(float(x) + (score[of] if of >= 0 else 0.0))

    children(-1)
    frontier = list(range(len(parent)))
    level = 1
    while len(parent) < n_cand and frontier and (max_depth is None or level < max_depth):
        level += 1
        best = sorted(frontier, key=lambda v: -score[v])[:k]
        start = len(parent)
        for v in best:
            children(v)
        frontier = list(range(start, len(parent)))
    return np.array(parent, np.int32), np.array(logp, np.float32)


def draw_rollouts(cfg: Config, round_index: int = 0, batch: int | None = None, n_cand: int = 64, k: int = 4):
    """Candidate sets of one round for every sequence: parent, logp [B][n_cand]."""
    B = cfg.batch if batch is None else batch
    rng = _rng(base_seed(cfg), round_index, 6)
    rows = [rollout(rng, n_cand, k) for _ in range(B)]
    return np.stack([r[0] for r in rows]), np.stack([r[1] for r in rows])
