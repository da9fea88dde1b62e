"""Oracle for the draft-side pruning and packing of SpecLA §6.1 and the
proposal converter of §7 (tree mask -> parent array).

TEST INFRASTRUCTURE ONLY: imported by ``tests/`` and by the benchmark's
CPU-baseline leg.  It shares no code with the HIP library.  Plain Python
loops over at most a few hundred candidates; numpy float32 scalars wherever a
floating-point value decides which node is kept, so that the decisions are
taken in the precision the library takes them in (fp32).

Definitions followed (§6.1, "Tree pruning"):
  * after the drafter's rollout every candidate v has a parent (-1: a child of
    the committed state) and the log-probability of its token given its path;
  * its score is the path's joint log-probability, summed along the root path
    from the root down:  q(v) = q(parent(v)) + logp(v), q = logp at a root;
  * with q* = max_v q(v) and a margin tau, the window keeps q(v) >= q* - tau;
  * a token budget T truncates the score-ranked selection; each retained
    candidate's missing ancestors are joined, until T is used up.
Readings (where the text is silent): ranking is by score, ties by the lower
index; a candidate is taken together with its missing ancestors only if they
all fit in the budget, and the selection stops at the first one that does
not; the window compares q(v) against the fp32 value q* - tau.

Packing (§7, the proposal converter feeding the verifier): the kept nodes keep
their relative (topological) order, are renumbered 0..m-1, and their parents
are renumbered accordingly; index_map[new] = old.

Tree mask -> parent array (§7; the mask M_tree of §4.2): row i of the mask
marks the ancestors of i, i included.  The parent of i is its deepest strict
ancestor, i.e. the strict ancestor whose own row marks the most nodes.
"""
from __future__ import annotations

import numpy as np

OK = 0
ERR_SHAPE = -2
ERR_TOPOLOGY = -4
ERR_SCORE = -10

F32 = np.float32


def _valid_parent(parent):
    n = len(parent)
    return all(-1 <= int(parent[j]) < j for j in range(n))


def scores(parent, logp):
    """q(v) in fp32, summed root first along the root path: returns (q, status).
    status ERR_SCORE for a log-probability above 0 or NaN (q must not increase
    along a path), ERR_TOPOLOGY for a parent array out of topological order."""
    parent = [int(p) for p in parent]
    n = len(parent)
    if not _valid_parent(parent):
        return None, ERR_TOPOLOGY
    lp = [F32(x) for x in logp]
    if any(not (x <= F32(0.0)) for x in lp):
        return None, ERR_SCORE
    q = []
    for v in range(n):
        path = []
        a = v
        while a != -1:
            path.append(a)
            a = parent[a]
        s = None
        for a in reversed(path):  # root first
            s = lp[a] if s is None else F32(s + lp[a])
        q.append(s)
    return np.array(q, np.float32), OK


def prune(parent, logp, tau, budget):
    """Kept candidates (sorted original indices), their scores and a status.
    budget <= 0 means no budget."""
    q, st = scores(parent, logp)
    if st != OK:
        return None, None, st
    n = len(q)
    qstar = F32(max(q))
    thr = F32(qstar - F32(tau))
    window = [v for v in range(n) if q[v] >= thr]
    if budget <= 0 or len(window) <= budget:
        return window, q, OK
    ranked = sorted(window, key=lambda v: (-float(q[v]), v))
    kept = set()
    for v in ranked:
        missing = []
        a = v
        while a != -1 and a not in kept:
            missing.append(a)
            a = int(parent[a])
        if len(kept) + len(missing) > budget:
            break
        kept.update(missing)
    return sorted(kept), q, OK


def pack(parent, keep):
    """(packed parent array, index_map): kept nodes renumbered in their order."""
    new = {old: i for i, old in enumerate(keep)}
    packed = []
    for old in keep:
        p = int(parent[old])
        if p != -1 and p not in new:
            raise ValueError("kept set is not ancestor-closed")
        packed.append(-1 if p == -1 else new[p])
    return np.array(packed, np.int32), np.array(keep, np.int32)


def mask_to_parent(mask):
    """Parent array from a tree mask given as boolean rows [n][n] (row i marks
    the ancestors of i, i included).  Returns (parent, status); status
    ERR_TOPOLOGY when the mask is not a tree mask in topological order (a
    missing diagonal, an ancestor after its descendant, ancestors that do not
    form one chain, or a row that is not closed under ancestry)."""
    m = np.asarray(mask, bool)
    n = m.shape[0]
    if m.shape != (n, n) or n < 1:
        return None, ERR_SHAPE
    depth = [int(np.count_nonzero(m[i])) for i in range(n)]
    parent = []
    for i in range(n):
        if not m[i, i]:
            return None, ERR_TOPOLOGY
        strict = [j for j in range(n) if j != i and m[i, j]]
        if any(j > i for j in strict):
            return None, ERR_TOPOLOGY
        # strict ancestors must form one chain: their depths are 1..len
        if sorted(depth[j] for j in strict) != list(range(1, len(strict) + 1)):
            return None, ERR_TOPOLOGY
        p = -1
        for j in strict:
            if p == -1 or depth[j] > depth[p]:
                p = j
        # the row is the parent's row plus i itself
        want = np.zeros(n, bool) if p == -1 else m[p].copy()
        want[i] = True
        if not np.array_equal(want, m[i]):
            return None, ERR_TOPOLOGY
        parent.append(p)
    return np.array(parent, np.int32), OK
