"""Models of the paper's speculative Procedures 4 and 5: TEST INFRASTRUCTURE ONLY.

Section 3.3 (Procedure 4, "Speculative Parallel Tree Evaluation"): one processor per tree
node evaluates its node for the record and stores the index of the chosen child in a
shared array ``path``; leaves are made to choose themselves.  The processors then
repeatedly replace their entry by the entry of their successor (pointer jumping) until
``path[0]`` names a leaf; that leaf's class is the record's class.

Section 3.4 (Procedure 5, the improved version): processors exist only for decision
nodes, mapped to them through a per-tree table; the leaf entries of ``path`` are set once
from a static table; each loop trip performs several jumps at once (the paper shows three
reads, ``path[path[path[i]]]``).

These models evaluate the same records as the plain oracle by a completely different
route, so agreement pins both.  They use this library's comparison (``x < t`` -> left,
i.e. the chosen child is ``left + (not x < t)``).  Readings taken where the paper is
unclear:
  * leaves choose themselves (the paper's "threshold -inf, child = own index" is
    inconsistent as printed, so the model sets ``path[leaf] = leaf`` directly);
  * the static initialisation covers all N entries of ``path`` (the printed loop over
    ``2 p_n`` and ``2 p_n + 1`` for ``p_n < (N-1)/2`` reaches only N-1 of them);
  * the outcome does not depend on the jump schedule: any order of in-place updates
    reaches the same terminal leaf (checked by ``procedure5_async``).
"""
from __future__ import annotations

import numpy as np


def _split(nodes):
    feat = np.asarray(nodes["feature"], dtype=np.int64)
    thr = np.asarray(nodes["threshold"], dtype=np.float32)
    left = np.asarray(nodes["left"], dtype=np.int64)
    cls = np.asarray(nodes["cls"], dtype=np.int64)
    internal = cls < 0
    return feat, thr, left, cls, internal


def _node_evaluation(x, feat, thr, left, internal):
    """path after the node-evaluation step, one row per record (internal nodes only)."""
    n_rec = x.shape[0]
    n_nodes = len(feat)
    path = np.tile(np.arange(n_nodes, dtype=np.int64), (n_rec, 1))   # leaves -> themselves
    idx = np.nonzero(internal)[0]
    xv = x[:, feat[idx]]                                    # [n_rec, n_internal]
    go_right = ~(xv < thr[idx][None, :])
    path[:, idx] = left[idx][None, :] + go_right.astype(np.int64)
    return path


def procedure4(nodes, x: np.ndarray):
    """Procedure 4: synchronous single jumps until path[0] is a leaf.

    Returns (leaf index per record, number of jump rounds per record).
    """
    feat, thr, left, cls, internal = _split(nodes)
    path = _node_evaluation(np.asarray(x, dtype=np.float32), feat, thr, left, internal)
    rows = np.arange(path.shape[0])
    rounds = np.zeros(path.shape[0], dtype=np.int64)
    for _ in range(len(feat) + 1):
        active = internal[path[:, 0]]
        if not active.any():
            break
        # every processor copies its successor's entry; all reads see the old array (barrier)
        new = np.take_along_axis(path, path, axis=1)
        path[active] = new[active]
        rounds += active
    else:
        raise RuntimeError("path reduction did not terminate")
    return path[rows, 0], rounds


def procedure5(nodes, x: np.ndarray, hops: int = 2):
    """Procedure 5: processors on decision nodes only, static leaf entries, ``hops`` jumps
    per trip (path[i] <- path^(hops)[i] read from the array of the previous trip).

    The paper's printed line reads three levels of ``path`` (two jumps on top of the
    entry itself); ``hops=2`` models that line.
    """
    feat, thr, left, cls, internal = _split(nodes)
    n_nodes = len(feat)
    leaf_paths = np.arange(n_nodes, dtype=np.int64)         # static: leaf -> itself
    proc_node_map = np.nonzero(internal)[0]                 # processor p -> its node
    x = np.asarray(x, dtype=np.float32)
    path = np.tile(leaf_paths, (x.shape[0], 1))
    ev = _node_evaluation(x, feat, thr, left, internal)
    path[:, proc_node_map] = ev[:, proc_node_map]
    rows = np.arange(x.shape[0])
    for _ in range(n_nodes + 1):
        active = internal[path[:, 0]]
        if not active.any():
            break
        old = path.copy()
        cur = old[:, proc_node_map]
        for _ in range(hops):
            cur = np.take_along_axis(old, cur, axis=1)
        upd = path[:, proc_node_map]
        upd[active] = cur[active]
        path[:, proc_node_map] = upd
    else:
        raise RuntimeError("path reduction did not terminate")
    return path[rows, 0]


def procedure5_async(nodes, x: np.ndarray, rng: np.random.Generator, hops: int = 2):
    """Procedure 5 with the barrier removed: processors update ``path`` in place, one at
    a time, in a random order each trip.  Every entry always names a node on the record's
    own root-to-leaf path below its owner, so any schedule ends at the same leaf."""
    feat, thr, left, cls, internal = _split(nodes)
    n_nodes = len(feat)
    proc_node_map = np.nonzero(internal)[0]
    x = np.asarray(x, dtype=np.float32)
    out = np.empty(x.shape[0], dtype=np.int64)
    for r in range(x.shape[0]):
        path = np.arange(n_nodes, dtype=np.int64)
        for i in proc_node_map:
            path[i] = left[i] + (0 if x[r, feat[i]] < thr[i] else 1)
        for _ in range(4 * n_nodes + 4):
            if not internal[path[0]]:
                break
            for i in rng.permutation(proc_node_map):
                v = path[i]
                for _ in range(hops):
                    v = path[v]
                path[i] = v
        else:
            raise RuntimeError("asynchronous path reduction did not terminate")
        out[r] = path[0]
    return out
