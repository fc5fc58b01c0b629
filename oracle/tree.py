"""Ball-tree ordering of a point cloud (oracle; test infrastructure only).

The paper orders an unordered point set with the ball tree of Erwin so that contiguous,
aligned runs of the sequence are spatial balls, the leaf level being the full sequence
(Section 1, Section 2.1 "Ball Tree Attention", Section 2.2). It does not spell out the
construction, so the oracle uses this reading:

  node(S, C): S = set of real point indices, C = capacity (a power of two).
    * C == 1: the slot holds S's single point, or -1 (a dummy) if S is empty.
    * otherwise: split axis = argmax over axes of (max - min) of S's coordinates; the
      extremes are exact float32 values and the subtraction is done in float64; equal
      spreads go to the lowest axis. S is ordered by (coordinate on that axis, original
      index), with -0.0 equal to +0.0. The first ceil(|S|/2) points form the left child
      and the rest the right child, each of capacity C/2.

The recursion runs down to single points, so every aligned power-of-two run of slots
(a ball, a compression block, a selection block, a query group) is a subtree. Dummies
(padding up to the power-of-two length) spread evenly over the tree.
"""
from __future__ import annotations

import numpy as np


def build_ball_tree(points: np.ndarray, n_pad: int) -> np.ndarray:
    """Slot -> point permutation of one cloud.

    points: [n_real, D] float32 coordinates. n_pad: power of two >= n_real.
    Returns int64 [n_pad]; slot s holds the index of the point placed there, or -1.
    """
    pts = np.asarray(points, dtype=np.float32)
    n_real, dim = pts.shape
    if n_pad < 1 or n_pad & (n_pad - 1):
        raise ValueError("n_pad must be a power of two")
    if n_real > n_pad:
        raise ValueError("more points than slots")
    perm = np.full(n_pad, -1, dtype=np.int64)

    def node(idx: np.ndarray, start: int, cap: int) -> None:
        if idx.size == 0:
            return
        if cap == 1:
            perm[start] = idx[0]
            return
        sub = pts[idx]
        spread = sub.max(axis=0).astype(np.float64) - sub.min(axis=0).astype(np.float64)
        axis = int(np.argmax(spread))          # first maximum = lowest axis on ties
        key = sub[:, axis] + np.float32(0.0)   # -0.0 + 0.0 == +0.0
        order = np.lexsort((idx, key))         # by coordinate, then by original index
        srt = idx[order]
        n_left = (srt.size + 1) // 2
        node(srt[:n_left], start, cap // 2)
        node(srt[n_left:], start + cap // 2, cap // 2)

    node(np.arange(n_real, dtype=np.int64), 0, n_pad)
    return perm


def permute_rows(x: np.ndarray, perm: np.ndarray) -> np.ndarray:
    """Gather rows into slot order: out[s] = x[perm[s]], zero rows where perm[s] == -1."""
    out = np.zeros((perm.shape[0],) + x.shape[1:], dtype=x.dtype)
    real = perm >= 0
    out[real] = x[perm[real]]
    return out
