"""Pins for the oracle's ball-tree ordering (CPU only).

The paper gives no worked tree, so the oracle is pinned by: two hand-worked cases
(tests/golden/tree_hand_2d.txt), the one-dimensional case reducing to a stable argsort,
the bijection, the per-node split invariants checked by independent code, the even
spreading of dummies, and invariance of the ordered coordinates under input shuffling.
"""
import os

import numpy as np
import pytest

from oracle.tree import build_ball_tree, permute_rows
from workloads import CONFIGS, make_points

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tree_hand_2d.txt")


def _read_cases():
    cases, cur = [], None
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, *vals = line.split()
        if key == "case":
            cur = {"points": [], "name": vals[0]}
            cases.append(cur)
        elif key == "n_pad":
            cur["n_pad"] = int(vals[0])
        elif key == "point":
            cur["points"].append([float(x) for x in vals])
        elif key == "perm":
            cur["perm"] = [int(x) for x in vals]
    return cases


@pytest.mark.parametrize("case", _read_cases(), ids=lambda c: c["name"])
def test_hand_worked(case):
    pts = np.array(case["points"], dtype=np.float32)
    perm = build_ball_tree(pts, case["n_pad"])
    assert perm.tolist() == case["perm"]


def test_1d_full_is_stable_argsort():
    rng = np.random.default_rng(0)
    x = rng.integers(0, 40, 256).astype(np.float32)   # many equal coordinates
    perm = build_ball_tree(x[:, None], 256)
    assert np.array_equal(perm, np.argsort(x, kind="stable"))


def _split_counts_ok(perm):
    """Every node's left half holds ceil(cnt/2) of its real points."""
    real = (perm >= 0).astype(np.int64)
    n = perm.size
    c = n
    while c >= 2:
        blocks = real.reshape(n // c, 2, c // 2).sum(axis=2)
        left, right = blocks[:, 0], blocks[:, 1]
        if not np.all((left - right == 0) | (left - right == 1)):
            return False
        c //= 2
    return True


def test_1d_with_dummies():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(300).astype(np.float32)
    perm = build_ball_tree(x[:, None], 512)
    assert np.array_equal(perm[perm >= 0], np.argsort(x, kind="stable"))
    assert _split_counts_ok(perm)


def _node_invariants(pts, perm):
    n = perm.size
    c = n
    while c >= 2:
        for s in range(0, n, c):
            ids = perm[s:s + c]
            ids = ids[ids >= 0]
            if ids.size < 2:
                continue
            sub = pts[ids].astype(np.float64)
            spread = [sub[:, a].max() - sub[:, a].min() for a in range(pts.shape[1])]
            best = max(spread)
            axis = min(a for a in range(len(spread)) if spread[a] == best)
            left = perm[s:s + c // 2]
            right = perm[s + c // 2:s + c]
            left, right = left[left >= 0], right[right >= 0]
            assert left.size == (ids.size + 1) // 2
            kl = [(float(pts[i, axis]) + 0.0, int(i)) for i in left]
            kr = [(float(pts[i, axis]) + 0.0, int(i)) for i in right]
            if kr:
                assert max(kl) < min(kr)
        c //= 2


@pytest.mark.parametrize("n_real,n_pad", [(64, 64), (50, 64), (33, 64), (1, 8), (0, 8)])
def test_node_invariants_3d(n_real, n_pad):
    rng = np.random.default_rng(n_real)
    pts = rng.uniform(0, 1, (n_real, 3)).astype(np.float32)
    pts[: n_real // 3, 1] = np.round(pts[: n_real // 3, 1] * 4) / 4   # coordinate ties
    perm = build_ball_tree(pts, n_pad)
    assert sorted(perm[perm >= 0].tolist()) == list(range(n_real))
    assert int((perm < 0).sum()) == n_pad - n_real
    assert _split_counts_ok(perm)
    _node_invariants(pts, perm)


def test_config2_cloud_invariants():
    cfg = CONFIGS[2]
    pts = make_points(cfg)[0]
    perm = build_ball_tree(pts, cfg.n_pad)
    assert sorted(perm[perm >= 0].tolist()) == list(range(cfg.n_real))
    assert _split_counts_ok(perm)
    # 3586 of 4096 slots are real: every aligned block of 8 holds at least 7 real points.
    assert (perm >= 0).reshape(-1, 8).sum(axis=1).min() >= 7


def test_shuffle_invariance():
    rng = np.random.default_rng(7)
    pts = rng.standard_normal((200, 3)).astype(np.float32)
    perm = build_ball_tree(pts, 256)
    sh = rng.permutation(200)
    perm2 = build_ball_tree(pts[sh], 256)
    a = permute_rows(pts, perm)
    b = permute_rows(pts[sh], perm2)
    assert np.array_equal(a, b)
    assert np.array_equal(perm < 0, perm2 < 0)


def test_permute_rows():
    x = np.arange(12, dtype=np.float32).reshape(4, 3)
    out = permute_rows(x, np.array([2, -1, 0, 3, -1, 1, -1, -1]))
    assert np.array_equal(out[0], x[2]) and np.array_equal(out[5], x[1])
    assert not out[1].any() and not out[7].any()
