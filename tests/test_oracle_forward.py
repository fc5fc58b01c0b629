"""Pins for the oracle's forward pass (CPU only).

No printed value in the paper pins a layer output, so each step is tied to something
outside the oracle: full attention from torch's scaled_dot_product_attention (float64,
CPU) wherever a branch reduces to it, softmax rows summing to one, the pooled-query
score against explicitly averaged per-token scores (Eq. 11 vs Eq. 12), a brute-force
top-k, one-hot MLP weights exposing the block flatten order, and gate saturation.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.special import logsumexp

from oracle import bsa
from oracle.bsa import Params


def sdpa(q, k, v, mask=None):
    """torch SDPA in float64; mask [Nq, Nk] bool, True = may attend."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))[None, None]
    m = None if mask is None else torch.from_numpy(mask)[None, None]
    return F.scaled_dot_product_attention(t(q), t(k), t(v), attn_mask=m)[0, 0].numpy()


def rnd(rng, *shape):
    return rng.standard_normal(shape)


@pytest.fixture
def rng():
    return np.random.default_rng(1234)


def test_attend_matches_sdpa_and_lse(rng):
    q, k, v = rnd(rng, 12, 8), rnd(rng, 20, 8), rnd(rng, 20, 8)
    kv = rng.random(20) > 0.3
    o, lse = bsa.attend(q, k, v, kv, 1 / math.sqrt(8))
    mask = np.repeat(kv[None], 12, 0)
    assert np.allclose(o, sdpa(q, k, v, mask), atol=1e-12)
    ref = logsumexp((q @ k.T / math.sqrt(8))[:, kv], axis=1)
    assert np.allclose(lse, ref, atol=1e-12)


def test_ball_branch_one_ball_is_full_attention(rng):
    n, d = 64, 16
    q, k, v = rnd(rng, n, d), rnd(rng, n, d), rnd(rng, n, d)
    valid = np.ones(n, bool)
    o, _ = bsa.ball_branch(q, k, v, valid, Params(ball=n, cmp_block=4, slc_block=8, topk=2, group=4))
    assert np.allclose(o, sdpa(q, k, v), atol=1e-12)


def test_ball_branch_blocks_and_dummies(rng):
    n, d, m = 64, 8, 16
    q, k, v = rnd(rng, n, d), rnd(rng, n, d), rnd(rng, n, d)
    valid = rng.random(n) > 0.25
    o, lse = bsa.ball_branch(q, k, v, valid, Params(ball=m, cmp_block=4, slc_block=8, topk=2, group=4))
    ball = np.arange(n) // m
    mask = (ball[:, None] == ball[None, :]) & valid[None, :]
    ref = sdpa(q, k, v, mask)
    assert np.allclose(o[valid], ref[valid], atol=1e-12)
    assert not o[~valid].any() and np.all(np.isneginf(lse[~valid]))
    # rows sum to one: with V = 1 every real query outputs exactly 1
    o1, _ = bsa.ball_branch(q, k, np.ones((n, d)), valid,
                            Params(ball=m, cmp_block=4, slc_block=8, topk=2, group=4))
    assert np.allclose(o1[valid], 1.0, atol=1e-14)


def test_mean_pool_l1_compression_is_full_attention(rng):
    n, d = 48, 8
    q, k, v = rnd(rng, n, d), rnd(rng, n, d), rnd(rng, n, d)
    valid = np.ones(n, bool)
    P = Params(ball=16, cmp_block=1, slc_block=4, topk=2, group=4, kv_pool="mean")
    kc, _ = bsa.compress(k, valid, None, P)
    vc, _ = bsa.compress(v, valid, None, P)
    o, _ = bsa.compression_branch(q, kc, vc, bsa.block_valid(valid, 1), valid, P)
    assert np.allclose(o, sdpa(q, k, v), atol=1e-12)


def test_mlp_matches_torch_and_flatten_order(rng):
    l, d, n = 4, 8, 32
    x = rnd(rng, n, d)
    valid = rng.random(n) > 0.2
    phi = {"w1": rnd(rng, l * d, d) * 0.1, "b1": rnd(rng, d) * 0.1,
           "w2": rnd(rng, d, d) * 0.1, "b2": rnd(rng, d) * 0.1}
    P = Params(ball=16, cmp_block=l, slc_block=8, topk=2, group=4)
    out, _ = bsa.compress(x, valid, phi, P)
    t = lambda a: torch.from_numpy(a)
    xz = t(np.where(valid[:, None], x, 0.0)).reshape(n // l, l * d)
    ref = F.linear(F.gelu(F.linear(xz, t(phi["w1"]).T, t(phi["b1"])), approximate="none"),
                   t(phi["w2"]).T, t(phi["b2"]))
    assert np.allclose(out, ref.numpy(), atol=1e-13)
    # one-hot first layer: hidden unit j reads token tj, channel cj of its block
    w1 = np.zeros((l * d, d))
    picks = [(j % l, (3 * j) % d) for j in range(d)]
    for j, (tt, c) in enumerate(picks):
        w1[tt * d + c, j] = 1.0
    phi1 = {"w1": w1, "b1": np.zeros(d), "w2": np.eye(d), "b2": np.zeros(d)}
    out1, cache = bsa.compress(x, np.ones(n, bool), phi1, P)
    for blk in range(n // l):
        for j, (tt, c) in enumerate(picks):
            assert cache["pre"][blk, j] == x[blk * l + tt, c]
    assert np.allclose(out1, bsa.gelu(cache["pre"]), atol=0)


def _scores_per_token_mean(q, kc, valid, P):
    """Eq. 6 then Eq. 12: per-token scores averaged over each group, written out."""
    n, d = q.shape
    g, l, ls = P.group, P.cmp_block, P.slc_block
    ncb = kc.shape[0]
    out = np.zeros((n // g, n // ls))
    for p in range(n // g):
        s_bar = np.zeros(ncb)
        for t in range(p * g, (p + 1) * g):
            if valid[t]:
                s_bar += np.array([np.dot(q[t], kc[c]) for c in range(ncb)])
        s_bar /= g
        r = ls // l
        for j in range(n // ls):
            out[p, j] = sum(s_bar[j * r:(j + 1) * r]) / r
    return out


def test_group_scores_pooled_equals_averaged(rng):
    n, d = 64, 8
    P = Params(ball=32, cmp_block=4, slc_block=8, topk=3, group=8, mask_own_ball=False)
    q = rnd(rng, n, d)
    kc = rnd(rng, n // 4, d)
    valid = rng.random(n) > 0.1
    valid[-8:] = True
    s = bsa.group_block_scores(q, kc, valid, P)
    ref = _scores_per_token_mean(q, kc, valid, P)
    blk_ok = valid.reshape(-1, 8).any(axis=1)
    assert np.allclose(s[:, blk_ok], ref[:, blk_ok], atol=1e-13)
    assert np.all(np.isneginf(s[:, ~blk_ok]))


def test_own_ball_mask(rng):
    n, d = 64, 8
    P = Params(ball=16, cmp_block=4, slc_block=8, topk=3, group=4)
    s = bsa.group_block_scores(rnd(rng, n, d), rnd(rng, n // 4, d), np.ones(n, bool), P)
    for p in range(n // 4):
        for j in range(n // 8):
            own = (p * 4) // 16 == (j * 8) // 16
            assert np.isneginf(s[p, j]) == own


def test_topk_brute_force(rng):
    s = np.round(rng.standard_normal((40, 30)), 1)          # many exact ties
    s[rng.random(s.shape) < 0.2] = -np.inf
    s[3, :] = -np.inf
    s[4, :27] = -np.inf
    k = 5
    got = bsa.topk_blocks(s, k)
    for p in range(s.shape[0]):
        cand = sorted(((-s[p, j], j) for j in range(s.shape[1]) if np.isfinite(s[p, j])))
        exp = sorted(j for _, j in cand[:k])
        exp += [-1] * (k - len(exp))
        assert got[p].tolist() == exp


def test_g1_is_per_token_topk(rng):
    n, d = 32, 8
    P = Params(ball=16, cmp_block=4, slc_block=4, topk=2, group=1, mask_own_ball=False)
    q, kc = rnd(rng, n, d), rnd(rng, n // 4, d)
    sel = bsa.topk_blocks(bsa.group_block_scores(q, kc, np.ones(n, bool), P), 2)
    for t in range(n):
        sc = q[t] @ kc.T                                   # Eq. 6, one row
        assert sel[t].tolist() == sorted(np.argsort(-sc, kind="stable")[:2].tolist())


def test_selection_all_blocks_is_full_attention(rng):
    n, d = 64, 8
    P = Params(ball=16, cmp_block=4, slc_block=8, topk=8, group=4, mask_own_ball=False)
    q, k, v = rnd(rng, n, d), rnd(rng, n, d), rnd(rng, n, d)
    valid = np.ones(n, bool)
    sel = bsa.topk_blocks(bsa.group_block_scores(q, rnd(rng, n // 4, d), valid, P), P.topk)
    assert np.all(sel >= 0)
    o, _ = bsa.selection_branch(q, k, v, valid, sel, P)
    assert np.allclose(o, sdpa(q, k, v), atol=1e-12)


def test_per_token_selection_all_blocks_is_full_attention(rng):
    # g = 1: every query selects on its own scores (Eq. 7); with all blocks selected each
    # query attends to every key
    n, d = 64, 8
    P = Params(ball=16, cmp_block=4, slc_block=8, topk=8, group=1, mask_own_ball=False)
    q, k, v = rnd(rng, n, d), rnd(rng, n, d), rnd(rng, n, d)
    valid = np.ones(n, bool)
    sel = bsa.topk_blocks(bsa.group_block_scores(q, rnd(rng, n // 4, d), valid, P), P.topk)
    assert sel.shape == (n, 8) and np.all(sel >= 0)
    o, _ = bsa.selection_branch(q, k, v, valid, sel, P)
    assert np.allclose(o, sdpa(q, k, v), atol=1e-12)


def test_per_token_selection_is_a_block_mask(rng):
    # g = 1 with k* < blocks: query t attends exactly to the keys of its own selected blocks
    n, d, ls = 64, 8, 8
    P = Params(ball=16, cmp_block=4, slc_block=ls, topk=3, group=1)
    q, k, v = rnd(rng, n, d), rnd(rng, n, d), rnd(rng, n, d)
    valid = rng.random(n) > 0.2
    sel = bsa.topk_blocks(bsa.group_block_scores(q, rnd(rng, n // 4, d), valid, P), P.topk)
    mask = np.zeros((n, n), bool)
    for t in range(n):
        for j in sel[t]:
            if j >= 0:
                mask[t, j * ls:(j + 1) * ls] = True
    mask &= valid[None, :]
    o, _ = bsa.selection_branch(q, k, v, valid, sel, P)
    rows = valid & mask.any(axis=1)
    assert np.allclose(o[rows], sdpa(q, k, v, mask)[rows], atol=1e-12)
    assert not o[~valid].any()


def test_selection_all_candidates_masks_own_ball(rng):
    n, d = 64, 8
    P = Params(ball=16, cmp_block=4, slc_block=8, topk=6, group=4)
    q, k, v = rnd(rng, n, d), rnd(rng, n, d), rnd(rng, n, d)
    valid = np.ones(n, bool)
    sel = bsa.topk_blocks(bsa.group_block_scores(q, rnd(rng, n // 4, d), valid, P), P.topk)
    o, _ = bsa.selection_branch(q, k, v, valid, sel, P)
    ball = np.arange(n) // 16
    assert np.allclose(o, sdpa(q, k, v, ball[:, None] != ball[None, :]), atol=1e-12)


def test_selection_too_few_candidates(rng):
    n, d = 32, 8
    P = Params(ball=16, cmp_block=4, slc_block=8, topk=3, group=4)
    valid = np.ones(n, bool)
    s = bsa.group_block_scores(rnd(rng, n, d), rnd(rng, n // 4, d), valid, P)
    sel = bsa.topk_blocks(s, 3)
    assert np.all(sel[:, 2] == -1) and np.all(sel[:, :2] >= 0)


def _tiny_inputs(rng, B=2, H=2, n=64, d=8, n_real=53):
    P = Params(ball=16, cmp_block=4, slc_block=8, topk=2, group=4)
    valid = np.zeros((B, n), bool)
    for b in range(B):
        valid[b, rng.choice(n, n_real, replace=False)] = True
    x = lambda *s: rng.standard_normal(s)
    phi = lambda: {"w1": x(P.cmp_block * d, d) * 0.2, "b1": x(d) * 0.2, "w2": x(d, d) * 0.2, "b2": x(d) * 0.2}
    return P, x(B, H, n, d), x(B, H, n, d), x(B, H, n, d), valid, x(B, n, 3), phi(), phi()


def test_gate_saturation_isolates_branches(rng):
    P, q, k, v, valid, gate, pk, pv = _tiny_inputs(rng)
    out = bsa.forward(q, k, v, valid, np.full_like(gate, 40.0), pk, pv, P)
    assert np.allclose(out["o"], out["o_branch"].sum(axis=0), atol=1e-14)
    for br in range(3):
        g = np.full_like(gate, -40.0)
        g[..., br] = 40.0
        ob = bsa.forward(q, k, v, valid, g, pk, pv, P)
        assert np.allclose(ob["o"], out["o_branch"][br], atol=1e-15)
    # dummy query rows are zero in every branch
    for b in range(q.shape[0]):
        assert not out["o"][b][:, ~valid[b]].any()


# ---- query coarsening (Eq. 13-14) and group compression (Eq. 15) ----

def _isolate_cmp(gate):
    g = np.full_like(gate, -40.0)
    g[..., 1] = 40.0
    return g


def test_group_compression_l1_is_full_attention(rng):
    # l = g = 1 with mean pooling: every query is its own coarse query and every key its
    # own compressed token, so Eq. 15 is plain attention
    B, H, n, d = 1, 2, 32, 8
    P = Params(ball=16, cmp_block=1, slc_block=4, topk=2, group=1, kv_pool="mean",
               group_compression=True)
    q, k, v = rnd(rng, B, H, n, d), rnd(rng, B, H, n, d), rnd(rng, B, H, n, d)
    out = bsa.forward(q, k, v, np.ones((B, n), bool), _isolate_cmp(rnd(rng, B, n, 3)), None, None, P)
    for h in range(H):
        assert np.allclose(out["o"][0, h], sdpa(q[0, h], k[0, h], v[0, h]), atol=1e-12)


def test_group_compression_block_constant_queries_equal_regular(rng):
    # queries equal within each block of l: the block mean is each of them, so Eq. 15
    # gives what the per-token compression branch gives
    B, H, n, d, l = 1, 2, 64, 8, 4
    base = dict(ball=16, cmp_block=l, slc_block=8, topk=2, group=l)
    q = np.repeat(rnd(rng, B, H, n // l, d), l, axis=2)
    k, v = rnd(rng, B, H, n, d), rnd(rng, B, H, n, d)
    phi = lambda: {"w1": rnd(rng, l * d, d) * 0.2, "b1": rnd(rng, d) * 0.2, "w2": rnd(rng, d, d) * 0.2,
                   "b2": rnd(rng, d) * 0.2}
    pk, pv = phi(), phi()
    valid = np.ones((B, n), bool)
    gate = rnd(rng, B, n, 3)
    reg = bsa.forward(q, k, v, valid, gate, pk, pv, Params(**base))
    grp = bsa.forward(q, k, v, valid, gate, pk, pv, Params(**base, group_compression=True))
    assert np.allclose(grp["o_branch"][1], reg["o_branch"][1], atol=1e-12)
    assert np.allclose(grp["lse"][1], reg["lse"][1], atol=1e-12)
    assert np.array_equal(grp["sel"], reg["sel"])


def test_group_compression_copies_to_real_rows(rng):
    B, H, n, d, l = 1, 1, 64, 8, 4
    P = Params(ball=16, cmp_block=l, slc_block=8, topk=2, group=l, group_compression=True)
    q, k, v = rnd(rng, B, H, n, d), rnd(rng, B, H, n, d), rnd(rng, B, H, n, d)
    valid = rng.random((B, n)) > 0.3
    valid[0, 8:12] = False                                   # one block with no real token
    phi = lambda: {"w1": rnd(rng, l * d, d) * 0.2, "b1": rnd(rng, d) * 0.2, "w2": rnd(rng, d, d) * 0.2,
                   "b2": rnd(rng, d) * 0.2}
    out = bsa.forward(q, k, v, valid, rnd(rng, B, n, 3), phi(), phi(), P)
    o1, lse1 = out["o_branch"][1, 0, 0], out["lse"][1, 0, 0]
    for c in range(n // l):
        rows = [t for t in range(c * l, (c + 1) * l) if valid[0, t]]
        for t in rows:
            assert np.array_equal(o1[t], o1[rows[0]]) and lse1[t] == lse1[rows[0]]
    assert not o1[~valid[0]].any() and np.all(np.isneginf(lse1[~valid[0]]))
    # V = 1: every real row of a block with a real key outputs exactly 1 (rows sum to one)
    vc_one = bsa.group_compression_branch(out["qc"][0, 0], out["kc"][0, 0], np.ones((n // l, d)),
                                          bsa.block_valid(valid[0], l), valid[0], P)[0]
    assert np.allclose(vc_one[valid[0]], 1.0, atol=1e-14)


def test_mlp_coarsening_with_a_mean_mlp_equals_mean_coarsening(rng):
    # phi_q whose first layer averages the block and shifts it by +1000 (where exact-erf
    # GELU is the identity in float64), second layer identity with bias -1000: the MLP
    # form of Eq. 13 then computes the mean form, so outputs and selections agree
    B, H, n, d, l = 1, 2, 64, 8, 4
    base = dict(ball=16, cmp_block=l, slc_block=8, topk=2, group=l, group_compression=True)
    q, k, v = rnd(rng, B, H, n, d), rnd(rng, B, H, n, d), rnd(rng, B, H, n, d)
    valid = rng.random((B, n)) > 0.2
    phi = lambda: {"w1": rnd(rng, l * d, d) * 0.2, "b1": rnd(rng, d) * 0.2, "w2": rnd(rng, d, d) * 0.2,
                   "b2": rnd(rng, d) * 0.2}
    pk, pv = phi(), phi()
    pq = {"w1": np.tile(np.eye(d), (l, 1)) / l, "b1": np.full(d, 1000.0), "w2": np.eye(d),
          "b2": np.full(d, -1000.0)}
    gate = rnd(rng, B, n, 3)
    mean = bsa.forward(q, k, v, valid, gate, pk, pv, Params(**base))
    mlp = bsa.forward(q, k, v, valid, gate, pk, pv, Params(**base, q_coarsen="mlp"), phi_q=pq)
    assert np.allclose(mlp["qc"], mean["qc"], atol=1e-12)
    assert np.array_equal(mlp["sel"], mean["sel"])
    assert np.allclose(mlp["o"], mean["o"], atol=1e-11)


def test_block_coarsening_needs_group_equal_block():
    with pytest.raises(ValueError):
        Params(ball=16, cmp_block=4, slc_block=8, topk=2, group=8, group_compression=True)
    with pytest.raises(ValueError):
        Params(ball=16, cmp_block=4, slc_block=8, topk=2, group=8, q_coarsen="mlp")
