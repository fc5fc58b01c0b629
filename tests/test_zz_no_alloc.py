"""The allocation-free tree build (bsa_build_ball_tree_noalloc, for callers that cannot
allocate) against the workspace entry point bsa_build_ball_tree: bit-exact orderings on
two calls in a row, the second on a smaller input (the static scratch keeps the first
call's contents), and a size beyond the scratch's limit rejected before any launch."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2506_12541_amd import _lib
from paper_2506_12541_amd import bsa as gb
from workloads import CONFIGS, make_points

pytestmark = pytest.mark.gpu


def _both(pts_np, n_pad):
    pts = torch.from_numpy(np.ascontiguousarray(pts_np, dtype=np.float32)).cuda()
    ref = gb.build_ball_tree(pts, n_pad)
    perm = torch.full((pts.shape[0], n_pad), -7, dtype=torch.int32, device="cuda")
    gb.build_ball_tree_noalloc(pts, perm)
    torch.cuda.synchronize()
    return ref.cpu().numpy(), perm.cpu().numpy()


def test_noalloc_tree_matches_workspace_tree():
    lib = _lib.load()
    # first call: the 65536-point Gaussian-mixture cloud (65536 slots)
    cfg = CONFIGS[3]
    print("allocation-free tree: 1 x 65536 points", flush=True)
    ref, got = _both(make_points(cfg), cfg.n_pad)
    assert np.array_equal(ref, got)
    # second call, smaller: 2 clouds of 900 points in 1024 slots, 2-D, with ties
    rng = np.random.default_rng(5)
    pts = rng.uniform(-1, 1, (2, 900, 2)).astype(np.float32)
    pts[:, :200, 0] = np.round(pts[:, :200, 0] * 3)
    print("allocation-free tree: 2 x 900 points in 1024 slots", flush=True)
    ref2, got2 = _both(pts, 1024)
    assert np.array_equal(ref2, got2)
    # the limit: 2 x 131072 slots is rejected on the host, nothing launched
    fake = C.c_void_p(256)
    st = lib.bsa_build_ball_tree_noalloc(fake, 100000, 3, 1 << 17, 2, fake, None)
    assert st == _lib.BSA_ERR_UNSUPPORTED
    assert "limit" in lib.bsa_last_error().decode()
