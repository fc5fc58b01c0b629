"""Host-side logic, CPU only: the benchmark's one-GPU guard, its FLOP model against the
formulas it documents, the committed traffic summary's source check, the binding failing
loudly without the library, and the seeded generators."""
import dataclasses
import importlib
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_algorithmic_flops_scaling_workload():
    import bench
    from workloads import CONFIGS
    cfg = CONFIGS[3]
    fwd, bwd = bench.algorithmic_flops(cfg)
    # per head: ball 4 N m d, MLP 2 * 2 (N/l)(l d d + d d), compressed 4 N (N/l) d, scoring
    # 2 (N/g)(N/l) d, selection 4 N k* l' d; backward 2.5x attention, 2x MLP, no scoring
    N, d, H = 65536, 64, 8
    m, l, ls, k, g = 256, 16, 32, 16, 16
    f = {"ball": 4 * N * m * d, "mlp": 4 * (N / l) * (l * d * d + d * d), "cmp": 4 * N * (N / l) * d,
         "score": 2 * (N / g) * (N / l) * d, "slc": 4 * N * k * ls * d}
    for name, v in f.items():
        assert fwd[name] == pytest.approx(v * H)
    total = sum(fwd.values()) + sum(bwd.values())
    assert sum(fwd.values()) == pytest.approx(679.1e9, rel=1e-3)
    assert total == pytest.approx(2329.5e9, rel=1e-3)
    # group compression: the compressed branch attends from N/l coarse rows
    fg, _ = bench.algorithmic_flops(cfg, "group_cmp")
    assert fg["cmp"] == pytest.approx(4 * (N / l) * (N / l) * d * H)


def test_block_flops():
    import bench
    fwd, bwd = bench.block_flops(65536, 512, 2048)
    assert fwd == pytest.approx(2 * 65536 * 512 * (3 * 512 + 512 + 2 * 2048 + 2048))
    assert bwd == pytest.approx(2 * fwd)


def test_traffic_summary_tracks_its_sources(tmp_path, monkeypatch):
    import bench
    # a summary is reported while the sources it names hash as recorded, and not once one
    # of them changes (a summary of the same form as the committed ones, on a scratch file)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic_{phase}_{workload}.txt"))
    src = tmp_path / "kernel.hip"
    src.write_text("// kernel source\n")
    (tmp_path / "traffic_bwd_kv_cmp_scaling_65536.txt").write_text(
        "# HBM traffic\nphase: bwd.kv_cmp\nworkload: scaling_65536\ntraffic_bytes_per_launch: 1234\n"
        f"sources: kernel.hip\nsources_sha256: {bench._sources_sha(['kernel.hip'])}\n")
    assert bench.measured_traffic("bwd.kv_cmp", "scaling_65536") == 1234
    src.write_text("// kernel source, changed\n")
    assert bench.measured_traffic("bwd.kv_cmp", "scaling_65536") is None


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    from paper_2506_12541_amd import _lib
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        _lib.load()


def test_generators_are_seeded_and_padding_is_zero():
    from workloads import CONFIGS, make_block_inputs, make_inputs
    cfg = dataclasses.replace(CONFIGS[1], n_real=1000)
    a = make_inputs(cfg, seed=5)
    b = make_inputs(cfg, seed=5)
    c = make_inputs(cfg, seed=6)
    assert np.array_equal(a["q"], b["q"]) and not np.array_equal(a["q"], c["q"])
    valid = np.ones((cfg.batch, cfg.n_pad), bool)
    valid[0, 100:124] = False
    blk = make_block_inputs(cfg, valid, seed=5)
    assert blk["x"].shape == (cfg.batch, cfg.n_pad, cfg.heads * cfg.head_dim)
    assert not np.any(blk["x"][0, 100:124]) and not np.any(blk["dy"][0, 100:124])
    assert np.all(np.any(blk["x"][0, :100] != 0, axis=-1))
    assert blk["W"]["w1"].shape == (blk["ffn"], cfg.heads * cfg.head_dim)


def test_rising_inputs_move_the_reference_in_every_tile():
    """Premise of the rising-maxima forward parity test: on its inputs every query's
    maximum over a 64-key tile exceeds its running maximum over the earlier tiles by more
    than the lazy-rescale margin (8 log2 units) in every tile after the first, in the ball
    branch (a middle ball of each head) and in the compressed branch (mean-pooled blocks of
    16 keys, every query). float64 on the inputs of both storage types."""
    from rising import rising_config, rising_inputs
    for dtype in ("bf16", "f32"):
        _check_rising(rising_config(dtype), rising_inputs(rising_config(dtype)))


def _check_rising(cfg, inp):
    d, m, n, l = cfg.head_dim, cfg.ball, cfg.n_pad, cfg.cmp_block
    sl2 = 1.0 / np.sqrt(d) / np.log(2.0)    # softmax scale in log2 units

    def tile_rises(s):
        tmax = s.reshape(s.shape[0], -1, 64).max(-1)
        return tmax[:, 1:] - np.maximum.accumulate(tmax, axis=1)[:, :-1]

    for h in range(cfg.heads):
        q = inp["q"][0, h].astype(np.float64)
        k = inp["k"][0, h].astype(np.float64)
        b0 = (n // m // 2) * m
        ball = q[b0:b0 + m] @ k[b0:b0 + m].T * sl2
        assert tile_rises(ball).min() > 8.0
        kc = k.reshape(n // l, l, d).mean(1)
        assert tile_rises(q @ kc.T * sl2).min() > 8.0
