"""Determinism and shape of the seeded synthetic workloads (CPU)."""
from __future__ import annotations

import hashlib

import numpy as np
import pytest

from workloads import configs, generators as gen
from workloads.rng import Stream


def _digest(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def test_stream_is_deterministic_and_counter_based():
    a = Stream(5, "x").uniform(1000)
    b = Stream(5, "x").uniform(1000)
    assert np.array_equal(a, b)
    s = Stream(5, "x")
    c = np.concatenate([s.uniform(300), s.uniform(700)])
    assert np.array_equal(a, c)
    assert not np.array_equal(a, Stream(6, "x").uniform(1000))
    assert not np.array_equal(a, Stream(5, "y").uniform(1000))
    assert a.min() >= 0.0 and a.max() < 1.0
    z = Stream(1, "n").normal(200_000)
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1.0) < 0.01


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 6, 7, 8, 9])
def test_config_shapes_and_determinism(cfg):
    a = configs.make(cfg)
    b = configs.make(cfg)
    assert _digest(a.positions) == _digest(b.positions)
    assert _digest(a.features) == _digest(b.features)
    assert a.positions.dtype == np.float32 and a.positions.shape[1] == 3
    assert np.isfinite(a.positions).all()
    expect_m = {1: 4096, 2: 2048, 3: 200_000, 4: 120_000, 6: 120_000, 7: 120_000, 8: 120_000, 9: 200_000}[cfg]
    assert a.m == expect_m
    for name, w in a.weights.items():
        assert w.shape[0] == configs.TAPS
    # every buffer column range written or read fits its buffer
    for op in a.ops:
        for key in ("src", "dst"):
            if key in op:
                buf, c0, cc = op[key]
                assert c0 + cc <= a.buffers[buf][1]


def test_object_is_normalised_to_unit_sphere():
    p = configs.make(2).positions.astype(np.float64)
    assert abs(np.linalg.norm(p, axis=1).max() - 1.0) < 1e-6
    assert np.abs(p.mean(axis=0)).max() < 1e-5


def test_lidar_geometry():
    p = configs.make(4).positions.astype(np.float64)
    r = np.linalg.norm(p[:, :2], axis=1)
    assert r.max() <= 50.0 + 0.1
    assert (p[:, 2] > -0.2).all()
    assert np.mean(np.abs(p[:, 2]) < 0.1) > 0.5          # mostly ground hits


def test_bf16_rounding_of_inputs():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5e-3, np.inf], np.float32)
    r = gen.bf16_bits_to_f32(gen.to_bf16_bits(x))
    assert r[0] == 1.0 and r[1] == 1.0 and r[2] == np.float32(1.0 + 2 ** -6) and np.isinf(r[4])


@pytest.mark.slow
def test_config5_small_variant():
    wl = configs.config5(m=20_000)
    assert wl.dtype == "bf16" and wl.levels == 4
    assert np.array_equal(gen.bf16_bits_to_f32(gen.to_bf16_bits(wl.features)), wl.features)


def test_bench_default_layout():
    """The bench's pipeline layout per workload: three pipelines on one build
    stream for the 120k-point LiDAR workloads and the multi-level 200k-point
    LatticeNet, two with a build stream each for the single-level room and
    the training step, two on one build stream for the 1M-point clouds."""
    import bench
    expect = {3: (2, False), 4: (3, True), 5: (2, True), 6: (3, True), 7: (2, False), 8: (3, True),
              9: (3, True), 10: (2, True)}
    for cfg, layout in expect.items():
        assert bench.default_layout(configs.make(cfg)) == layout, cfg
