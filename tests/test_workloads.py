"""The seeded input recipes (CPU only)."""
import numpy as np
import pytest

from paper_2608_25332_amd import workloads as W


def _neighbour_cos(x, grid=24):
    n = x / np.linalg.norm(x, axis=-1, keepdims=True)
    g = n.reshape(grid, grid, -1)
    right = np.sum(g[:, :-1] * g[:, 1:], -1)
    down = np.sum(g[:-1] * g[1:], -1)
    return float(np.mean(np.concatenate([right.ravel(), down.ravel()])))


def test_bf16_rounding_rne():
    x = np.array([1.0, 1.00390625, 1.005859375, -2.5, 3.0e38, 1e-40], np.float32)
    bits = W.bf16_bits(x)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa (1.0) wins
    assert bits[1] == 0x3F80
    # 1 + 3*2^-9 rounds up to 1 + 2^-7
    assert bits[2] == 0x3F81
    assert W.bf16_from_bits(bits)[3] == -2.5
    y = W.bf16_round(np.random.default_rng(0).standard_normal(1000).astype(np.float32))
    assert np.array_equal(W.bf16_round(y), y)


def test_tiny_recipe():
    w = W.make_workload(1)
    assert w.vis.shape == (1, 64, 256) and w.vis.dtype == np.float32
    for a, b in w.dup_pairs:
        assert a < b and np.array_equal(w.vis[0, a], w.vis[0, b])
    assert len({int(x) for x in w.dup_pairs.ravel()}) == 16
    assert w.heads.tolist() == [[1]]
    assert (w.N1, w.N2) == (32, 16)
    w2 = W.make_workload(1)
    assert np.array_equal(w.vis, w2.vis) and np.array_equal(w.q, w2.q)


def test_llava_recipe():
    w = W.make_workload(2)
    assert w.vis.shape == (1, 576, 4096)
    assert np.array_equal(W.bf16_round(w.vis), w.vis)
    c = _neighbour_cos(w.vis[0].astype(np.float64))
    assert abs(c - 0.80) < 0.01, c
    assert w.q.shape == (1, 32, 64, 128) and w.k_full.shape == (1, 32, 576, 128)
    assert len(set(w.heads[0].tolist())) == 4 and w.heads.max() < 32


@pytest.mark.slow
def test_hires_followers():
    w = W.make_workload(4, B=1, with_kv=False)
    f = w.followers[0]
    assert len(f) >= 50
    x = w.vis[0].astype(np.float64)
    n = x / np.linalg.norm(x, axis=-1, keepdims=True)
    cos = np.sum(n[f[:, 0]] * n[f[:, 1]], -1)
    assert np.all(cos > 0.98), cos.min()


def test_multiframe_recipe():
    w = W.make_workload(5, B=1, with_kv=False)
    x = w.vis[0].reshape(8, 576, 5120).astype(np.float64)
    d = x[1:] - x[:1]
    assert abs(float(d.std()) - 0.1) < 0.01
