"""The radix top-k (pv_select_topk) against the oracle's rank-count top-k on
score vectors chosen to stress a radix select: ties of every size, all-equal
rows, signed zeros, keys that differ only in the last bit, scores packed
into one exponent, and sizes at the edges of the per-thread key counts.
Index results must match bit for bit."""

from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_25332_amd import provip
    provip.load()


def scores(kind: str, n: int, seed: int) -> np.ndarray:
    g = np.random.default_rng(seed)
    if kind == "normal":
        x = g.standard_normal(n)
    elif kind == "ties":
        x = g.choice(np.array([-1.5, 0.25, 0.5, 0.75, 3.0]), size=n)
    elif kind == "equal":
        x = np.full(n, 0.3)
    elif kind == "two":
        x = np.where(g.random(n) < 0.5, 1.0, 2.0)
    elif kind == "signed_zero":
        x = g.choice(np.array([0.0, -0.0, 1e-3, -1e-3]), size=n)
    elif kind == "lowbit":
        base = np.float32(0.8125)
        x = base + g.integers(0, 6, size=n).astype(np.float32) * np.spacing(base)
    elif kind == "packed":
        x = 1.0 + 1e-6 * g.standard_normal(n)
    elif kind == "negative":
        x = -np.abs(g.standard_normal(n)) - 1.0
    elif kind == "wide":
        x = g.choice([-1.0, 1.0], size=n) * 10.0 ** g.uniform(-30, 30, size=n)
    elif kind == "ascending":
        x = np.arange(n, dtype=np.float64)
    elif kind == "descending":
        x = -np.arange(n, dtype=np.float64)
    else:
        raise ValueError(kind)
    return np.ascontiguousarray(x, np.float32)


def run(sc: np.ndarray, k: int):
    from paper_2608_25332_amd import provip
    t = torch.from_numpy(sc).cuda()
    r = provip.pv_select_topk(t, k, want_rest=True, want_slot=True)
    torch.cuda.synchronize()
    return {key: v.cpu().numpy() for key, v in r.items()}


def check(sc2: np.ndarray, k: int, r: dict):
    B, n = sc2.shape
    for b in range(B):
        want = oracle.topk(sc2[b].astype(np.float64), k)
        np.testing.assert_array_equal(r["kept"][b], want)
        rest = np.setdiff1d(np.arange(n), want)
        np.testing.assert_array_equal(r["rest"][b], rest)
        slot = np.full(n, -1, np.int32)
        slot[want] = np.arange(k, dtype=np.int32)
        np.testing.assert_array_equal(r["slot_of"][b], slot)


KINDS = ["normal", "ties", "equal", "two", "signed_zero", "lowbit", "packed", "negative", "wide",
         "ascending", "descending"]
SIZES = [1, 2, 63, 64, 65, 192, 576, 1024, 1025, 2880, 4096, 4097, 4608, 5120, 5121]


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("kind", KINDS)
def test_topk_against_oracle(kind, n):
    for k in sorted({1, max(1, n // 3), max(1, n - 1), n}):
        sc = scores(kind, n, seed=1000 + n + k)
        print(f"topk kind={kind} n={n} k={k}", flush=True)
        r = run(sc[None], k)
        check(sc[None], k, r)


@pytest.mark.parametrize("kind", ["normal", "ties", "packed", "equal"])
def test_topk_max_tokens(kind):
    n = 16384
    for k in (1, 5461, n):
        sc = scores(kind, n, seed=7 + k)
        print(f"topk kind={kind} n={n} k={k}", flush=True)
        r = run(sc[None], k)
        check(sc[None], k, r)


def test_topk_batched_rows_independent():
    kinds = ["normal", "ties", "equal", "signed_zero", "lowbit", "packed", "wide", "two"]
    n, k = 576, 192
    sc = np.stack([scores(kd, n, seed=50 + i) for i, kd in enumerate(kinds)])
    sys.stdout.flush()
    r = run(sc, k)
    check(sc, k, r)


def test_topk_one_dimensional_input():
    sc = scores("normal", 100, seed=11)
    r = run(sc, 30)
    assert r["kept"].shape == (30,) and r["rest"].shape == (70,) and r["slot_of"].shape == (100,)
    check(sc[None], 30, {key: v[None] for key, v in r.items()})


def test_topk_deterministic():
    sc = scores("ties", 2880, seed=3)[None]
    a = run(sc, 960)
    b = run(sc, 960)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
