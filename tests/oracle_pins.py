"""Pins of the CPU oracle to facts that do not come from the oracle itself.

Every pin is a plain function taking the loaded oracle library (a ctypes
handle).  ``test_oracle_pins.py`` runs them against the real oracle;
``test_oracle_mutants.py`` runs them against copies of the oracle with a
planted mistake and requires that at least one pin fails for each.

Sources of truth used here: closed forms (cosines of constructed angles,
the logistic function), hand-worked examples (``golden/worked_examples.json``),
invariants that follow from the equations (row sums, shift invariance,
permutation equivariance), brute-force enumeration on tiny inputs, and
special cases that reduce to a library routine (numpy stable argsort,
torch.softmax in float64 on the CPU).
"""

from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np

import oracle as O

GOLDEN = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                     "worked_examples.json")))


def _rot(d, rng):
    q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    return q


# ----------------------------------------------------------- Eq. r, T -----

def pin_critical_text_two_tokens(lib):
    """Sec. 4.2 on two orthogonal text tokens of squared norms a and b: the
    logits are [[a, 0], [0, b]], so with s(x) the logistic function
    r = ((s(a) + 1 - s(b)) / 2, (1 - s(a) + s(b)) / 2), and T holds the token
    of larger norm alone (r[0] > 1/2 exactly when a > b)."""
    for a, b in ((1.5, 0.25), (0.2, 2.0), (3.0, 2.9)):
        E = np.zeros((1, 2, 3))
        E[0, 0, 0] = math.sqrt(a)
        E[0, 1, 2] = math.sqrt(b)
        r, mask, count = O.critical_text(E, lib=lib)
        sg = lambda x: 1.0 / (1.0 + math.exp(-x))
        want = np.array([(sg(a) + 1 - sg(b)) / 2, (1 - sg(a) + sg(b)) / 2])
        assert np.max(np.abs(r[0] - want)) < 1e-15
        assert mask[0].tolist() == ([1, 0] if a > b else [0, 1]) and count[0] == 1


def pin_critical_text_strictly_above_mean(lib):
    """Sec. 4.2, equation for T keeps tokens strictly above the mean.  Four
    integer vectors whose logit gaps (>= 2048) make every softmax row exact
    in float64: rows (1,0,0,0), (1/2,1/2,0,0), (1/2,0,1/2,0), (0,1/2,1/2,0),
    so r = (1/2, 1/4, 1/4, 0) and the mean is 1/4: T = {0} only."""
    E = np.array([[[256.0, 0, 0], [128, 128, 0], [128, 0, 128], [0, 32, 32]]])
    r, mask, count = O.critical_text(E, lib=lib)
    assert r[0].tolist() == [0.5, 0.25, 0.25, 0.0]
    assert mask[0].tolist() == [1, 0, 0, 0] and count[0] == 1


def pin_critical_text_library_and_fallback(lib):
    """r is the column mean of torch.softmax(E E^T) in float64 (no scale),
    sums to 1, and permuting the tokens permutes r and T; when every r is
    equal (orthogonal rows of equal norm: each row's softmax is the same up
    to a shift and one-hot in float64) no token is above the mean and T is
    every token."""
    import torch
    rng = np.random.default_rng(35)
    E = rng.standard_normal((3, 9, 12)) * 0.4
    r, mask, count = O.critical_text(E, lib=lib)
    for b in range(3):
        t = torch.from_numpy(E[b])
        want = torch.softmax(t @ t.T, dim=-1).mean(dim=0).numpy()
        assert np.max(np.abs(r[b] - want)) < 1e-15
        assert abs(r[b].sum() - 1.0) < 1e-14
        assert np.array_equal(mask[b], (want > want.mean()).astype(np.int32))
        assert count[b] == mask[b].sum() and 0 < count[b] < 9
    perm = rng.permutation(9)
    rp, mp, _ = O.critical_text(E[:, perm], lib=lib)
    assert np.max(np.abs(rp - r[:, perm])) < 1e-15 and np.array_equal(mp, mask[:, perm])
    Q = _rot(8, rng) * 100.0            # 8 orthogonal rows, squared norm 1e4
    r2, m2, c2 = O.critical_text(Q[None], lib=lib)
    assert np.all(r2 == 0.125)
    assert c2[0] == 8 and np.all(m2 == 1)


# ------------------------------------------------------------------ Eq. M --

def pin_cosine_known_angles(lib):
    """Sec. 4.3, equation for M.  Anchors and visual tokens lie in a rotated
    plane at known angles with arbitrary positive lengths, so
    M[i][j] = cos(alpha_i - beta_j) exactly."""
    rng = np.random.default_rng(11)
    d, nt, nv = 24, 5, 9
    R = _rot(d, rng)
    e1, e2 = R[0], R[1]
    alpha = rng.uniform(-math.pi, math.pi, nt)
    beta = rng.uniform(-math.pi, math.pi, nv)
    ra = rng.uniform(0.1, 20.0, nt)
    rb = rng.uniform(0.1, 20.0, nv)
    A = (ra[:, None] * (np.cos(alpha)[:, None] * e1 + np.sin(alpha)[:, None] * e2))
    V = (rb[:, None] * (np.cos(beta)[:, None] * e1 + np.sin(beta)[:, None] * e2))
    M = O.cosine(A, V, lib=lib)
    want = np.cos(alpha[:, None] - beta[None, :])
    assert M.shape == (nt, nv)
    assert np.max(np.abs(M - want)) < 1e-12


def pin_cosine_zero_rule_and_bounds(lib):
    """Zero vectors give 0 (reading of the equation for M); |M| <= 1; M is
    unchanged by positive row scaling and flips sign with the visual token."""
    rng = np.random.default_rng(12)
    A = rng.standard_normal((4, 16))
    V = rng.standard_normal((7, 16))
    A[2] = 0.0
    V[5] = 0.0
    M = O.cosine(A, V, lib=lib)
    assert np.all(M[2] == 0.0) and np.all(M[:, 5] == 0.0)
    assert np.all(np.abs(M) <= 1.0 + 1e-15)
    M2 = O.cosine(A * rng.uniform(0.5, 3.0, (4, 1)), V * rng.uniform(0.01, 9.0, (7, 1)), lib=lib)
    assert np.max(np.abs(M2 - M)) < 1e-13
    M3 = O.cosine(A, -V, lib=lib)
    assert np.max(np.abs(M3 + M)) < 1e-15
    # parallel vectors have cosine 1
    M4 = O.cosine(V[:1] * 3.0, V[:1] * 0.25, lib=lib)
    assert abs(M4[0, 0] - 1.0) < 1e-14


# -------------------------------------------------------------- Eq. M-hat --

def pin_center_worked_example(lib):
    g = GOLDEN["center"]
    out = O.center(np.array(g["M"]), lib=lib)
    assert np.array_equal(out, np.array(g["Mhat"]))


def pin_center_row_properties(lib):
    """Each row of M-hat sums to zero and differs from M by a per-row
    constant (together these fix M-hat = M - row mean)."""
    rng = np.random.default_rng(13)
    M = rng.uniform(-1, 1, (6, 11))
    Mh = O.center(M, lib=lib)
    assert np.max(np.abs(Mh.sum(axis=1))) < 1e-13
    diff = M - Mh
    assert np.max(np.abs(diff - diff[:, :1])) < 1e-14


# ------------------------------------------------------------------ Eq. p --

def pin_maxpool_worked_example(lib):
    g = GOLDEN["maxpool"]
    p = O.maxpool(np.array(g["Mhat"]), lib=lib)
    assert np.array_equal(p, np.array(g["p"]))


def pin_maxpool_properties(lib):
    rng = np.random.default_rng(14)
    Mh = rng.standard_normal((7, 13))
    p = O.maxpool(Mh, lib=lib)
    assert p.shape == (13,)
    assert np.all(p[None, :] >= Mh)
    assert all(p[j] in Mh[:, j] for j in range(13))


# ---------------------------------------------------------------- top-k ----

def _brute_topk(score, k):
    """Enumerate every size-k subset; keep the largest score sum, breaking
    ties by the lexicographically smallest index tuple.  Integer scores keep
    the sums exact."""
    best, best_sum = None, None
    for comb in itertools.combinations(range(len(score)), k):
        s = sum(score[c] for c in comb)
        if best is None or s > best_sum or (s == best_sum and comb < best):
            best, best_sum = comb, s
    return np.array(best, np.int32)


def pin_topk_bruteforce(lib):
    rng = np.random.default_rng(15)
    for trial in range(60):
        n = int(rng.integers(1, 11))
        k = int(rng.integers(1, n + 1))
        score = rng.integers(-3, 4, n).astype(np.float64)  # many ties
        got = O.topk(score, k, lib=lib)
        assert np.array_equal(got, _brute_topk(list(score), k)), (score, k, got)


def pin_topk_library_and_edges(lib):
    """Stable argsort of -score (numpy) is the same total order; k = n is the
    identity; +0 and -0 tie; output strictly increasing with exactly k."""
    rng = np.random.default_rng(16)
    for _ in range(20):
        n = int(rng.integers(1, 300))
        k = int(rng.integers(1, n + 1))
        score = np.round(rng.standard_normal(n), 1)
        got = O.topk(score, k, lib=lib)
        want = np.sort(np.argsort(-score, kind="stable")[:k])
        assert np.array_equal(got, want)
        assert got.shape == (k,) and np.all(np.diff(got) > 0)
    s = rng.standard_normal(17)
    assert np.array_equal(O.topk(s, 17, lib=lib), np.arange(17))
    z = np.array([1.0, -0.0, 0.0, -0.0, -1.0])
    assert np.array_equal(O.topk(z, 2, lib=lib), [0, 1])
    assert np.array_equal(O.topk(z, 3, lib=lib), [0, 1, 2])


# ----------------------------------------------------- nearest centroid ----

def pin_assign_constructed(lib):
    """Sec. 4.3, last paragraph.  Each pruned token is a positive multiple of
    one centroid plus a small perturbation, so its nearest centroid is known
    by construction.  Decoy centroids with 100x the norm and a moderate
    cosine (0.5) would win under an unnormalised dot product."""
    rng = np.random.default_rng(17)
    d, n1 = 64, 6
    R = _rot(d, rng)
    cents = R[:n1] * rng.uniform(0.5, 2.0, (n1, 1))
    nv = 40
    vis = np.zeros((nv, d))
    kept = np.sort(rng.choice(nv, n1, replace=False)).astype(np.int32)
    for s, j in enumerate(kept):
        vis[j] = cents[s]
    # make the last two centroids huge decoys
    vis[kept[-1]] = 100.0 * R[n1 + 0]
    vis[kept[-2]] = 100.0 * R[n1 + 1]
    want = {}
    for j in range(nv):
        if j in kept:
            continue
        s = int(rng.integers(0, n1 - 2))
        u = R[s] * rng.uniform(0.1, 5.0)
        # a component towards a decoy: cosine to the decoy ~0.5, to its own ~0.85
        u = u + 0.55 * np.linalg.norm(u) * R[n1 + 0] + 0.01 * rng.standard_normal(d)
        vis[j] = u
        want[j] = s
    a, b1, b2 = O.assign(vis, kept, lib=lib)
    for j, s in want.items():
        assert a[j] == s, (j, a[j], s)
        assert b1[j] > b2[j]
    for s, j in enumerate(kept):
        assert a[j] == s


def pin_assign_twins_and_ties(lib):
    """An exact copy of a kept token has cosine 1 to it (the maximum);
    two identical centroids tie and the lower slot wins."""
    rng = np.random.default_rng(18)
    d = 32
    vis = rng.standard_normal((8, d))
    vis[6] = vis[2]          # twin of kept token 2
    vis[4] = vis[1]          # kept tokens 1 and 4 are identical centroids
    vis[7] = vis[1] * 2.0    # parallel to both -> tie -> lower slot (token 1)
    kept = np.array([1, 2, 4, 5], np.int32)
    a, b1, _ = O.assign(vis, kept, lib=lib)
    assert a[6] == 1 and abs(b1[6] - 1.0) < 1e-14
    assert a[7] == 0
    assert list(a[kept]) == [0, 1, 2, 3]


def pin_assign_subset_rows(lib):
    rng = np.random.default_rng(19)
    vis = rng.standard_normal((30, 16))
    kept = np.array([0, 3, 9, 20, 29], np.int32)
    full, f1, f2 = O.assign(vis, kept, lib=lib)
    rows = np.array([28, 1, 7, 3], np.int32)
    sub, s1, s2 = O.assign(vis, kept, rows, lib=lib)
    assert np.array_equal(sub, full[rows])
    assert np.array_equal(s1, f1[rows]) and np.array_equal(s2, f2[rows])


# ----------------------------------------------------------------- merge ---

def pin_merge_reading(lib):
    """Pinned only to the reading (unweighted mean of centroid and members);
    a centroid with no members is unchanged bit for bit."""
    g = GOLDEN["merge"]
    out = O.merge(np.array(g["vis"]), np.array(g["kept"]), np.array(g["assign"]), lib=lib)
    assert np.array_equal(out, np.array(g["merged"]))
    rng = np.random.default_rng(20)
    vis = rng.standard_normal((9, 12))
    vis[5] = vis[1]
    kept = np.array([1, 3, 7], np.int32)
    asg = np.array([0, 0, 0, 1, 1, 0, 2, 2, 2], np.int32)   # 1 absorbs its twin 5 and 0, 2
    out = O.merge(vis, kept, asg, lib=lib)
    assert np.array_equal(out[2], (vis[7] + vis[6] + vis[8]) / 3.0)
    asg2 = np.array([1, 0, 1, 1, 1, 0, 1, 2, 1], np.int32)
    out2 = O.merge(vis, kept, asg2, lib=lib)
    assert np.array_equal(out2[2], vis[7])                  # no members: unchanged
    assert np.array_equal(out2[0], vis[1])                  # absorbing an exact twin


# ------------------------------------------------------- softmax / Eq. v ---

def pin_attention_two_keys(lib):
    g = GOLDEN["two_key_softmax"]
    A = O.attention(np.array(g["q"]), np.array(g["k"]), lib=lib)
    e = math.e
    assert abs(A[0, 0] - e / (1 + e)) < 1e-15 and abs(A[0, 1] - 1 / (1 + e)) < 1e-15


def pin_attention_invariants(lib):
    """Rows sum to 1; adding one vector to every key shifts each row's
    logits by a constant and leaves the row unchanged; Q = 0 is uniform."""
    rng = np.random.default_rng(21)
    q = rng.standard_normal((5, 16)) * 2
    k = rng.standard_normal((23, 16)) * 2
    A = O.attention(q, k, lib=lib)
    assert np.max(np.abs(A.sum(1) - 1.0)) < 1e-14 and np.all(A > 0)
    w = rng.standard_normal(16) * 3
    A2 = O.attention(q, k + w[None, :], lib=lib)
    assert np.max(np.abs(A2 - A)) < 1e-12
    U = O.attention(np.zeros((3, 16)), k, lib=lib)
    assert np.max(np.abs(U - 1.0 / 23)) < 1e-16


def pin_attention_library(lib):
    """Special case reducing to a library routine: torch.softmax in float64
    on the CPU over q k^T / sqrt(hd)."""
    import torch
    rng = np.random.default_rng(22)
    q = rng.standard_normal((7, 32))
    k = rng.standard_normal((19, 32))
    want = torch.softmax(torch.from_numpy(q) @ torch.from_numpy(k).T / math.sqrt(32), dim=-1).numpy()
    A = O.attention(q, k, lib=lib)
    assert np.max(np.abs(A - want)) < 1e-14


def _torch_all_head_mean(q, k):
    """FastV-style importance: attention averaged over every head and every
    text row, computed independently with torch (float64, CPU)."""
    import torch
    Q = torch.from_numpy(q)
    K = torch.from_numpy(k)
    A = torch.softmax(Q @ K.transpose(1, 2).contiguous() / math.sqrt(q.shape[-1]), dim=-1)
    return A.mean(dim=(0, 1)).numpy()


def pin_head_aware_all_heads_baseline(lib):
    """Sec. 4.4: with V = every head the head-aware score is the all-head
    aggregation of attention-based pruning (the paper's 'All Attention
    Heads' configuration)."""
    rng = np.random.default_rng(23)
    H, nt, n, hd = 6, 9, 31, 16
    q = rng.standard_normal((H, nt, hd)) * 1.5
    k = rng.standard_normal((H, n, hd)) * 1.5
    v = O.head_aware_score(q, k, list(range(H)), lib=lib)
    assert np.max(np.abs(v - _torch_all_head_mean(q, k))) < 1e-15


def pin_head_aware_subset(lib):
    """Only the listed heads are read; one head gives that head's column
    mean; the order of the list does not matter; v sums to 1; permuting
    the keys permutes v."""
    import torch
    rng = np.random.default_rng(24)
    H, nt, n, hd = 5, 6, 17, 8
    q = rng.standard_normal((H, nt, hd)) * 2
    k = rng.standard_normal((H, n, hd)) * 2
    v = O.head_aware_score(q, k, [3, 1], lib=lib)
    assert abs(v.sum() - 1.0) < 1e-14
    k2 = k.copy()
    k2[0] = rng.standard_normal((n, hd))
    k2[4] = 0.0
    assert np.array_equal(O.head_aware_score(q, k2, [3, 1], lib=lib), v)
    assert np.max(np.abs(O.head_aware_score(q, k, [1, 3], lib=lib) - v)) < 1e-16
    one = O.head_aware_score(q, k, [2], lib=lib)
    A2 = torch.softmax(torch.from_numpy(q[2]) @ torch.from_numpy(k[2]).T / math.sqrt(hd), -1)
    assert np.max(np.abs(one - A2.mean(0).numpy())) < 1e-15
    two = _torch_all_head_mean(q[[1, 3]], k[[1, 3]])
    assert np.max(np.abs(v - two)) < 1e-15
    perm = rng.permutation(n)
    vp = O.head_aware_score(q, k[:, perm], [3, 1], lib=lib)
    assert np.max(np.abs(vp - v[perm])) < 1e-15


def pin_head_aware_topk(lib):
    rng = np.random.default_rng(25)
    B, H, nt, n, hd = 2, 4, 5, 12, 8
    q = rng.standard_normal((B, H, nt, hd))
    k = rng.standard_normal((B, H, n, hd))
    heads = np.array([[0, 2], [3, 1]], np.int32)
    kept, v = O.head_aware(q, k, heads, 5, lib=lib)
    for b in range(B):
        assert np.array_equal(kept[b], np.sort(np.argsort(-v[b], kind="stable")[:5]))


# ----------------------------------------- in-model softmax domain --------

def pin_in_model_is_the_visual_slice(lib):
    """The in-model map is the visual slice of one softmax over explicit
    non-visual keys and the visual keys (torch, float64): the non-visual keys
    enter only through the log-sum-exp of their scaled logits."""
    import torch
    rng = np.random.default_rng(36)
    nt, n, n_other, hd = 6, 11, 7, 16
    q = rng.standard_normal((nt, hd)) * 2
    k = rng.standard_normal((n, hd)) * 2
    k_other = rng.standard_normal((n_other, hd)) * 2
    Q, K, Ko = (torch.from_numpy(x) for x in (q, k, k_other))
    full = torch.softmax(torch.cat([Q @ Ko.T, Q @ K.T], dim=1) / math.sqrt(hd), dim=-1)
    want = full[:, n_other:].numpy()
    lse = torch.logsumexp(Q @ Ko.T / math.sqrt(hd), dim=1).numpy()
    A = O.attention_in_model(q, k, lse, lib=lib)
    assert np.max(np.abs(A - want)) < 1e-15
    # every row's visual mass is below 1 by the other keys' share
    assert np.all(A.sum(1) < 1.0)
    assert np.max(np.abs(A.sum(1) - want.sum(1))) < 1e-15


def pin_in_model_closed_forms(lib):
    """lse = -inf is the plain map; one visual key with scaled logit s and
    lse = t gives the logistic s(s - t); adding c to every logit and to lse
    leaves A unchanged."""
    rng = np.random.default_rng(37)
    q = rng.standard_normal((4, 8)) * 2
    k = rng.standard_normal((9, 8)) * 2
    A0 = O.attention_in_model(q, k, np.full(4, -np.inf), lib=lib)
    assert np.array_equal(A0, O.attention(q, k, lib=lib))
    hd = 4
    ts = np.array([-1.5, 0.0, 2.25])
    qq = np.zeros((3, hd))
    qq[:, 0] = math.sqrt(hd)            # scaled logit of the key = 0.7
    kk = np.zeros((1, hd))
    kk[0, 0] = 0.7
    A1 = O.attention_in_model(qq, kk, ts, lib=lib)
    want = 1.0 / (1.0 + np.exp(-(0.7 - ts)))
    assert np.max(np.abs(A1[:, 0] - want)) < 1e-15
    lse = rng.standard_normal(4)
    w = rng.standard_normal(8)
    A2 = O.attention_in_model(q, k, lse, lib=lib)
    # a key shift by w adds q.w / sqrt(hd) to every visual logit of a row
    shift = q @ w / math.sqrt(8)
    A3 = O.attention_in_model(q, k + w[None, :], lse + shift, lib=lib)
    assert np.max(np.abs(A3 - A2)) < 1e-13


def pin_head_aware_in_model(lib):
    """v on the in-model map: heads outside the list are never read, and the
    plain head-aware score is the case lse = -inf."""
    rng = np.random.default_rng(38)
    B, H, nt, n, hd = 2, 4, 5, 12, 8
    q = rng.standard_normal((B, H, nt, hd))
    k = rng.standard_normal((B, H, n, hd))
    heads = np.array([[0, 2], [3, 1]], np.int32)
    lse = rng.standard_normal((B, H, nt)) + 1.0
    kept, v = O.head_aware_in_model(q, k, heads, lse, 4, lib=lib)
    k2 = k.copy()
    k2[0, 1] = 0.0
    k2[1, 0] = 5.0
    lse2 = lse.copy()
    lse2[0, 3] = 9.0
    kept2, v2 = O.head_aware_in_model(q, k2, heads, lse2, 4, lib=lib)
    assert np.array_equal(v, v2) and np.array_equal(kept, kept2)
    for b in range(B):
        A = [O.attention_in_model(q[b, h], k[b, h], lse[b, h], lib=lib) for h in heads[b]]
        want = np.mean([a.mean(0) for a in A], axis=0)
        assert np.max(np.abs(v[b] - want)) < 1e-15
    _, vp = O.head_aware_in_model(q, k, heads, np.full((B, H, nt), -np.inf), 4, lib=lib)
    _, vplain = O.head_aware(q, k, heads, 4, lib=lib)
    assert np.array_equal(vp, vplain)


# ------------------------------------------------------- Eq. C^h, V_l ------

def pin_confidence_closed_forms(lib):
    """Sec. 4.4, equation for C^h, on rows whose variance is known exactly:
    Q = 0 gives uniform rows (variance 0); two keys with logits 0 and t give
    the row (1 - s, s) with s the logistic of t, whose population variance
    is (s - 1/2)^2; a dominant key (one-hot row) gives (n - 1) / n^2."""
    hd = 4
    # head 0: Q = 0 over 7 keys; head 1: two keys, logit difference per row
    q = np.zeros((2, 3, hd))
    k = np.zeros((2, 7, hd))
    k[0] = np.random.default_rng(31).standard_normal((7, hd))
    ts = np.array([0.5, -1.25, 2.0])
    q[1, :, 0] = ts * math.sqrt(hd)   # logit of key 1 minus key 0 = t
    k[1, 1, 0] = 1.0
    c2 = O.head_confidence(q, k[:, :7], lib=lib)
    assert abs(c2[0]) < 1e-30
    # head 1 has only two meaningful keys: redo with n = 2
    q2 = q[1:2]
    k2 = k[1:2, :2]
    c = O.head_confidence(q2, k2, lib=lib)
    want = sum((1.0 / (1.0 + math.exp(-t)) - 0.5) ** 2 for t in ts)
    assert abs(c[0] - want) < 1e-15
    # one dominant key per row: logits differ by 800 -> exactly one-hot in fp64
    n = 9
    q3 = np.zeros((1, 4, hd))
    k3 = np.zeros((1, n, hd))
    q3[0, :, 0] = 800.0 * math.sqrt(hd)
    k3[0, 5, 0] = 1.0
    c3 = O.head_confidence(q3, k3, lib=lib)
    assert abs(c3[0] - 4 * (n - 1) / n ** 2) < 1e-15


def pin_confidence_library(lib):
    """Special case reducing to library routines: numpy's population
    variance (np.var) of torch.softmax rows in float64, summed per head."""
    import torch
    rng = np.random.default_rng(32)
    H, nt, n, hd = 5, 6, 21, 16
    q = rng.standard_normal((H, nt, hd)) * 2
    k = rng.standard_normal((H, n, hd)) * 2
    A = torch.softmax(torch.from_numpy(q) @ torch.from_numpy(k).transpose(1, 2).contiguous()
                      / math.sqrt(hd), dim=-1).numpy()
    want = np.var(A, axis=2).sum(axis=1)
    c = O.head_confidence(q, k, lib=lib)
    assert np.max(np.abs(c - want)) < 1e-15 * max(1.0, want.max())


def pin_confidence_invariants(lib):
    """The confidence does not depend on the order of the keys or of the
    text rows; heads are independent (permuting heads permutes C); adding
    one vector to every key of a head leaves its C unchanged."""
    rng = np.random.default_rng(33)
    H, nt, n, hd = 4, 5, 13, 8
    q = rng.standard_normal((H, nt, hd)) * 2
    k = rng.standard_normal((H, n, hd)) * 2
    c = O.head_confidence(q, k, lib=lib)
    assert np.all(c > 0)
    ck = O.head_confidence(q, k[:, rng.permutation(n)], lib=lib)
    cq = O.head_confidence(q[:, rng.permutation(nt)], k, lib=lib)
    perm = rng.permutation(H)
    ch = O.head_confidence(q[perm], k[perm], lib=lib)
    w = rng.standard_normal(hd) * 3
    cs = O.head_confidence(q, k + w[None, None, :], lib=lib)
    assert np.max(np.abs(ck - c)) < 1e-15 and np.max(np.abs(cq - c)) < 1e-15
    assert np.array_equal(ch, c[perm])
    assert np.max(np.abs(cs - c)) < 1e-13


def pin_visual_heads_topk(lib):
    """Sec. 4.4, equation for V_l: the N_vis heads of largest C, ascending;
    the same total order as the token top-k (numpy stable argsort); N_vis = H
    keeps every head.  A head whose queries are zero (uniform attention,
    C = 0) is never chosen while another head has C > 0."""
    rng = np.random.default_rng(34)
    B, H, nt, n, hd = 3, 8, 5, 11, 8
    q = rng.standard_normal((B, H, nt, hd)) * 2
    k = rng.standard_normal((B, H, n, hd)) * 2
    q[:, 6] = 0.0
    for nv in (1, 3, H - 1, H):
        heads, conf = O.visual_heads(q, k, nv, lib=lib)
        for b in range(B):
            assert np.array_equal(heads[b], np.sort(np.argsort(-conf[b], kind="stable")[:nv]))
            assert abs(conf[b, 6]) < 1e-30
            if nv < H:
                assert 6 not in heads[b]
        if nv == H:
            assert np.array_equal(heads, np.tile(np.arange(H), (B, 1)))


# ------------------------------- Eq. C^h on the model's softmax domain -----

def _slice_logits(q, k, ko, hd):
    import torch
    Q, K, Ko = (torch.from_numpy(x) for x in (q, k, ko))
    lo = torch.matmul(Q, Ko.transpose(-1, -2).contiguous()) / math.sqrt(hd)
    lv = torch.matmul(Q, K.transpose(-1, -2).contiguous()) / math.sqrt(hd)
    return lo, lv


def pin_confidence_in_model_visual_slice(lib):
    """Sec. 4.4, equation for C^h on A^cross as the model has it: numpy's
    population variance (np.var) of the visual slice of one torch softmax
    (float64) over explicit non-visual keys and the visual keys, summed over
    the rows.  The other keys enter only through their log-sum-exp, and
    their share of each row changes C."""
    import torch
    rng = np.random.default_rng(41)
    H, nt, n, n_other, hd = 4, 6, 13, 9, 16
    q = rng.standard_normal((H, nt, hd)) * 2
    k = rng.standard_normal((H, n, hd)) * 2
    ko = rng.standard_normal((H, n_other, hd)) * 2
    lo, lv = _slice_logits(q, k, ko, hd)
    full = torch.softmax(torch.cat([lo, lv], dim=-1), dim=-1).numpy()
    want = np.var(full[..., n_other:], axis=2).sum(axis=1)
    lse = torch.logsumexp(lo, dim=-1).numpy()
    c = O.head_confidence_in_model(q, k, lse, lib=lib)
    assert np.max(np.abs(c - want)) < 1e-15 * max(1.0, want.max())
    c_plain = O.head_confidence(q, k, lib=lib)
    assert np.max(np.abs(c - c_plain)) > 1e-3 * c_plain.max()


def pin_confidence_in_model_closed_forms(lib):
    """lse = -inf everywhere is the plain confidence, bit for bit; two
    visual keys with scaled logits 0 and b and lse = t give the slice
    (1, e^b) / (1 + e^b + e^t), whose population variance is
    ((A_1 - A_2) / 2)^2; permuting the visual keys leaves C unchanged."""
    rng = np.random.default_rng(42)
    H, nt, n, hd = 3, 5, 11, 8
    q = rng.standard_normal((H, nt, hd)) * 2
    k = rng.standard_normal((H, n, hd)) * 2
    c0 = O.head_confidence_in_model(q, k, np.full((H, nt), -np.inf), lib=lib)
    assert np.array_equal(c0, O.head_confidence(q, k, lib=lib))
    lse = rng.standard_normal((H, nt))
    c1 = O.head_confidence_in_model(q, k, lse, lib=lib)
    cp = O.head_confidence_in_model(q, k[:, rng.permutation(n)], lse, lib=lib)
    assert np.max(np.abs(cp - c1)) < 1e-15
    hd2 = 4
    bs = np.array([0.5, -1.0, 2.0, 0.0])
    ts = np.array([1.0, -0.5, 3.0, -2.0])
    q2 = np.zeros((1, 4, hd2))
    q2[0, :, 0] = bs * math.sqrt(hd2)   # key 1's scaled logit is b; key 0's is 0
    k2 = np.zeros((1, 2, hd2))
    k2[0, 1, 0] = 1.0
    c2 = O.head_confidence_in_model(q2, k2, ts[None], lib=lib)
    den = 1.0 + np.exp(bs) + np.exp(ts)
    want = np.sum(((1.0 - np.exp(bs)) / den / 2.0) ** 2)
    assert abs(c2[0] - want) < 1e-16


def pin_visual_heads_in_model_topk(lib):
    """Sec. 4.4, equation for V_l on the in-model confidence: the N_vis heads
    of largest C (numpy stable argsort order), ascending; with lse = -inf the
    plain visual heads."""
    rng = np.random.default_rng(43)
    B, H, nt, n, hd = 2, 7, 4, 9, 8
    q = rng.standard_normal((B, H, nt, hd)) * 2
    k = rng.standard_normal((B, H, n, hd)) * 2
    lse = rng.standard_normal((B, H, nt)) + 1.5
    for nv in (1, 3, H):
        heads, conf = O.visual_heads_in_model(q, k, lse, nv, lib=lib)
        for b in range(B):
            assert np.array_equal(heads[b], np.sort(np.argsort(-conf[b], kind="stable")[:nv]))
            assert np.array_equal(conf[b], O.head_confidence_in_model(q[b], k[b], lse[b], lib=lib))
    hp, cp = O.visual_heads_in_model(q, k, np.full((B, H, nt), -np.inf), 3, lib=lib)
    hv, cv = O.visual_heads(q, k, 3, lib=lib)
    assert np.array_equal(hp, hv) and np.array_equal(cp, cv)


# ---------------------------------------------------------------- gather ---

def pin_gather_bytes(lib):
    rng = np.random.default_rng(26)
    src = rng.integers(0, 255, (3, 4, 11, 16), dtype=np.uint8)
    idx = np.stack([np.sort(rng.choice(11, 5, replace=False)) for _ in range(3)]).astype(np.int32)
    out = O.gather(src, idx, lib=lib)
    want = np.stack([src[b][:, idx[b]] for b in range(3)])
    assert np.array_equal(out, want)
    h = rng.standard_normal((2, 9, 6)).astype(np.float32)
    idx2 = np.array([[0, 4, 8], [1, 2, 3]], np.int32)
    assert np.array_equal(O.gather(h, idx2, lib=lib), np.stack([h[0][[0, 4, 8]], h[1][[1, 2, 3]]]))


# ------------------------------------------------------- stage A end to end

def pin_dedup_axes(lib):
    g = GOLDEN["dedup_axes"]
    A = np.array(g["anchors"])[None]
    V = np.array(g["vis"])[None]
    r = 1.0 / math.sqrt(2.0)
    want_p = np.array([1 - (1 + r) / 5, 0.8, -0.2, -0.2, r - (1 + r) / 5])
    for n1, key in ((2, "kept_top2"), (3, "kept_top3"), (4, "kept_top4")):
        res = O.dedup(A, V, n1, lib=lib)
        assert np.max(np.abs(res["p"][0] - want_p)) < 1e-15
        assert np.array_equal(res["kept"][0], g[key])


def pin_dedup_twins(lib):
    """Exact twins get bit-identical p; if the higher twin is kept the lower
    one is too; a pruned twin whose twin is kept is absorbed by it."""
    rng = np.random.default_rng(27)
    B, nv, d, nt = 1, 40, 24, 6
    vis = rng.standard_normal((B, nv, d))
    pairs = [(2, 30), (5, 6), (11, 39), (17, 18)]
    for a, b in pairs:
        vis[0, b] = vis[0, a]
    anchors = rng.standard_normal((B, nt, d))
    res = O.dedup(anchors, vis, 20, lib=lib)
    kept = set(res["kept"][0].tolist())
    for a, b in pairs:
        assert res["p"][0, a] == res["p"][0, b]
        if b in kept:
            assert a in kept
        if a in kept and b not in kept:
            slot = list(res["kept"][0]).index(a)
            assert res["assign"][0, b] == slot
    assert len(kept) == 20 and np.all(np.diff(res["kept"][0]) > 0)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_") and callable(v)]
