"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: published
test vectors, closed forms, brute force on tiny inputs, invariants stated in
the paper, or independent library routines (torch CPU attention, eigh).
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import park_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed=0):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- init -----
def test_splitmix64_published_vectors():
    with open(os.path.join(GOLDEN, "splitmix64.txt")) as f:
        rows = [l.split() for l in f if l.strip() and not l.startswith("#")]
    assert rows
    for row in rows:
        seed, expect = int(row[0]), [int(x) for x in row[1:]]
        g = O.SplitMix64(seed)
        assert [g.next() for _ in expect] == expect


def test_init_indices_distinct_prefix_and_permutation():
    N = 1000
    a = O.init_indices(N, 37, seed=5, head=3, side=1)
    assert len(set(a.tolist())) == 37 and a.min() >= 0 and a.max() < N
    # Fisher-Yates: a shorter draw is a prefix of a longer one
    b = O.init_indices(N, 200, seed=5, head=3, side=1)
    assert np.array_equal(a, b[:37])
    full = O.init_indices(N, N, seed=5, head=3, side=1)
    assert sorted(full.tolist()) == list(range(N))
    # heads and sides draw different streams
    assert not np.array_equal(a, O.init_indices(N, 37, 5, 3, 0))
    assert not np.array_equal(a, O.init_indices(N, 37, 5, 4, 1))


def test_init_indices_uniform():
    # each token is picked with probability C/N (chi-square over many seeds)
    N, C, S = 20, 5, 4000
    cnt = np.zeros(N)
    for s in range(S):
        cnt[O.init_indices(N, C, seed=s, head=0, side=0)] += 1
    exp = S * C / N
    chi2 = ((cnt - exp) ** 2 / exp).sum()
    assert chi2 < 45.0  # 19 dof, p ~ 1e-3
    # first pick is uniform too
    first = np.bincount([O.init_indices(N, 1, s, 0, 0)[0] for s in range(S)], minlength=N)
    chi2 = ((first - S / N) ** 2 / (S / N)).sum()
    assert chi2 < 45.0


# ------------------------------------------------------ query metric ------
def test_metric_closed_form_diagonal():
    # rows are scaled basis vectors: G is diagonal with known entries
    d, L = 4, 8
    Q = np.zeros((L, d))
    sig = np.array([1.0, 2.0, 3.0, 4.0])
    for i in range(L):
        Q[i, i % d] = sig[i % d]
    m = O.query_metric(Q, alpha=0.05, eps=1e-6)
    G = np.diag(sig ** 2 * 2 / L)
    assert np.allclose(m["G"], G, rtol=0, atol=1e-15)
    s = np.trace(G) / d
    assert m["s"] == pytest.approx(s, rel=1e-15)
    gbar = 0.95 * G + (0.05 + 1e-6) * s * np.eye(d)
    assert np.allclose(m["Gbar"], gbar, rtol=1e-14, atol=0)
    assert np.allclose(m["R"], np.sqrt(gbar), rtol=1e-14, atol=0)


def test_metric_factor_and_alpha_one():
    Q = rng(1).standard_normal((300, 16)) * np.linspace(0.1, 3, 16)
    m = O.query_metric(Q, alpha=0.05, eps=1e-6)
    R = m["R"]
    assert np.allclose(R, np.tril(R))
    assert np.all(np.diag(R) > 0)
    assert np.abs(R @ R.T - m["Gbar"]).max() <= 1e-12 * np.abs(m["Gbar"]).max()
    # G is PSD: x^T G x = |Q x|^2 / L
    x = rng(2).standard_normal(16)
    assert x @ m["G"] @ x == pytest.approx(np.sum((Q @ x) ** 2) / 300, rel=1e-12)
    # alpha = 1 gives an isotropic metric
    m1 = O.query_metric(Q, alpha=1.0, eps=1e-6)
    assert np.allclose(m1["R"], math.sqrt((1 + 1e-6) * m1["s"]) * np.eye(16), rtol=1e-13, atol=1e-15)


def test_metric_scale_floor_and_failure():
    Z = np.zeros((50, 8))
    m = O.query_metric(Z)
    assert m["s"] == 1e-12
    assert np.allclose(m["Gbar"], (0.05 + 1e-6) * 1e-12 * np.eye(8), rtol=1e-14, atol=0)
    # rank-deficient queries without shrinkage: Cholesky must fail
    Q = np.zeros((40, 8))
    Q[:, :3] = rng(3).standard_normal((40, 3))
    with pytest.raises(np.linalg.LinAlgError):
        O.query_metric(Q, alpha=0.0, eps=0.0)


def test_transformed_distance_equivalences():
    # |R^T delta|^2 = delta^T Gbar delta = |Gbar^(1/2) delta|^2; with alpha=eps=0
    # also = |Q delta|^2 / L (the direct L-dimensional map)
    L, d = 200, 12
    Q = rng(4).standard_normal((L, d)) @ rng(5).standard_normal((d, d))
    K = rng(6).standard_normal((30, d))
    m = O.query_metric(Q, alpha=0.0, eps=0.0)
    Kt = O.transform_keys(K, m["R"])
    w, U = np.linalg.eigh(m["Gbar"])
    S = U @ np.diag(np.sqrt(np.maximum(w, 0))) @ U.T
    for j in range(30):
        for c in range(0, 30, 7):
            delta = K[j] - K[c]
            a = np.sum((Kt[j] - Kt[c]) ** 2)
            b = delta @ m["Gbar"] @ delta
            e = np.sum((S @ delta) ** 2)
            f = np.sum((Q @ delta) ** 2) / L
            assert a == pytest.approx(b, rel=1e-11)
            assert a == pytest.approx(e, rel=1e-10)
            assert a == pytest.approx(f, rel=1e-10)


# ------------------------------------------------------------ k-means -----
def brute_assign(X, mu):
    z = []
    for x in X:
        best, bi = None, -1
        for v, m in enumerate(mu):
            dist = sum((xa - ma) ** 2 for xa, ma in zip(x, m))
            if best is None or dist < best:
                best, bi = dist, v
        z.append(bi)
    return np.array(z)


def brute_mean(X, z, mu):
    out = mu.copy()
    for v in range(len(mu)):
        rows = [X[j] for j in range(len(X)) if z[j] == v]
        if rows:
            out[v] = [sum(r[a] for r in rows) / len(rows) for a in range(X.shape[1])]
    return out


def test_assign_and_update_brute_force():
    X = rng(7).standard_normal((60, 5))
    mu = rng(8).standard_normal((7, 5))
    z = O.assign(X, mu)
    assert np.array_equal(z, brute_assign(X, mu))
    new = O.update(X, z, mu)
    assert np.allclose(new, brute_mean(X, z, mu), rtol=1e-14, atol=1e-15)


def test_assign_ties_lowest_id_and_empty_keeps_centroid():
    X = np.array([[0.0, 0.0], [2.0, 0.0], [10.0, 10.0]])
    mu = np.array([[1.0, 0.0], [1.0, 0.0], [-50.0, -50.0], [10.0, 10.0]])
    z = O.assign(X, mu)
    assert z.tolist() == [0, 0, 3]  # equal distances -> lowest id
    new = O.update(X, z, mu)
    assert np.array_equal(new[1], mu[1]) and np.array_equal(new[2], mu[2])
    assert np.array_equal(new[0], [1.0, 0.0])


def test_kmeans_objective_non_increasing():
    X = rng(9).standard_normal((400, 6)) + np.repeat(rng(10).standard_normal((8, 6)) * 3, 50, 0)
    init = O.init_indices(400, 10, 0, 0, 0)
    mu = X[init].copy()
    prev = np.inf
    for t in range(8):
        z = O.assign(X, mu)
        J = np.sum((X - mu[z]) ** 2)
        assert J <= prev + 1e-9
        prev = J
        mu = O.update(X, z, mu)


def test_kmeans_singletons_when_C_equals_N():
    X = rng(11).standard_normal((40, 4))
    init = O.init_indices(40, 40, 1, 0, 0)
    z, _ = O.kmeans(X, 40, 3, init)
    # every token seeds its own cluster and keeps it
    assert np.array_equal(init[z], np.arange(40))


def test_qrkc_alpha_one_equals_euclidean_kmeans():
    Q = rng(12).standard_normal((300, 8)) * np.linspace(0.2, 4, 8)
    K = rng(13).standard_normal((300, 8)) + np.repeat(rng(14).standard_normal((6, 8)) * 2, 50, 0)
    ck = O.cluster_keys(K, Q, C=12, T=6, seed=3, head=2, alpha=1.0)
    init = O.init_indices(300, 12, 3, 2, 1)
    z, _ = O.kmeans(K, 12, 6, init)
    assert np.array_equal(ck["labels"], z)


def test_qrkc_objective_identities():
    # Jbar = (1-a) J + (a+eps) s J_euc, and the G-form of J equals the
    # explicit average over queries of squared score errors.
    L, d = 80, 6
    Q = rng(15).standard_normal((L, d)) * np.array([0.3, 1, 2, 0.5, 1.5, 3])
    K = rng(16).standard_normal((L, d))
    z = rng(17).integers(0, 5, L)
    c = np.array([K[z == v].mean(0) for v in range(5)])
    a, eps = 0.05, 1e-6
    m = O.query_metric(Q, a, eps)
    delta = K - c[z]
    J = np.einsum("ja,ab,jb->", delta, m["G"], delta)
    J_explicit = sum((Q[i] @ delta[j]) ** 2 for i in range(L) for j in range(L)) / L
    assert J == pytest.approx(J_explicit, rel=1e-11)
    Jeuc = np.sum(delta ** 2)
    Kt = O.transform_keys(K, m["R"])
    ct = np.array([Kt[z == v].mean(0) for v in range(5)])
    Jbar = np.sum((Kt - ct[z]) ** 2)
    assert Jbar == pytest.approx((1 - a) * J + (a + eps) * m["s"] * Jeuc, rel=1e-11)
    # transformed centroids are the transforms of the centroids (linearity)
    assert np.allclose(ct, c @ m["R"], rtol=1e-12, atol=1e-13)


# -------------------------------------------------------- permutation -----
def test_stable_argsort_properties():
    z = rng(18).integers(0, 9, 500)
    z[z == 4] = 5  # force an empty cluster
    perm, off = O.stable_argsort(z, 9)
    assert sorted(perm.tolist()) == list(range(500))
    zs = z[perm]
    assert np.all(np.diff(zs) >= 0)
    for v in range(9):
        seg = perm[off[v]:off[v + 1]]
        assert np.all(z[seg] == v)
        assert np.all(np.diff(seg) > 0)  # stable: original order inside a block
    assert off[4] == off[5] and off[-1] == 500


def test_block_centroids_brute_force_and_zero_residual():
    K = rng(19).standard_normal((100, 8)).astype(np.float32).astype(np.float64)
    z = rng(20).integers(0, 6, 100)
    z[z == 2] = 3
    perm, off = O.stable_argsort(z, 6)
    c, n = O.block_centroids(K[perm], off)
    assert c.dtype == np.float32 and n.tolist() == np.bincount(z, minlength=6).tolist()
    assert np.all(c[2] == 0)
    for v in range(6):
        if n[v]:
            exact = K[z == v].sum(0) / n[v]
            assert np.array_equal(c[v], exact.astype(np.float32))
            # residuals about the (unrounded) centroid sum to zero
            assert np.abs((K[z == v] - exact).sum(0)).max() < 1e-12


# --------------------------------------------------------------- PAMA -----
def test_pama_hand_computed():
    # two queries, key blocks: block 0 has 1 key at (2,0), block 1 has 3
    # keys averaging (0,0), block 2 empty.  d = 2.
    Qp = np.array([[1.0, 0.0], [0.0, 1.0]])
    c = np.array([[2.0, 0.0], [0.0, 0.0], [9.0, 9.0]], dtype=np.float32)
    n = np.array([1, 3, 0])
    S = O.pama_scores(Qp, c, n)
    r2 = math.sqrt(2.0)
    assert S[0, 0] == pytest.approx(2 / r2, rel=1e-15)
    assert S[0, 1] == pytest.approx(math.log(3), rel=1e-15)
    assert S[1, 0] == pytest.approx(0.0, abs=1e-15)
    assert np.isneginf(S[:, 2]).all()
    p00 = math.exp(2 / r2) / (math.exp(2 / r2) + 3)
    p10 = 1 / (1 + 3)
    W = O.pama(Qp, np.array([0, 2]), c, n)
    assert W[0, 0] == pytest.approx((p00 + p10) / 2, rel=1e-14)
    assert W[0, 1] == pytest.approx(((1 - p00) + (1 - p10)) / 2, rel=1e-14)
    assert W[0, 2] == 0.0


def test_pama_rows_sum_to_one_and_jensen():
    Qp = rng(21).standard_normal((64, 16))
    Kp = rng(22).standard_normal((90, 16))
    koff = np.array([0, 10, 10, 35, 36, 90])
    c, n = O.block_centroids(Kp, koff)
    S = O.pama_scores(Qp, c, n)
    P = O.softmax_rows(S)
    assert np.allclose(P.sum(1), 1, atol=1e-14)
    W = O.pama(Qp, np.array([0, 20, 20, 64]), c, n)
    assert np.allclose(W[[0, 2]].sum(1), 1, atol=1e-14) and np.all(W[1] == 0)
    # key-centroid estimate is a lower bound of the exact log-mass (Jensen)
    Kp32 = Kp.copy()
    # compare with centroids that are exact means (use float64 means here)
    cexact = np.array([Kp[koff[v]:koff[v + 1]].mean(0) if n[v] else np.zeros(16)
                       for v in range(5)])
    Shat = (Qp @ cexact.T) / 4.0 + np.log(np.maximum(n, 1))
    Sstar = O.exact_log_mass(Qp, Kp32, koff)
    for v in range(5):
        if n[v]:
            assert np.all(Shat[:, v] <= Sstar[:, v] + 1e-12)


def test_pama_block_size_one_equals_attention():
    # singleton key and query blocks: W^ is exactly the dense attention
    # matrix (log 1 = 0, centroid = key), checked against torch's softmax.
    N, d = 48, 8
    Q = rng(23).standard_normal((N, d)).astype(np.float32).astype(np.float64)
    K = rng(24).standard_normal((N, d)).astype(np.float32).astype(np.float64)
    qp = rng(25).permutation(N)
    kp = rng(26).permutation(N)
    off = np.arange(N + 1)
    c, n = O.block_centroids(K[kp], off)
    W = O.pama(Q[qp], off, c, n)
    A = torch.softmax(torch.from_numpy(Q) @ torch.from_numpy(K).T / math.sqrt(d), dim=1).numpy()
    assert np.abs(W - A[np.ix_(qp, kp)]).max() < 1e-14


def test_pama_identical_keys_equals_exact_importance():
    # when every key of a block equals its centroid, S^ = S* exactly and
    # PAMA equals the exact block importance of Eq. (3) (pins log n_v and the
    # softmax-then-average order).
    d = 8
    base = rng(27).standard_normal((5, d)).astype(np.float32).astype(np.float64)
    sizes = [3, 1, 7, 2, 5]
    Kp = np.concatenate([np.repeat(base[v:v + 1], s, 0) for v, s in enumerate(sizes)])
    koff = np.concatenate([[0], np.cumsum(sizes)])
    Qp = rng(28).standard_normal((30, d)) * 2
    qoff = np.array([0, 4, 4, 17, 30])
    c, n = O.block_centroids(Kp, koff)
    W = O.pama(Qp, qoff, c, n)
    Wex = O.exact_block_importance(Qp, Kp, qoff, koff)
    assert np.abs(W - Wex).max() < 1e-13


def test_pama_identical_queries_equals_centroid_estimate():
    d = 6
    Kp = rng(29).standard_normal((40, d))
    koff = np.array([0, 5, 19, 40])
    c, n = O.block_centroids(Kp, koff)
    q = rng(30).standard_normal(d)
    Qp = np.repeat(q[None], 9, 0)
    W = O.pama(Qp, np.array([0, 9]), c, n)
    S = (c.astype(np.float64) @ q) / math.sqrt(d) + np.log(n)
    e = np.exp(S - S.max())
    assert np.allclose(W[0], e / e.sum(), rtol=1e-14, atol=0)


# ---------------------------------------------------------- selection -----
def brute_select(w, valid, mode, param):
    items = sorted([(-w[v], v) for v in range(len(w)) if valid[v]])
    if mode == "topk":
        k = max(1, min(math.ceil(param * len(w) - 1e-9), len(items)))
        return sorted(v for _, v in items[:k])
    tot = 0.0
    out = []
    for negw, v in items:
        out.append(v)
        tot += -negw
        if tot >= param:
            break
    return sorted(out)


def test_select_brute_force():
    r = rng(31)
    for trial in range(200):
        C = int(r.integers(1, 40))
        w = r.random(C) ** 4
        w[r.random(C) < 0.2] = 0.0
        if trial % 5 == 0:
            w = np.round(w * 4) / 4  # many ties
        valid = r.random(C) < 0.85
        if not valid.any():
            valid[0] = True
        w = np.where(valid, w, 0.0)
        w = w / w.sum() if w.sum() > 0 else w
        for mode, param in (("topk", r.random()), ("topp", r.random())):
            got, _, _ = O.select_row(w, valid, mode, param)
            assert got.tolist() == brute_select(w, valid, mode, param)


def test_select_extremes_and_monotone():
    r = rng(32)
    w = r.random(50) ** 3
    w /= w.sum()
    valid = np.ones(50, bool)
    valid[[3, 9]] = False
    w[[3, 9]] = 0
    allv = np.nonzero(valid)[0].tolist()
    assert O.select_row(w, valid, "topk", 1.0)[0].tolist() == allv
    assert O.select_row(w, valid, "topp", 1.0)[0].tolist() == allv
    prev = set()
    for p in np.linspace(0.05, 1.0, 20):
        cur = set(O.select_row(w, valid, "topp", p)[0].tolist())
        assert prev <= cur
        prev = cur
    prev = set()
    for rho in np.linspace(0.02, 1.0, 20):
        cur = set(O.select_row(w, valid, "topk", rho)[0].tolist())
        assert prev <= cur
        prev = cur
    # top-k counts: ceil(rho * N_K)
    assert len(O.select_row(w, valid, "topk", 0.2)[0]) == 10
    assert O.topk_count(0.2, 256, 256) == 52 and O.topk_count(0.1, 1861, 1861) == 187


# ---------------------------------------------------------- attention -----
def test_all_blocks_kept_is_dense_attention():
    N, d = 70, 16
    r = rng(33)
    Q, K, V = (r.standard_normal((N, d)) for _ in range(3))
    qperm, kperm = r.permutation(N), r.permutation(N)
    qoff = np.array([0, 13, 13, 40, 70])
    koff = np.array([0, 7, 30, 30, 52, 70])
    rows = [np.array([0, 1, 3, 4])] * 4  # block 2 is empty, the rest all kept
    Ob = O.block_sparse_attention(Q[qperm], K[kperm], V[kperm], qoff, koff, rows, qperm)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q)[None], torch.from_numpy(K)[None], torch.from_numpy(V)[None])[0]
    assert np.abs(Ob - ref.numpy()).max() < 1e-12
    assert np.abs(O.dense_attention(Q, K, V) - ref.numpy()).max() < 1e-12


def test_sparse_attention_ignores_unselected_and_renormalises():
    N, d = 40, 8
    r = rng(34)
    Q, K, V = (r.standard_normal((N, d)) for _ in range(3))
    qoff = np.array([0, 20, 40])
    koff = np.array([0, 10, 25, 40])
    rows = [np.array([1]), np.array([0, 2])]
    perm = np.arange(N)
    O1 = O.block_sparse_attention(Q, K, V, qoff, koff, rows, perm)
    V2 = V.copy()
    V2[0:10] += 100.0  # block 0 not selected by query block 0
    O2 = O.block_sparse_attention(Q, K, V2, qoff, koff, rows, perm)
    assert np.array_equal(O1[:20], O2[:20])
    # query block 0 attends to keys 10..24 only, softmax renormalised there
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q[:20])[None], torch.from_numpy(K[10:25])[None],
        torch.from_numpy(V[10:25])[None])[0].numpy()
    assert np.abs(O1[:20] - ref).max() < 1e-12


# --------------------------------------------------------- whole path -----
def test_tiny_layer_end_to_end_sanity():
    from paper_2609_38978_amd import synth
    cfg = synth.CONFIGS["tiny"]
    q, k, v = synth.make_head(cfg, 0)
    res = O.park_head(q, k, v, cfg.C, cfg.C, cfg.iters, "topk", cfg.ratio)
    assert all(len(r) == 16 for r in res["rows"] if len(r))
    assert res["q"]["offsets"][-1] == cfg.N and res["k"]["offsets"][-1] == cfg.N
    qoff, koff = res["q"]["offsets"], res["k"]["offsets"]
    rec = O.recall(res["Qp"], res["Kp"], qoff, koff, res["rows"])
    assert rec > 0.9  # clustered inputs: 25% of blocks hold most of the mass
    # the mask keeps most of the exact importance of each query block
    Wex = O.exact_block_importance(res["Qp"], res["Kp"], qoff, koff)
    assert np.allclose(Wex[np.diff(qoff) > 0].sum(1), 1, atol=1e-12)


# ------------------------------------------- query-centroid estimate -----
def test_query_centroid_estimate_equals_pama_for_constant_blocks():
    # Sec. 4.1: the query-centroid gap is driven by the within-block query
    # covariance; with identical queries in every block it vanishes, and the
    # estimate is PAMA itself.  Rows sum to one; empty query blocks are zero.
    d = 8
    Kp = rng(60).standard_normal((50, d))
    koff = np.array([0, 9, 9, 31, 50])
    c, n = O.block_centroids(Kp, koff)
    base = rng(61).standard_normal((3, d)).astype(np.float32).astype(np.float64)
    sizes = [4, 0, 7, 2]
    Qp = np.concatenate([np.repeat(base[min(u, 2):min(u, 2) + 1], s, 0)
                         for u, s in enumerate(sizes)])
    qoff = np.concatenate([[0], np.cumsum(sizes)])
    Wc = O.query_centroid_estimate(Qp, qoff, c, n)
    Wp = O.pama(Qp, qoff, c, n)
    assert np.abs(Wc - Wp).max() < 1e-15
    assert np.all(Wc[1] == 0)
    nz = np.array(sizes) > 0
    assert np.abs(Wc[nz].sum(axis=1) - 1).max() < 1e-14
    assert np.all(Wc[:, 1] == 0)  # the empty key block gets no weight


def test_query_centroid_estimate_gap_is_second_order():
    # Sec. 4.1 / App. C: W - W^centroid = 1/2 <H_phi(qbar), Sigma_Q> + higher
    # order, so for the block {qbar + e delta, qbar - e delta} the gap shrinks
    # by ~4 when e halves (a first-order mistake, e.g. scoring one query
    # instead of the mean, would shrink it by ~2).
    d = 8
    Kp = rng(62).standard_normal((40, d)) * 2
    koff = np.array([0, 10, 25, 40])
    c, n = O.block_centroids(Kp, koff)
    qbar = rng(63).standard_normal(d).astype(np.float32).astype(np.float64)
    delta = rng(64).standard_normal(d)
    gaps = []
    for e in (2.0 ** -6, 2.0 ** -7):
        Qp = np.stack([qbar + e * delta, qbar - e * delta])
        Qp = Qp.astype(np.float32).astype(np.float64)
        off = np.array([0, 2])
        Wp = O.pama(Qp, off, c, n)
        Wc = O.query_centroid_estimate(Qp, off, c, n)
        gaps.append(np.abs(Wp - Wc).max())
    assert 3.5 < gaps[0] / gaps[1] < 4.5


def test_query_centroid_estimate_single_tokens_is_attention():
    # singleton query and key blocks: qbar = q, c = k, log 1 = 0, so the
    # estimate is the dense attention matrix (torch softmax).
    N, d = 40, 8
    Q = rng(65).standard_normal((N, d)).astype(np.float32).astype(np.float64)
    K = rng(66).standard_normal((N, d)).astype(np.float32).astype(np.float64)
    qp, kp = rng(67).permutation(N), rng(68).permutation(N)
    off = np.arange(N + 1)
    c, n = O.block_centroids(K[kp], off)
    W = O.query_centroid_estimate(Q[qp], off, c, n)
    A = torch.softmax(torch.from_numpy(Q) @ torch.from_numpy(K).T / math.sqrt(d), dim=1).numpy()
    assert np.abs(W - A[np.ix_(qp, kp)]).max() < 1e-14


# -------------------------------------------------- fixed-tile blocks -----
@pytest.mark.parametrize("N,C", [(4096, 64), (75600, 1182), (100, 30), (129, 2), (7, 7)])
def test_fixed_tile_offsets_partition(N, C):
    # blocks of b = ceil(N / C) consecutive tokens, a shorter last block, and
    # empty blocks only at the end; together a partition of range(N)
    off = O.fixed_tile_offsets(N, C)
    b = -(-N // C)
    sz = np.diff(off)
    assert len(off) == C + 1 and off[0] == 0 and off[-1] == N
    assert np.all(sz >= 0) and np.all(sz <= b)
    full = np.nonzero(sz)[0]
    assert np.all(sz[full[:-1]] == b) and np.all(sz[full[-1] + 1:] == 0)
    assert len(full) == -(-N // b)


def test_fixed_tiles_end_to_end_pins():
    # fixed tiles with every key block kept: dense attention (torch SDPA);
    # with one token per block (C = N): W^ is the exact attention mass.
    N, d = 96, 8
    r = rng(69)
    Q, K, V = (r.standard_normal((N, d)) for _ in range(3))
    out = O.park_head(Q, K, V, 12, 12, 3, "topk", 1.0, blocks="fixed")
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q)[None], torch.from_numpy(K)[None], torch.from_numpy(V)[None])[0]
    assert np.abs(out["O"] - ref.numpy()).max() < 1e-12
    assert np.array_equal(out["q"]["offsets"], np.arange(13) * 8)
    Qs, Ks = (x.astype(np.float32).astype(np.float64) for x in (Q[:24], K[:24]))
    one = O.park_head(Qs, Ks, V[:24], 24, 24, 2, "topk", 0.5, blocks="fixed")
    A = torch.softmax(torch.from_numpy(Qs) @ torch.from_numpy(Ks).T / math.sqrt(d), 1).numpy()
    assert np.abs(one["W"] - A[np.ix_(one["q"]["perm"], one["k"]["perm"])]).max() < 1e-13


# -------------------------------------- symmetric-square-root metric -----
def test_sqrt_realisation_same_distances_and_rank_deficient():
    # App. D: |Gbar^(1/2) delta|^2 = delta^T Gbar delta = |R^T delta|^2, and
    # the square root exists where Cholesky does not (rank-deficient Gbar).
    r = rng(70)
    Q = r.standard_normal((300, 12)) @ np.diag(np.linspace(0.2, 3.0, 12))
    ch, sq = O.query_metric(Q), O.query_metric_sqrt(Q)
    S = sq["R"]
    assert np.array_equal(ch["Gbar"], sq["Gbar"])
    assert np.abs(S - S.T).max() == 0 or np.abs(S - S.T).max() < 1e-14
    assert np.abs(S @ S - sq["Gbar"]).max() < 1e-12 * np.abs(sq["Gbar"]).max()
    delta = r.standard_normal((20, 12))
    qf = np.einsum("nd,de,ne->n", delta, sq["Gbar"], delta)
    assert np.allclose((delta @ S) ** 2 @ np.ones(12), qf, rtol=1e-12)
    assert np.allclose(((delta @ ch["R"]) ** 2).sum(1), qf, rtol=1e-12)
    # three informative feature directions, no shrinkage: rank 3
    Qd = np.zeros((200, 10))
    Qd[:, :3] = r.standard_normal((200, 3))
    with pytest.raises(np.linalg.LinAlgError):
        O.query_metric(Qd, alpha=0.0, eps=0.0)
    m = O.query_metric_sqrt(Qd, alpha=0.0, eps=0.0)
    assert np.linalg.matrix_rank(m["R"], tol=1e-10) == 3
    assert np.abs(m["R"] @ m["R"] - m["Gbar"]).max() < 1e-12
    d2 = r.standard_normal((15, 10))
    assert np.allclose(((d2 @ m["R"]) ** 2).sum(1),
                       np.einsum("nd,de,ne->n", d2, m["Gbar"], d2), rtol=1e-10, atol=1e-13)


def test_sqrt_and_cholesky_cluster_alike():
    # the two realisations give the same QRKC objective (App. D), hence the
    # same k-means labels on well-separated data
    r = rng(71)
    cen = r.standard_normal((6, 8)) * 6
    K = np.repeat(cen, 20, 0) + r.standard_normal((120, 8)) * 0.3
    Q = r.standard_normal((120, 8))
    a = O.cluster_keys(K, Q, 6, 5, 3, 0)
    b = O.cluster_keys(K, Q, 6, 5, 3, 0, realisation="sqrt")
    assert np.array_equal(a["labels"], b["labels"])
    assert np.array_equal(a["perm"], b["perm"])


# ------------------------------------- recall and exact log-mass pins -----
def _brute_attention(Q, K):
    """Row softmax of Q K^T / sqrt(d) by explicit loops over math.exp."""
    n, d = Q.shape
    A = np.zeros((n, K.shape[0]))
    for i in range(n):
        s = [sum(Q[i, t] * K[j, t] for t in range(d)) / math.sqrt(d) for j in range(K.shape[0])]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        z = sum(e)
        A[i] = [x / z for x in e]
    return A


def test_recall_all_blocks_kept_is_one():
    Qp = rng(70).standard_normal((30, 8))
    Kp = rng(71).standard_normal((40, 8))
    qoff = np.array([0, 7, 7, 30])
    koff = np.array([0, 5, 5, 22, 40])
    every = [np.array([0, 1, 2, 3]), np.array([], dtype=np.int64), np.array([0, 1, 2, 3])]
    assert O.recall(Qp, Kp, qoff, koff, every) == pytest.approx(1.0, abs=1e-14)
    assert O.recall(Qp, Kp, qoff, koff, [np.array([], dtype=np.int64)] * 3) == 0.0


def test_recall_hand_sized_brute_force():
    # Eq. (4): the attention mass inside the mask over the total (= number of
    # queries, since each row of A sums to one), on a case where the two query
    # blocks keep different, asymmetric key blocks: swapping the roles of u
    # and v, or summing the wrong block's columns, changes the value
    Q = np.array([[1.0, 0.0], [0.8, 0.3], [0.0, 1.0], [-0.5, 0.9], [0.2, -0.7]])
    K = np.array([[2.0, 0.0], [0.0, 1.5], [-1.0, 1.0], [0.5, 0.5]])
    qoff = np.array([0, 2, 5])
    koff = np.array([0, 1, 3, 4])
    rows = [np.array([0]), np.array([1, 2])]
    A = _brute_attention(Q, K)
    want = (A[0:2, 0:1].sum() + A[2:5, 1:3].sum() + A[2:5, 3:4].sum()) / 5.0
    assert O.recall(Q, K, qoff, koff, rows) == pytest.approx(want, rel=1e-13)
    swapped = (A[0:2, 1:4].sum() + A[2:5, 0:1].sum()) / 5.0
    assert abs(want - swapped) > 0.05


def test_recall_block_size_one_is_kept_attention_mass():
    # singleton blocks: recall is the sum of the kept entries of A over N
    Q = rng(72).standard_normal((6, 3))
    K = rng(73).standard_normal((6, 3))
    off = np.arange(7)
    rows = [np.array([0, 2]), np.array([5]), np.array([1, 3, 4]), np.array([0]),
            np.array([2, 3]), np.array([])]
    A = _brute_attention(Q, K)
    want = sum(A[i, j] for i, r in enumerate(rows) for j in r) / 6.0
    assert O.recall(Q, K, off, off, [np.asarray(r, dtype=np.int64) for r in rows]) == \
        pytest.approx(want, rel=1e-13)


def test_exact_log_mass_closed_forms():
    d = 4
    Q = rng(74).standard_normal((9, d))
    # a singleton block: S* is the raw scaled score
    K1 = rng(75).standard_normal((3, d))
    S = O.exact_log_mass(Q, K1, np.array([0, 1, 2, 3]))
    assert np.allclose(S, Q @ K1.T / math.sqrt(d), rtol=0, atol=1e-14)
    # n identical keys: S* = score + log n
    k = rng(76).standard_normal(d)
    Kid = np.tile(k, (5, 1))
    S = O.exact_log_mass(Q, Kid, np.array([0, 5]))
    assert np.allclose(S[:, 0], Q @ k / math.sqrt(d) + math.log(5), rtol=0, atol=1e-13)
    # two keys c +- eps e: S* - S^ = log cosh(eps q.e / sqrt(d)) (the key-side
    # error of Sec. 4.2 in closed form), S^ = q.c / sqrt(d) + log 2
    c, e, eps = rng(77).standard_normal(d), rng(78).standard_normal(d), 0.7
    K2 = np.stack([c + eps * e, c - eps * e])
    S = O.exact_log_mass(Q, K2, np.array([0, 2]))[:, 0]
    Shat = Q @ c / math.sqrt(d) + math.log(2)
    b = eps * (Q @ e) / math.sqrt(d)
    assert np.allclose(S - Shat, np.log(np.cosh(b)), rtol=0, atol=1e-13)
    # empty block
    S = O.exact_log_mass(Q, K2, np.array([0, 0, 2]))
    assert np.isneginf(S[:, 0]).all()


# ------------------------------------------- mismatch diagnostics pins -----
def test_tv_error_hand_example():
    # block 0 (3 queries): rows [1,0,0] vs [0,1,0] -> TV 1; block 1 (1 query):
    # [0.5,0.5,0] vs [0.5,0.25,0.25] -> TV 0.25; empty block 2 has no weight
    Wh = np.array([[1.0, 0.0, 0.0], [0.5, 0.5, 0.0], [0.0, 0.0, 0.0]])
    W = np.array([[0.0, 1.0, 0.0], [0.5, 0.25, 0.25], [0.3, 0.3, 0.4]])
    assert O.tv_error(Wh, W, np.array([3, 1, 0])) == pytest.approx(3 / 4 * 1 + 1 / 4 * 0.25)
    assert O.tv_error(W, W, np.array([3, 1, 0])) == 0.0
    # symmetric, in [0, 1] for distributions
    assert O.tv_error(W, Wh, np.array([3, 1, 0])) == O.tv_error(Wh, W, np.array([3, 1, 0]))


def test_tv_zero_when_pama_is_exact():
    # identical keys in every key block make PAMA the exact block importance
    # (Eq. (3)), so its TV error vanishes; the query-centroid estimate does not
    d = 6
    Q = rng(80).standard_normal((24, d))
    base = rng(81).standard_normal((4, d))
    Kp = np.repeat(base, [3, 5, 1, 7], axis=0)
    koff = np.array([0, 3, 8, 9, 16])
    qoff = np.array([0, 10, 24])
    c = O.block_means(Kp, koff)
    n = np.diff(koff)
    W = O.exact_block_importance(Q, Kp, qoff, koff)
    S = O.log_mass_estimate(Q, c, n)
    Wp = np.stack([O.softmax_rows(S[a:b]).mean(0) for a, b in ((0, 10), (10, 24))])
    assert O.tv_error(Wp, W, np.diff(qoff)) < 1e-14
    Wc = O.query_centroid_full_keys(Q, qoff, Kp, koff)
    assert O.tv_error(Wc, W, np.diff(qoff)) > 1e-3


def test_query_centroid_full_keys_brute_force():
    Q = rng(82).standard_normal((7, 3))
    K = rng(83).standard_normal((9, 3))
    qoff = np.array([0, 4, 4, 7])
    koff = np.array([0, 2, 6, 9])
    W = O.query_centroid_full_keys(Q, qoff, K, koff)
    for u, (a, b) in enumerate(((0, 4), (4, 4), (4, 7))):
        if b == a:
            assert np.all(W[u] == 0)
            continue
        A = _brute_attention(Q[a:b].mean(0, keepdims=True), K)[0]
        assert np.allclose(W[u], [A[0:2].sum(), A[2:6].sum(), A[6:9].sum()], atol=1e-14)
    # with one query per block it is the exact block importance
    off = np.arange(8)
    assert np.allclose(O.query_centroid_full_keys(Q, off, K, koff),
                       O.exact_block_importance(Q, K, off, koff), atol=1e-14)


def test_centred_log_mass_rmse_closed_forms():
    # hand example: one query with Delta = [3, 1] (mean 2, delta = [1, -1]) and
    # one with Delta = [0, 4] (delta = [-2, 2]): E_LM = (1 + 2) / 2
    Sstar = np.array([[3.0, 1.0, -np.inf], [0.0, 4.0, -np.inf]])
    Shat = np.zeros((2, 3))
    Shat[:, 2] = -np.inf
    assert O.centred_log_mass_rmse(Sstar, Shat) == pytest.approx(1.5)
    # a per-query offset does not count
    assert O.centred_log_mass_rmse(Sstar, Shat + np.array([[7.0], [-2.0]])) == pytest.approx(1.5)
    # two-key blocks c_v +- eps e_v: Delta = log cosh(eps q.e_v / sqrt(d)) exactly
    d = 4
    Q = rng(84).standard_normal((5, d))
    cs = rng(85).standard_normal((3, d))
    es = rng(86).standard_normal((3, d))
    Kp = np.concatenate([np.stack([cs[v] + 0.5 * es[v], cs[v] - 0.5 * es[v]]) for v in range(3)])
    off = np.array([0, 2, 4, 6])
    Sstar = O.exact_log_mass(Q, Kp, off)
    Shat = O.log_mass_estimate(Q, O.block_means(Kp, off), np.diff(off))
    Dl = np.log(np.cosh(0.5 * (Q @ es.T) / math.sqrt(d)))
    want = np.sqrt(((Dl - Dl.mean(1, keepdims=True)) ** 2).mean(1)).mean()
    assert O.centred_log_mass_rmse(Sstar, Shat) == pytest.approx(want, rel=1e-12)
    # singleton blocks: the estimate is exact
    Sstar = O.exact_log_mass(Q, Kp, np.arange(7))
    Shat = O.log_mass_estimate(Q, Kp, np.ones(6, dtype=int))
    assert O.centred_log_mass_rmse(Sstar, Shat) < 1e-14


def test_key_space_errors_brute_force_and_objective():
    d = 3
    Q = rng(87).standard_normal((6, d))
    K = rng(88).standard_normal((8, d))
    z = np.array([0, 1, 0, 2, 1, 1, 0, 2])
    c = np.stack([K[z == v].mean(0) for v in range(3)])
    dk, dq = O.key_space_errors(K, Q, z, c)
    bk = sum(sum((K[j, t] - c[z[j], t]) ** 2 for t in range(d)) for j in range(8)) / 8
    bq = sum(sum(Q[i, t] * (K[j, t] - c[z[j], t]) for t in range(d)) ** 2 / d
             for i in range(6) for j in range(8)) / 48
    assert dk == pytest.approx(bk, rel=1e-13) and dq == pytest.approx(bq, rel=1e-13)
    # D_QK is the QRKC objective of Eq. (10) (metric G_Q = Q^T Q / L_Q,
    # no stabilisation) divided by L_K d
    G = Q.T @ Q / 6
    J = sum((K[j] - c[z[j]]) @ G @ (K[j] - c[z[j]]) for j in range(8))
    assert dq == pytest.approx(J / (8 * d), rel=1e-13)
    # singletons: no error; one cluster: D_key is the total variance
    assert O.key_space_errors(K, Q, np.arange(8), K) == (0.0, 0.0)
    dk1, _ = O.key_space_errors(K, Q, np.zeros(8, dtype=int), K.mean(0, keepdims=True))
    assert dk1 == pytest.approx(((K - K.mean(0)) ** 2).sum() / 8, rel=1e-13)


def test_mismatch_directions():
    # The paper's directional claims (App. A, App. B) where they must hold.
    # (1) Clustered layer from the seeded generator: per-query PAMA has a far
    # lower TV error than the query-centroid estimate (M1).
    from paper_2609_38978_amd import synth
    cfg = synth.CONFIGS["tiny"].with_(grid=(2, 16, 32))
    q, k, _ = synth.make_head(cfg, 0)
    rep = O.mismatch_report(q, k, cfg.C, cfg.C, 6)
    print("generator", rep)
    assert rep["tv_per_query"] < 0.5 * rep["tv_query_centroid"]
    # (2) Queries spread along two directions only, keys in blobs: QRKC
    # clusters keys by QK-score error, so it lowers D_QK and the centred
    # log-mass error and raises the raw-key MSE relative to Euclidean k-means
    # (M2, App. B).  With isotropic queries the two metrics nearly coincide.
    r = rng(90)
    d, N = 16, 768
    basis = np.linalg.qr(r.standard_normal((d, 2)))[0]
    Q = 3.0 * r.standard_normal((N, 2)) @ basis.T + 0.05 * r.standard_normal((N, d))
    cent = 2.0 * r.standard_normal((24, d))
    K = cent[r.integers(0, 24, N)] + 0.5 * r.standard_normal((N, d))
    rep = O.mismatch_report(Q, K, 12, 24, 8)
    print("anisotropic queries", rep)
    assert rep["d_qk_qrkc"] < 0.5 * rep["d_qk_euclid"]
    assert rep["d_key_qrkc"] > rep["d_key_euclid"]
    assert rep["log_mass_rmse_qrkc"] < 0.5 * rep["log_mass_rmse_euclid"]


def test_alpha_sweep_of_the_key_metric():
    # App. D: alpha moves the key metric from the query-response metric
    # (alpha -> 0) to the isotropic one (alpha = 1).  At alpha = 1 the key
    # partition is Euclidean k-means' (a scaled metric, the same init), so
    # every diagnostic equals the Euclidean one; at the paper's alpha the
    # partition follows the queries' directions (lower D_QK and log-mass
    # error, higher raw-key MSE than alpha = 1).  Same anisotropic layer as
    # the directional test above.
    r = rng(90)
    d, N = 16, 768
    basis = np.linalg.qr(r.standard_normal((d, 2)))[0]
    Q = 3.0 * r.standard_normal((N, 2)) @ basis.T + 0.05 * r.standard_normal((N, d))
    cent = 2.0 * r.standard_normal((24, d))
    K = cent[r.integers(0, 24, N)] + 0.5 * r.standard_normal((N, d))
    rows = {}
    for alpha in (0.0, 0.05, 0.25, 0.5, 1.0):
        rep = O.mismatch_report(Q, K, 12, 24, 8, alpha=alpha)
        rows[alpha] = rep
        print(f"alpha={alpha:<5} D_QK={rep['d_qk_qrkc']:.4g} D_key={rep['d_key_qrkc']:.4g} "
              f"log-mass RMSE={rep['log_mass_rmse_qrkc']:.4g}  (Euclidean: "
              f"{rep['d_qk_euclid']:.4g}, {rep['d_key_euclid']:.4g}, "
              f"{rep['log_mass_rmse_euclid']:.4g})")
    one = rows[1.0]
    for key in ("d_qk", "d_key", "log_mass_rmse"):
        assert one[f"{key}_qrkc"] == pytest.approx(one[f"{key}_euclid"], rel=1e-12)
    small = rows[0.05]
    assert small["d_qk_qrkc"] < 0.5 * one["d_qk_qrkc"]
    assert small["d_key_qrkc"] > one["d_key_qrkc"]
    assert small["log_mass_rmse_qrkc"] < 0.5 * one["log_mass_rmse_qrkc"]


def test_block_sparse_lse_pins():
    from scipy.special import logsumexp
    d = 8
    Q = rng(95).standard_normal((30, d))
    K = rng(96).standard_normal((25, d))
    qoff = np.array([0, 12, 12, 30])
    koff = np.array([0, 4, 4, 13, 25])
    perm = rng(97).permutation(30)
    # every block kept: the dense row log-sum-exp (scipy), un-permuted
    every = [np.array([0, 1, 2, 3])] * 3
    lse = O.block_sparse_lse(Q, K, qoff, koff, every, perm)
    want = np.empty(30)
    want[perm] = logsumexp(Q @ K.T / math.sqrt(d), axis=1)
    assert np.allclose(lse, want, rtol=0, atol=1e-13)
    # a selection: the log-sum-exp over the kept blocks of their exact
    # log-masses S*_iv (Eq. (6)); nothing kept gives -inf
    rows = [np.array([0, 3]), np.array([], dtype=np.int64), np.array([1, 2])]
    lse = O.block_sparse_lse(Q, K, qoff, koff, rows, perm)
    S = O.exact_log_mass(Q, K, koff)
    assert np.allclose(lse[perm[:12]], logsumexp(S[:12][:, [0, 3]], axis=1), atol=1e-13)
    assert np.allclose(lse[perm[12:]], logsumexp(S[12:][:, [2]], axis=1), atol=1e-13)
    rows[0] = np.array([1])  # an empty key block only: nothing kept
    lse = O.block_sparse_lse(Q, K, qoff, koff, rows, perm)
    assert np.isneginf(lse[perm[:12]]).all()


# ------------------------------------------------------------ warm start -----
def test_warm_start_pins():
    X = rng(100).standard_normal((300, 5))
    init = O.init_indices(300, 12, seed=4, head=0, side=0)
    # starting from the seeded centroids is the seeded run
    z1, mu1 = O.kmeans(X, 12, 6, init)
    z2, mu2 = O.kmeans(X, 12, 6, init, mu0=X[init])
    assert np.array_equal(z1, z2) and np.array_equal(mu1, mu2)
    # final means: brute force, empty clusters keep their centroid
    z = z1.copy()
    z[z == 3] = 4
    m = O.final_means(X, z, mu1)
    for v in range(12):
        want = X[z == v].mean(0) if np.any(z == v) else mu1[v]
        assert np.allclose(m[v], want, rtol=0, atol=1e-14)
    # a warm start at a fixed point of Lloyd's iteration stays there
    zc, muc = O.kmeans(X, 12, 60, init)
    fixed = O.final_means(X, zc, muc)
    z3, mu3 = O.kmeans(X, 12, 3, init, mu0=fixed)
    assert np.array_equal(z3, zc) and np.allclose(mu3, fixed, atol=1e-14)
    # keys: a warm start in the original key space is transformed by R
    Q = rng(101).standard_normal((300, 5))
    K = rng(102).standard_normal((300, 5))
    r = O.cluster_keys(K, Q, 12, 4, 0, 0)
    mu_in = O.final_means(K, r["labels"], r["mu"] @ np.linalg.inv(r["R"]))
    r2 = O.cluster_keys(K, Q, 12, 2, 0, 0, mu0=mu_in)
    zt = O.assign(r["Kt"], mu_in @ r["R"])
    assert np.array_equal(r2["labels"], O.assign(r["Kt"], O.update(r["Kt"], zt, mu_in @ r["R"])))
