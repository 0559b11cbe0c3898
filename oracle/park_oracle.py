"""PARK sparse-attention forward -- plain CPU oracle (float64 NumPy).

TEST INFRASTRUCTURE ONLY.  This module is imported by ``tests/``, by
``__graft_entry__.smoke()`` and by the ``cpu_baseline`` leg of ``bench.py``,
nothing else.  The HIP library never imports, links or calls it, and it
imports nothing from the library.  It shares no code with the GPU path except
that both consume the seeded tensors of ``paper_2609_38978_amd.synth``.

Everything is computed per attention head in float64; bf16/fp32 inputs are
upcast exactly.  Each function follows one passage of the paper (PARK:
Accurate Block Retrieval for Sparse Attention in Video Diffusion
Transformers), cited in its docstring by section, equation or algorithm.

Readings taken where the paper is silent (the same list is kept with the
design notes of the repository):

* blocks are k-means clusters, ``C = ceil(N / B)`` of them per side;
* k-means init: ``C`` distinct token indices from a partial Fisher-Yates
  shuffle driven by SplitMix64, seeded with
  ``seed XOR (0x9E3779B97F4A7C15 * (2*head + side + 1)) mod 2^64``, where
  ``side`` is 0 for queries and 1 for keys;
* k-means runs exactly ``T`` (assign, update) rounds, the labels are those of
  the T-th assignment; argmin ties go to the lowest cluster id; an empty
  cluster keeps its previous centroid;
* the token permutation is the stable argsort of the labels;
* the stability constant is ``eps = 1e-6`` and ``s_min = 1e-12``;
* key-block centroids are rounded to float32 before PAMA scores them;
* empty key blocks get no score (they are left out of the softmax and are
  never selected); empty query blocks get no mask row;
* top-p keeps the shortest prefix (descending estimated importance, ties by
  ascending block id) whose float64 cumulative sum is >= p, all nonempty
  blocks if rounding never reaches p, and at least one block; top-k keeps
  ``ceil(rho * N_K - 1e-9)`` blocks clamped to [1, #nonempty];
* sparse attention renormalises the softmax over the selected keys (the
  block-sparse flash-attention semantics); with every block kept this is
  exactly full attention.
"""
from __future__ import annotations

import math

import numpy as np

_M64 = (1 << 64) - 1
_GOLDEN = 0x9E3779B97F4A7C15


# --------------------------------------------------------------------------
# seeded k-means initialisation (the paper only says "initialize from K~")
# --------------------------------------------------------------------------
class SplitMix64:
    """SplitMix64 generator (Steele, Lea & Flood, OOPSLA 2014), as published."""

    def __init__(self, seed: int):
        self.state = seed & _M64

    def next(self) -> int:
        self.state = (self.state + _GOLDEN) & _M64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
        return z ^ (z >> 31)


def init_seed(seed: int, head: int, side: int) -> int:
    return (seed ^ ((_GOLDEN * (2 * head + side + 1)) & _M64)) & _M64


def init_indices(N: int, C: int, seed: int, head: int, side: int) -> np.ndarray:
    """First C entries of a Fisher-Yates shuffle of range(N) (distinct tokens).

    Step i swaps position i with position ``i + (next() mod (N - i))``.
    """
    if not 1 <= C <= N:
        raise ValueError("need 1 <= C <= N")
    rng = SplitMix64(init_seed(seed, head, side))
    a = list(range(N))
    for i in range(C):
        j = i + rng.next() % (N - i)
        a[i], a[j] = a[j], a[i]
    return np.array(a[:C], dtype=np.int64)


# --------------------------------------------------------------------------
# QRKC: query metric, Cholesky factor, key transform (Sec. 5.2, App. D.2, Alg. 3)
# --------------------------------------------------------------------------
def query_metric(Q: np.ndarray, alpha: float = 0.05, eps: float = 1e-6, s_min: float = 1e-12):
    """Stabilised query second moment and its Cholesky factor (Alg. 3).

    G = Q^T Q / L, symmetrised; s = max(tr(G)/d, s_min);
    Gbar = (1 - alpha) G + alpha s I + eps s I; Gbar = R R^T with R lower.
    Raises ``np.linalg.LinAlgError`` when Gbar is not positive definite.
    """
    Q = np.asarray(Q, dtype=np.float64)
    L, d = Q.shape
    G = (Q.T @ Q) / L
    G = (G + G.T) / 2.0
    s = max(np.trace(G) / d, s_min)
    eye = np.eye(d)
    Gbar = (1.0 - alpha) * G + alpha * s * eye + eps * s * eye
    R = np.linalg.cholesky(Gbar)
    return {"G": G, "s": s, "Gbar": Gbar, "R": R}


def query_metric_sqrt(Q: np.ndarray, alpha: float = 0.05, eps: float = 1e-6,
                      s_min: float = 1e-12):
    """The same Gbar with its symmetric square root (App. D).

    Gbar = U Lambda U^T (eigh), Gbar^(1/2) = U Lambda^(1/2) U^T; eigenvalues
    that rounding leaves below zero are taken as zero.  Unlike the Cholesky
    factor it exists for a rank-deficient Gbar.  k~ = Gbar^(1/2) k, and since
    the root is symmetric the row form is K~ = K Gbar^(1/2).
    """
    Q = np.asarray(Q, dtype=np.float64)
    L, d = Q.shape
    G = (Q.T @ Q) / L
    G = (G + G.T) / 2.0
    s = max(np.trace(G) / d, s_min)
    eye = np.eye(d)
    Gbar = (1.0 - alpha) * G + alpha * s * eye + eps * s * eye
    lam, U = np.linalg.eigh(Gbar)
    S = (U * np.sqrt(np.maximum(lam, 0.0))) @ U.T
    return {"G": G, "s": s, "Gbar": Gbar, "R": S}


def transform_keys(K: np.ndarray, R: np.ndarray) -> np.ndarray:
    """Row form of k~ = R^T k (Eq. (12)): K~ = K R."""
    return np.asarray(K, dtype=np.float64) @ R


# --------------------------------------------------------------------------
# Euclidean k-means (Sec. 5.2 "standard Euclidean K-means", Alg. 3 loop)
# --------------------------------------------------------------------------
def sq_distances(X: np.ndarray, mu: np.ndarray) -> np.ndarray:
    """Squared Euclidean distances ``[n, C]`` = |x|^2 - 2 x.mu + |mu|^2."""
    x2 = np.einsum("ij,ij->i", X, X)
    m2 = np.einsum("ij,ij->i", mu, mu)
    return x2[:, None] - 2.0 * (X @ mu.T) + m2[None, :]


def assign(X: np.ndarray, mu: np.ndarray, chunk: int = 8192) -> np.ndarray:
    """z_j = argmin_v |x_j - mu_v|^2, ties to the lowest v."""
    z = np.empty(X.shape[0], dtype=np.int64)
    for a in range(0, X.shape[0], chunk):
        z[a:a + chunk] = np.argmin(sq_distances(X[a:a + chunk], mu), axis=1)
    return z


def update(X: np.ndarray, z: np.ndarray, mu: np.ndarray) -> np.ndarray:
    """mu_v = mean{x_j : z_j = v}; an empty cluster keeps its centroid."""
    C = mu.shape[0]
    cnt = np.bincount(z, minlength=C)
    sums = np.zeros_like(mu)
    np.add.at(sums, z, X)
    new = mu.copy()
    nz = cnt > 0
    new[nz] = sums[nz] / cnt[nz, None]
    return new


def kmeans(X: np.ndarray, C: int, T: int, init: np.ndarray, labels_hook=None, mu0=None):
    """T rounds of (assign, update) from centroids X[init], or from the given
    centroids ``mu0`` (a warm start, e.g. the previous recomputation's means).

    Returns the labels of the T-th assignment and the centroids it used.
    ``labels_hook(t, z, mu)`` may return replacement labels for round t
    (parity tests use it to follow another implementation's near-tie flips).
    """
    X = np.asarray(X, dtype=np.float64)
    mu = (X[np.asarray(init)] if mu0 is None else np.asarray(mu0, dtype=np.float64)).copy()
    z = None
    for t in range(T):
        z = assign(X, mu)
        if labels_hook is not None:
            z = labels_hook(t, z, mu)
        if t + 1 < T:
            mu = update(X, z, mu)
    return z, mu


def final_means(X, z, mu_last):
    """Means of the final clusters, an empty cluster keeping mu_last (its
    centroid in the last assignment): the starting centroids a warm-started
    recomputation takes from the previous one (clusters change little between
    adjacent diffusion steps, Sec. 5.2)."""
    return update(np.asarray(X, dtype=np.float64), np.asarray(z), np.asarray(mu_last, np.float64))


# --------------------------------------------------------------------------
# permutation and block layout (Alg. 3 tail; App. E "queries stored contiguously")
# --------------------------------------------------------------------------
def stable_argsort(z: np.ndarray, C: int):
    """pi = stable argsort(z); offsets o[0..C] with o[v+1] - o[v] = n_v."""
    z = np.asarray(z)
    perm = np.argsort(z, kind="stable")
    counts = np.bincount(z, minlength=C)
    offsets = np.concatenate([[0], np.cumsum(counts)])
    return perm.astype(np.int64), offsets.astype(np.int64)


def fixed_tile_offsets(N: int, C: int) -> np.ndarray:
    """Blocks as fixed chunks of the cluster-sorted order: o_v = min(v b, N).

    The literal reading of a block size with a padded last block: b =
    ceil(N / C) tokens per block, a shorter last block, and empty trailing
    blocks when C b - N >= b.  The tokens keep the order of the stable
    argsort of the cluster labels (Alg. 3).
    """
    b = -(-N // C)
    return np.minimum(np.arange(C + 1, dtype=np.int64) * b, N)


def block_centroids(Kp: np.ndarray, offsets: np.ndarray):
    """c_v = (1/n_v) sum of the original keys of block v (Eq. (8), Alg. 3).

    Kp are the permuted keys.  The centroids are rounded to float32 (the
    precision the retrieval kernel scores them in); empty blocks give 0.
    """
    Kp = np.asarray(Kp, dtype=np.float64)
    C = len(offsets) - 1
    c = np.zeros((C, Kp.shape[1]), dtype=np.float64)
    n = np.diff(offsets).astype(np.int64)
    for v in range(C):
        if n[v] > 0:
            c[v] = Kp[offsets[v]:offsets[v + 1]].sum(axis=0) / n[v]
    return c.astype(np.float32), n


# --------------------------------------------------------------------------
# PAMA (Sec. 5.1, Eqs. (8)-(9))
# --------------------------------------------------------------------------
def pama_scores(Qp: np.ndarray, c: np.ndarray, n: np.ndarray) -> np.ndarray:
    """S^_iv = q_i . c_v / sqrt(d) + log n_v; -inf for empty key blocks."""
    Qp = np.asarray(Qp, dtype=np.float64)
    d = Qp.shape[1]
    S = (Qp @ np.asarray(c, dtype=np.float64).T) / math.sqrt(d)
    with np.errstate(divide="ignore"):
        logn = np.where(n > 0, np.log(np.maximum(n, 1).astype(np.float64)), -np.inf)
    return S + logn[None, :]


def softmax_rows(S: np.ndarray) -> np.ndarray:
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    return E / E.sum(axis=1, keepdims=True)


def pama(Qp: np.ndarray, q_offsets: np.ndarray, c: np.ndarray, n: np.ndarray) -> np.ndarray:
    """W^_uv = (1/n_u) sum_{i in Q_u} softmax_v(S^_i.)_v  (Eq. (9)).

    Rows of empty query blocks are zero.
    """
    CQ = len(q_offsets) - 1
    W = np.zeros((CQ, len(n)), dtype=np.float64)
    for u in range(CQ):
        a, b = int(q_offsets[u]), int(q_offsets[u + 1])
        if b > a:
            P = softmax_rows(pama_scores(Qp[a:b], c, n))
            W[u] = P.sum(axis=0) / (b - a)
    return W


def query_centroid_estimate(Qp: np.ndarray, q_offsets: np.ndarray, c: np.ndarray,
                            n: np.ndarray) -> np.ndarray:
    """W^centroid_uv = phi_v(qbar_u), the query-centroid estimate (Sec. 4.1).

    The queries of block u are replaced by their mean before the softmax:
    phi_v(q) is the weight a single query q gives key block v under the
    PAMA score of Eq. (8), so the row is softmax_v(qbar_u . c_v / sqrt(d) +
    log n_v).  This is the "w/o PAMA" variant of the ablation (Sec. 6).
    qbar_u is rounded to float32, like the key-block centroids.  Rows of
    empty query blocks are zero.
    """
    Qp = np.asarray(Qp, dtype=np.float64)
    CQ = len(q_offsets) - 1
    W = np.zeros((CQ, len(n)), dtype=np.float64)
    for u in range(CQ):
        a, b = int(q_offsets[u]), int(q_offsets[u + 1])
        if b > a:
            qbar = (Qp[a:b].sum(axis=0) / (b - a)).astype(np.float32)
            W[u] = softmax_rows(pama_scores(qbar[None, :], c, n))[0]
    return W


# --------------------------------------------------------------------------
# mask selection (Sec. 3.2 top-p; App. J top-k)
# --------------------------------------------------------------------------
def descending_order(w: np.ndarray, valid: np.ndarray) -> np.ndarray:
    """Valid block ids by decreasing w, ties by increasing id."""
    ids = np.nonzero(valid)[0]
    return ids[np.lexsort((ids, -w[ids]))]


def topk_count(rho: float, n_blocks: int, n_valid: int) -> int:
    k = math.ceil(rho * n_blocks - 1e-9)
    return max(1, min(k, n_valid))


def select_row(w: np.ndarray, valid: np.ndarray, mode: str, param: float):
    """Selected key-block ids of one query block, ascending.

    Also returns the descending order and the cut (number kept) so callers
    can inspect near-ties.
    """
    order = descending_order(w, valid)
    if len(order) == 0:
        return np.zeros(0, dtype=np.int64), order, 0
    if mode == "topk":
        m = topk_count(param, len(w), len(order))
    elif mode == "topp":
        cs = np.cumsum(w[order])
        hit = np.nonzero(cs >= param)[0]
        m = int(hit[0]) + 1 if len(hit) else len(order)
    else:
        raise ValueError(mode)
    return np.sort(order[:m]), order, m


def select(W: np.ndarray, q_sizes: np.ndarray, k_sizes: np.ndarray, mode: str, param: float):
    """Block mask as a list of ascending key-block id arrays per query block."""
    valid = np.asarray(k_sizes) > 0
    rows = []
    for u in range(W.shape[0]):
        if q_sizes[u] == 0:
            rows.append(np.zeros(0, dtype=np.int64))
        else:
            rows.append(select_row(W[u], valid, mode, param)[0])
    return rows


# --------------------------------------------------------------------------
# attention (Eqs. (1)-(2))
# --------------------------------------------------------------------------
def dense_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """O = softmax(Q K^T / sqrt(d)) V (Eq. (1))."""
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    A = softmax_rows((Q @ K.T) / math.sqrt(Q.shape[1]))
    return A @ V


def block_sparse_attention(Qp, Kp, Vp, q_offsets, k_offsets, rows, q_perm) -> np.ndarray:
    """Attention of each query block over the union of its selected key blocks.

    The softmax is renormalised over the kept keys; row i of the permuted
    queries is written to position q_perm[i] (un-permutation).
    """
    Qp, Kp, Vp = (np.asarray(a, dtype=np.float64) for a in (Qp, Kp, Vp))
    N, d = Qp.shape
    O = np.zeros((N, Vp.shape[1]), dtype=np.float64)
    for u, sel in enumerate(rows):
        a, b = int(q_offsets[u]), int(q_offsets[u + 1])
        if b == a:
            continue
        keys = np.concatenate([np.arange(k_offsets[v], k_offsets[v + 1]) for v in sel])
        A = softmax_rows((Qp[a:b] @ Kp[keys].T) / math.sqrt(d))
        O[np.asarray(q_perm[a:b])] = A @ Vp[keys]
    return O


def block_sparse_lse(Qp, Kp, q_offsets, k_offsets, rows, q_perm) -> np.ndarray:
    """Natural-log normaliser of each row of the block-sparse attention.

    lse_i = log sum_j exp(q_i . k_j / sqrt(d)) over the keys of the selected
    key blocks of i's query block (the denominator of Eq. (2) renormalised over
    the kept keys), stored at position q_perm[i]; -inf when nothing is kept.
    """
    Qp, Kp = (np.asarray(a, dtype=np.float64) for a in (Qp, Kp))
    N, d = Qp.shape
    out = np.full(N, -np.inf)
    for u, sel in enumerate(rows):
        a, b = int(q_offsets[u]), int(q_offsets[u + 1])
        if b == a or len(sel) == 0:
            continue
        keys = np.concatenate([np.arange(k_offsets[v], k_offsets[v + 1]) for v in sel])
        if len(keys) == 0:
            continue
        Z = (Qp[a:b] @ Kp[keys].T) / math.sqrt(d)
        m = Z.max(axis=1)
        out[np.asarray(q_perm[a:b])] = m + np.log(np.exp(Z - m[:, None]).sum(axis=1))
    return out


# --------------------------------------------------------------------------
# whole head (Alg. 3 + Sec. 5.1 + Eq. (2))
# --------------------------------------------------------------------------
def cluster_queries(Q, C, T, seed, head, mu0=None):
    """Euclidean k-means on the queries and their permutation (Sec. 5.2);
    ``mu0`` replaces the seeded init by given starting centroids."""
    Q = np.asarray(Q, dtype=np.float64)
    init = init_indices(Q.shape[0], C, seed, head, side=0)
    z, mu = kmeans(Q, C, T, init, mu0=mu0)
    perm, off = stable_argsort(z, C)
    return {"labels": z, "perm": perm, "offsets": off, "mu": mu, "init": init}


def cluster_keys(K, Q, C, T, seed, head, alpha=0.05, eps=1e-6, s_min=1e-12,
                 realisation="cholesky", mu0=None):
    """QRKC (Alg. 3): k-means on K R, with Gbar = R R^T from the queries.

    realisation "sqrt" uses the symmetric square root instead of the
    Cholesky factor (App. D): the same distances, and defined for a
    rank-deficient Gbar.  ``mu0`` (original key space) replaces the seeded
    init: the transformed starting centroids are mu0 R."""
    met = (query_metric if realisation == "cholesky" else query_metric_sqrt)(Q, alpha, eps, s_min)
    Kt = transform_keys(K, met["R"])
    init = init_indices(Kt.shape[0], C, seed, head, side=1)
    z, mu = kmeans(Kt, C, T, init, mu0=None if mu0 is None else transform_keys(mu0, met["R"]))
    perm, off = stable_argsort(z, C)
    return {"labels": z, "perm": perm, "offsets": off, "mu": mu, "init": init,
            "Kt": Kt, **met}


def park_head(Q, K, V, CQ, CK, T, mode, param, seed=0, head=0, alpha=0.05, eps=1e-6,
              s_min=1e-12, estimator="pama", blocks="cluster", key_metric="qrkc"):
    """PARK forward of one head; returns every intermediate and O.

    estimator: "pama" (Eqs. (8)-(9)) or "qcentroid" (the query-centroid
    estimate, the "w/o PAMA" ablation).  blocks: "cluster" (block v is
    cluster v) or "fixed" (fixed chunks of the cluster-sorted order).
    key_metric: "qrkc" (Alg. 3) or "euclid" (the "w/o QRKC" ablation).
    """
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    cq = cluster_queries(Q, CQ, T, seed, head)
    if key_metric == "qrkc":
        ck = cluster_keys(K, Q, CK, T, seed, head, alpha, eps, s_min)
    else:
        init = init_indices(K.shape[0], CK, seed, head, side=1)
        z, mu = kmeans(K, CK, T, init)
        perm, off = stable_argsort(z, CK)
        ck = {"labels": z, "perm": perm, "offsets": off, "mu": mu, "init": init}
    if blocks == "fixed":
        cq = {**cq, "offsets": fixed_tile_offsets(Q.shape[0], CQ)}
        ck = {**ck, "offsets": fixed_tile_offsets(K.shape[0], CK)}
    elif blocks != "cluster":
        raise ValueError(blocks)
    Qp, Kp, Vp = Q[cq["perm"]], K[ck["perm"]], V[ck["perm"]]
    c, n = block_centroids(Kp, ck["offsets"])
    if estimator == "pama":
        W = pama(Qp, cq["offsets"], c, n)
    elif estimator == "qcentroid":
        W = query_centroid_estimate(Qp, cq["offsets"], c, n)
    else:
        raise ValueError(estimator)
    rows = select(W, np.diff(cq["offsets"]), n, mode, param)
    O = block_sparse_attention(Qp, Kp, Vp, cq["offsets"], ck["offsets"], rows, cq["perm"])
    return {"q": cq, "k": ck, "Qp": Qp, "Kp": Kp, "Vp": Vp, "centroids": c, "sizes": n,
            "W": W, "rows": rows, "O": O}


# --------------------------------------------------------------------------
# diagnostics of Secs. 3.2 / App. A (used as checks, not on the hot path)
# --------------------------------------------------------------------------
def exact_block_importance(Qp, Kp, q_offsets, k_offsets) -> np.ndarray:
    """W_uv = (1/n_u) sum_{i in Q_u} sum_{j in K_v} A_ij  (Eq. (3))."""
    A = softmax_rows((np.asarray(Qp, np.float64) @ np.asarray(Kp, np.float64).T)
                     / math.sqrt(Qp.shape[1]))
    CQ, CK = len(q_offsets) - 1, len(k_offsets) - 1
    W = np.zeros((CQ, CK))
    for u in range(CQ):
        a, b = q_offsets[u], q_offsets[u + 1]
        if b == a:
            continue
        for v in range(CK):
            W[u, v] = A[a:b, k_offsets[v]:k_offsets[v + 1]].sum() / (b - a)
    return W


def recall(Qp, Kp, q_offsets, k_offsets, rows) -> float:
    """Attention recall sum(A * M) / sum(A) of a block mask (Eq. (4))."""
    A = softmax_rows((np.asarray(Qp, np.float64) @ np.asarray(Kp, np.float64).T)
                     / math.sqrt(Qp.shape[1]))
    kept = 0.0
    for u, sel in enumerate(rows):
        a, b = q_offsets[u], q_offsets[u + 1]
        for v in sel:
            kept += A[a:b, k_offsets[v]:k_offsets[v + 1]].sum()
    return kept / A.sum()


def exact_log_mass(Qp, Kp, k_offsets) -> np.ndarray:
    """S*_iv = log sum_{j in K_v} exp(q_i . k_j / sqrt(d))  (Eq. (6))."""
    Z = (np.asarray(Qp, np.float64) @ np.asarray(Kp, np.float64).T) / math.sqrt(Qp.shape[1])
    CK = len(k_offsets) - 1
    S = np.full((Z.shape[0], CK), -np.inf)
    for v in range(CK):
        a, b = k_offsets[v], k_offsets[v + 1]
        if b > a:
            m = Z[:, a:b].max(axis=1)
            S[:, v] = m + np.log(np.exp(Z[:, a:b] - m[:, None]).sum(axis=1))
    return S


# --------------------------------------------------------------------------
# mismatch diagnostics (App. A "Direct Evaluation of Retrieval Mismatches",
# App. B "Key-Space and QK-Score Approximation Errors"); reported on
# synthetic layers, never on the hot path
# --------------------------------------------------------------------------
def block_means(Kp, offsets) -> np.ndarray:
    """Float64 mean of the keys of every block (0 for an empty block)."""
    Kp = np.asarray(Kp, dtype=np.float64)
    C = len(offsets) - 1
    c = np.zeros((C, Kp.shape[1]))
    for v in range(C):
        a, b = int(offsets[v]), int(offsets[v + 1])
        if b > a:
            c[v] = Kp[a:b].sum(axis=0) / (b - a)
    return c


def tv_error(W_hat, W, q_sizes) -> float:
    """Attention-weight TV error of one head (App. A, M1).

    E_TV = sum_u (n_u / L) * (1/2) sum_v |W^_uv - W_uv|: the total-variation
    distance between the estimated and the exact block-weight distribution of
    each query block, weighted by the block's share of the L queries.
    """
    W_hat = np.asarray(W_hat, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    n = np.asarray(q_sizes, dtype=np.float64)
    L = n.sum()
    per_block = 0.5 * np.abs(W_hat - W).sum(axis=1)
    return float((n / L * per_block).sum())


def centred_log_mass_rmse(S_star, S_hat) -> float:
    """Mean centred log-mass RMSE of one head (App. A, M2).

    Delta_iv = S*_iv - S^_iv on the nonempty key blocks (the columns where
    S* is finite); delta_iv = Delta_iv minus its mean over those blocks (a
    per-query offset does not change a softmax); E_LM = (1/L) sum_i
    sqrt(mean_v delta_iv^2).
    """
    S_star = np.asarray(S_star, dtype=np.float64)
    S_hat = np.asarray(S_hat, dtype=np.float64)
    valid = np.isfinite(S_star[0])
    Delta = S_star[:, valid] - S_hat[:, valid]
    delta = Delta - Delta.mean(axis=1, keepdims=True)
    return float(np.sqrt((delta ** 2).mean(axis=1)).mean())


def log_mass_estimate(Qp, c, n) -> np.ndarray:
    """S^_iv = q_i . c_v / sqrt(d) + log n_v with float64 centroids c (Eq. (8));
    -inf for an empty block."""
    Qp = np.asarray(Qp, dtype=np.float64)
    S = (Qp @ np.asarray(c, dtype=np.float64).T) / math.sqrt(Qp.shape[1])
    n = np.asarray(n)
    with np.errstate(divide="ignore"):
        logn = np.where(n > 0, np.log(np.maximum(n, 1).astype(np.float64)), -np.inf)
    return S + logn[None, :]


def key_space_errors(K, Q, labels, c):
    """Raw-key MSE and QK-score squared error of a key clustering (App. B).

    D_key = (1/L_K) sum_j |k_j - c_v(j)|^2 (not divided by d);
    D_QK = (1/(L_Q L_K)) sum_i sum_j [q_i . (k_j - c_v(j)) / sqrt(d)]^2.
    ``c`` are the clusters' centroids in the original key space.  Returns
    (D_key, D_QK); the double sum is taken over query chunks.
    """
    K = np.asarray(K, dtype=np.float64)
    Q = np.asarray(Q, dtype=np.float64)
    R = K - np.asarray(c, dtype=np.float64)[np.asarray(labels)]
    Lk, d = K.shape
    Lq = Q.shape[0]
    d_key = float((R ** 2).sum() / Lk)
    tot = 0.0
    for a in range(0, Lq, 512):
        E = (Q[a:a + 512] @ R.T) / math.sqrt(d)
        tot += float((E ** 2).sum())
    return d_key, tot / (Lq * Lk)


def query_centroid_full_keys(Qp, q_offsets, Kp, k_offsets) -> np.ndarray:
    """W^_uv = phi_v(qbar_u) with every original key (App. A, the query-centroid
    error with full keys): the block's mean query attends over all keys and
    the weights of each key block are summed.  Rows of empty query blocks are
    zero."""
    Qp = np.asarray(Qp, dtype=np.float64)
    Kp = np.asarray(Kp, dtype=np.float64)
    CQ, CK = len(q_offsets) - 1, len(k_offsets) - 1
    W = np.zeros((CQ, CK))
    for u in range(CQ):
        a, b = int(q_offsets[u]), int(q_offsets[u + 1])
        if b == a:
            continue
        qbar = Qp[a:b].sum(axis=0) / (b - a)
        p = softmax_rows((qbar[None, :] @ Kp.T) / math.sqrt(Qp.shape[1]))[0]
        for v in range(CK):
            W[u, v] = p[int(k_offsets[v]):int(k_offsets[v + 1])].sum()
    return W


def mismatch_report(Q, K, CQ, CK, T, seed=0, head=0, alpha=0.05, eps=1e-6, s_min=1e-12):
    """The App. A / App. B diagnostics of one head on given Q, K.

    M1: Euclidean query and key partitions; TV of PAMA (per-query), of the
    query-centroid estimate, and of the query centroid with full keys, each
    against the exact block importance (Eq. (3)).  M2: all original queries;
    centred log-mass RMSE under the Euclidean and the QRKC key partition,
    each against the exact log-mass of its own partition (Eq. (6)).  App. B:
    D_key and D_QK of both key partitions.  Everything in float64.
    """
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    N = Q.shape[0]
    cq = cluster_queries(Q, CQ, T, seed, head)
    ke = kmeans(K, CK, T, init_indices(N, CK, seed, head, side=1))[0]
    kq = cluster_keys(K, Q, CK, T, seed, head, alpha, eps, s_min)["labels"]
    out = {}
    # M1 on the Euclidean partitions
    Qp = Q[cq["perm"]]
    perm_e, off_e = stable_argsort(ke, CK)
    Kp = K[perm_e]
    c = block_means(Kp, off_e)
    n = np.diff(off_e)
    W_exact = exact_block_importance(Qp, Kp, cq["offsets"], off_e)
    qs = np.diff(cq["offsets"])
    S_hat = log_mass_estimate(Qp, c, n)
    W_per = np.zeros_like(W_exact)
    W_cen = np.zeros_like(W_exact)
    for u in range(CQ):
        a, b = int(cq["offsets"][u]), int(cq["offsets"][u + 1])
        if b > a:
            W_per[u] = softmax_rows(S_hat[a:b]).sum(axis=0) / (b - a)
            qbar = Qp[a:b].sum(axis=0) / (b - a)
            W_cen[u] = softmax_rows(log_mass_estimate(qbar[None, :], c, n))[0]
    W_full = query_centroid_full_keys(Qp, cq["offsets"], Kp, off_e)
    out["tv_per_query"] = tv_error(W_per, W_exact, qs)
    out["tv_query_centroid"] = tv_error(W_cen, W_exact, qs)
    out["tv_query_centroid_full_keys"] = tv_error(W_full, W_exact, qs)
    # M2 and App. B for both key partitions
    for name, z in (("euclid", ke), ("qrkc", kq)):
        perm, off = stable_argsort(z, CK)
        Kp = K[perm]
        c = block_means(Kp, off)
        out[f"log_mass_rmse_{name}"] = centred_log_mass_rmse(
            exact_log_mass(Q, Kp, off), log_mass_estimate(Q, c, np.diff(off)))
        d_key, d_qk = key_space_errors(K, Q, z, c)
        out[f"d_key_{name}"] = d_key
        out[f"d_qk_{name}"] = d_qk
    return out
