"""End-to-end GPU parity of park_forward with the oracle's whole pipeline."""
import numpy as np
import pytest
import torch

import parity as PT
from oracle import park_oracle as O
from paper_2609_38978_amd import park as P
from paper_2609_38978_amd import synth

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": ("tiny", None, None, None),
    "medium": ("medium", None, [0, 3, 7], None),  # GPU runs 3 heads of the 8-head layer
    "ragged_topp": ("medium", (3, 11, 13), [0, 1], ("topp", 0.9)),
    "hunyuan_small_topk": ("hunyuan", (2, 9, 16), [0], None),
}


@pytest.mark.parametrize("tag", list(CASES))
@pytest.mark.parametrize("out_dtype", [P.PARK_F32, P.PARK_BF16])
def test_forward_matches_oracle(tag, out_dtype):
    name, grid, heads, sel = CASES[tag]
    cfg = synth.CONFIGS[name]
    if grid is not None:
        cfg = cfg.with_(grid=grid)
    mode, param = sel if sel else (cfg.select, cfg.ratio if cfg.select == "topk" else cfg.topp)
    q, k, v = synth.make_layer(cfg, heads)
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (q, k, v))
    C = cfg.C
    prm = P.make_params(C, C, T=cfg.iters, select=mode, ratio=param, topp=param, seed=0,
                        out_dtype=out_dtype)
    ws = P.workspace(Q, C, C)
    st = P.make_state(Q, C, C, want_W=True)
    Og, st = P.park_forward(Q, K, V, prm, state=st, ws=ws)
    P.park_check(ws)
    Og = PT.np64(Og)
    hs = heads if heads is not None else range(cfg.H)
    for i, h in enumerate(hs):
        ref = O.park_head(q[i], k[i], v[i], C, C, cfg.iters, mode, param, seed=0, head=i)
        qp = st["q_perm"][i].cpu().numpy()
        kp = st["k_perm"][i].cpu().numpy()
        same_q = np.array_equal(qp, ref["q"]["perm"])
        same_k = np.array_equal(kp, ref["k"]["perm"])
        print(f"[{tag} h={h}] q_perm equal={same_q} k_perm equal={same_k}")
        assert same_q and same_k
        kvc = st["kv_count"][i].cpu().numpy()
        kvi = st["kv_index"][i].cpu().numpy()
        nd, nb = PT.compare_masks(ref["W"], ref["sizes"], np.diff(ref["q"]["offsets"]), mode,
                                  param, kvc, kvi)
        print(f"[{tag} h={h}] mask rows differing={nd} not-exempt={nb}")
        assert nb == 0
        # attention on the GPU's own mask
        Oref = O.block_sparse_attention(ref["Qp"], ref["Kp"], ref["Vp"], ref["q"]["offsets"],
                                        ref["k"]["offsets"], PT.rows_from_csr(kvc, kvi),
                                        ref["q"]["perm"])
        tol = PT.attn_tol(cfg.dtype, out_dtype == P.PARK_BF16, Oref)
        err = np.abs(Og[i] - Oref)
        print(f"[{tag} h={h}] attention max-abs err {err.max():.3g}")
        assert np.all(err <= tol)
        ok, werr = PT.w_error_ok(cfg.dtype, st["W"][i].cpu().numpy(), ref["W"])
        print(f"[{tag} h={h}] W max-abs err {werr:.3g}")
        assert ok


def test_reuse_modes():
    cfg = synth.CONFIGS["medium"].with_(grid=(2, 16, 32))
    q, k, v = synth.make_layer(cfg, [0, 1])
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (q, k, v))
    C = cfg.C
    prm = P.make_params(C, C, T=5, select="topp", topp=0.9)
    ws = P.workspace(Q, C, C)
    O1, st = P.park_forward(Q, K, V, prm, ws=ws)
    perm_before = st["q_perm"].clone()
    mask_before = st["kv_index"].clone()
    # next diffusion step: drifted Q and K
    q2 = np.stack([synth.perturb_head(cfg, h, q[h], k[h])[0] for h in range(2)])
    k2 = np.stack([synth.perturb_head(cfg, h, q[h], k[h])[1] for h in range(2)])
    Q2, K2 = PT.to_dev(q2, cfg.dtype), PT.to_dev(k2, cfg.dtype)
    O2, st = P.park_forward(Q2, K2, V, prm, reuse=P.PARK_REUSE_CLUSTERS, state=st, ws=ws)
    P.park_check(ws)
    assert torch.equal(st["q_perm"], perm_before)
    O3, st = P.park_forward(Q2, K2, V, prm, reuse=P.PARK_REUSE_CLUSTERS_AND_MASK, state=st, ws=ws)
    P.park_check(ws)
    assert torch.equal(O2, O3)  # same clusters, same mask, same tensors
    for i in range(2):
        qp = st["q_perm"][i].cpu().numpy()
        kp = st["k_perm"][i].cpu().numpy()
        qoff = st["q_offsets"][i].cpu().numpy()
        koff = st["k_offsets"][i].cpu().numpy()
        c, n = O.block_centroids(k2[i][kp], koff)
        W = O.pama(q2[i][qp], qoff, c, n)
        kvc = st["kv_count"][i].cpu().numpy()
        kvi = st["kv_index"][i].cpu().numpy()
        nd, nb = PT.compare_masks(W, n, np.diff(qoff), "topp", 0.9, kvc, kvi)
        assert nb == 0
        Oref = O.block_sparse_attention(q2[i][qp], k2[i][kp], v[i][kp], qoff, koff,
                                        PT.rows_from_csr(kvc, kvi), qp)
        assert np.abs(PT.np64(O2)[i] - Oref).max() <= 2e-2


# Ablation variants and the fixed-tile block mode through park_forward:
# (config, grid override, heads, selection, estimator, block mode, key metric)
VARIANTS = {
    "qcentroid_tiny": ("tiny", None, None, None, "qcentroid", "cluster", "qrkc"),
    "qcentroid_medium_topp": ("medium", (2, 16, 32), [0, 5], ("topp", 0.9), "qcentroid",
                              "cluster", "qrkc"),
    "fixed_tiny": ("tiny", None, None, None, "pama", "fixed", "qrkc"),
    "fixed_ragged_topp": ("medium", (3, 11, 13), [0, 1], ("topp", 0.9), "pama", "fixed", "qrkc"),
    "fixed_qcentroid_hunyuan": ("hunyuan", (2, 9, 16), [0], None, "qcentroid", "fixed", "qrkc"),
    # 150 query blocks: two full 64-block tiles of the query-centroid kernel and a ragged 22
    "qcentroid_ragged_150": ("medium", (3, 20, 160), [3], ("topk", 0.2), "qcentroid", "cluster",
                             "qrkc"),
    "euclid_keys_medium": ("medium", (2, 16, 32), [1, 2], None, "pama", "cluster", "euclid"),
}


@pytest.mark.parametrize("tag", list(VARIANTS))
def test_forward_variants_match_oracle(tag):
    name, grid, heads, sel, est, blocks, metric = VARIANTS[tag]
    cfg = synth.CONFIGS[name]
    if grid is not None:
        cfg = cfg.with_(grid=grid)
    mode, param = sel if sel else (cfg.select, cfg.ratio if cfg.select == "topk" else cfg.topp)
    q, k, v = synth.make_layer(cfg, heads)
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (q, k, v))
    C = cfg.C
    prm = P.make_params(C, C, T=cfg.iters, select=mode, ratio=param, topp=param, seed=0,
                        out_dtype=P.PARK_F32,
                        estimator={"pama": P.PARK_EST_PAMA, "qcentroid": P.PARK_EST_QCENTROID}[est],
                        block_mode={"cluster": P.PARK_BLOCKS_CLUSTER,
                                    "fixed": P.PARK_BLOCKS_FIXED}[blocks],
                        key_metric={"qrkc": P.PARK_METRIC_QRKC,
                                    "euclid": P.PARK_METRIC_EUCLID}[metric])
    ws = P.workspace(Q, C, C)
    st = P.make_state(Q, C, C, want_W=True)
    Og, st = P.park_forward(Q, K, V, prm, state=st, ws=ws)
    P.park_check(ws)
    Og = PT.np64(Og)
    hs = heads if heads is not None else range(cfg.H)
    for i, h in enumerate(hs):
        print(f"[{tag} h={h}] N={cfg.N} C={C} {mode} {param}", flush=True)
        ref = O.park_head(q[i], k[i], v[i], C, C, cfg.iters, mode, param, seed=0, head=i,
                          estimator=est, blocks=blocks, key_metric=metric)
        assert np.array_equal(st["q_perm"][i].cpu().numpy(), ref["q"]["perm"])
        assert np.array_equal(st["k_perm"][i].cpu().numpy(), ref["k"]["perm"])
        assert np.array_equal(st["q_offsets"][i].cpu().numpy(), ref["q"]["offsets"])
        assert np.array_equal(st["k_offsets"][i].cpu().numpy(), ref["k"]["offsets"])
        assert np.array_equal(st["k_sizes"][i].cpu().numpy(), ref["sizes"])
        kvc = st["kv_count"][i].cpu().numpy()
        kvi = st["kv_index"][i].cpu().numpy()
        nd, nb = PT.compare_masks(ref["W"], ref["sizes"], np.diff(ref["q"]["offsets"]), mode,
                                  param, kvc, kvi)
        print(f"[{tag} h={h}] mask rows differing={nd} not-exempt={nb}")
        assert nb == 0
        Oref = O.block_sparse_attention(ref["Qp"], ref["Kp"], ref["Vp"], ref["q"]["offsets"],
                                        ref["k"]["offsets"], PT.rows_from_csr(kvc, kvi),
                                        ref["q"]["perm"])
        err = np.abs(Og[i] - Oref)
        print(f"[{tag} h={h}] attention max-abs err {err.max():.3g}")
        assert np.all(err <= PT.attn_tol(cfg.dtype, False, Oref))
        ok, werr = PT.w_error_ok(cfg.dtype, st["W"][i].cpu().numpy(), ref["W"])
        print(f"[{tag} h={h}] W max-abs err {werr:.3g}")
        assert ok


def test_schedule_drives_recompute_and_reuse():
    # a short denoising run with recomputation set {1, 3}: the mode of each
    # step comes from park_schedule_step; reused steps keep the clustering and
    # mask of the last recompute and match the oracle's attention on them
    cfg = synth.CONFIGS["medium"].with_(grid=(2, 16, 32))
    q, k, v = synth.make_layer(cfg, [0, 1])
    C = cfg.C
    prm = P.make_params(C, C, T=4, select="topp", topp=0.9)
    Q0, V = PT.to_dev(q, cfg.dtype), PT.to_dev(v, cfg.dtype)
    ws = P.workspace(Q0, C, C)
    st = P.make_state(Q0, C, C)
    sched = [1, 3]
    qs, ks = q, k
    last = None
    for step in range(5):
        mode = P.park_schedule_step(step, sched)
        print(f"[schedule] step {step} mode {mode}", flush=True)
        if step > 0:  # the next denoising step's drifted queries and keys (fresh drift per step)
            pq = [synth.perturb_head(cfg, h, qs[h], ks[h], step=step) for h in range(2)]
            qs = np.stack([a for a, _ in pq])
            ks = np.stack([b for _, b in pq])
        if mode == P.PARK_STEP_DENSE:
            assert step == 0
            continue
        Q, K = PT.to_dev(qs, cfg.dtype), PT.to_dev(ks, cfg.dtype)
        Og, st = P.park_forward(Q, K, V, prm, reuse=mode, state=st, ws=ws)
        P.park_check(ws)
        if mode == P.PARK_RECOMPUTE:
            last = (st["q_perm"].clone(), st["kv_index"].clone())
            continue
        assert mode == P.PARK_REUSE_CLUSTERS_AND_MASK and step in (2, 4)
        assert torch.equal(st["q_perm"], last[0]) and torch.equal(st["kv_index"], last[1])
        for i in range(2):
            qp = st["q_perm"][i].cpu().numpy()
            kp = st["k_perm"][i].cpu().numpy()
            Oref = O.block_sparse_attention(
                PT.np64(Q)[i][qp], PT.np64(K)[i][kp], v[i][kp], st["q_offsets"][i].cpu().numpy(),
                st["k_offsets"][i].cpu().numpy(),
                PT.rows_from_csr(st["kv_count"][i].cpu().numpy(), st["kv_index"][i].cpu().numpy()),
                qp)
            assert np.abs(PT.np64(Og)[i] - Oref).max() <= 2e-2


@pytest.mark.parametrize("name,grid,block", [("medium", (2, 16, 32), 64), ("medium", (2, 32, 64), 8)])
def test_warm_start_matches_oracle(name, grid, block):
    # a recomputation leaves the means of its final clusters in the state; the
    # next one (drifted Q, K) starts both k-means from them.  Block 8 puts the
    # layer above 512 clusters, where the rounds after the first are filtered.
    cfg = synth.CONFIGS[name].with_(grid=grid, block=block)
    q, k, v = synth.make_layer(cfg, [0, 1])
    C, T = cfg.C, 4
    print(f"[warm start N={cfg.N} C={C}]", flush=True)
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (q, k, v))
    prm = P.make_params(C, C, T=T, select="topp", topp=0.9)
    ws = P.workspace(Q, C, C)
    st = P.make_state(Q, C, C, want_mu=True)
    _, st = P.park_forward(Q, K, V, prm, state=st, ws=ws)
    P.park_check(ws)
    qmu, kmu = st["q_mu"].cpu().numpy(), st["k_mu"].cpu().numpy()
    for i in range(2):  # stored means: the means of the final clusters
        for X, side in ((q[i], "q"), (k[i], "k")):
            perm = st[f"{side}_perm"][i].cpu().numpy()
            off = st[f"{side}_offsets"][i].cpu().numpy()
            mu = (qmu if side == "q" else kmu)[i]
            for u in range(C):
                if off[u + 1] > off[u]:
                    want = X[perm[off[u]:off[u + 1]]].astype(np.float64).mean(0)
                    assert np.allclose(mu[u], want, rtol=1e-12, atol=1e-12), (side, u)
    # next step, warm-started from those means
    pq = [synth.perturb_head(cfg, h, q[h], k[h], step=1) for h in range(2)]
    q2, k2 = np.stack([a for a, _ in pq]), np.stack([b for _, b in pq])
    Q2, K2 = PT.to_dev(q2, cfg.dtype), PT.to_dev(k2, cfg.dtype)
    warm = P.make_params(C, C, T=T, select="topp", topp=0.9, init=P.PARK_INIT_WARM)
    Og, st = P.park_forward(Q2, K2, V, warm, state=st, ws=ws)
    P.park_check(ws)
    for i in range(2):
        rq = O.cluster_queries(q2[i], C, T, 0, i, mu0=qmu[i])
        rk = O.cluster_keys(k2[i], q2[i], C, T, 0, i, mu0=kmu[i])
        for side, r, X in (("q", rq, q2[i].astype(np.float64)), ("k", rk, rk["Kt"])):
            perm = st[f"{side}_perm"][i].cpu().numpy()
            off = st[f"{side}_offsets"][i].cpu().numpy()
            z = np.empty(cfg.N, np.int64)
            for u in range(C):
                z[perm[off[u]:off[u + 1]]] = u
            nm, nb, worst = PT.label_flips(X, r["mu"], z, r["labels"])
            print(f"[warm start h={i} {side}] label mismatches={nm} not-exempt={nb}", flush=True)
            assert nb == 0
            p2, o2 = O.stable_argsort(z, C)
            assert np.array_equal(p2, perm) and np.array_equal(o2, off)
        kvc = st["kv_count"][i].cpu().numpy()
        kvi = st["kv_index"][i].cpu().numpy()
        qp, kp = st["q_perm"][i].cpu().numpy(), st["k_perm"][i].cpu().numpy()
        qoff, koff = st["q_offsets"][i].cpu().numpy(), st["k_offsets"][i].cpu().numpy()
        Oref = O.block_sparse_attention(q2[i][qp], k2[i][kp], v[i][kp], qoff, koff,
                                        PT.rows_from_csr(kvc, kvi), qp)
        assert np.abs(PT.np64(Og)[i] - Oref).max() <= 2e-2
