"""GPU parity of each stage of the C ABI against the CPU oracle.

Every stage is fed the same inputs as the oracle stage (so an earlier
legitimate near-tie cannot cascade) and compared element by element.
"""
import math

import numpy as np
import pytest
import torch

import parity as PT
from oracle import park_oracle as O
from paper_2609_38978_amd import park as P
from paper_2609_38978_amd import synth

pytestmark = pytest.mark.gpu


def setup_module(module):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    P.lib()


def small(name, grid=None, heads=None, **kw):
    cfg = synth.CONFIGS[name]
    if grid is not None:
        cfg = cfg.with_(grid=grid)
    if kw:
        cfg = cfg.with_(**kw)
    q, k, v = synth.make_layer(cfg, heads)
    return cfg, q, k, v


CASES = {
    # name: (config, grid override, heads) -- sizes span several tiles plus a ragged tail
    "tiny": ("tiny", None, None),
    "medium2": ("medium", None, [0, 5]),
    "ragged_bf16": ("medium", (3, 11, 13), [1, 2, 3]),  # N = 429, not a multiple of 64
    "hunyuan_small": ("hunyuan", (1, 9, 16), [0, 1]),   # text tokens appended
    "tiny_bf16_d64": ("tiny", (2, 16, 32), None, {"dtype": "bf16"}),  # bf16 at head_dim 64
}


@pytest.fixture(scope="module", params=list(CASES))
def case(request):
    name, grid, heads, *kw = CASES[request.param]
    cfg, q, k, v = small(name, grid, heads, **(kw[0] if kw else {}))
    return request.param, cfg, q, k, v


def test_metric_factor_and_transform(case):
    tag, cfg, q, k, v = case
    Q, K = PT.to_dev(q, cfg.dtype), PT.to_dev(k, cfg.dtype)
    C = cfg.C
    out = P.park_cluster_keys(K, C, 1, seed=0, side=1, metric=P.PARK_METRIC_QRKC, Qmetric=Q,
                              want_R=True, want_Xt=True)
    P.park_check(out["ws"])
    R = out["R"].cpu().numpy()
    Xt = out["Xt"].cpu().numpy()
    for h in range(q.shape[0]):
        m = O.query_metric(q[h].astype(np.float64))
        assert np.abs(R[h] - m["R"]).max() <= 1e-12 * np.abs(m["R"]).max()
        ref = O.transform_keys(k[h], m["R"])
        err = np.abs(Xt[h].astype(np.float64) - ref)
        assert np.all(err <= 2.0 ** -23 * np.abs(ref) + 1e-30), (tag, err.max())


@pytest.mark.parametrize("side", [0, 1])
def test_kmeans_labels_permutation_offsets(case, side):
    tag, cfg, q, k, v = case
    Q, K = PT.to_dev(q, cfg.dtype), PT.to_dev(k, cfg.dtype)
    C, T = cfg.C, cfg.iters
    if side == 0:
        out = P.park_cluster_keys(Q, C, T, seed=7, side=0, metric=P.PARK_METRIC_EUCLID)
    else:
        out = P.park_cluster_keys(K, C, T, seed=7, side=1, metric=P.PARK_METRIC_QRKC, Qmetric=Q)
    P.park_check(out["ws"])
    lab = out["labels"].cpu().numpy()
    perm = out["perm"].cpu().numpy()
    off = out["offsets"].cpu().numpy()
    for h in range(q.shape[0]):
        if side == 0:
            res = O.cluster_queries(q[h], C, T, 7, h)
            X = q[h].astype(np.float64)
        else:
            res = O.cluster_keys(k[h], q[h], C, T, 7, h)
            X = res["Kt"]
        # init indices are generated independently on both sides
        n_mis, n_bad, worst = PT.label_flips(X, res["mu"], lab[h], res["labels"])
        print(f"[{tag} side={side} h={h}] label mismatches={n_mis} not-exempt={n_bad} "
              f"worst-gap={worst:.3g}")
        assert n_bad == 0
        if n_mis == 0:
            assert np.array_equal(perm[h], res["perm"])
            assert np.array_equal(off[h], res["offsets"])
        # permutation is the stable argsort of the GPU's own labels in any case
        p2, o2 = O.stable_argsort(lab[h], C)
        assert np.array_equal(perm[h], p2) and np.array_equal(off[h], o2)


def test_gather_and_centroids(case):
    tag, cfg, q, k, v = case
    K = PT.to_dev(k, cfg.dtype)
    H, N, d = k.shape
    C = cfg.C
    rng = np.random.default_rng(3)
    z = rng.integers(0, C, size=(H, N))
    z[:, z[0] == 1] = 2  # force an empty cluster
    perms, offs = zip(*[O.stable_argsort(z[h], C) for h in range(H)])
    perm = torch.from_numpy(np.stack(perms).astype(np.int32)).cuda()
    off = torch.from_numpy(np.stack(offs).astype(np.int32)).cuda()
    Kp = P.park_gather_rows(K, perm)
    assert torch.equal(Kp.cpu(), K.cpu()[torch.arange(H)[:, None], perm.cpu().long()])
    cen, sizes = P.park_block_centroids(K, perm, off, C)
    cen2, sizes2 = P.park_block_centroids(Kp, torch.arange(N, dtype=torch.int32).repeat(H, 1).cuda(),
                                          off, C)
    assert torch.equal(cen, cen2) and torch.equal(sizes, sizes2)
    cen, sizes = cen.cpu().numpy(), sizes.cpu().numpy()
    for h in range(H):
        c_o, n_o = O.block_centroids(k[h][perms[h]], offs[h])
        assert np.array_equal(sizes[h], n_o)
        # identical up to float64 summation order, then rounded to float32
        ulp = np.spacing(np.abs(c_o).astype(np.float32))
        assert np.all(np.abs(cen[h] - c_o) <= ulp), tag


@pytest.mark.parametrize("mode", ["topk", "topp"])
def test_retrieval_matches_oracle(case, mode):
    tag, cfg, q, k, v = case
    H, N, d = q.shape
    CQ = CK = cfg.C
    param = cfg.ratio if mode == "topk" else 0.9
    qps, qoffs, cens, ns, Ws = [], [], [], [], []
    for h in range(H):
        rq = O.cluster_queries(q[h], CQ, 3, 1, h)
        rk = O.cluster_keys(k[h], q[h], CK, 3, 1, h)
        c, n = O.block_centroids(k[h][rk["perm"]], rk["offsets"])
        Qp = q[h][rq["perm"]]
        qps.append(Qp)
        qoffs.append(rq["offsets"])
        cens.append(c)
        ns.append(n)
        Ws.append(O.pama(Qp, rq["offsets"], c, n))
    Qp = PT.to_dev(np.stack(qps), cfg.dtype)
    qoff = torch.from_numpy(np.stack(qoffs).astype(np.int32)).cuda()
    cen = torch.from_numpy(np.stack(cens)).cuda()
    ksz = torch.from_numpy(np.stack(ns).astype(np.int32)).cuda()
    sel = P.PARK_SELECT_TOPK if mode == "topk" else P.PARK_SELECT_TOPP
    kvc, kvi, W = P.park_retrieve_blocks(Qp, qoff, cen, ksz, CQ, CK, sel, param, want_W=True)
    kvc, kvi, W = kvc.cpu().numpy(), kvi.cpu().numpy(), W.cpu().numpy()
    # without W^ the top-k rows the bound cannot settle take the band path
    kvc2, kvi2, _ = P.park_retrieve_blocks(Qp, qoff, cen, ksz, CQ, CK, sel, param)
    kvc2, kvi2 = kvc2.cpu().numpy(), kvi2.cpu().numpy()
    for h in range(H):
        ok, werr = PT.w_error_ok(cfg.dtype, W[h], Ws[h])
        print(f"[{tag} {mode} h={h}] W max-abs err {werr:.3g}")
        assert ok, (tag, werr)
        qs = np.diff(qoffs[h])
        for kc, ki in ((kvc[h], kvi[h]), (kvc2[h], kvi2[h])):
            nd, nb = PT.compare_masks(Ws[h], ns[h], qs, mode, param, kc, ki)
            print(f"[{tag} {mode} h={h}] mask rows differing={nd} not-exempt={nb}")
            assert nb == 0
        # both paths give the same masks
        assert np.array_equal(kvc[h], kvc2[h])
        for u in range(CQ):
            assert np.array_equal(kvi[h][u, :kvc[h][u]], kvi2[h][u, :kvc2[h][u]]), (h, u)


@pytest.mark.parametrize("mode", ["topk", "topp"])
def test_retrieval_small_query_blocks(mode):
    # query blocks of 0-40 rows and a few of 100-300 (bf16): a wavefront's
    # two 32-query chunks often belong to different blocks, blocks end on
    # odd chunk counts, and empty blocks sit between them
    rng = np.random.default_rng(21)
    H, N, d, CQ, CK = 2, 3000, 128, 160, 96
    param = 0.2 if mode == "topk" else 0.9
    qps, qoffs, cens, ns, Ws = [], [], [], [], []
    for h in range(H):
        sizes = rng.choice([0, 1, 5, 17, 31, 33, 40, 150, 300], size=CQ,
                           p=[0.1, 0.1, 0.15, 0.15, 0.1, 0.1, 0.1, 0.1, 0.1]).astype(np.int64)
        while sizes.sum() > N:
            i = int(np.argmax(sizes))
            sizes[i] -= min(sizes[i], sizes.sum() - N)
        sizes[-1] += N - sizes.sum()
        off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
        Qp = synth.bf16_round(rng.standard_normal((N, d)).astype(np.float32) * 1.5)
        kz = rng.integers(0, CK, N)
        Kx = rng.standard_normal((N, d)).astype(np.float32)
        pk, ok = O.stable_argsort(kz, CK)
        c, n = O.block_centroids(Kx[pk], ok)
        qps.append(Qp)
        qoffs.append(off)
        cens.append(c)
        ns.append(n)
        Ws.append(O.pama(Qp, off, c, n))
    Qd = PT.to_dev(np.stack(qps), "bf16")
    qoff = torch.from_numpy(np.stack(qoffs).astype(np.int32)).cuda()
    cen = torch.from_numpy(np.stack(cens)).cuda()
    ksz = torch.from_numpy(np.stack(ns).astype(np.int32)).cuda()
    sel = P.PARK_SELECT_TOPK if mode == "topk" else P.PARK_SELECT_TOPP
    kvc, kvi, W = P.park_retrieve_blocks(Qd, qoff, cen, ksz, CQ, CK, sel, param, want_W=True)
    kvc2, kvi2, _ = P.park_retrieve_blocks(Qd, qoff, cen, ksz, CQ, CK, sel, param)
    kvc, kvi, W = kvc.cpu().numpy(), kvi.cpu().numpy(), W.cpu().numpy()
    kvc2, kvi2 = kvc2.cpu().numpy(), kvi2.cpu().numpy()
    for h in range(H):
        ok, werr = PT.w_error_ok("bf16", W[h], Ws[h])
        print(f"[small query blocks {mode} h={h}] W max-abs err {werr:.3g}")
        assert ok, werr
        qs = np.diff(qoffs[h])
        assert np.all(W[h][qs == 0] == 0.0)
        for kc, ki in ((kvc[h], kvi[h]), (kvc2[h], kvi2[h])):
            nd, nb = PT.compare_masks(Ws[h], ns[h], qs, mode, param, kc, ki)
            print(f"[small query blocks {mode} h={h}] mask rows differing={nd} not-exempt={nb}")
            assert nb == 0


@pytest.mark.parametrize("out_dtype", [P.PARK_F32, P.PARK_BF16])
def test_attention_matches_oracle(case, out_dtype):
    tag, cfg, q, k, v = case
    H, N, d = q.shape
    C = cfg.C
    rng = np.random.default_rng(11)
    qperm, kperm, qoff, koff, kvc, kvi, rows = [], [], [], [], [], [], []
    for h in range(H):
        zq = rng.integers(0, C, N)
        zk = rng.integers(0, C, N)
        zk[zk == 3] = 4  # an empty key block
        pq, oq = O.stable_argsort(zq, C)
        pk, ok = O.stable_argsort(zk, C)
        cnt = np.zeros(C, np.int32)
        idx = np.zeros((C, C), np.int32)
        rr = []
        for u in range(C):
            m = int(rng.integers(1, max(2, C // 3)))
            s = np.sort(rng.choice(C, size=m, replace=False))
            s = s[np.diff(ok)[s] > 0]  # selected blocks are nonempty
            if len(s) == 0:
                s = np.array([int(np.argmax(np.diff(ok)))])
            cnt[u] = len(s)
            idx[u, :len(s)] = s
            rr.append(s)
        qperm.append(pq); kperm.append(pk); qoff.append(oq); koff.append(ok)
        kvc.append(cnt); kvi.append(idx); rows.append(rr)
    t = lambda a: torch.from_numpy(np.stack(a).astype(np.int32)).cuda()
    Qp = PT.to_dev(np.stack([q[h][qperm[h]] for h in range(H)]), cfg.dtype)
    Kp = PT.to_dev(np.stack([k[h][kperm[h]] for h in range(H)]), cfg.dtype)
    Vp = PT.to_dev(np.stack([v[h][kperm[h]] for h in range(H)]), cfg.dtype)
    Ot, Lt = P.park_block_sparse_attn(Qp, Kp, Vp, t(qoff), t(koff), t(kvc), t(kvi), t(qperm), C,
                                      C, out_dtype, want_lse=True)
    Og = PT.np64(Ot)
    Lg = Lt.double().cpu().numpy()
    for h in range(H):
        args = (q[h][qperm[h]], k[h][kperm[h]])
        ref = O.block_sparse_attention(*args, v[h][kperm[h]], qoff[h], koff[h], rows[h], qperm[h])
        tol = PT.attn_tol(cfg.dtype, out_dtype == P.PARK_BF16, ref)
        err = np.abs(Og[h] - ref)
        print(f"[{tag} out={out_dtype} h={h}] attention max-abs err {err.max():.3g}")
        assert np.all(err <= tol), (tag, err.max())
        lref = O.block_sparse_lse(*args, qoff[h], koff[h], rows[h], qperm[h])
        ok, worst = PT.lse_ok(Lg[h], lref, PT.lse_tol(*args, qoff[h], koff[h], rows[h], qperm[h],
                                                      lref))
        print(f"[{tag} out={out_dtype} h={h}] lse worst err / bound {worst:.3g}")
        assert ok, (tag, worst)


@pytest.mark.parametrize("d", [64, 128])
def test_attention_many_small_query_blocks(d):
    # query blocks of 0-3 rows (a group of rows then holds more query blocks
    # than one selection word), a few large ones, and empty selections
    rng = np.random.default_rng(5)
    H, N, C = 2, 1500, 700
    q = rng.standard_normal((H, N, d)).astype(np.float32)
    k = rng.standard_normal((H, N, d)).astype(np.float32)
    v = rng.standard_normal((H, N, d)).astype(np.float32)
    q, k, v = (synth.bf16_round(a) for a in (q, k, v))
    qperm, kperm, qoff, koff, kvc, kvi, rows = [], [], [], [], [], [], []
    CK = 48
    for h in range(H):
        sizes = rng.choice([0, 1, 2, 3, 150], size=C, p=[0.2, 0.35, 0.25, 0.15, 0.05])
        sizes[-1] += N - sizes.sum() if sizes.sum() < N else 0
        while sizes.sum() > N:
            i = int(np.argmax(sizes)); sizes[i] -= min(sizes[i], sizes.sum() - N)
        zq = np.repeat(np.arange(C), sizes)
        zq = zq[rng.permutation(N)]
        zk = rng.integers(0, CK, N)
        pq, oq = O.stable_argsort(zq, C)
        pk, ok = O.stable_argsort(zk, CK)
        cnt = np.zeros(C, np.int32)
        idx = np.zeros((C, CK), np.int32)
        rr = []
        for u in range(C):
            m = int(rng.integers(0, 10))  # 0: an empty selection
            s = np.sort(rng.choice(CK, size=m, replace=False))
            cnt[u] = len(s)
            idx[u, :len(s)] = s
            rr.append(s)
        qperm.append(pq); kperm.append(pk); qoff.append(oq); koff.append(ok)
        kvc.append(cnt); kvi.append(idx); rows.append(rr)
    t = lambda a: torch.from_numpy(np.stack(a).astype(np.int32)).cuda()
    Qp = PT.to_dev(np.stack([q[h][qperm[h]] for h in range(H)]), "bf16")
    Kp = PT.to_dev(np.stack([k[h][kperm[h]] for h in range(H)]), "bf16")
    Vp = PT.to_dev(np.stack([v[h][kperm[h]] for h in range(H)]), "bf16")
    Ot, Lt = P.park_block_sparse_attn(Qp, Kp, Vp, t(qoff), t(koff), t(kvc), t(kvi), t(qperm), C,
                                      CK, P.PARK_F32, want_lse=True)
    Og = PT.np64(Ot)
    Lg = Lt.double().cpu().numpy()
    for h in range(H):
        # the oracle needs a selection per block: give the empty ones a
        # placeholder, then expect zero rows for them
        rr = [s if len(s) else np.array([0]) for s in rows[h]]
        ref = O.block_sparse_attention(q[h][qperm[h]], k[h][kperm[h]], v[h][kperm[h]], qoff[h],
                                       koff[h], rr, qperm[h])
        for u, s in enumerate(rows[h]):
            if len(s) == 0:
                ref[qperm[h][qoff[h][u]:qoff[h][u + 1]]] = 0.0
        tol = PT.attn_tol("bf16", False, ref)
        err = np.abs(Og[h] - ref)
        print(f"[small blocks d={d} h={h}] attention max-abs err {err.max():.3g}")
        assert np.all(err <= tol), err.max()
        # empty selections have lse = -inf
        args = (q[h][qperm[h]], k[h][kperm[h]])
        lref = O.block_sparse_lse(*args, qoff[h], koff[h], rows[h], qperm[h])
        ok, worst = PT.lse_ok(Lg[h], lref, PT.lse_tol(*args, qoff[h], koff[h], rows[h], qperm[h],
                                                      lref))
        print(f"[small blocks d={d} h={h}] lse worst err / bound {worst:.3g}")
        assert ok, worst


def test_attention_plan_selection_families():
    # query blocks drawn from a few families of nearly equal selections: the
    # plan's family of block u is the smallest v <= u with Jaccard(S_u, S_v)
    # > 1/2, the blocks of one family are neighbours in the plan's order, and
    # the output still matches the oracle
    rng = np.random.default_rng(11)
    H, N, d, CQ, CK = 2, 3000, 128, 90, 120
    q, k, v = (synth.bf16_round(rng.standard_normal((H, N, d)).astype(np.float32))
               for _ in range(3))
    qperm, kperm, qoff, koff, kvc, kvi, rows, fams = [], [], [], [], [], [], [], []
    for h in range(H):
        zq = rng.integers(0, CQ, N)
        zk = rng.integers(0, CK, N)
        pq, oq = O.stable_argsort(zq, CQ)
        pk, ok = O.stable_argsort(zk, CK)
        base = [rng.choice(CK, size=30, replace=False) for _ in range(6)]
        cnt = np.zeros(CQ, np.int32)
        idx = np.zeros((CQ, CK), np.int32)
        rr, sets = [], []
        for u in range(CQ):
            s = set(base[int(rng.integers(0, 6))].tolist())
            drop = rng.choice(sorted(s), size=int(rng.integers(0, 12)), replace=False)
            s -= set(drop.tolist())
            s |= set(rng.choice(CK, size=int(rng.integers(0, 12)), replace=False).tolist())
            s = np.array(sorted(s))
            cnt[u] = len(s)
            idx[u, :len(s)] = s
            rr.append(s)
            sets.append(set(s.tolist()))
        fam = np.arange(CQ)
        for u in range(CQ):
            for w in range(u):
                inter = len(sets[u] & sets[w])
                if 3 * inter > len(sets[u]) + len(sets[w]):
                    fam[u] = w
                    break
        qperm.append(pq); kperm.append(pk); qoff.append(oq); koff.append(ok)
        kvc.append(cnt); kvi.append(idx); rows.append(rr); fams.append(fam)
    t = lambda a: torch.from_numpy(np.stack(a).astype(np.int32)).cuda()
    Qp = PT.to_dev(np.stack([q[h][qperm[h]] for h in range(H)]), "bf16")
    Kp = PT.to_dev(np.stack([k[h][kperm[h]] for h in range(H)]), "bf16")
    Vp = PT.to_dev(np.stack([v[h][kperm[h]] for h in range(H)]), "bf16")
    ws = P.workspace(Qp, CQ, CK)
    Ot = P.park_block_sparse_attn(Qp, Kp, Vp, t(qoff), t(koff), t(kvc), t(kvi), t(qperm), CQ, CK,
                                  P.PARK_F32, ws=ws)
    torch.cuda.synchronize()
    # plan layout after the 256-byte status region: order [H][CQ], row
    # prefix [H][CQ+1], groups int4 [H][GPH] (16-byte aligned), families [H][CQ]
    W = -(-N // 128)
    GPH = W + -(-(CQ + W) // 16) + 1
    goff = ((H * CQ + H * (CQ + 1)) * 4 + 15) & ~15
    raw = ws.cpu().numpy()[256:].view(np.uint8)
    order = raw[:H * CQ * 4].view(np.int32).reshape(H, CQ)
    fam_dev = raw[goff + H * GPH * 16:goff + H * GPH * 16 + H * CQ * 4].view(np.int32).reshape(H, CQ)
    Og = PT.np64(Ot)
    for h in range(H):
        assert np.array_equal(fam_dev[h], fams[h])
        lab = fams[h][fams[h]]
        seq = lab[order[h][order[h] >= 0]]
        # each label occupies one contiguous run of the order
        runs = [int(x) for i, x in enumerate(seq) if i == 0 or seq[i - 1] != x]
        assert len(runs) == len(set(runs)), runs
        ref = O.block_sparse_attention(q[h][qperm[h]], k[h][kperm[h]], v[h][kperm[h]], qoff[h],
                                       koff[h], rows[h], qperm[h])
        err = np.abs(Og[h] - ref)
        print(f"[families h={h}] {len(set(lab.tolist()))} families, attention max-abs err "
              f"{err.max():.3g}")
        assert np.all(err <= PT.attn_tol("bf16", False, ref)), err.max()


def test_dense_when_every_block_kept():
    cfg = synth.CONFIGS["tiny"]
    q, k, v = synth.make_layer(cfg)
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (q, k, v))
    prm = P.make_params(cfg.C, cfg.C, T=3, select="topk", ratio=1.0)
    O_, st = P.park_forward(Q, K, V, prm)
    torch.cuda.synchronize()
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).double(), torch.from_numpy(k).double(), torch.from_numpy(v).double())
    err = (O_.cpu().double() - ref).abs().max().item()
    assert err <= 1e-4, err
    assert (st["kv_count"] == (st["k_sizes"] > 0).sum(1, keepdim=True)).all()


def test_block_size_one_gives_exact_attention_mass():
    # C = N: singleton blocks; W^ equals the dense attention matrix
    cfg = synth.CONFIGS["tiny"].with_(grid=(1, 8, 24))  # N = 192
    q, k, v = synth.make_layer(cfg)
    N = q.shape[1]
    Q, K = PT.to_dev(q, "f32"), PT.to_dev(k, "f32")
    rq = P.park_cluster_keys(Q, N, 2, seed=0, side=0, metric=P.PARK_METRIC_EUCLID)
    rk = P.park_cluster_keys(K, N, 2, seed=0, side=1, metric=P.PARK_METRIC_QRKC, Qmetric=Q)
    assert torch.all(rq["offsets"][:, 1:] - rq["offsets"][:, :-1] == 1)
    Qp = P.park_gather_rows(Q, rq["perm"])
    cen, sz = P.park_block_centroids(K, rk["perm"], rk["offsets"], N)
    kvc, kvi, W = P.park_retrieve_blocks(Qp, rq["offsets"], cen, sz, N, N, P.PARK_SELECT_TOPP, 0.5,
                                         want_W=True)
    A = torch.softmax(torch.from_numpy(q[0]).double() @ torch.from_numpy(k[0]).double().T
                      / math.sqrt(q.shape[2]), dim=1).numpy()
    pq, pk = rq["perm"][0].cpu().numpy(), rk["perm"][0].cpu().numpy()
    err = np.abs(W[0].cpu().numpy() - A[np.ix_(pq, pk)])
    assert err.max() <= 1e-6


def test_forward_is_deterministic():
    cfg = synth.CONFIGS["medium"].with_(grid=(2, 16, 32))
    q, k, v = synth.make_layer(cfg, [0, 1])
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (q, k, v))
    prm = P.make_params(cfg.C, cfg.C, T=5, select="topp", topp=0.9, out_dtype=P.PARK_BF16)
    O1, s1 = P.park_forward(Q, K, V, prm)
    O2, s2 = P.park_forward(Q, K, V, prm)
    torch.cuda.synchronize()
    assert torch.equal(O1, O2)
    for key in ("q_perm", "k_perm", "kv_count", "k_centroids", "k_sizes"):
        assert torch.equal(s1[key], s2[key]), key
    # only the first kv_count entries of a kv_index row are defined
    kvc = s1["kv_count"].cpu()
    a, b = s1["kv_index"].cpu(), s2["kv_index"].cpu()
    for h in range(kvc.shape[0]):
        for u in range(kvc.shape[1]):
            n = int(kvc[h, u])
            assert torch.equal(a[h, u, :n], b[h, u, :n])


def test_duplicate_tokens_make_empty_clusters():
    cfg = synth.CONFIGS["tiny"].with_(grid=(1, 16, 16))
    q, k, v = synth.make_layer(cfg)
    q[:, 128:] = q[:, :1]  # half the tokens identical
    k[:, 128:] = k[:, :1]
    Q, K, V = (PT.to_dev(a, "f32") for a in (q, k, v))
    C = 32
    prm = P.make_params(C, C, T=4, select="topp", topp=0.9)
    O_, st = P.park_forward(Q, K, V, prm)
    torch.cuda.synchronize()
    res = O.park_head(q[0], k[0], v[0], C, C, 4, "topp", 0.9)
    assert np.array_equal(st["q_perm"][0].cpu().numpy(), res["q"]["perm"])
    assert np.array_equal(st["k_perm"][0].cpu().numpy(), res["k"]["perm"])
    assert (st["k_sizes"][0] == 0).any()
    err = np.abs(PT.np64(O_)[0] - res["O"]).max()
    assert err <= 1e-4


def test_numeric_failure_is_reported():
    # rank-deficient queries with no shrinkage: the metric is not positive definite
    H, N, d = 1, 256, 64
    Q = torch.zeros(H, N, d, device="cuda")
    Q[..., :3] = torch.randn(H, N, 3, device="cuda")
    K = torch.randn(H, N, d, device="cuda")
    # (only the Cholesky factor needs positive definiteness: ask for it)
    out = P.park_cluster_keys(K, 8, 2, side=1, metric=P.PARK_METRIC_QRKC, Qmetric=Q, alpha=0.0,
                              eps=0.0, want_R=True)
    with pytest.raises(P.ParkError) as ei:
        P.park_check(out["ws"])
    assert ei.value.status == P.PARK_ERR_NUMERIC
    # with the paper's shrinkage the same queries factorise fine
    out = P.park_cluster_keys(K, 8, 2, side=1, metric=P.PARK_METRIC_QRKC, Qmetric=Q)
    P.park_check(out["ws"])


@pytest.mark.parametrize("mode,param", [("topk", 0.3), ("topp", 0.7)])
def test_retrieval_exact_ties_take_the_float64_path(mode, param):
    # duplicated key blocks give exactly tied W^: the float bound cannot order
    # them, so those rows are recomputed in float64 and ties go to the lower id
    cfg = synth.CONFIGS["medium"].with_(grid=(2, 16, 32))
    q, k, v = synth.make_layer(cfg, [0])
    CQ = CK = cfg.C
    rq = O.cluster_queries(q[0], CQ, 3, 1, 0)
    rk = O.cluster_keys(k[0], q[0], CK, 3, 1, 0)
    c, n = O.block_centroids(k[0][rk["perm"]], rk["offsets"])
    for a_, b_ in ((0, 1), (2, 3), (4, 5), (6, 7)):
        c[b_] = c[a_]
        n[b_] = n[a_]
    Qp = q[0][rq["perm"]]
    Wo = O.pama(Qp, rq["offsets"], c, n)
    sel = P.PARK_SELECT_TOPK if mode == "topk" else P.PARK_SELECT_TOPP
    args = (PT.to_dev(Qp[None], "bf16"),
            torch.from_numpy(rq["offsets"][None].astype(np.int32)).cuda(),
            torch.from_numpy(c[None]).cuda(), torch.from_numpy(n[None].astype(np.int32)).cuda(),
            CQ, CK, sel, param)
    # with W^ asked for (float64 rows whole) and without (top-k: only the
    # band of ambiguous blocks in float64)
    for want_W in (True, False):
        kvc, kvi, W = P.park_retrieve_blocks(*args, want_W=want_W)
        kvc, kvi = kvc.cpu().numpy()[0], kvi.cpu().numpy()[0]
        nd, nb = PT.compare_masks(Wo, n, np.diff(rq["offsets"]), mode, param, kvc, kvi)
        assert nb == 0 and nd == 0, want_W


@pytest.mark.parametrize("sizes", [
    [700, 60, 240, 1, 299, 600, 50, 50],  # work items of 8 chunks: two rows split in two
    [150] + [10] * 63,                    # one item per chunk: a row of three items
    [0, 64, 65, 3000, 128],               # an empty block; 47 chunks cut into items of 16
], ids=["m8", "m1", "m16"])
def test_retrieval_float64_work_items(sizes):
    # every key block has an exact twin and k is odd, so the k-th and (k+1)-th
    # scores of every row tie: each query block goes through the float64 pass,
    # whose work items (whole chunks of 64 queries) are summed in item order
    rng = np.random.default_rng(11)
    d, CK = 128, 32
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N, CQ = int(offs[-1]), len(sizes)
    Qp = torch.from_numpy(rng.standard_normal((N, d)).astype(np.float32)).bfloat16().float().numpy()
    c = (0.3 * rng.standard_normal((CK, d))).astype(np.float32)
    n = rng.integers(1, 100, CK)
    c[1::2] = c[0::2]
    n[1::2] = n[0::2]
    Wo = O.pama(Qp, offs, c, n)
    param = 11 / 32  # k = 11
    kvc, kvi, W = P.park_retrieve_blocks(
        PT.to_dev(Qp[None], "bf16"), torch.from_numpy(offs[None].astype(np.int32)).cuda(),
        torch.from_numpy(c[None]).cuda(), torch.from_numpy(n[None].astype(np.int32)).cuda(),
        CQ, CK, P.PARK_SELECT_TOPK, param, want_W=True)
    W = W.cpu().numpy()[0]
    # float64 rows rounded once to float32: within one float32 ulp of the oracle
    ref = Wo.astype(np.float32)
    assert np.all(np.abs(W - ref) <= np.spacing(np.abs(ref))), np.abs(W - ref).max()
    nd, nb = PT.compare_masks(Wo, n, np.diff(offs), "topk", param, kvc.cpu().numpy()[0],
                              kvi.cpu().numpy()[0])
    assert nb == 0 and nd == 0


@pytest.mark.parametrize("mode,param", [("topk", 21 / 64), ("topp", 0.9)])
def test_retrieval_float64_normaliser_leaves_out_negligible_blocks(mode, param):
    # tight query blocks and long centroids spread each block's logits over
    # tens of nats, so most blocks of a row weigh far below 2^-33 / (n_u CK)
    # and the float64 pass leaves them out of its normalisers; twin blocks
    # send every row to that pass.  The left-out mass is below 2^-33 of each
    # normaliser, so the float64 rows still round to within one float32 ulp
    # of the oracle
    rng = np.random.default_rng(5)
    d, CK = 128, 64
    sizes = [700, 60, 240, 1, 299, 600, 50, 50, 0, 130]
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N, CQ = int(offs[-1]), len(sizes)
    mu = rng.standard_normal((CQ, d))
    q = mu[np.repeat(np.arange(CQ), sizes)] + 0.3 * rng.standard_normal((N, d))
    Qp = torch.from_numpy(q.astype(np.float32)).bfloat16().float().numpy()
    c = (30.0 * rng.standard_normal((CK, d))).astype(np.float32)
    n = rng.integers(1, 100, CK)
    n[7] = 0  # an empty block
    c[1::2] = c[0::2]
    n[1::2] = n[0::2]
    Wo = O.pama(Qp, offs, c, n)
    nu = np.diff(offs).astype(np.float64)
    small = (Wo * nu[:, None] * CK < 2.0 ** -34) & (n[None, :] > 0)
    live = nu > 0
    print(f"[{mode}] blocks below the drop threshold: {small[live].mean():.2f} of each row",
          flush=True)
    assert small[live].mean() > 0.3
    sel = P.PARK_SELECT_TOPK if mode == "topk" else P.PARK_SELECT_TOPP
    args = (PT.to_dev(Qp[None], "bf16"), torch.from_numpy(offs[None].astype(np.int32)).cuda(),
            torch.from_numpy(c[None]).cuda(), torch.from_numpy(n[None].astype(np.int32)).cuda(),
            CQ, CK, sel, param)
    for want_W in (True, False):
        kvc, kvi, W = P.park_retrieve_blocks(*args, want_W=want_W)
        if want_W:
            W = W.cpu().numpy()[0]
            ref = Wo.astype(np.float32)
            err = np.abs(W - ref)
            assert np.all(err <= np.spacing(np.abs(ref))), err.max()
        nd, nb = PT.compare_masks(Wo, n, nu, mode, param, kvc.cpu().numpy()[0],
                                  kvi.cpu().numpy()[0])
        assert nb == 0 and nd == 0, want_W


@pytest.mark.parametrize("dtype,N,d,C", [("fp32", 256, 64, 8), ("bf16", 2048, 128, 32)])
def test_rank_deficient_metric_clusters_like_the_square_root(dtype, N, d, C):
    # App. D: the symmetric square root realises the metric when Gbar is
    # rank deficient; the k-means (which uses Gbar's quadratic form) runs and
    # matches the oracle's square-root path label for label (up to exempt
    # near-ties).  Queries span three feature directions, no shrinkage.
    r = np.random.default_rng(11)
    q = np.zeros((1, N, d), dtype=np.float32)
    q[0, :, :3] = r.standard_normal((N, 3))
    k = (r.standard_normal((1, N, d)) * 2).astype(np.float32)
    Q, K = PT.to_dev(q, dtype), PT.to_dev(k, dtype)
    qh = PT.np64(Q)[0]
    kh = PT.np64(K)[0]
    T = 4
    print(f"[rank-deficient {dtype} N={N} d={d} C={C}]", flush=True)
    out = P.park_cluster_keys(K, C, T, seed=5, side=1, metric=P.PARK_METRIC_QRKC, Qmetric=Q,
                              alpha=0.0, eps=0.0)
    P.park_check(out["ws"])
    lab = out["labels"][0].cpu().numpy()
    res = O.cluster_keys(kh, qh, C, T, 5, 0, alpha=0.0, eps=0.0, realisation="sqrt")
    n_mis, n_bad, worst = PT.label_flips(res["Kt"], res["mu"], lab, res["labels"])
    print(f"label mismatches={n_mis} not-exempt={n_bad} worst-gap={worst:.3g}")
    assert n_bad == 0
    p2, o2 = O.stable_argsort(lab, C)
    assert np.array_equal(out["perm"][0].cpu().numpy(), p2)
    assert np.array_equal(out["offsets"][0].cpu().numpy(), o2)
    # and the whole layer runs on the same metric
    prm = P.make_params(C, C, T=T, select="topk", ratio=0.25, alpha=0.0, eps=0.0, seed=5)
    ws = P.workspace(Q, C, C)
    Og, st = P.park_forward(Q, K, K, prm, ws=ws)
    P.park_check(ws)
    assert np.array_equal(st["k_perm"][0].cpu().numpy(), out["perm"][0].cpu().numpy())


# App. D: the shrinkage alpha moves the key metric from the query-response
# metric (alpha = 0) to the isotropic one (alpha = 1).  Queries spread along
# two directions make the partitions differ along the sweep; C = 640 runs the
# candidate filter.  At alpha = 1 the partition is the Euclidean one.
@pytest.mark.parametrize("alpha,C", [(0.0, 64), (0.05, 64), (0.25, 64), (0.5, 64), (1.0, 64),
                                     (0.25, 640)])
def test_alpha_sweep_key_clustering_matches_oracle(alpha, C):
    r = np.random.default_rng(21)
    H, N, d, T = 2, 4096, 128, 5
    basis = np.linalg.qr(r.standard_normal((d, 2)))[0]
    q = 3.0 * r.standard_normal((H, N, 2)) @ basis.T + 0.05 * r.standard_normal((H, N, d))
    cent = 2.0 * r.standard_normal((48, d))
    k = cent[r.integers(0, 48, (H, N))] + 0.5 * r.standard_normal((H, N, d))
    Q, K = PT.to_dev(q.astype(np.float32), "bf16"), PT.to_dev(k.astype(np.float32), "bf16")
    qh, kh = PT.np64(Q), PT.np64(K)
    print(f"[alpha sweep alpha={alpha} N={N} C={C}]", flush=True)
    out = P.park_cluster_keys(K, C, T, seed=3, side=1, metric=P.PARK_METRIC_QRKC, Qmetric=Q,
                              alpha=alpha)
    P.park_check(out["ws"])
    for h in range(H):
        res = O.cluster_keys(kh[h], qh[h], C, T, 3, h, alpha=alpha)
        lab = out["labels"][h].cpu().numpy()
        n_mis, n_bad, worst = PT.label_flips(res["Kt"], res["mu"], lab, res["labels"])
        print(f"  head {h}: label mismatches={n_mis} not-exempt={n_bad} worst-gap={worst:.3g}")
        assert n_bad == 0
        p2, o2 = O.stable_argsort(lab, C)
        assert np.array_equal(out["perm"][h].cpu().numpy(), p2)
        assert np.array_equal(out["offsets"][h].cpu().numpy(), o2)
        if alpha == 1.0:
            # the Euclidean k-means of the raw keys from the same init
            ze, me = O.kmeans(kh[h], C, T, O.init_indices(N, C, 3, h, side=1))
            n_mis, n_bad, _ = PT.label_flips(kh[h], me, lab, ze)
            print(f"  head {h}: against Euclidean k-means mismatches={n_mis} not-exempt={n_bad}")
            assert n_bad == 0


# The exact candidate filter of the k-means rounds after the first runs where
# C >= 512; small layers with many clusters exercise it (and clusters with a
# single or no token, and centroids pulled far apart by the 2N(0,1) centres).
@pytest.mark.parametrize("name,grid,C,side", [("medium", (2, 32, 64), 600, 0),
                                              ("medium", (2, 32, 64), 600, 1),
                                              ("hunyuan", (2, 16, 32), 700, 1),
                                              ("medium", (1, 32, 32), 1024, 1)])
def test_kmeans_candidate_filter_matches_oracle_and_dense(name, grid, C, side):
    import os
    cfg = synth.CONFIGS[name].with_(grid=grid)
    q, k, _ = synth.make_layer(cfg, [0, 1])
    Q, K = PT.to_dev(q, cfg.dtype), PT.to_dev(k, cfg.dtype)
    T = 6
    print(f"[filter {name} N={cfg.N} C={C} side={side}]", flush=True)

    def run():
        if side == 0:
            o = P.park_cluster_keys(Q, C, T, seed=3, side=0, metric=P.PARK_METRIC_EUCLID)
        else:
            o = P.park_cluster_keys(K, C, T, seed=3, side=1, metric=P.PARK_METRIC_QRKC, Qmetric=Q)
        P.park_check(o["ws"])
        return o["labels"].cpu().numpy(), o["perm"].cpu().numpy(), o["offsets"].cpu().numpy()

    lab, perm, off = run()
    os.environ["PARK_KMEANS_FILTER"] = "0"
    try:
        lab_d, perm_d, off_d = run()
    finally:
        del os.environ["PARK_KMEANS_FILTER"]
    # radii measured every round instead of bounded from the previous round
    os.environ["PARK_KFILTER_EXACT_RADIUS"] = "1"
    try:
        lab_r, perm_r, off_r = run()
    finally:
        del os.environ["PARK_KFILTER_EXACT_RADIUS"]
    # the filter and its radii change which centroids are scored, never the labels
    for lb, pb, ob in ((lab_d, perm_d, off_d), (lab_r, perm_r, off_r)):
        assert np.array_equal(lab, lb) and np.array_equal(perm, pb)
        assert np.array_equal(off, ob)
    for h in range(2):
        if side == 0:
            res = O.cluster_queries(q[h], C, T, 3, h)
            X = q[h].astype(np.float64)
        else:
            res = O.cluster_keys(k[h], q[h], C, T, 3, h)
            X = res["Kt"]
        n_mis, n_bad, worst = PT.label_flips(X, res["mu"], lab[h], res["labels"])
        print(f"[filter h={h}] label mismatches={n_mis} not-exempt={n_bad} worst-gap={worst:.3g}; "
              f"empty clusters={int((np.diff(off[h]) == 0).sum())}", flush=True)
        assert n_bad == 0
        p2, o2 = O.stable_argsort(lab[h], C)
        assert np.array_equal(perm[h], p2) and np.array_equal(off[h], o2)
