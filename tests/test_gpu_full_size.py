"""GPU parity at the full layer sizes.

The GPU runs the whole layer (every head) in the launch configuration the
benchmark uses; the oracle recomputes a sample of heads.  Heads are
independent, so a sampled head is checked exactly as if it were run alone.
Oracle clusterings are cached per (layer, block size, iterations, head): the
selection sweep and the output dtypes reuse them.
"""
import functools
import os

import numpy as np
import pytest
import torch

import parity as PT
from oracle import park_oracle as O
from paper_2609_38978_amd import park as P
from paper_2609_38978_amd import synth

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=2)
def layer(name):
    cfg = synth.CONFIGS[name]
    print(f"[{name}] generating H={cfg.H} N={cfg.N}", flush=True)
    q, k, v = synth.make_layer(cfg, workers=16)
    return q, k, v


@functools.lru_cache(maxsize=4)
def device_layer(name):
    cfg = synth.CONFIGS[name]
    return tuple(PT.to_dev(a, cfg.dtype) for a in layer(name))


@functools.lru_cache(maxsize=64)
def oracle_clusters(name, block, T, h):
    q, k, _ = layer(name)
    C = synth.CONFIGS[name].with_(block=block).C
    print(f"[oracle] {name} B={block} T={T} head {h}: k-means of both sides", flush=True)
    return O.cluster_queries(q[h], C, T, 0, h), O.cluster_keys(k[h], q[h], C, T, 0, h)


def run_layer(name, mode, param, T=None, out_dtype=P.PARK_BF16, block=None, Q=None, K=None):
    cfg = synth.CONFIGS[name]
    cfg = cfg if block is None else cfg.with_(block=block)
    Qd, Kd, Vd = device_layer(name)
    Q = Qd if Q is None else Q
    K = Kd if K is None else K
    C = cfg.C
    T = cfg.iters if T is None else T
    prm = P.make_params(C, C, T=T, select=mode, ratio=param, topp=param, seed=0,
                        out_dtype=out_dtype)
    ws = P.workspace(Q, C, C)
    st = P.make_state(Q, C, C)
    Og, st = P.park_forward(Q, K, Vd, prm, state=st, ws=ws)
    P.park_check(ws)
    torch.cuda.synchronize()
    return cfg, C, T, Og, st, prm, ws


def labels_of(perm, off):
    z = np.empty(len(perm), np.int64)
    for u in range(len(off) - 1):
        z[perm[off[u]:off[u + 1]]] = u
    return z


def check_clustering(tag, name, cfg, C, T, h, st):
    q, k, _ = layer(name)
    rq, rk = oracle_clusters(name, cfg.block, T, h)
    qperm, kperm = st["q_perm"][h].cpu().numpy(), st["k_perm"][h].cpu().numpy()
    qoff, koff = st["q_offsets"][h].cpu().numpy(), st["k_offsets"][h].cpu().numpy()
    zq, zk = labels_of(qperm, qoff), labels_of(kperm, koff)
    nq, bq, _ = PT.label_flips(q[h].astype(np.float64), rq["mu"], zq, rq["labels"])
    nk, bk, _ = PT.label_flips(rk["Kt"], rk["mu"], zk, rk["labels"])
    print(f"[{tag} h={h}] label mismatches q={nq} (not exempt {bq}) k={nk} (not exempt {bk})",
          flush=True)
    assert bq == 0 and bk == 0
    # the permutation is the stable argsort of the labels
    for z, perm, off in ((zq, qperm, qoff), (zk, kperm, koff)):
        p2, o2 = O.stable_argsort(z, C)
        assert np.array_equal(p2, perm) and np.array_equal(o2, off)


def check_downstream(tag, cfg, C, mode, param, q, k, v, h, st, Og, out_dtype, nsample=48):
    """Centroids, mask and sampled attention of head h on the GPU's own clustering."""
    qperm, kperm = st["q_perm"][h].cpu().numpy(), st["k_perm"][h].cpu().numpy()
    qoff, koff = st["q_offsets"][h].cpu().numpy(), st["k_offsets"][h].cpu().numpy()
    Qp, Kp, Vp = q[qperm], k[kperm], v[kperm]
    c, n = O.block_centroids(Kp, koff)
    cg = st["k_centroids"][h].cpu().numpy()
    assert np.array_equal(st["k_sizes"][h].cpu().numpy(), n)
    assert np.all(np.abs(cg - c) <= np.spacing(np.abs(c)))
    W = O.pama(Qp, qoff, c, n)
    kvc = st["kv_count"][h].cpu().numpy()
    kvi = st["kv_index"][h].cpu().numpy()
    nd, nb = PT.compare_masks(W, n, np.diff(qoff), mode, param, kvc, kvi)
    print(f"[{tag} h={h}] mask rows differing={nd} not-exempt={nb}; "
          f"mean kept blocks={kvc[np.diff(qoff) > 0].mean():.1f}", flush=True)
    assert nb == 0
    # attention on a sample of query blocks (the largest, the smallest
    # nonempty and random ones), each computed by the oracle
    sizes = np.diff(qoff)
    nonempty = np.nonzero(sizes)[0]
    rng = np.random.default_rng(h)
    sample = set(rng.choice(nonempty, size=min(nsample, len(nonempty)), replace=False).tolist())
    sample |= {int(nonempty[np.argmax(sizes[nonempty])]), int(nonempty[np.argmin(sizes[nonempty])])}
    rows = PT.rows_from_csr(kvc, kvi)
    Oh = PT.np64(Og[h])
    worst = 0.0
    for u in sorted(sample):
        a, b = qoff[u], qoff[u + 1]
        ref = O.block_sparse_attention(Qp[a:b], Kp, Vp, np.array([0, b - a]), koff, [rows[u]],
                                       np.arange(b - a))
        err = np.abs(Oh[qperm[a:b]] - ref)
        worst = max(worst, float(err.max()))
        assert np.all(err <= PT.attn_tol(cfg.dtype, out_dtype == P.PARK_BF16, ref)), (tag, h, u)
    print(f"[{tag} h={h}] attention max-abs err over {len(sample)} query blocks {worst:.3g} "
          f"(output {'bf16' if out_dtype == P.PARK_BF16 else 'fp32, flat bar'})", flush=True)


def wan_scale_extremes():
    # the Wan-shaped layer scales Q by s_h ~ U[0.5, 2]: the heads with the
    # smallest and the largest scale (flattest and most peaked attention)
    q, _, _ = layer("wan")
    rms = np.sqrt((q[:, :4096] ** 2).mean(axis=(1, 2)))
    return int(np.argmin(rms)), int(np.argmax(rms))


@pytest.mark.parametrize("out_dtype", [P.PARK_BF16, P.PARK_F32])
@pytest.mark.parametrize("name", ["wan", "hunyuan"])
def test_full_layer_sampled_heads(name, out_dtype):
    base = synth.CONFIGS[name]
    mode = base.select
    param = base.ratio if mode == "topk" else base.topp
    heads = ((0, 39) + wan_scale_extremes()) if name == "wan" else (0, 11, 23)
    if os.environ.get("PARK_FULL_ALL_HEADS") == "1":
        heads = tuple(range(base.H))  # every head (an extended run, ~10 min per layer)
    cfg, C, T, Og, st, _, _ = run_layer(name, mode, param, out_dtype=out_dtype)
    q, k, v = layer(name)
    for h in dict.fromkeys(heads):
        check_clustering(name, name, cfg, C, T, h, st)
        check_downstream(name, cfg, C, mode, param, q[h], k[h], v[h], h, st, Og, out_dtype)


SWEEP = [(b, 10, p) for b in (64, 128) for p in (0.8, 0.9, 0.95)] + [(64, 5, 0.9), (64, 20, 0.9)]


@pytest.mark.parametrize("block,T,p", SWEEP)
def test_wan_sweep_points(block, T, p):
    tag = f"sweep B={block} T={T} p={p}"
    cfg, C, T, Og, st, _, _ = run_layer("wan", "topp", p, T=T, block=block)
    q, k, v = layer("wan")
    h = cfg.H // 2
    check_clustering(tag, "wan", cfg, C, T, h, st)
    check_downstream(tag, cfg, C, "topp", p, q[h], k[h], v[h], h, st, Og, P.PARK_BF16,
                     nsample=16)


def test_wan_reuse_modes():
    # the next denoising step (Q, K drifted by N(0, 0.05^2)) reusing the
    # clustering, then the clustering and the mask, of the recompute step
    name = "wan"
    cfg, C, T, Og, st, prm, ws = run_layer(name, "topp", 0.9)
    q, k, v = layer(name)
    q2, k2 = synth.perturb_layer(cfg, q, k, workers=16)
    Q2, K2 = PT.to_dev(q2, cfg.dtype), PT.to_dev(k2, cfg.dtype)
    _, _, Vd = device_layer(name)
    perm = (st["q_perm"].clone(), st["k_perm"].clone(), st["q_offsets"].clone(),
            st["k_offsets"].clone())
    O2, st = P.park_forward(Q2, K2, Vd, prm, reuse=P.PARK_REUSE_CLUSTERS, state=st, ws=ws)
    P.park_check(ws)
    assert all(torch.equal(a, b) for a, b in zip(perm, (st["q_perm"], st["k_perm"],
                                                         st["q_offsets"], st["k_offsets"])))
    for h in (0, 21):
        check_downstream("reuse clusters", cfg, C, "topp", 0.9, q2[h], k2[h], v[h], h, st, O2,
                         P.PARK_BF16, nsample=24)
    mask = (st["kv_count"].clone(), st["kv_index"].clone())
    # reuse the mask too, on the next step's tensors
    q3, k3 = np.empty_like(q2), np.empty_like(k2)
    for h in range(cfg.H):
        q3[h], k3[h] = synth.perturb_head(cfg, h, q2[h], k2[h], step=2)
    Q3, K3 = PT.to_dev(q3, cfg.dtype), PT.to_dev(k3, cfg.dtype)
    O3, st = P.park_forward(Q3, K3, Vd, prm, reuse=P.PARK_REUSE_CLUSTERS_AND_MASK, state=st,
                            ws=ws)
    P.park_check(ws)
    torch.cuda.synchronize()
    assert torch.equal(mask[0], st["kv_count"]) and torch.equal(mask[1], st["kv_index"])
    O3h = PT.np64(O3)
    for h in (0, 21):
        qperm, kperm = st["q_perm"][h].cpu().numpy(), st["k_perm"][h].cpu().numpy()
        qoff, koff = st["q_offsets"][h].cpu().numpy(), st["k_offsets"][h].cpu().numpy()
        rows = PT.rows_from_csr(st["kv_count"][h].cpu().numpy(), st["kv_index"][h].cpu().numpy())
        Qp, Kp, Vp = q3[h][qperm], k3[h][kperm], v[h][kperm]
        rng = np.random.default_rng(h)
        worst = 0.0
        for u in rng.choice(np.nonzero(np.diff(qoff))[0], size=24, replace=False):
            a, b = qoff[u], qoff[u + 1]
            ref = O.block_sparse_attention(Qp[a:b], Kp, Vp, np.array([0, b - a]), koff, [rows[u]],
                                           np.arange(b - a))
            err = np.abs(O3h[h][qperm[a:b]] - ref)
            worst = max(worst, float(err.max()))
            assert np.all(err <= PT.attn_tol(cfg.dtype, True, ref))
        print(f"[reuse clusters+mask h={h}] attention max-abs err {worst:.3g}", flush=True)
