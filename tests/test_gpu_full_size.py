"""GPU parity at the full layer sizes.

The GPU runs the whole layer (every head) in the launch configuration the
benchmark uses; the oracle recomputes a sample of heads end to end.  Heads are
independent, so a sampled head is checked exactly as if it were run alone.
"""
import numpy as np
import pytest
import torch

import parity as PT
from oracle import park_oracle as O
from paper_2609_38978_amd import park as P
from paper_2609_38978_amd import synth

pytestmark = pytest.mark.gpu


def run_layer(cfg, mode, param, T=None, out_dtype=P.PARK_BF16, block=None):
    cfg = cfg if block is None else cfg.with_(block=block)
    q, k, v = synth.make_layer(cfg)
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (q, k, v))
    C = cfg.C
    T = cfg.iters if T is None else T
    prm = P.make_params(C, C, T=T, select=mode, ratio=param, topp=param, seed=0,
                        out_dtype=out_dtype)
    ws = P.workspace(Q, C, C)
    st = P.make_state(Q, C, C)
    Og, st = P.park_forward(Q, K, V, prm, state=st, ws=ws)
    P.park_check(ws)
    torch.cuda.synchronize()
    return cfg, C, T, q, k, v, Og, st


def check_head(tag, h, cfg, C, T, mode, param, q, k, v, Og, st, out_dtype):
    qh, kh, vh = q[h], k[h], v[h]
    # clustering: labels equal to the oracle's up to near-ties
    rq = O.cluster_queries(qh, C, T, 0, h)
    rk = O.cluster_keys(kh, qh, C, T, 0, h)
    qperm = st["q_perm"][h].cpu().numpy()
    kperm = st["k_perm"][h].cpu().numpy()
    qoff = st["q_offsets"][h].cpu().numpy()
    koff = st["k_offsets"][h].cpu().numpy()
    zq = np.empty(len(qperm), np.int64)
    zk = np.empty(len(kperm), np.int64)
    for u in range(C):
        zq[qperm[qoff[u]:qoff[u + 1]]] = u
        zk[kperm[koff[u]:koff[u + 1]]] = u
    nq, bq, wq = PT.label_flips(qh.astype(np.float64), rq["mu"], zq, rq["labels"])
    nk, bk, wk = PT.label_flips(rk["Kt"], rk["mu"], zk, rk["labels"])
    print(f"[{tag} h={h}] label mismatches q={nq} (not exempt {bq}) k={nk} (not exempt {bk})")
    assert bq == 0 and bk == 0
    # the permutation is the stable argsort of the labels
    p2, o2 = O.stable_argsort(zq, C)
    assert np.array_equal(p2, qperm) and np.array_equal(o2, qoff)
    p2, o2 = O.stable_argsort(zk, C)
    assert np.array_equal(p2, kperm) and np.array_equal(o2, koff)
    # downstream stages on the GPU's own clustering
    Qp, Kp, Vp = qh[qperm], kh[kperm], vh[kperm]
    c, n = O.block_centroids(Kp, koff)
    cg = st["k_centroids"][h].cpu().numpy()
    assert np.array_equal(st["k_sizes"][h].cpu().numpy(), n)
    assert np.all(np.abs(cg - c) <= np.spacing(np.abs(c)))
    W = O.pama(Qp, qoff, c, n)
    kvc = st["kv_count"][h].cpu().numpy()
    kvi = st["kv_index"][h].cpu().numpy()
    nd, nb = PT.compare_masks(W, n, np.diff(qoff), mode, param, kvc, kvi)
    print(f"[{tag} h={h}] mask rows differing={nd} not-exempt={nb}; "
          f"mean kept blocks={kvc[np.diff(qoff) > 0].mean():.1f}")
    assert nb == 0
    # attention on a sample of query blocks (every size class: the largest,
    # the smallest nonempty, and random ones), each computed by the oracle
    sizes = np.diff(qoff)
    nonempty = np.nonzero(sizes)[0]
    rng = np.random.default_rng(h)
    sample = set(rng.choice(nonempty, size=min(48, len(nonempty)), replace=False).tolist())
    sample |= {int(nonempty[np.argmax(sizes[nonempty])]), int(nonempty[np.argmin(sizes[nonempty])])}
    rows = PT.rows_from_csr(kvc, kvi)
    Oh = PT.np64(Og[h])
    worst = 0.0
    for u in sorted(sample):
        a, b = qoff[u], qoff[u + 1]
        ref = O.block_sparse_attention(Qp[a:b], Kp, Vp, np.array([0, b - a]), koff, [rows[u]],
                                       np.arange(b - a))
        got = Oh[qperm[a:b]]
        err = np.abs(got - ref)
        worst = max(worst, float(err.max()))
        assert np.all(err <= PT.attn_tol(cfg.dtype, out_dtype == P.PARK_BF16, ref)), (tag, h, u)
    print(f"[{tag} h={h}] attention max-abs err over {len(sample)} query blocks {worst:.3g}")


@pytest.mark.parametrize("name,heads", [("wan", (0, 39)), ("hunyuan", (23,))])
def test_full_layer_sampled_heads(name, heads):
    base = synth.CONFIGS[name]
    mode = base.select
    param = base.ratio if mode == "topk" else base.topp
    cfg, C, T, q, k, v, Og, st = run_layer(base, mode, param)
    for h in heads:
        check_head(name, h, cfg, C, T, mode, param, q, k, v, Og, st, P.PARK_BF16)


@pytest.mark.parametrize("block,T,p", [(128, 5, 0.8), (64, 20, 0.95)])
def test_wan_sweep_points(block, T, p):
    base = synth.CONFIGS["wan_sweep"]
    cfg, C, T, q, k, v, Og, st = run_layer(base, "topp", p, T=T, block=block)
    check_head(f"sweep B={block} T={T} p={p}", cfg.H // 2, cfg, C, T, "topp", p, q, k, v, Og,
               st, P.PARK_BF16)
