"""Non-finite inputs: every kernel finishes normally, park_check reports
PARK_ERR_NUMERIC, and the next call on the same workspace starts clean.

Traced through the kernels before running: a non-finite token gets no fast
label (its scores are NaN or infinite), is refined against every centroid,
gets label 0 with the non-finite status raised; a non-finite centroid never
wins a comparison; non-finite block weights rank as 0 in the selection, and
every index read from the mask is bounds-checked."""
import numpy as np
import pytest
import torch

import parity as PT
from oracle import park_oracle as O
from paper_2609_38978_amd import park as P
from paper_2609_38978_amd import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,where,value", [("medium", "q", np.nan), ("medium", "k", np.inf),
                                              ("tiny", "q", -np.inf), ("tiny", "k", np.nan)])
def test_nonfinite_input_is_reported(name, where, value):
    cfg = synth.CONFIGS[name].with_(grid=(2, 16, 32))
    q, k, v = synth.make_layer(cfg, [0, 1])
    C = cfg.C
    prm = P.make_params(C, C, T=3, select="topk", ratio=0.25)
    print(f"[nonfinite {name} {where}={value}] N={cfg.N} C={C}", flush=True)
    bad_q, bad_k = q.copy(), k.copy()
    (bad_q if where == "q" else bad_k)[1, 37, 5] = value
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (bad_q, bad_k, v))
    ws = P.workspace(Q, C, C)
    out, st = P.park_forward(Q, K, V, prm, ws=ws)
    with pytest.raises(P.ParkError) as e:
        P.park_check(ws)
    assert e.value.status == P.PARK_ERR_NUMERIC
    assert "non-finite" in str(e.value)
    # labels stayed in range: the permutation and offsets are well formed
    for h in range(2):
        for side in ("q", "k"):
            perm = st[f"{side}_perm"][h].cpu().numpy()
            off = st[f"{side}_offsets"][h].cpu().numpy()
            assert np.array_equal(np.sort(perm), np.arange(cfg.N))
            assert off[0] == 0 and off[-1] == cfg.N and np.all(np.diff(off) >= 0)
        kvc = st["kv_count"][h].cpu().numpy()
        assert np.all((kvc >= 0) & (kvc <= C))
    # the clean head is unaffected and matches the oracle
    ref = O.park_head(q[0], k[0], v[0], C, C, 3, "topk", 0.25, seed=0, head=0)
    assert np.array_equal(st["q_perm"][0].cpu().numpy(), ref["q"]["perm"])
    assert np.array_equal(st["k_perm"][0].cpu().numpy(), ref["k"]["perm"])
    # the next call on the same workspace starts with a clear status
    Q2, K2 = PT.to_dev(q, cfg.dtype), PT.to_dev(k, cfg.dtype)
    P.park_forward(Q2, K2, V, prm, state=st, ws=ws)
    P.park_check(ws)
    torch.cuda.synchronize()
