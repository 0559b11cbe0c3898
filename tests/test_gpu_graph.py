"""park_forward captured in a HIP graph: every replay equals the eager result.

The forward launches only kernels on the caller's stream (no memsets, copies,
allocations or host synchronisation), so it can be captured.  Each replay is
separated by eager work and a synchronisation, and compared bit for bit with
the eager call on the same inputs.
"""
import numpy as np
import pytest
import torch

import parity as PT
from paper_2609_38978_amd import park as P
from paper_2609_38978_amd import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,grid,sel", [("medium", (2, 16, 32), "topk"),
                                           ("wan", (3, 9, 16), "topp")])
def test_forward_graph_replays_match_eager(name, grid, sel):
    cfg = synth.CONFIGS[name].with_(grid=grid)
    q, k, v = synth.make_layer(cfg, [0, 1, 2])
    Q, K, V = (PT.to_dev(a, cfg.dtype) for a in (q, k, v))
    C = cfg.C
    param = cfg.ratio if sel == "topk" else cfg.topp
    prm = P.make_params(C, C, T=cfg.iters, select=sel, ratio=param, topp=param, seed=0,
                        out_dtype=P.PARK_BF16)
    ws = P.workspace(Q, C, C)
    st = P.make_state(Q, C, C)
    out = torch.empty(Q.shape, dtype=torch.bfloat16, device="cuda")
    P.park_forward(Q, K, V, prm, state=st, out=out, ws=ws)
    P.park_check(ws)
    torch.cuda.synchronize()
    keys = ("q_perm", "k_perm", "q_offsets", "k_offsets", "k_sizes", "kv_count")
    ref = {n: st[n].clone() for n in keys}
    kvc = st["kv_count"].cpu().numpy()
    kvi_ref = st["kv_index"].cpu().numpy()
    O_ref = out.clone()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        P.park_forward(Q, K, V, prm, state=st, out=out, ws=ws)
    for rep in range(3):
        # eager work between replays: scribble over the outputs
        out.fill_(float("nan"))
        for n in keys:
            st[n].fill_(-7)
        st["kv_index"].fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        P.park_check(ws)
        print(f"[{name} replay {rep}] checking")
        assert torch.equal(out.view(torch.int16), O_ref.view(torch.int16)), rep
        for n in keys:
            assert torch.equal(st[n], ref[n]), (rep, n)
        kvi = st["kv_index"].cpu().numpy()
        H, CQ = kvc.shape
        for h in range(H):
            for u in range(CQ):
                assert np.array_equal(kvi[h, u, :kvc[h, u]], kvi_ref[h, u, :kvc[h, u]]), (rep, h, u)
    del graph
