"""park_block_sparse_attn_static (no workspace, static device scratch) against
park_block_sparse_attn (caller workspace): the same kernels, so O and lse must
be bit-identical; also within the oracle's bar.  Two calls in a row, the
second on a smaller input, so the scratch keeps the first call's plan when
the second starts."""
import ctypes as C

import numpy as np
import pytest
import torch

import parity as PT
from oracle import park_oracle as O
from paper_2609_38978_amd import park as P
from paper_2609_38978_amd import synth

pytestmark = pytest.mark.gpu


def _case(seed, H, N, CQ, CK, d):
    rng = np.random.default_rng(seed)
    q, k, v = (synth.bf16_round(rng.standard_normal((H, N, d)).astype(np.float32) * 1.5)
               for _ in range(3))
    qperm, kperm, qoff, koff, kvc, kvi, rows = [], [], [], [], [], [], []
    for h in range(H):
        pq, oq = O.stable_argsort(rng.integers(0, CQ, N), CQ)
        pk, ok = O.stable_argsort(rng.integers(0, CK, N), CK)
        cnt = np.zeros(CQ, np.int32)
        idx = np.zeros((CQ, CK), np.int32)
        rr = []
        for u in range(CQ):
            s = np.sort(rng.choice(CK, size=int(rng.integers(1, max(2, CK // 3))), replace=False))
            cnt[u], idx[u, :len(s)] = len(s), s
            rr.append(s)
        qperm.append(pq); kperm.append(pk); qoff.append(oq); koff.append(ok)
        kvc.append(cnt); kvi.append(idx); rows.append(rr)
    t = lambda a: torch.from_numpy(np.stack(a).astype(np.int32)).cuda()
    dev = dict(Qp=PT.to_dev(np.stack([q[h][qperm[h]] for h in range(H)]), "bf16"),
               Kp=PT.to_dev(np.stack([k[h][kperm[h]] for h in range(H)]), "bf16"),
               Vp=PT.to_dev(np.stack([v[h][kperm[h]] for h in range(H)]), "bf16"),
               qo=t(qoff), ko=t(koff), kc=t(kvc), ki=t(kvi), qp=t(qperm))
    host = dict(q=q, k=k, v=v, qperm=qperm, kperm=kperm, qoff=qoff, koff=koff, rows=rows)
    return dev, host


def _run_both(dev, CQ, CK, out_dtype):
    args = (dev["Qp"], dev["Kp"], dev["Vp"], dev["qo"], dev["ko"], dev["kc"], dev["ki"], dev["qp"],
            CQ, CK, out_dtype)
    O_ws, L_ws = P.park_block_sparse_attn(*args, want_lse=True)
    # the static entry point through the C ABI, into preallocated outputs
    O_st = torch.full_like(O_ws, float("nan"))
    L_st = torch.full_like(L_ws, float("nan"))
    H, N, d = dev["Qp"].shape
    dims = P.Dims(H, N, d, P.PARK_BF16)
    ptr = lambda x: C.c_void_p(x.data_ptr())
    r = P.lib().park_block_sparse_attn_static(
        ptr(dev["Qp"]), ptr(dev["Kp"]), ptr(dev["Vp"]), ptr(dev["qo"]), ptr(dev["ko"]),
        ptr(dev["kc"]), ptr(dev["ki"]), ptr(dev["qp"]), C.byref(dims), CQ, CK, ptr(O_st),
        out_dtype, ptr(L_st), C.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert r == P.PARK_OK, P.lib().park_last_error()
    torch.cuda.synchronize()
    return O_ws, L_ws, O_st, L_st


def _check(tag, dev, host, CQ, CK, out_dtype):
    O_ws, L_ws, O_st, L_st = _run_both(dev, CQ, CK, out_dtype)
    assert torch.equal(O_ws, O_st), tag
    assert torch.equal(L_ws, L_st), tag
    Og = PT.np64(O_st)
    for h in range(Og.shape[0]):
        Qh, Kh = host["q"][h][host["qperm"][h]], host["k"][h][host["kperm"][h]]
        ref = O.block_sparse_attention(Qh, Kh, host["v"][h][host["kperm"][h]], host["qoff"][h],
                                       host["koff"][h], host["rows"][h], host["qperm"][h])
        err = np.abs(Og[h] - ref)
        print(f"[{tag} h={h}] static == workspace entry point; max-abs err vs oracle "
              f"{err.max():.3g}", flush=True)
        assert np.all(err <= PT.attn_tol("bf16", out_dtype == P.PARK_BF16, ref))


def test_static_scratch_matches_workspace_entry_point_twice():
    dev, host = _case(1, 3, 2000, 40, 36, 128)
    _check("first call H=3 N=2000", dev, host, 40, 36, P.PARK_F32)
    dev, host = _case(2, 1, 700, 15, 12, 64)
    _check("second call H=1 N=700", dev, host, 15, 12, P.PARK_BF16)


def test_static_scratch_rejects_a_plan_that_does_not_fit():
    # host-side check: nothing is enqueued
    fake = C.c_void_p(1 << 20)
    dims = P.Dims(64, 1 << 20, 64, P.PARK_BF16)
    r = P.lib().park_block_sparse_attn_static(fake, fake, fake, fake, fake, fake, fake, fake,
                                              C.byref(dims), 2048, 2048, fake, P.PARK_F32, None,
                                              None)
    assert r == P.PARK_ERR_WORKSPACE
    assert b"static scratch" in P.lib().park_last_error()
