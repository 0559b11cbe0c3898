"""The C ABI loads, exports every symbol include/park.h declares, and rejects
bad arguments on the host before anything is enqueued (no GPU needed)."""
import ctypes as C
import os
import re

import pytest

from paper_2609_38978_amd import park as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "park.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(park_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_binding_exports():
    assert declared_symbols() == sorted(P.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = P.lib()
    for name in declared_symbols():
        assert hasattr(L, name), name
    # the symbols are C, unmangled
    out = os.popen(f"nm -D --defined-only {P.LIB_PATH}").read()
    for name in declared_symbols():
        assert re.search(rf"\bT {name}$", out, re.M), name


def test_status_strings():
    L = P.lib()
    for s in range(6):
        assert L.park_status_string(s)
    assert L.park_status_string(99) == b"unknown status"


FAKE = 1 << 20  # 16-byte aligned fake device address, never dereferenced


def _dims(H=2, N=1000, d=128, dtype=P.PARK_BF16):
    return P.Dims(H, N, d, dtype)


def test_workspace_size_monotone_and_validated():
    L = P.lib()
    out = C.c_size_t()
    assert L.park_workspace_size(C.byref(_dims()), 16, 16, C.byref(out)) == P.PARK_OK
    a = out.value
    assert L.park_workspace_size(C.byref(_dims()), 16, 32, C.byref(out)) == P.PARK_OK
    assert out.value >= a > 0
    assert L.park_workspace_size(C.byref(_dims(d=96)), 16, 16, C.byref(out)) == P.PARK_ERR_UNSUPPORTED
    assert L.park_workspace_size(C.byref(_dims()), 0, 16, C.byref(out)) == P.PARK_ERR_INVALID_ARG
    assert L.park_workspace_size(C.byref(_dims()), 1001, 16, C.byref(out)) == P.PARK_ERR_INVALID_ARG
    assert L.park_workspace_size(C.byref(_dims(N=5000)), 2049, 16, C.byref(out)) == P.PARK_ERR_UNSUPPORTED
    assert L.park_workspace_size(C.byref(_dims(dtype=7)), 16, 16, C.byref(out)) == P.PARK_ERR_INVALID_ARG
    assert b"dtype" in L.park_last_error()


def _cluster(**kw):
    a = dict(X=FAKE, Q=FAKE, dims=_dims(), C=16, T=10, seed=0, side=1, metric=P.PARK_METRIC_QRKC,
             alpha=0.05, eps=1e-6, s_min=1e-12, labels=None, perm=FAKE, offsets=FAKE, R=None,
             Xt=None, ws=FAKE, ws_bytes=1 << 40)
    a.update(kw)
    return P.lib().park_cluster_keys(a["X"], a["Q"], C.byref(a["dims"]), a["C"], a["T"], a["seed"],
                                     a["side"], a["metric"], a["alpha"], a["eps"], a["s_min"],
                                     a["labels"], a["perm"], a["offsets"], a["R"], a["Xt"], a["ws"],
                                     a["ws_bytes"], None)


def test_cluster_argument_errors():
    assert _cluster(X=None) == P.PARK_ERR_INVALID_ARG
    assert _cluster(X=FAKE + 4) == P.PARK_ERR_INVALID_ARG  # misaligned
    assert b"aligned" in P.lib().park_last_error()
    assert _cluster(Q=None) == P.PARK_ERR_INVALID_ARG  # QRKC needs the queries
    assert _cluster(C=0) == P.PARK_ERR_INVALID_ARG
    assert _cluster(C=1001) == P.PARK_ERR_INVALID_ARG  # C > N
    assert _cluster(T=0) == P.PARK_ERR_INVALID_ARG
    assert _cluster(side=2) == P.PARK_ERR_INVALID_ARG
    assert _cluster(metric=5) == P.PARK_ERR_INVALID_ARG
    assert _cluster(alpha=1.5) == P.PARK_ERR_INVALID_ARG
    assert _cluster(alpha=float("nan")) == P.PARK_ERR_INVALID_ARG
    assert _cluster(s_min=0.0) == P.PARK_ERR_INVALID_ARG
    assert _cluster(dims=_dims(d=32)) == P.PARK_ERR_UNSUPPORTED
    assert _cluster(ws_bytes=100) == P.PARK_ERR_WORKSPACE
    assert _cluster(metric=P.PARK_METRIC_EUCLID, R=FAKE) == P.PARK_ERR_INVALID_ARG


def test_retrieve_and_attention_argument_errors():
    L = P.lib()
    d = _dims()

    def retr(sel=P.PARK_SELECT_TOPP, param=0.9, CQ=16, CK=16, ws_bytes=1 << 40):
        return L.park_retrieve_blocks(FAKE, FAKE, FAKE, FAKE, C.byref(d), CQ, CK, sel, param, None,
                                      FAKE, FAKE, FAKE, ws_bytes, None)

    assert retr(param=0.0) == P.PARK_ERR_INVALID_ARG
    assert retr(param=1.5) == P.PARK_ERR_INVALID_ARG
    assert retr(sel=9) == P.PARK_ERR_INVALID_ARG
    assert retr(CK=3000) == P.PARK_ERR_INVALID_ARG
    assert retr(ws_bytes=8) == P.PARK_ERR_WORKSPACE
    def attn(V=FAKE, out_dtype=P.PARK_F32, lse=None, ws_bytes=1 << 30):
        return L.park_block_sparse_attn(FAKE, FAKE, V, FAKE, FAKE, FAKE, FAKE, FAKE, C.byref(d), 16,
                                        16, FAKE, out_dtype, lse, FAKE, ws_bytes, None)

    assert attn(out_dtype=7) == P.PARK_ERR_INVALID_ARG
    assert attn(V=None) == P.PARK_ERR_INVALID_ARG
    assert attn(lse=FAKE + 4) == P.PARK_ERR_INVALID_ARG  # lse misaligned
    assert b"lse" in L.park_last_error()
    assert attn(ws_bytes=8) == P.PARK_ERR_WORKSPACE


def test_state_sizes():
    # one entry per park_state member, matching the buffers the binding allocates
    L = P.lib()
    H, N, d, CQ, CK = 3, 1000, 128, 16, 24
    n = len(P.STATE_FIELDS)
    out = (C.c_size_t * n)()
    assert L.park_state_sizes(C.byref(_dims(H, N, d, P.PARK_BF16)), CQ, CK, out, n) == P.PARK_OK
    want = {"q_perm": H * N * 4, "k_perm": H * N * 4, "q_offsets": H * (CQ + 1) * 4,
            "k_offsets": H * (CK + 1) * 4, "k_centroids": H * CK * d * 4, "k_sizes": H * CK * 4,
            "kv_count": H * CQ * 4, "kv_index": H * CQ * CK * 4, "Qp": H * N * d * 2,
            "Kp": H * N * d * 2, "Vp": H * N * d * 2, "W": H * CQ * CK * 4,
            "q_mu": H * CQ * d * 8, "k_mu": H * CK * d * 8}
    assert dict(zip(P.STATE_FIELDS, out)) == want
    assert [f for f, _ in P.State._fields_] == list(P.STATE_FIELDS)
    assert L.park_state_sizes(C.byref(_dims(H, N, 64, P.PARK_F32)), CQ, CK, out, n) == P.PARK_OK
    assert out[8] == H * N * 64 * 4
    assert L.park_state_sizes(C.byref(_dims()), 16, 16, out, n - 1) == P.PARK_ERR_INVALID_ARG
    assert L.park_state_sizes(C.byref(_dims()), 16, 16, None, n) == P.PARK_ERR_INVALID_ARG
    assert L.park_state_sizes(C.byref(_dims()), 0, 16, out, n) == P.PARK_ERR_INVALID_ARG


def test_forward_argument_errors():
    L = P.lib()
    d = _dims()
    prm = P.make_params(16, 16)
    st = P.State(*([FAKE] * 11 + [None]))

    def fwd(params=prm, reuse=0, state=st, ws_bytes=1 << 40):
        return L.park_forward(FAKE, FAKE, FAKE, C.byref(d), C.byref(params), reuse, C.byref(state),
                              FAKE, FAKE, ws_bytes, None)

    assert fwd(reuse=3) == P.PARK_ERR_INVALID_ARG
    bad = P.make_params(16, 16, select="topk", ratio=0.0)
    assert fwd(params=bad) == P.PARK_ERR_INVALID_ARG
    bad = P.make_params(16, 16, out_dtype=3)
    assert fwd(params=bad) == P.PARK_ERR_INVALID_ARG
    bad = P.make_params(16, 16, T=0)
    assert fwd(params=bad) == P.PARK_ERR_INVALID_ARG
    st2 = P.State(*([FAKE] * 10 + [None, None]))  # Vp missing
    assert fwd(state=st2) == P.PARK_ERR_INVALID_ARG
    assert fwd(ws_bytes=64) == P.PARK_ERR_WORKSPACE
    assert L.park_forward(FAKE, FAKE, FAKE, C.byref(d), None, 0, C.byref(st), FAKE, FAKE, 1 << 40,
                          None) == P.PARK_ERR_INVALID_ARG
    # a warm-started recomputation needs the centroid buffers of the state
    warm = P.make_params(16, 16, init=P.PARK_INIT_WARM)
    assert fwd(params=warm) == P.PARK_ERR_INVALID_ARG
    assert b"q_mu" in L.park_last_error()
    assert fwd(params=P.make_params(16, 16, init=5)) == P.PARK_ERR_INVALID_ARG
    st3 = P.State(*([FAKE] * 11 + [None, FAKE + 8, FAKE]))  # q_mu misaligned
    assert fwd(state=st3) == P.PARK_ERR_INVALID_ARG


def test_schedule_step_host_logic():
    # clustering and mask computed at the steps of the set, reused between
    # them, dense attention before the first (no GPU involved)
    sched = [10, 20, 30]
    modes = [P.park_schedule_step(t, sched) for t in range(50)]
    assert all(m == P.PARK_STEP_DENSE for m in modes[:10])
    for t in range(10, 50):
        want = P.PARK_RECOMPUTE if t in sched else P.PARK_REUSE_CLUSTERS_AND_MASK
        assert modes[t] == want, t
    assert P.park_schedule_step(0, [0]) == P.PARK_RECOMPUTE
    for bad_step, bad_sched in ((-1, [3]), (4, [3, 3]), (4, [5, 2]), (4, [-1, 2]), (1, [])):
        with pytest.raises(P.ParkError) as ei:
            P.park_schedule_step(bad_step, bad_sched)
        assert ei.value.status == P.PARK_ERR_INVALID_ARG


def test_probe_argument_errors():
    L = P.lib()
    assert L.park_probe_exp2(FAKE, FAKE, -1, None) == P.PARK_ERR_INVALID_ARG
    assert L.park_probe_exp2(None, FAKE, 5, None) == P.PARK_ERR_INVALID_ARG
    assert L.park_probe_exp2(None, None, 0, None) == P.PARK_OK  # nothing to do
    for K in (0, 8, 24, 4112):
        assert L.park_probe_mfma_bf16(FAKE, FAKE, FAKE, FAKE, 1, K, None) == P.PARK_ERR_INVALID_ARG
    assert L.park_probe_mfma_bf16(FAKE, FAKE, FAKE + 8, FAKE, 1, 32, None) == P.PARK_ERR_INVALID_ARG
    assert L.park_probe_mfma_bf16(FAKE, FAKE, FAKE, FAKE, -1, 32, None) == P.PARK_ERR_INVALID_ARG
