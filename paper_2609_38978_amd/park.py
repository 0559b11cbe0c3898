"""Python binding of libpark (ctypes).  Argument marshalling only.

Every function here has the name of the C entry point it calls, takes torch
tensors that live on the GPU, allocates its outputs with torch (PyTorch is
used for device memory and streams only) and launches on torch's current
stream.  All computation happens in the HIP kernels of libpark.so; when the
library is missing every call raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes as C
import json
import os

import torch

PARK_OK, PARK_ERR_INVALID_ARG, PARK_ERR_UNSUPPORTED, PARK_ERR_WORKSPACE = 0, 1, 2, 3
PARK_ERR_HIP, PARK_ERR_NUMERIC = 4, 5
PARK_F32, PARK_BF16 = 0, 1
PARK_METRIC_EUCLID, PARK_METRIC_QRKC = 0, 1
PARK_SELECT_TOPK, PARK_SELECT_TOPP = 0, 1
PARK_RECOMPUTE, PARK_REUSE_CLUSTERS, PARK_REUSE_CLUSTERS_AND_MASK = 0, 1, 2
PARK_EST_PAMA, PARK_EST_QCENTROID = 0, 1
PARK_BLOCKS_CLUSTER, PARK_BLOCKS_FIXED = 0, 1
PARK_INIT_SEEDED, PARK_INIT_WARM = 0, 1

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpark.so")

# names of every entry point declared in include/park.h
EXPORTS = (
    "park_workspace_size", "park_cluster_keys", "park_gather_rows", "park_block_centroids",
    "park_retrieve_blocks", "park_block_sparse_attn", "park_forward", "park_check",
    "park_status_string", "park_last_error", "park_profile_enable", "park_profile_reset",
    "park_profile_read", "park_schedule_step", "park_state_sizes", "park_probe_exp2",
    "park_probe_mfma_bf16", "park_block_sparse_attn_static",
)


class ParkError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"park status {status}: {msg}")
        self.status = status


class Dims(C.Structure):
    _fields_ = [("H", C.c_int32), ("N", C.c_int32), ("d", C.c_int32), ("dtype", C.c_int32)]


class Params(C.Structure):
    _fields_ = [("CQ", C.c_int32), ("CK", C.c_int32), ("T", C.c_int32), ("select", C.c_int32),
                ("topk_ratio", C.c_double), ("topp", C.c_double), ("alpha", C.c_double),
                ("eps", C.c_double), ("s_min", C.c_double), ("seed", C.c_uint64),
                ("key_metric", C.c_int32), ("out_dtype", C.c_int32),
                ("estimator", C.c_int32), ("block_mode", C.c_int32), ("init", C.c_int32)]


class State(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("q_perm", "k_perm", "q_offsets", "k_offsets",
                                          "k_centroids", "k_sizes", "kv_count", "kv_index",
                                          "Qp", "Kp", "Vp", "W", "q_mu", "k_mu")]


_lib = None


def lib():
    """The loaded libpark.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    L = C.CDLL(LIB_PATH)
    vp, i32, u64, f64, sz = C.c_void_p, C.c_int32, C.c_uint64, C.c_double, C.c_size_t
    pd = C.POINTER(Dims)
    sig = {
        "park_workspace_size": [pd, i32, i32, C.POINTER(C.c_size_t)],
        "park_cluster_keys": [vp, vp, pd, i32, i32, u64, i32, i32, f64, f64, f64, vp, vp, vp, vp,
                              vp, vp, sz, vp],
        "park_gather_rows": [vp, vp, pd, vp, vp],
        "park_block_centroids": [vp, vp, vp, pd, i32, vp, vp, vp],
        "park_retrieve_blocks": [vp, vp, vp, vp, pd, i32, i32, i32, f64, vp, vp, vp, vp, sz, vp],
        "park_block_sparse_attn": [vp, vp, vp, vp, vp, vp, vp, vp, pd, i32, i32, vp, i32, vp, vp,
                                   sz, vp],
        "park_block_sparse_attn_static": [vp, vp, vp, vp, vp, vp, vp, vp, pd, i32, i32, vp, i32,
                                          vp, vp],
        "park_state_sizes": [pd, i32, i32, C.POINTER(C.c_size_t), i32],
        "park_forward": [vp, vp, vp, pd, C.POINTER(Params), i32, C.POINTER(State), vp, vp, sz,
                         vp],
        "park_check": [vp, vp],
        "park_probe_exp2": [vp, vp, C.c_int64, vp],
        "park_probe_mfma_bf16": [vp, vp, vp, vp, i32, i32, vp],
        "park_schedule_step": [i32, C.POINTER(C.c_int32), i32, C.POINTER(C.c_int32)],
        "park_status_string": [i32],
        "park_last_error": [],
        "park_profile_enable": [i32],
        "park_profile_reset": [],
        "park_profile_read": [C.c_char_p, sz],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = C.c_char_p if name in ("park_status_string", "park_last_error") else C.c_int
    _lib = L
    return L


def _check(status: int):
    if status != PARK_OK:
        raise ParkError(status, lib().park_last_error().decode())


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return PARK_F32
    if t.dtype == torch.bfloat16:
        return PARK_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dims(X: torch.Tensor) -> Dims:
    if X.dim() != 3 or not X.is_cuda or not X.is_contiguous():
        raise ValueError("expected a contiguous [H, N, d] CUDA tensor")
    H, N, d = X.shape
    return Dims(H, N, d, _dtype_code(X))


def _dev(X):
    return dict(device=X.device)


def park_workspace_size(H: int, N: int, d: int, dtype: int, CQ: int, CK: int) -> int:
    out = C.c_size_t(0)
    dims = Dims(H, N, d, dtype)
    _check(lib().park_workspace_size(C.byref(dims), CQ, CK, C.byref(out)))
    return out.value


def workspace(X: torch.Tensor, CQ: int, CK: int) -> torch.Tensor:
    H, N, d = X.shape
    n = park_workspace_size(H, N, d, _dtype_code(X), CQ, CK)
    return torch.empty(n, dtype=torch.uint8, device=X.device)


def park_cluster_keys(X, C_: int, T: int, seed: int = 0, side: int = 1,
                      metric: int = PARK_METRIC_QRKC, Qmetric=None, alpha: float = 0.05,
                      eps: float = 1e-6, s_min: float = 1e-12, want_R: bool = False,
                      want_Xt: bool = False, ws=None):
    """k-means of one side; returns dict(labels, perm, offsets[, R, Xt])."""
    dims = _dims(X)
    H, N, d = X.shape
    ws = workspace(X, C_, C_) if ws is None else ws
    out = {"labels": torch.empty(H, N, dtype=torch.int32, **_dev(X)),
           "perm": torch.empty(H, N, dtype=torch.int32, **_dev(X)),
           "offsets": torch.empty(H, C_ + 1, dtype=torch.int32, **_dev(X))}
    if want_R:
        out["R"] = torch.empty(H, d, d, dtype=torch.float64, **_dev(X))
    if want_Xt:
        out["Xt"] = torch.empty(H, N, d, dtype=torch.float32, **_dev(X))
    _check(lib().park_cluster_keys(
        _ptr(X), _ptr(Qmetric), C.byref(dims), C_, T, seed, side, metric, alpha, eps, s_min,
        _ptr(out["labels"]), _ptr(out["perm"]), _ptr(out["offsets"]), _ptr(out.get("R")),
        _ptr(out.get("Xt")), _ptr(ws), ws.numel(), _stream()))
    out["ws"] = ws
    return out


def park_gather_rows(X, perm):
    dims = _dims(X)
    Xp = torch.empty_like(X)
    _check(lib().park_gather_rows(_ptr(X), _ptr(perm), C.byref(dims), _ptr(Xp), _stream()))
    return Xp


def park_block_centroids(X, perm, offsets, C_: int):
    dims = _dims(X)
    H, N, d = X.shape
    cen = torch.empty(H, C_, d, dtype=torch.float32, **_dev(X))
    sizes = torch.empty(H, C_, dtype=torch.int32, **_dev(X))
    _check(lib().park_block_centroids(_ptr(X), _ptr(perm), _ptr(offsets), C.byref(dims), C_,
                                      _ptr(cen), _ptr(sizes), _stream()))
    return cen, sizes


def park_retrieve_blocks(Qp, q_offsets, centroids, k_sizes, CQ: int, CK: int, select: int,
                         param: float, want_W: bool = False, ws=None):
    """Returns (kv_count [H,CQ], kv_index [H,CQ,CK], W [H,CQ,CK] or None)."""
    dims = _dims(Qp)
    H = Qp.shape[0]
    ws = workspace(Qp, CQ, CK) if ws is None else ws
    kv_count = torch.empty(H, CQ, dtype=torch.int32, **_dev(Qp))
    kv_index = torch.empty(H, CQ, CK, dtype=torch.int32, **_dev(Qp))
    W = torch.empty(H, CQ, CK, dtype=torch.float32, **_dev(Qp)) if want_W else None
    _check(lib().park_retrieve_blocks(_ptr(Qp), _ptr(q_offsets), _ptr(centroids), _ptr(k_sizes),
                                      C.byref(dims), CQ, CK, select, param, _ptr(W),
                                      _ptr(kv_count), _ptr(kv_index), _ptr(ws), ws.numel(),
                                      _stream()))
    return kv_count, kv_index, W


def park_block_sparse_attn(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm,
                           CQ: int, CK: int, out_dtype: int = PARK_F32, ws=None,
                           want_lse: bool = False):
    """Returns O, or (O, lse [H, N] float32) when want_lse."""
    dims = _dims(Qp)
    O = torch.empty(Qp.shape, dtype=torch.float32 if out_dtype == PARK_F32 else torch.bfloat16,
                    **_dev(Qp))
    lse = torch.empty(Qp.shape[:2], dtype=torch.float32, **_dev(Qp)) if want_lse else None
    ws = workspace(Qp, CQ, CK) if ws is None else ws
    _check(lib().park_block_sparse_attn(_ptr(Qp), _ptr(Kp), _ptr(Vp), _ptr(q_offsets),
                                        _ptr(k_offsets), _ptr(kv_count), _ptr(kv_index),
                                        _ptr(q_perm), C.byref(dims), CQ, CK, _ptr(O), out_dtype,
                                        _ptr(lse), _ptr(ws), ws.numel(), _stream()))
    return (O, lse) if want_lse else O


def park_block_sparse_attn_static(Qp, Kp, Vp, q_offsets, k_offsets, kv_count, kv_index, q_perm,
                                  CQ: int, CK: int, out_dtype: int = PARK_F32, O=None, lse=None):
    """The workspace-free entry point: writes into the given O (and lse) tensors,
    allocating nothing when both are given; returns (O, lse)."""
    dims = _dims(Qp)
    if O is None:
        O = torch.empty(Qp.shape, dtype=torch.float32 if out_dtype == PARK_F32
                        else torch.bfloat16, **_dev(Qp))
    _check(lib().park_block_sparse_attn_static(_ptr(Qp), _ptr(Kp), _ptr(Vp), _ptr(q_offsets),
                                               _ptr(k_offsets), _ptr(kv_count), _ptr(kv_index),
                                               _ptr(q_perm), C.byref(dims), CQ, CK, _ptr(O),
                                               out_dtype, _ptr(lse), _stream()))
    return O, lse


STATE_FIELDS = ("q_perm", "k_perm", "q_offsets", "k_offsets", "k_centroids", "k_sizes",
                "kv_count", "kv_index", "Qp", "Kp", "Vp", "W", "q_mu", "k_mu")


def park_state_sizes(H: int, N: int, d: int, dtype: int, CQ: int, CK: int) -> dict:
    """Bytes of each park_state buffer, keyed by member name."""
    n = len(STATE_FIELDS)
    out = (C.c_size_t * n)()
    dims = Dims(H, N, d, dtype)
    _check(lib().park_state_sizes(C.byref(dims), CQ, CK, out, n))
    return dict(zip(STATE_FIELDS, out))


def make_params(CQ, CK, T=10, select="topk", ratio=0.25, topp=0.9, alpha=0.05, eps=1e-6,
                s_min=1e-12, seed=0, key_metric=PARK_METRIC_QRKC, out_dtype=PARK_F32,
                estimator=PARK_EST_PAMA, block_mode=PARK_BLOCKS_CLUSTER,
                init=PARK_INIT_SEEDED) -> Params:
    sel = PARK_SELECT_TOPK if select in ("topk", PARK_SELECT_TOPK) else PARK_SELECT_TOPP
    return Params(CQ, CK, T, sel, ratio, topp, alpha, eps, s_min, seed, key_metric, out_dtype,
                  estimator, block_mode, init)


def make_state(Q, CQ: int, CK: int, want_W: bool = False, want_mu: bool = False) -> dict:
    """Caller-owned device buffers for park_forward (a dict of tensors); want_mu
    adds the float64 centroids a warm-started recomputation reads and every
    recomputation writes."""
    H, N, d = Q.shape
    i32 = dict(dtype=torch.int32, **_dev(Q))
    st = {"q_perm": torch.empty(H, N, **i32), "k_perm": torch.empty(H, N, **i32),
          "q_offsets": torch.empty(H, CQ + 1, **i32), "k_offsets": torch.empty(H, CK + 1, **i32),
          "k_centroids": torch.empty(H, CK, d, dtype=torch.float32, **_dev(Q)),
          "k_sizes": torch.empty(H, CK, **i32), "kv_count": torch.empty(H, CQ, **i32),
          "kv_index": torch.empty(H, CQ, CK, **i32), "Qp": torch.empty_like(Q),
          "Kp": torch.empty_like(Q), "Vp": torch.empty_like(Q),
          "W": torch.empty(H, CQ, CK, dtype=torch.float32, **_dev(Q)) if want_W else None,
          "q_mu": torch.empty(H, CQ, d, dtype=torch.float64, **_dev(Q)) if want_mu else None,
          "k_mu": torch.empty(H, CK, d, dtype=torch.float64, **_dev(Q)) if want_mu else None}
    return st


def _state_struct(st: dict) -> State:
    return State(*[(None if st.get(n) is None else st[n].data_ptr()) for n, _ in State._fields_])


def park_forward(Q, K, V, params: Params, reuse: int = PARK_RECOMPUTE, state: dict | None = None,
                 out=None, ws=None):
    """Whole layer; returns (O, state).  `state` is a dict from make_state."""
    dims = _dims(Q)
    state = make_state(Q, params.CQ, params.CK) if state is None else state
    ws = workspace(Q, params.CQ, params.CK) if ws is None else ws
    if out is None:
        out = torch.empty(Q.shape, dtype=torch.float32 if params.out_dtype == PARK_F32
                          else torch.bfloat16, **_dev(Q))
    s = _state_struct(state)
    _check(lib().park_forward(_ptr(Q), _ptr(K), _ptr(V), C.byref(dims), C.byref(params), reuse,
                              C.byref(s), _ptr(out), _ptr(ws), ws.numel(), _stream()))
    return out, state


PARK_STEP_DENSE = -1


def park_schedule_step(step: int, steps) -> int:
    """Mode of denoising step `step` under the recomputation set `steps`:
    PARK_RECOMPUTE, PARK_REUSE_CLUSTERS_AND_MASK or PARK_STEP_DENSE."""
    arr = (C.c_int32 * len(steps))(*steps)
    out = C.c_int32(0)
    _check(lib().park_schedule_step(int(step), arr, len(steps), C.byref(out)))
    return out.value


def park_probe_exp2(x):
    """2^x by the device's v_exp_f32 (x: float32 CUDA tensor)."""
    x = x.contiguous()
    y = torch.empty_like(x)
    _check(lib().park_probe_exp2(_ptr(x), _ptr(y), x.numel(), _stream()))
    return y


def park_probe_mfma_bf16(A, Bt, C0):
    """C0 + A Bt^T by a chain of 32x32x16 bf16 MFMAs (A, Bt: [P, 32, K] bf16, C0: [P, 32, 32])."""
    A, Bt, C0 = A.contiguous(), Bt.contiguous(), C0.contiguous()
    out = torch.empty_like(C0)
    _check(lib().park_probe_mfma_bf16(_ptr(A), _ptr(Bt), _ptr(C0), _ptr(out), A.shape[0],
                                      A.shape[2], _stream()))
    return out


def park_check(ws):
    """Synchronises and raises ParkError if the last call on `ws` failed on the device."""
    _check(lib().park_check(_ptr(ws), _stream()))


def park_profile_enable(on: bool = True):
    _check(lib().park_profile_enable(1 if on else 0))


def park_profile_reset():
    _check(lib().park_profile_reset())


def park_profile_read() -> dict:
    buf = C.create_string_buffer(1 << 16)
    _check(lib().park_profile_read(buf, len(buf)))
    return json.loads(buf.value.decode())
