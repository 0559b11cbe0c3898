"""Parity helpers: compare the HIP path with the CPU oracle.

Bars (stated by the method's specification):
* labels, permutations, masks: bit-exact, except where the oracle's own
  distance / score gap is below 1e-6 relative;
* attention outputs: 1e-4 max-abs (fp32 inputs), 2e-2 max-abs (bf16 inputs).
"""
from __future__ import annotations

import math

import numpy as np
import torch

from oracle import park_oracle as O

REL_GAP = 1e-6
FLT_MIN = float(np.finfo(np.float32).tiny)
ATOL = {"f32": 1e-4, "bf16": 2e-2}


def to_dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    t = t.to(torch.bfloat16) if dtype == "bf16" else t
    return t.cuda().contiguous()


def np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def label_flips(X: np.ndarray, mu: np.ndarray, z_gpu: np.ndarray, z_or: np.ndarray):
    """Mismatched tokens and whether each is a near-tie of the oracle's distances.

    Returns (n_mismatch, n_not_exempt, worst relative gap).
    """
    bad = np.nonzero(z_gpu != z_or)[0]
    worst = 0.0
    n_not = 0
    for j in bad:
        da = np.sum((X[j] - mu[z_gpu[j]]) ** 2)
        db = np.sum((X[j] - mu[z_or[j]]) ** 2)
        rel = (da - db) / max(db, 1e-300)
        worst = max(worst, rel)
        if rel > REL_GAP:
            n_not += 1
    return len(bad), n_not, worst


def mask_row_exempt(w: np.ndarray, valid: np.ndarray, mode: str, param: float,
                    got: set, want: set) -> bool:
    """A differing mask row is acceptable only at a near-tie of the oracle.

    Top-p: when the oracle's cumulative mass at the cut lies within 1e-6 p
    of p, the next block (order[m]) may be added; when the mass one block
    earlier does, the last kept block (order[m-1]) may be dropped -- only that
    block.  Beyond that, a near-tie in value can only swap blocks: the two
    rows must keep as many blocks, and every block in which they differ must
    have an oracle weight within 1e-6 (relative) of the cut weight (or both
    below FLT_MIN).
    """
    if got == want:
        return True
    sel, order, m = O.select_row(w, valid, mode, param)
    cut = w[order[m - 1]] if m > 0 else 0.0
    got, want = set(got), set(want)
    if mode == "topp" and m > 0:
        cs = np.cumsum(w[order])
        if abs(cs[m - 1] - param) <= REL_GAP * param and m < len(order):
            extra = int(order[m])
            if extra in got and extra not in want:
                got.discard(extra)
        if m >= 2 and abs(cs[m - 2] - param) <= REL_GAP * param:
            last = int(order[m - 1])
            if last in want and last not in got:
                want.discard(last)
    if len(got) != len(want):
        return False
    for v in got ^ want:
        if w[v] < FLT_MIN and cut < FLT_MIN:
            continue
        if abs(w[v] - cut) > REL_GAP * max(cut, FLT_MIN):
            return False
    return True


def compare_masks(W: np.ndarray, k_sizes: np.ndarray, q_sizes: np.ndarray, mode: str,
                  param: float, kv_count: np.ndarray, kv_index: np.ndarray):
    """(n_rows_differing, n_not_exempt) for one head."""
    valid = k_sizes > 0
    n_diff = n_bad = 0
    for u in range(W.shape[0]):
        got = set(kv_index[u, :kv_count[u]].tolist())
        if q_sizes[u] == 0:
            assert kv_count[u] == 0
            continue
        want = set(O.select_row(W[u], valid, mode, param)[0].tolist())
        ids = kv_index[u, :kv_count[u]]
        assert np.all(np.diff(ids) > 0), "kv_index row not ascending"
        if got != want:
            n_diff += 1
            if not mask_row_exempt(W[u], valid, mode, param, got, want):
                n_bad += 1
    return n_diff, n_bad


def attn_tol(dtype: str, out_bf16: bool, ref: np.ndarray) -> np.ndarray:
    """Per-element tolerance: the dtype bar, plus half an ulp of bf16 output."""
    tol = np.full(ref.shape, ATOL[dtype])
    if out_bf16:
        e = np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126)))
        tol = tol + 2.0 ** (e - 8)
    return tol


def lse_tol(Qp: np.ndarray, Kp: np.ndarray, q_offsets, k_offsets, rows, q_perm,
            lse_ref: np.ndarray) -> np.ndarray:
    """Per-row bound on the error of a float32 log-normaliser (in token order).

    A score q.k / sqrt(d) accumulated in float32 over d products (exact for
    bf16 operands, one rounding for float32 ones) errs by at most
    (d + 1) 2^-23 sum_t |q_t k_t| / sqrt(d); a log-sum-exp moves by at most
    the largest score error.  The float32 sum of the probabilities (each from
    one exp, relative error <= 2^-22) adds about (n_keys / 4 + 16) 2^-23
    relative, and the final scale, log and add 2^-22 (|lse| + 1).
    """
    Qp, Kp = np.abs(np.asarray(Qp, np.float64)), np.abs(np.asarray(Kp, np.float64))
    N, d = Qp.shape
    tol = np.zeros(N)
    for u, sel in enumerate(rows):
        a, b = int(q_offsets[u]), int(q_offsets[u + 1])
        if b == a or len(sel) == 0:
            continue
        keys = np.concatenate([np.arange(k_offsets[v], k_offsets[v + 1]) for v in sel])
        if len(keys) == 0:
            continue
        smax = (Qp[a:b] @ Kp[keys].T).max(axis=1) / math.sqrt(d)
        t = (d + 1) * 2.0 ** -23 * smax + (len(keys) / 4 + 16) * 2.0 ** -23
        tol[np.asarray(q_perm[a:b])] = t
    return tol + 2.0 ** -22 * (np.where(np.isfinite(lse_ref), np.abs(lse_ref), 0.0) + 1.0)


def lse_ok(got: np.ndarray, ref: np.ndarray, tol: np.ndarray) -> tuple[bool, float]:
    """-inf exactly where the reference is -inf, else within tol; (ok, worst err / tol)."""
    inf_r, inf_g = np.isneginf(ref), np.isneginf(got)
    if not np.array_equal(inf_r, inf_g) or not np.all(np.isfinite(got[~inf_g])):
        return False, float("inf")
    if inf_r.all():
        return True, 0.0
    ratio = np.abs(got[~inf_r] - ref[~inf_r]) / tol[~inf_r]
    return bool(ratio.max() <= 1.0), float(ratio.max())


def w_error_ok(dtype: str, W: np.ndarray, ref: np.ndarray) -> tuple[bool, float]:
    """Block-score matrix W^ against the oracle's float64 value.

    float32 inputs: W^ is computed in float64 and rounded once to float.
    bf16 inputs: rows are computed on bf16 MFMA with a certified per-row
    relative bound (about 1e-3 in the worst case, far smaller in practice),
    rows the bound cannot settle are recomputed in float64.
    """
    err = np.abs(W.astype(np.float64) - ref)
    if dtype == "f32":
        return bool(np.all(err <= 2.0 ** -23 * ref + 1e-40)), float(err.max())
    return bool(err.max() <= 1e-4 and np.all(err <= 4e-3 * ref + 1e-30)), float(err.max())


def rows_from_csr(kv_count: np.ndarray, kv_index: np.ndarray):
    return [kv_index[u, :kv_count[u]].astype(np.int64) for u in range(len(kv_count))]
