"""Measures the two hardware error models the certified fast paths rest on.

* v_exp_f32 (PAMA's and attention's exponentials): for an exactly known float
  argument x in PAMA's range, relative error <= 2^-23 (2 + 1.5 |x|) where the
  result is a normal float (the retrieval bound charges 1.5 |x| for the
  rounding of the argument it computes; the instruction alone is measured
  here), and at most FLT_MIN absolute below the normal range (the selection's
  absolute term).
* v_mfma_f32_32x32x16_bf16 accumulation chains (k-means and PAMA scores): the
  bounds assume every addition errs by at most 2^-23 of the magnitudes
  involved, i.e. |C^ - C| <= (K + 1) 2^-23 (|C0| + sum_k |a_k b_k|) for a
  chain of K products started from C0.

The references are float64 (exp2 of the float argument; products of bf16
values are exact in float64 and summed with compensation)."""
import numpy as np
import pytest
import torch

from paper_2609_38978_amd import park as P
from paper_2609_38978_amd import synth

pytestmark = pytest.mark.gpu

FLT_MIN = float(np.finfo(np.float32).tiny)
U23 = 2.0 ** -23


def test_exp2_relative_error_model():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.uniform(-150.0, 8.0, 1 << 22).astype(np.float32),
        np.arange(-150, 9, dtype=np.float32),                     # integers
        np.nextafter(np.arange(-150, 9, dtype=np.float32), np.float32(np.inf)),
        np.nextafter(np.arange(-150, 9, dtype=np.float32), np.float32(-np.inf)),
        rng.uniform(-1e-3, 1e-3, 1 << 16).astype(np.float32),      # near zero
    ])
    y = P.park_probe_exp2(torch.from_numpy(x).cuda()).cpu().numpy().astype(np.float64)
    ref = np.exp2(x.astype(np.float64))
    normal = ref >= FLT_MIN
    rel = np.abs(y[normal] - ref[normal]) / ref[normal]
    bound = U23 * (2.0 + 1.5 * np.abs(x[normal].astype(np.float64)))
    worst_ulp = float((rel / U23).max())
    print(f"[exp2] {normal.sum()} normal results: worst relative error {worst_ulp:.3f} x 2^-23; "
          f"worst error / model bound {float((rel / bound).max()):.3g}")
    assert np.all(rel <= bound)
    sub = ~normal
    err_sub = np.abs(y[sub] - ref[sub])
    print(f"[exp2] {sub.sum()} subnormal results: worst absolute error {err_sub.max():.3g} "
          f"(FLT_MIN {FLT_MIN:.3g})")
    assert np.all(err_sub <= FLT_MIN)


def _exact_chain(A, Bt, C0):
    """C0 + sum_k A[:, i, k] Bt[:, j, k] in float64 with Neumaier compensation,
    and sum_k |a_k b_k|."""
    A64, B64 = A.astype(np.float64), Bt.astype(np.float64)
    s = C0.astype(np.float64).copy()
    comp = np.zeros_like(s)
    mag = np.abs(s)
    for k in range(A.shape[2]):
        p = A64[:, :, k][:, :, None] * B64[:, :, k][:, None, :]  # exact products
        t = s + p
        comp += np.where(np.abs(s) >= np.abs(p), (s - t) + p, (p - t) + s)
        s = t
        mag = mag + np.abs(p)
    return s + comp, mag


def _bf16(a):
    return synth.bf16_round(np.asarray(a, np.float32))


@pytest.mark.parametrize("kind", ["random", "cancel", "wide", "on_top"])
@pytest.mark.parametrize("K", [128, 384])
def test_mfma_bf16_chain_error_model(kind, K):
    rng = np.random.default_rng(K + len(kind))
    Pn = 96
    if kind == "wide":  # products spread over 2^-24 .. 2^24
        A = rng.standard_normal((Pn, 32, K)) * 2.0 ** rng.integers(-12, 13, (Pn, 32, K))
        B = rng.standard_normal((Pn, 32, K)) * 2.0 ** rng.integers(-12, 13, (Pn, 32, K))
    else:
        A = rng.standard_normal((Pn, 32, K))
        B = rng.standard_normal((Pn, 32, K))
    A, B = _bf16(A), _bf16(B)
    if kind == "cancel":  # the second half cancels the first up to one small term
        h = K // 2
        A[:, :, h:] = -A[:, :, :h]
        B[:, :, h:] = B[:, :, :h]
        A[:, :, -1] = _bf16(A[:, :, -1] * 2.0 ** -10)
    C0 = np.zeros((Pn, 32, 32), np.float32)
    if kind == "on_top":  # a chain continued on an accumulator (the split-part chains)
        C0 = (rng.standard_normal((Pn, 32, 32)) * 4.0).astype(np.float32)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    got = P.park_probe_mfma_bf16(t(A).to(torch.bfloat16), t(B).to(torch.bfloat16),
                                 t(C0)).cpu().numpy().astype(np.float64)
    exact, mag = _exact_chain(A, B, C0)
    err = np.abs(got - exact)
    ratio = err / (U23 * mag)
    print(f"[mfma {kind} K={K}] worst error {float(ratio.max()):.3f} x 2^-23 (|C0| + sum|ab|); "
          f"model allows {K + 1}")
    assert np.all(err <= (K + 1) * U23 * mag)
