"""Pass rule for the linear's fp16 outputs against the oracle's fp64 result.

TEST INFRASTRUCTURE ONLY (tests, smoke check, benchmark's parity line).

Tolerance: max abs error <= 1e-3 x RMS of the output.  The library rounds
each output once to fp16, and for outputs above ~2x RMS one fp16 half-ulp
already exceeds 1e-3 x RMS, so the bound is applied to the value before that
final rounding: an output passes when it is the round-to-nearest-even fp16
of some real value within tau = 1e-3 * rms of the exact result, i.e.

    fp16_rne(y_ref - tau) <= y_gpu <= fp16_rne(y_ref + tau).

The literal max |y_gpu - y_ref| / rms is reported alongside.
"""
import numpy as np

REL_TOL = 1e-3


def linear_check(y_gpu, y_ref, rel_tol: float = REL_TOL):
    y_gpu = np.asarray(y_gpu)
    assert y_gpu.dtype == np.float16
    y_ref = np.asarray(y_ref, dtype=np.float64)
    assert y_gpu.shape == y_ref.shape
    rms = float(np.sqrt(np.mean(y_ref ** 2))) if y_ref.size else 0.0
    tau = rel_tol * rms
    lo = (y_ref - tau).astype(np.float16)   # numpy rounds float64 -> float16 to nearest-even
    hi = (y_ref + tau).astype(np.float16)
    g = y_gpu.astype(np.float64)
    ok = (g >= lo.astype(np.float64)) & (g <= hi.astype(np.float64)) & np.isfinite(g)
    err = np.abs(g - y_ref)
    return {
        "ok": bool(ok.all()),
        "n_bad": int((~ok).sum()),
        "rms": rms,
        "tau": tau,
        "max_err_over_rms": float(err.max() / rms) if rms > 0 and err.size else float(err.max() if err.size else 0.0),
        "n_over_tau_literal": int((err > tau).sum()),
        "first_bad": None if ok.all() else tuple(int(i) for i in np.argwhere(~ok)[0]),
    }
