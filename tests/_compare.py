"""Parity tolerances and comparison helpers shared by the GPU tests and the mutation tests.

Binding tolerances on bf16 outputs: max-abs <= 2e-2 and mean-abs <= 2e-3.  The LSE (fp32 on the
GPU) must match to max-abs <= 1e-3: with N(0, 1) inputs long-context outputs are ~1e-2 in size,
so the output tolerances alone could not see a dropped page, but the LSE moves by about the
dropped probability mass.
"""
import numpy as np

TOL_MAX_ABS = 2e-2
TOL_MEAN_ABS = 2e-3
TOL_LSE_MAX_ABS = 1e-3


def report(o_test, o_ref, lse_test=None, lse_ref=None):
    o_test = np.asarray(o_test, dtype=np.float64)
    o_ref = np.asarray(o_ref, dtype=np.float64)
    err = np.abs(o_test - o_ref)
    rep = {
        "max_abs": float(err.max()) if err.size else 0.0,
        "mean_abs": float(err.mean()) if err.size else 0.0,
        "finite": bool(np.isfinite(o_test).all()),
    }
    if lse_test is not None and lse_ref is not None:
        le = np.abs(np.asarray(lse_test, dtype=np.float64) - np.asarray(lse_ref, dtype=np.float64))
        rep["lse_max_abs"] = float(le.max()) if le.size else 0.0
        rep["lse_finite"] = bool(np.isfinite(np.asarray(lse_test)).all())
    return rep


def passes(rep):
    ok = rep["finite"] and rep["max_abs"] <= TOL_MAX_ABS and rep["mean_abs"] <= TOL_MEAN_ABS
    if "lse_max_abs" in rep:
        ok = ok and rep["lse_finite"] and rep["lse_max_abs"] <= TOL_LSE_MAX_ABS
    return ok


def assert_parity(o_test, o_ref, lse_test=None, lse_ref=None, what=""):
    rep = report(o_test, o_ref, lse_test, lse_ref)
    assert passes(rep), f"parity failed {what}: {rep}"
    return rep


# ------------------------------------------------------------------------------------------------
# KDA chunked prefill
# ------------------------------------------------------------------------------------------------
# The chunkwise kernel rounds each operand of its contractions to bf16 (relative 2^-9) and keeps
# the state and every accumulation in fp32.  One output combines a handful of such products, and
# the state carries their errors over its memory horizon, where the decay damps them.  A CPU model
# of the kernel's rounding points against the fp64 oracle gives max-abs errors of ~0.6 % and
# mean-abs errors of ~0.45 % of the output's size, up to 4,096-token chunks and decays as slow as
# 0.9998 per token.  The tolerance is the attention one (2e-2 max, 2e-3 mean) on outputs of size up
# to 2, scaled with the output's size beyond that.

def kda_scale(ref):
    ref = np.asarray(ref, dtype=np.float64)
    return max(1.0, float(np.abs(ref).max()) / 2.0) if ref.size else 1.0


def kda_report(test, ref):
    rep = report(test, ref)
    s = kda_scale(ref)
    rep["scale"] = s
    rep["ok"] = rep["finite"] and rep["max_abs"] <= TOL_MAX_ABS * s and rep["mean_abs"] <= TOL_MEAN_ABS * s
    return rep


def assert_kda_parity(test, ref, what=""):
    rep = kda_report(test, ref)
    assert rep["ok"], f"KDA parity failed {what}: {rep}"
    return rep
