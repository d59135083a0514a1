"""Parity gates shared by the GPU tests (comparison only, no attention math).

bf16 in / fp32 accumulate: max-abs <= 2e-2 and mean-abs <= 2e-3 over all
checked elements, plus relative Frobenius error <= 1e-2 and |lse error| <= 1e-3
(the plain gates alone accept an all-zero output at long prefixes).
fp32: max-abs <= 1e-4 and relative Frobenius <= 1e-5.
"""
import numpy as np

BF16_MAX_ABS, BF16_MEAN_ABS, BF16_REL_FRO, LSE_ABS = 2e-2, 2e-3, 1e-2, 1e-3
F32_MAX_ABS, F32_REL_FRO = 1e-4, 1e-5


def _stats(out, lse, ref, ref_lse):
    out = np.asarray(out, np.float64)
    err = np.abs(out - ref)
    st = {
        "max_abs": float(err.max()) if err.size else 0.0,
        "mean_abs": float(err.mean()) if err.size else 0.0,
        "rel_fro": float(np.linalg.norm(out - ref) / max(np.linalg.norm(ref), 1e-300)),
        "finite": bool(np.isfinite(out).all()),
    }
    if lse is not None:
        st["lse_max_abs"] = float(np.abs(np.asarray(lse, np.float64) - ref_lse).max())
    return st


def check_bf16(out, lse, ref, ref_lse):
    st = _stats(out, lse, ref, ref_lse)
    ok = (st["finite"] and st["max_abs"] <= BF16_MAX_ABS and st["mean_abs"] <= BF16_MEAN_ABS
          and st["rel_fro"] <= BF16_REL_FRO and st.get("lse_max_abs", 0.0) <= LSE_ABS)
    return ok, st


def check_f32(out, lse, ref, ref_lse):
    st = _stats(out, lse, ref, ref_lse)
    ok = (st["finite"] and st["max_abs"] <= F32_MAX_ABS and st["rel_fro"] <= F32_REL_FRO
          and st.get("lse_max_abs", 0.0) <= F32_MAX_ABS)
    return ok, st
