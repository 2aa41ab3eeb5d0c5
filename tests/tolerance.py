"""Pass/fail rule for comparing an output against the fp64 oracle.

PASS requires both ``max|out - ref| <= max_abs`` and
``||out - ref||_2 / ||ref||_2 <= rel_l2`` over the whole output, in fp64.
bf16 inputs with fp32 accumulation: 2e-2 and 1e-2. fp32 inputs: 1e-5 and
1e-5. A max-abs bound alone would pass an all-zeros output, because with
N(0, 1) inputs the attention output shrinks like 1/sqrt(context), so the
relative L2 bound is the one that catches wrong results.
"""
import numpy as np

TOL = {"bf16": (2e-2, 1e-2), "f32": (1e-5, 1e-5)}


def compare(out, ref, dtype):
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert out.shape == ref.shape, (out.shape, ref.shape)
    d = out - ref
    max_abs = float(np.max(np.abs(d))) if d.size else 0.0
    nref = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(d)) / nref if nref > 0 else float(np.linalg.norm(d))
    tol_abs, tol_rel = TOL[dtype]
    finite = bool(np.all(np.isfinite(out)))
    return {"max_abs": max_abs, "rel_l2": rel, "finite": finite,
            "pass": finite and max_abs <= tol_abs and rel <= tol_rel}
