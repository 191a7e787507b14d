"""Float parity metrics shared by the GPU tests.

* normwise: max_i |g_i - r_i| / max_i |r_i|  (the bound the spec states:
  1e-5 for fp32, 2e-2 for bf16 / fp16 storage with fp32 accumulation);
* p999: the 99.9th percentile over elements of |g_i - r_i| / max(|r_i|, rms(r)),
  so that a localized error cannot hide under a large maximum.

Elementwise bounds (derived from the arithmetic, not fitted):
* one rounding to bf16 relative to a value is at most 2^-8 (half an ulp; an ulp is
  2^-7 of the leading power of two), so two roundings of values that differ only
  in fp32 accumulation order differ by at most one ulp, < 0.8%: single ops get 1e-2;
* a chain of L ops that each store their output in the 16-bit type adds at most one
  such flip per op, propagated through normalised layers with gain ~1: the block
  (three stored stages) gets 2e-2, the network (~40 stored stages, random-walk
  sqrt(40) ~ 6 ulps) 5e-2;
* fp32: accumulation order over at most ~10^4 terms, ~1e-6 relative: 1e-4.
"""
import json
import os

import numpy as np

NORMWISE = {"f32": 1e-5, "bf16": 2e-2, "f16": 2e-2}
ELEMWISE = {"op": {"f32": 1e-4, "bf16": 1e-2, "f16": 1e-2},
            "block": {"f32": 1e-4, "bf16": 2e-2, "f16": 2e-2},
            "network": {"f32": 1e-4, "bf16": 5e-2, "f16": 5e-2}}

_LOG = os.environ.get("SPV_PARITY_LOG")  # a path: one JSON line per comparison is appended


def errors(g, r, scale=None):
    """(normwise, p999) of g against r (float arrays of one shape); scale overrides max|r|."""
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    if r.size == 0:
        return 0.0, 0.0
    d = np.abs(g - r)
    mx = float(np.abs(r).max()) if scale is None else float(scale)
    nw = float(d.max() / max(mx, 1e-30))
    rms = float(np.sqrt(np.mean(r * r)))
    rel = d / np.maximum(np.abs(r), max(rms, 1e-30))
    return nw, float(np.percentile(rel, 99.9))


def check(g, r, dtype, kind="op", what="", normwise_tol=None, elemwise_tol=None, scale=None):
    """Assert both bounds; print (and optionally log) the two errors."""
    nw, p = errors(g, r, scale)
    tn = NORMWISE[dtype] if normwise_tol is None else normwise_tol
    te = ELEMWISE[kind][dtype] if elemwise_tol is None else elemwise_tol
    rec = {"what": what or os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0], "dtype": dtype, "kind": kind,
           "normwise": nw, "p999": p, "normwise_tol": tn, "p999_tol": te}
    print(f"parity {rec['what']}: normwise {nw:.3e} (<= {tn}), p99.9 {p:.3e} (<= {te})", flush=True)
    if _LOG:
        with open(_LOG, "a") as f:
            f.write(json.dumps(rec) + "\n")
    assert nw <= tn, f"normwise error {nw:.3e} > {tn}"
    assert p <= te, f"elementwise 99.9th percentile {p:.3e} > {te}"
    return nw
