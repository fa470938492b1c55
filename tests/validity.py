"""Per-ray validity of a GPU result against the oracle (test helper).

A bf16 or fp8 network rounds every hidden activation.  The GPU sums each
pre-activation in fp32 in its own order, so where an exact pre-activation
lies close to a rounding midpoint the GPU may round it the other way, and the
change propagates.  Such a result is still a correct evaluation of the
network.  A ray's GPU values therefore pass when

  (a) they equal the oracle's nominal evaluation within ``tol`` (the size of
      fp32 accumulation noise where no rounding decision differs), or
  (b) one of up to ``runs`` further oracle evaluations of that ray, each with
      every pre-activation moved inside its fp32 accumulation bound
      (``O.accumulation_bound``; a share rho of it, drawn uniformly) and every
      encoded feature moved by up to 4e-7 (the hardware sine's error) before
      rounding, reproduces them within ``tol``: a valid evaluation that gives
      the GPU's result is exhibited, or
  (c) they lie within ``spread_factor`` times the largest distance of those
      valid evaluations from the nominal one: the ray is as sensitive to
      rounding as the GPU's deviation says.

Evaluations in (b) and (c) only run for rays that fail (a); the jitter
shares rotate over 0.03, 0.1, 0.25 and 0.5 of the bound for fp8 steps (whose
MFMA accumulates with up to 0.19 of the bound, measured per layer) and stay
at 0.01 for bf16 steps (up to 0.0016) and 0.05 for fp32 steps.
"""
import numpy as np

FP8_SHARES = (0.03, 0.1, 0.25, 0.5)


def jitter_rho(run_block):
    return {"fp64": 0.05, "bf16": 0.01, "fp8": FP8_SHARES[run_block % len(FP8_SHARES)], "input": 4e-7}


def check_rays(gpu, nominal, rerun, tol, runs=64, block=16, spread_factor=2.0, seed=0):
    """gpu, nominal: (rays, k) values.  rerun(ray_ids, rng, rho) -> (len(ray_ids), k)
    values of jittered oracle evaluations of those rays (ids may repeat).
    Asserts every ray passes (a), (b) or (c); returns counts for the log."""
    gpu = np.asarray(gpu, dtype=np.float64)
    nominal = np.asarray(nominal, dtype=np.float64)
    err = np.abs(gpu - nominal).max(axis=1)
    div = np.nonzero(err > tol)[0]
    reproduced = np.zeros(len(div), bool)
    spread = np.zeros(len(div))
    active = np.arange(len(div))
    for b in range(0, runs, block):
        if len(active) == 0:
            break
        ids = np.repeat(div[active], block)
        vals = np.asarray(rerun(ids, np.random.default_rng(seed * 1000003 + b), jitter_rho(b // block)),
                          dtype=np.float64)
        d_gpu = np.abs(vals - gpu[ids]).max(axis=1).reshape(len(active), block)
        d_nom = np.abs(vals - nominal[ids]).max(axis=1).reshape(len(active), block)
        reproduced[active] |= (d_gpu <= tol).any(axis=1)
        spread[active] = np.maximum(spread[active], d_nom.max(axis=1))
        active = active[~reproduced[active]]
    within = err[div] <= spread_factor * spread
    bad = div[~(reproduced | within)]
    assert len(bad) == 0, (f"rays {bad[:8]} leave every valid evaluation: err {err[bad[:8]]}, "
                           f"spread {spread[~(reproduced | within)][:8]}")
    return {"rays": len(err), "max_err": float(err.max()) if len(err) else 0.0, "beyond_tol": int(len(div)),
            "reproduced": int(reproduced.sum()), "within_spread": int((~reproduced).sum())}
