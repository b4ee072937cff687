"""Empirical MatMul cost for the simulator's device model.

The paper's simulator gives matrix multiplications an empirical cost: a
linear regression in the sizes of the input tensors, fitted on timings of
that one op alone over a range of operand shapes (Sec. 4, implementation
notes); some coefficients then play the part of hardware parameters such as
launch overhead.  This module does that for the GPU it
runs on:

    python -m paper_2111_05426_amd.calibrate [--dtype fp16] [--reps 20] [--out FILE]

times one matrix multiplication C[m, n] = A[m, k] B[k, n] per shape (HIP
events around `reps` back-to-back products, operands resident in device
memory), and fits two forms:

* the paper's linear form (the baseline)

      t = c0 + c1 * flops + c2 * bytes,   flops = 2 m n k,
                                          bytes = e (m k + k n + m n)

  by non-negative least squares on relative error;

* the same with the reduction length k as a fourth regressor and a floor,

      t = max(floor, c0 + c1 * flops + c2 * bytes + c3 * k),

  fitted for the least worst relative error.  A product of few output tiles
  and a long k runs its k loop serially (64 x 256 x 12288 takes longer than
  2048 x 1536 x 1536, which has 96 times its flops), which neither flops nor
  bytes show; and products issued back to back from the host never finish
  faster than their dispatch, which the floor models.

Every coefficient must be >= 0 for the device model.  The result is a
5-tuple (c0, c1, c2, c3, floor) for `DeviceSpec.matmul` /
`dsim_device_model.mm_c*`, `mm_floor` (c3 = floor = 0 is the linear form).
The products are the measured op, not part of the simulator: they run
through the framework's matmul (hipBLASLt), as the op a simulated program
would call.
"""
import argparse
import json
import sys

import numpy as np

# (m, n, k): row counts of microbatches by hidden sizes of the models the
# simulator studies (MLP 256 .. 8192 wide, GPT-2 768, GPT-3 12288 with its
# tensor-parallel slices), from launch-bound to compute-bound
SHAPES = [(m, n, k) for m in (64, 512, 2048, 8192) for n in (256, 1536, 6144, 12288) for k in (256, 1536, 12288)]


def design(flops, nbytes):
    """Rows (1, flops, bytes) of the regression."""
    flops = np.asarray(flops, np.float64)
    nbytes = np.asarray(nbytes, np.float64)
    return np.stack([np.ones_like(flops), flops, nbytes], axis=1)


def fit(flops, nbytes, seconds):
    """Non-negative least squares of t = c0 + c1 flops + c2 bytes, each row
    weighted by 1 / t (relative error).  Returns ((c0, c1, c2), worst
    relative error of the fit over the samples)."""
    from scipy.optimize import nnls
    X = design(flops, nbytes)
    t = np.asarray(seconds, np.float64)
    w = 1.0 / t
    # scale the columns so the solver sees numbers of similar size
    scale = np.maximum(np.abs(X).max(axis=0), 1e-300)
    coef, _ = nnls(X * w[:, None] / scale, t * w)
    c = coef / scale
    pred = X @ c
    return tuple(float(v) for v in c), float(np.max(np.abs(pred - t) / t))


def _feasible(X, t, z, upper):
    """Non-negative c with X c <= t (1 + z) on every sample and X c >=
    t (1 - z) on the `upper` ones, or None (a linear program)."""
    from scipy.optimize import linprog
    scale = np.maximum(np.abs(X / t[:, None]).max(axis=0), 1e-300)
    A = X / t[:, None] / scale
    rows = [A, -A[upper]]
    rhs = [np.full(len(t), 1.0 + z), np.full(int(upper.sum()), -(1.0 - z))]
    r = linprog(np.zeros(X.shape[1]), A_ub=np.vstack(rows), b_ub=np.concatenate(rhs),
                bounds=[(0, None)] * X.shape[1], method="highs")
    return r.x / scale if r.status == 0 else None


def fit_max(flops, nbytes, k, seconds, tol=1e-5):
    """t = max(floor, c0 + c1 flops + c2 bytes + c3 k), every coefficient
    >= 0, with the least worst relative error over the samples.  For an
    error bound z the floor can carry every sample whose time is within
    t_min (1 + z) / (1 - z) (a floor in [t_j (1 - z), t_min (1 + z)] is
    within z of each of them); the rest need the linear part within z,
    which is a linear feasibility problem.  Carrying more samples on the
    floor only drops constraints, so bisection on z finds the minimax.
    Returns ((c0, c1, c2, c3, floor), worst relative error)."""
    t = np.asarray(seconds, np.float64)
    X = np.stack([np.ones_like(t), np.asarray(flops, np.float64), np.asarray(nbytes, np.float64),
                  np.asarray(k, np.float64)], axis=1)
    tmin = t.min()

    def attempt(z):
        upper = t * (1.0 - z) > tmin * (1.0 + z)
        c = _feasible(X, t, z, upper)
        if c is None:
            return None
        low = t[~upper]
        # the floor nearest to every floor-carried sample in relative terms
        floor = 2.0 * low.min() * low.max() / (low.min() + low.max()) if len(low) else 0.0
        return c, floor

    lo, hi = 0.0, 1.0
    best = attempt(hi)
    while best is None:
        hi *= 2.0
        best = attempt(hi)
    while hi - lo > tol:
        mid = 0.5 * (lo + hi)
        got = attempt(mid)
        if got is None:
            lo = mid
        else:
            hi, best = mid, got
    c, floor = best
    coef = tuple(float(v) for v in c) + (float(floor),)
    return coef, float(np.max(np.abs(predict(coef, flops, nbytes, k) - t) / t))


def predict(coef, flops, nbytes, k=0.0):
    """Seconds per product under (c0, c1, c2) or (c0, c1, c2, c3, floor), in
    the simulator's order of operations."""
    c = tuple(coef) + (0.0, 0.0)[:5 - len(coef)]
    flops, nbytes = np.asarray(flops, np.float64), np.asarray(nbytes, np.float64)
    lin = ((c[0] + c[1] * flops) + c[2] * nbytes) + c[3] * np.asarray(k, np.float64)
    return np.maximum(c[4], lin)


def shape_class(m, n, k, seconds):
    """Reporting classes of a measured product: dispatch-bound (under 25 us),
    long-k (k at least twice max(m, n)), and the rest."""
    if seconds < 25e-6:
        return "dispatch"
    if k >= 2 * max(m, n):
        return "long_k"
    return "large"


def error_by_class(rows, coef):
    """Worst relative error of a fit per shape class."""
    out = {}
    for m, n, k, fl, by, s in rows:
        e = abs(float(predict(coef, fl, by, k)) - s) / s
        c = shape_class(m, n, k, s)
        out[c] = max(out.get(c, 0.0), e)
    return out


def measure(shapes=SHAPES, dtype="fp16", reps=20, warmup=3):
    """Seconds per product for every (m, n, k); rows of
    (m, n, k, flops, bytes, seconds)."""
    import torch
    dt = {"fp16": torch.float16, "bf16": torch.bfloat16, "fp32": torch.float32}[dtype]
    e = torch.tensor([], dtype=dt).element_size()
    gen = torch.Generator(device="cuda").manual_seed(0)
    rows = []
    for m, n, k in shapes:
        a = torch.randn(m, k, device="cuda", dtype=dt, generator=gen)
        b = torch.randn(k, n, device="cuda", dtype=dt, generator=gen)
        c = torch.empty(m, n, device="cuda", dtype=dt)
        for _ in range(warmup):
            torch.matmul(a, b, out=c)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch.matmul(a, b, out=c)
        e1.record()
        torch.cuda.synchronize()
        s = e0.elapsed_time(e1) * 1e-3 / reps
        rows.append((m, n, k, 2 * m * n * k, e * (m * k + k * n + m * n), s))
        del a, b, c
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--dtype", default="fp16", choices=("fp16", "bf16", "fp32"))
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--out", default=None, help="write the samples and the fit as JSON")
    args = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():
        print("calibrate needs a GPU", file=sys.stderr)
        return 1
    rows = measure(dtype=args.dtype, reps=args.reps)
    fl, by, kk, sec = ([r[i] for r in rows] for i in (3, 4, 2, 5))
    lin, worst_lin = fit(fl, by, sec)
    coef, worst = fit_max(fl, by, kk, sec)
    out = {"device": torch.cuda.get_device_name(0), "dtype": args.dtype, "reps": args.reps,
           "matmul": {"c0": coef[0], "c1": coef[1], "c2": coef[2], "c3": coef[3], "floor": coef[4]},
           "worst_relative_error": worst, "worst_by_class": error_by_class(rows, coef),
           "linear": {"c0": lin[0], "c1": lin[1], "c2": lin[2], "worst_relative_error": worst_lin,
                      "worst_by_class": error_by_class(rows, lin)},
           "samples": [dict(m=r[0], n=r[1], k=r[2], flops=r[3], bytes=r[4], seconds=r[5],
                            fitted=float(predict(coef, r[3], r[4], r[2])), linear=float(predict(lin, r[3], r[4])))
                       for r in rows]}
    text = json.dumps(out, indent=1)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
    print(json.dumps({k: out[k] for k in ("device", "dtype", "matmul", "worst_relative_error", "worst_by_class",
                                          "linear")}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
