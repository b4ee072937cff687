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
memory), and fits

    t = c0 + c1 * flops + c2 * bytes,   flops = 2 m n k,
                                        bytes = e (m k + k n + m n)

by non-negative least squares on relative error (every coefficient must be
>= 0 for the device model).  The result is a (c0, c1, c2) triple for
`DeviceSpec.matmul` / `dsim_device_model.mm_c*`.  The products are the
measured op, not part of the simulator: they run through the framework's
matmul (hipBLASLt), as the op a simulated program would call.
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
    coef, worst = fit([r[3] for r in rows], [r[4] for r in rows], [r[5] for r in rows])
    out = {"device": torch.cuda.get_device_name(0), "dtype": args.dtype, "reps": args.reps,
           "matmul": {"c0": coef[0], "c1": coef[1], "c2": coef[2]}, "worst_relative_error": worst,
           "samples": [dict(m=r[0], n=r[1], k=r[2], flops=r[3], bytes=r[4], seconds=r[5]) for r in rows]}
    text = json.dumps(out, indent=1)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
    print(json.dumps({k: out[k] for k in ("device", "dtype", "matmul", "worst_relative_error")}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
