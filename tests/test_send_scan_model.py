"""The transform kernel's Send scan (`send_scan` in csrc/parametric.hip),
modelled lane by lane on the CPU and checked against the step-by-step walk
of the same slot (Sec. 2.1: a Send starts when both of its stages are free
and both end together; the slot's Sends run in ascending source order).

Both functions below restate, for one 64-lane wavefront, what the kernel
computes: `steps` the run-parallel loop, `scan` the segmented prefix scans
in integer ulps, each scan taken the way the kernel takes it (`seg_scan`:
rows of 16 lanes first, then the carries of row_bcast:15 and row_bcast:31).  Neither calls the library or the oracle; the GPU parity
tests check the kernel itself.  Here the model of the scan must give the
same doubles as the step walk whenever it does not decline, on random slots
with dead lanes, partial segments, both directions, pairs of opposite Sends,
half-way costs and clocks across binades."""
import math
import random

import numpy as np


def _shr(v, fill):   # lane i receives lane i - 1's value
    return [fill] + v[:-1]


def _shl(v, fill):   # lane i receives lane i + 1's value
    return v[1:] + [fill]


def _flags(W, P, live, sdir):
    s = [i % W for i in range(64)]
    l_dir, r_dir = _shr(sdir, 0), _shl(sdir, 0)
    from_left = [live[i] and s[i] >= 1 and l_dir[i] == 1 for i in range(64)]
    from_right = [live[i] and s[i] + 1 < P[i] and r_dir[i] == -1 for i in range(64)]
    return s, l_dir, from_left, from_right


def _positions(start_flags):
    pos, st = [], 0
    for i, f in enumerate(start_flags):
        if f:
            st = i
        pos.append(i - st)
    return pos


def seg_scan(v, spos, nlev, op):
    """`seg_scan` of the kernel, lane by lane: DPP row_shr:o moves stay inside
    rows of 16 lanes, row_bcast:15 hands lane 15 of rows 0 and 2 to rows 1
    and 3, row_bcast:31 hands lane 31 to rows 2 and 3."""
    v = list(v)
    sr = [min(spos[i], i & 15) for i in range(64)]
    for lev in range(min(nlev, 4)):
        o = 1 << lev
        up = [v[i - o] if (i & 15) >= o else 0 for i in range(64)]
        v = [op(v[i], up[i]) if sr[i] >= o else v[i] for i in range(64)]
    if any(spos[i] > (i & 15) for i in range(64)):
        up = [v[(i & ~15) - 1] if (i >> 4) in (1, 3) else 0 for i in range(64)]
        v = [op(v[i], up[i]) if ((i & 16) and spos[i] > (i & 15)) else v[i] for i in range(64)]
        up = [v[31] if i >= 32 else 0 for i in range(64)]
        v = [op(v[i], up[i]) if (i >= 32 and spos[i] >= i - 31) else v[i] for i in range(64)]
    return v


def plain_scan(v, spos, op):
    out = list(v)
    for i in range(64):
        if spos[i] > 0:
            out[i] = op(out[i - 1], v[i])
    return out


def steps(W, P, live, sdir, cost, clk):
    s, l_dir, from_left, from_right = _flags(W, P, live, sdir)
    l_cost, r_cost = _shr(cost, 0.0), _shl(cost, 0.0)
    linked = [s[i] >= 1 and s[i] < P[i] and (l_dir[i] == 1 or sdir[i] == -1) for i in range(64)]
    rpos = _positions([not x for x in linked])
    clk = list(clk)
    for r in range(max(rpos) + 1):
        cl, cr = _shr(clk, 0.0), _shl(clk, 0.0)
        new = list(clk)
        for i in range(64):
            src = rpos[i] == r and sdir[i] != 0
            tl = rpos[i] == r + 1 and from_left[i]
            tr = rpos[i] == r - 1 and from_right[i]
            a = cl[i] if ((src and sdir[i] < 0) or tl) else cr[i]
            if src or tl or tr:
                new[i] = max(a, clk[i]) + (cost[i] if src else (l_cost[i] if tl else r_cost[i]))
        clk = new
    return clk


def scan(W, P, live, sdir, cost, clk):
    """None where the kernel declines the scans (then it walks the steps)."""
    s, _, from_left, from_right = _flags(W, P, live, sdir)
    cl, cr = _shr(clk, 0.0), _shl(clk, 0.0)
    z = [max(clk[i], cr[i]) if sdir[i] > 0 else (max(clk[i], cl[i]) if sdir[i] < 0 else clk[i]) for i in range(64)]
    carry = [sdir[i] < 0 or from_left[i] for i in range(64)]
    involved = [sdir[i] != 0 or from_left[i] or from_right[i] for i in range(64)]
    spos = _positions([not c for c in carry])
    e = [0] * 64
    for i in range(64):
        if spos[i] == 0:
            if involved[i]:
                if not (0.0 < z[i] < math.inf):
                    return None
                e[i] = math.frexp(z[i])[1] - 1
                if e[i] < -1022:
                    return None
        else:
            e[i] = e[i - 1]
    K = [math.ldexp(z[i], 52 - e[i]) for i in range(64)]
    Wu = [0.0] * 64
    for i in range(64):
        if sdir[i] != 0:
            if not (0.0 <= cost[i] < math.inf):
                return None
            t = math.ldexp(cost[i], 52 - e[i])
            Wu[i] = float(np.rint(t))
            if abs(t - Wu[i]) == 0.5:
                return None
    nlev = max(spos).bit_length()   # 2^nlev > the largest position
    q = seg_scan(Wu, spos, nlev, lambda a, b: a + b)
    y = seg_scan([K[i] - (q[i] - Wu[i]) for i in range(64)], spos, nlev, max)
    v = [q[i] + y[i] for i in range(64)]
    if any(involved[i] and not v[i] < 2.0 ** 53 for i in range(64)):
        return None
    vd = [math.ldexp(v[i], e[i] - 52) for i in range(64)]
    vr = _shl(vd, 0.0)
    return [vr[i] if from_right[i] else (vd[i] if (sdir[i] != 0 or from_left[i]) else clk[i]) for i in range(64)]


def _random_slot(rng):
    W = rng.choice([1, 2, 4, 8, 16, 32, 64])
    P, live = [], []
    for _ in range(64 // W):
        p = rng.randint(1, W) if rng.random() < 0.8 else W
        alive = rng.random() < 0.95
        P += [p] * W
        live += [alive and j < p for j in range(W)]
    base = 2.0 ** rng.uniform(-12, 9)
    mode = rng.random()
    if mode < 0.2:
        clk = [base] * 64
    elif mode < 0.6:
        clk = [base * (1 + rng.uniform(0, 1e-3)) for _ in range(64)]
    else:
        clk = [base * rng.uniform(0.9, 1.1) for _ in range(64)]
    sdir = []
    for i in range(64):
        st = i % W
        opts = ([1] if st < P[i] - 1 else []) + ([-1] if st > 0 else [])
        if not live[i] or not opts or rng.random() < 0.1:
            sdir.append(0)
        elif mode < 0.4 and 1 in opts and rng.random() < 0.8:
            sdir.append(1)
        else:
            sdir.append(rng.choice(opts))
    sc = 2.0 ** rng.uniform(-30, -5) * base
    half_ulp = math.ldexp(1.0, math.frexp(base)[1] - 54)
    kind = rng.random()
    cost = []
    for d in sdir:
        if d == 0:
            cost.append(0.0)
        elif kind < 0.3:
            cost.append(sc)
        elif kind < 0.45:
            cost.append(rng.randint(0, 9) * half_ulp)   # half-way cases
        else:
            cost.append(sc * rng.uniform(0.5, 2))
    return W, P, live, sdir, cost, clk


def test_scan_model_equals_steps():
    rng = random.Random(20261202)
    taken = declined = 0
    for trial in range(3000):
        slot = _random_slot(rng)
        got = scan(*slot)
        if got is None:
            declined += 1
            continue
        taken += 1
        want = steps(*slot)
        assert got == want, trial
    assert taken > 2000 and declined > 100


def test_scan_model_long_forward_run():
    """Pipeline fill: stages 0..62 each send forward, one run of 63 Sends."""
    clk = [1.0 + i * 2.0 ** -20 for i in range(64)]
    sdir = [1] * 63 + [0]
    cost = [2.0 ** -12 + 3.0 * 2.0 ** -40] * 64
    slot = (64, [64] * 64, [True] * 64, sdir, cost, clk)
    got = scan(*slot)
    assert got is not None and got == steps(*slot)
    # stage s ends where its own Send ended; the last two share the last one
    assert got[63] == got[62] and got[0] < got[63]


def test_seg_scan_rows_and_carries():
    """The row-then-carry order gives the plain left-to-right segmented scan
    for sums of integers (exact) and for maxima, on random segments that
    start anywhere, span rows or cover the whole wavefront."""
    rng = random.Random(7)
    for trial in range(2000):
        mode = rng.random()
        if mode < 0.1:
            starts = [i == 0 for i in range(64)]
        else:
            p = rng.choice([0.02, 0.1, 0.3, 0.7])
            starts = [i == 0 or rng.random() < p for i in range(64)]
        spos = _positions(starts)
        nlev = max(spos).bit_length()
        vals = [float(rng.randint(0, 2 ** 40)) for _ in range(64)]
        assert seg_scan(vals, spos, nlev, lambda a, b: a + b) == plain_scan(vals, spos, lambda a, b: a + b), trial
        ivals = [rng.randint(-2 ** 31, 2 ** 31) for _ in range(64)]
        assert seg_scan(ivals, spos, nlev, max) == plain_scan(ivals, spos, max), trial
