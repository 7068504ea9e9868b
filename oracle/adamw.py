"""AdamW replay oracle for the optimizer-boundary check.

TEST INFRASTRUCTURE ONLY, like the rest of this package.

Sec. 9 (optimizer boundary) and Sec. 6.2 (optimizer recipe): at a scheduled
check each replica re-applies the same base optimizer step to a copied slice
of its parameter, gradient and optimizer state, and exact C3 compares the
updated slices across replicas.  The base optimizer of the paper's
experiments is PyTorch's AdamW (Sec. 10); the update here is AdamW with
decoupled weight decay (Loshchilov and Hutter) in the operation order of
PyTorch's single-tensor AdamW without amsgrad:

    p1 = p * (1 - lr wd)
    m1 = lerp(m, g, 1 - b1)
    v1 = v * b2 + (1 - b2) g g
    p2 = p1 - lr / (1 - b1^t) * m1 / (sqrt(v1) / sqrt(1 - b2^t) + eps)

written in numpy float32, one rounding per operation (numpy does not fuse
multiply-add), with each scalar factor formed in fp64 and rounded to fp32 as
PyTorch passes it to an fp32 kernel.  NaN results are stored as the quiet NaN
0x7FC00000 so the hashed bytes do not depend on NaN payload propagation.

Pinned (tests/test_oracle.py): against torch.optim.AdamW on the CPU in
float64 within a bound derived from the fp32 roundings, for both branches of
the interpolation, several steps, with and without weight decay; against
closed forms (zero gradient and state leave p * (1 - lr wd); a first step
moves every coordinate by about lr against the sign of its gradient); and
NaN/Inf propagation.
"""
import math

import numpy as np

from . import F32, localize, signature, vote_exact

CANONICAL_NAN = np.uint32(0x7FC00000)


def scalars(lr, beta1, beta2, eps, weight_decay, step):
    """fp32 factors of one step t = step (>= 1), each formed in fp64 first."""
    f = np.float32
    w = f(1.0 - beta1)
    return {
        "decay": f(1.0 - lr * weight_decay),
        "w": w,
        "one_minus_w": f(1.0) - w,                # formed in fp32 inside the lerp
        "beta2": f(beta2),
        "c2": f(1.0 - beta2),
        "s2": f(math.sqrt(1.0 - beta2 ** step)),
        "eps": f(eps),
        "step_size": f(lr / (1.0 - beta1 ** step)),
    }


def _canon(x):
    bits = x.view(np.uint32).copy()
    bits[np.isnan(x)] = CANONICAL_NAN
    return bits.view(np.float32)


def adamw_step(p, g, m, v, lr, beta1, beta2, eps, weight_decay, step):
    """One AdamW step on fp32 arrays; returns (p2, m1, v1) as new arrays."""
    p, g, m, v = (np.asarray(a, dtype=np.float32) for a in (p, g, m, v))
    s = scalars(lr, beta1, beta2, eps, weight_decay, step)
    with np.errstate(all="ignore"):
        p1 = p * s["decay"]
        if abs(s["w"]) < np.float32(0.5):
            m1 = m + s["w"] * (g - m)
        else:
            m1 = g - (g - m) * s["one_minus_w"]
        v1 = v * s["beta2"] + (s["c2"] * g) * g
        d = np.sqrt(v1) / s["s2"] + s["eps"]
        p2 = p1 + (-s["step_size"]) * (m1 / d)
    return _canon(p2), _canon(m1), _canon(v1)


def slice_bounds(k, numel, slice_elems):
    """Rotating slice k of a tensor of numel elements: the k-th window of
    slice_elems elements, wrapping after the last (possibly shorter) one."""
    if numel <= 0:
        return 0, 0
    n_slices = -(-numel // slice_elems)
    off = (k % n_slices) * slice_elems
    return off, min(slice_elems, numel - off)


def boundary_check(state, k, hp, slice_elems):
    """Check k of the optimizer boundary on R replicas.

    state: [param, grad, exp_avg, exp_avg_sq], each a list of R fp32 numpy
    arrays of one length.  Signs the four input slices and the three replayed
    outputs of every replica (one chunk per tensor, Sec. 5.2), votes exactly
    per tensor (Algorithm 1) and localizes the outliers (Sec. 5.1).
    """
    R, numel = len(state[0]), state[0][0].size
    off, n = slice_bounds(k, numel, slice_elems)
    reps = []
    for r in range(R):
        ins = [np.ascontiguousarray(x[r][off:off + n], np.float32) for x in state]
        outs = adamw_step(*ins, lr=hp["lr"], beta1=hp["betas"][0], beta2=hp["betas"][1],
                          eps=hp["eps"], weight_decay=hp["weight_decay"], step=hp["step"])
        reps.append([a.view(np.uint8) for a in ins + list(outs)])
    metas = [(F32, (n,))] * 7
    rec = signature(reps, metas, slice_elems * 4)
    st, bm, mj = vote_exact(rec["sig"])
    loc = localize(st, bm, mj, R)
    return dict(offset=off, n=n, records=rec, status=st, bitmap=bm, majority=mj, localize=loc,
                outputs=[[np.frombuffer(a, np.float32) for a in rep[4:]] for rep in reps])
