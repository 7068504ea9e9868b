"""Pins of the AdamW replay oracle (optimizer-boundary check, Sec. 9).

The update's fp32 rounding order is this implementation's reading; what the
mathematics fixes is pinned here:

* torch.optim.AdamW on the CPU in float64 (an independent implementation of
  the same update) agrees within a bound derived from the fp32 roundings;
  plausible mistakes (weight decay dropped or not scaled by lr, either bias
  correction dropped, eps inside the bias-corrected root, the interpolation
  weight swapped, the sign of the step) exceed it by orders of magnitude;
* closed forms: zero gradient and zero moments leave p * (1 - lr wd) bit for
  bit; a first step moves each coordinate by lr |g| / (|g| + eps) against
  the sign of g;
* NaN and Inf propagation, with the canonical NaN;
* the rotating slice covers every element once per cycle;
* the check attributes exactly the planted input faults, and its signature
  vote equals a vote on the raw bytes.
"""
import numpy as np
import pytest

import oracle
import workloads
from oracle import adamw

torch = pytest.importorskip("torch")

U = 2.0 ** -24


def _torch_adamw(p, g, m, v, lr, b1, b2, eps, wd, t, dtype=torch.float64):
    P = torch.nn.Parameter(torch.from_numpy(p).to(dtype))
    P.grad = torch.from_numpy(g).to(dtype)
    opt = torch.optim.AdamW([P], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd, foreach=False)
    st = opt.state[P]
    st["step"] = torch.tensor(float(t - 1))
    st["exp_avg"] = torch.from_numpy(m).to(dtype).clone()
    st["exp_avg_sq"] = torch.from_numpy(v).to(dtype).clone()
    opt.step()
    return (P.detach().numpy().astype(np.float64), st["exp_avg"].numpy().astype(np.float64),
            st["exp_avg_sq"].numpy().astype(np.float64))


def _bounds(p, g, m, v, lr, b1, b2, eps, wd, t, ref):
    """Per-element error bounds of the fp32 update against exact arithmetic:
    m1 from three roundings plus the rounded weight, v1 from four positive
    terms' roundings, p2 from the decay, the propagated m1 error through
    lr/(1 - b1^t) / d and about ten roundings of the quotient."""
    p, g, m, v = (a.astype(np.float64) for a in (p, g, m, v))
    p2, m1, v1 = ref
    e_m = 4 * U * (np.abs(m) + np.abs(g))
    e_v = 4 * U * (np.abs(v) + (1 - b2) * g * g)
    a = lr / (1 - b1 ** t)
    d = np.sqrt(np.maximum(v1, 0)) / np.sqrt(1 - b2 ** t) + eps
    upd = a * np.abs(m1) / d
    e_p = 2 * U * np.abs(p) + a * e_m / d + 10 * U * upd + U * np.abs(p2)
    return e_p, e_m, e_v


def _state(seed, n, first=False):
    rng = np.random.default_rng(seed)
    p = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    m = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    v = np.abs(rng.standard_normal(n) * 1e-7).astype(np.float32)
    g[:500] = 0                                   # eps-dominated denominators
    v[250:750] = 0
    if first:
        m[:] = 0
        v[:] = 0
    return p, g, m, v


CASES = [  # (beta1, beta2, weight_decay, step): both interpolation branches
    (0.9, 0.999, 0.1, 1), (0.9, 0.999, 0.0, 7), (0.9, 0.95, 0.1, 1000),
    (0.3, 0.999, 0.01, 3), (0.5, 0.99, 0.1, 2), (0.0, 0.999, 0.1, 5),
]


@pytest.mark.parametrize("b1,b2,wd,t", CASES)
def test_adamw_matches_torch_fp64_within_rounding_bound(b1, b2, wd, t):
    p, g, m, v = _state(t, 50000, first=(t == 1))
    args = (1e-3, b1, b2, 1e-8, wd, t)
    ref = _torch_adamw(p, g, m, v, *args)
    out = adamw.adamw_step(p, g, m, v, *args)
    for name, o, r, b in zip(("param", "exp_avg", "exp_avg_sq"), out, ref,
                             _bounds(p, g, m, v, *args, ref)):
        err = np.abs(o.astype(np.float64) - r)
        assert (err <= b).all(), f"{name}: worst {np.max(err / np.maximum(b, 1e-300)):.3g} of bound"


def _mutant(kind):
    f = np.float32

    def step(p, g, m, v, lr, b1, b2, eps, wd, t):
        s = adamw.scalars(lr, b1, b2, eps, wd, t)
        p1 = p * (f(1) if kind == "no_decay" else f(1 - wd) if kind == "decay_without_lr"
                  else s["decay"])
        w = s["one_minus_w"] if kind == "weight_swapped" else s["w"]
        m1 = m + w * (g - m)
        v1 = v * s["beta2"] + (s["c2"] * g) * g
        s2 = f(1) if kind == "no_bias2" else s["s2"]
        a = f(lr) if kind == "no_bias1" else s["step_size"]
        d = (np.sqrt(v1) + s["eps"]) / s2 if kind == "eps_inside" else np.sqrt(v1) / s2 + s["eps"]
        p2 = p1 + (a if kind == "sign" else -a) * (m1 / d)
        return p2, m1, v1
    return step


@pytest.mark.parametrize("kind", ["no_decay", "decay_without_lr", "weight_swapped", "no_bias2",
                                  "no_bias1", "eps_inside", "sign"])
def test_rounding_bound_rejects_plausible_mistakes(kind):
    worst = 0.0
    for b1, b2, wd, t in CASES[:4]:
        p, g, m, v = _state(t + 10, 20000, first=(t == 1))
        args = (1e-3, b1, b2, 1e-8, wd, t)
        ref = _torch_adamw(p, g, m, v, *args)
        with np.errstate(all="ignore"):
            out = _mutant(kind)(p, g, m, v, *args)
        for o, r, b in zip(out, ref, _bounds(p, g, m, v, *args, ref)):
            worst = max(worst, float(np.max(np.abs(o.astype(np.float64) - r) / np.maximum(b, 1e-300))))
    assert worst > 10.0, f"mutant {kind} stays within the bound ({worst:.3g})"


def test_zero_gradient_and_state_only_decay():
    rng = np.random.default_rng(3)
    p = (rng.standard_normal(4096) * 0.02).astype(np.float32)
    z = np.zeros_like(p)
    for wd in (0.0, 0.1, 0.5):
        p2, m1, v1 = adamw.adamw_step(p, z, z, z, 1e-3, 0.9, 0.999, 1e-8, wd, 4)
        assert np.array_equal(p2, p * np.float32(1 - 1e-3 * wd))
        assert not m1.any() and not v1.any()


def test_first_step_moves_by_lr_against_the_gradient():
    rng = np.random.default_rng(4)
    p = (rng.standard_normal(4096) * 0.02).astype(np.float32)
    g = (rng.standard_normal(4096) * 1e-2).astype(np.float32)
    z = np.zeros_like(p)
    lr, eps = 1e-3, 1e-8
    p2, m1, v1 = adamw.adamw_step(p, g, z, z, lr, 0.9, 0.999, eps, 0.0, 1)
    gd = g.astype(np.float64)
    expect = p.astype(np.float64) - lr * gd / (np.abs(gd) + eps)
    assert np.allclose(p2, expect, rtol=0, atol=4 * U * (np.abs(p) + lr).max())
    assert np.array_equal(m1, np.float32(1 - 0.9) * g)          # 0 + w (g - 0), one rounding
    assert np.array_equal(v1, (np.float32(1 - 0.999) * g) * g)


def test_nan_and_inf_propagate_as_canonical_nan():
    f = np.float32
    p = np.full(5, 0.5, f)
    g = np.array([np.nan, np.inf, -np.inf, 1e-3, 1e-3], f)
    m = np.zeros(5, f)
    v = np.array([0, 0, 0, -1e-3, 1e-6], f)                    # negative v: root of < 0
    g.view(np.uint32)[0] = 0xFFC12345                          # payload and sign to drop
    p2, m1, v1 = adamw.adamw_step(p, g, m, v, 1e-3, 0.9, 0.999, 1e-8, 0.0, 3)
    bits = np.uint32(0x7FC00000)
    assert p2.view(np.uint32)[0] == bits and m1.view(np.uint32)[0] == bits
    assert v1.view(np.uint32)[0] == bits
    assert m1[1] == np.inf and v1[1] == np.inf and p2.view(np.uint32)[1] == bits   # inf / inf
    assert m1[2] == -np.inf and v1[2] == np.inf and p2.view(np.uint32)[2] == bits
    assert v1[3] < 0 and p2.view(np.uint32)[3] == bits and np.isfinite(m1[3])
    assert np.isfinite(p2[4]) and p2[4] < 0.5


@pytest.mark.parametrize("numel,S", [(10, 4), (12, 4), (3, 4), (65536 * 3 + 1000, 65536), (1, 1)])
def test_rotating_slice_covers_every_element_once_per_cycle(numel, S):
    n_slices = -(-numel // S)
    seen = np.zeros(numel, np.int64)
    for k in range(n_slices):
        off, n = adamw.slice_bounds(k, numel, S)
        assert 0 < n <= S and off % S == 0
        seen[off:off + n] += 1
    assert (seen == 1).all()
    assert adamw.slice_bounds(n_slices, numel, S) == adamw.slice_bounds(0, numel, S)
    assert adamw.slice_bounds(5, 0, S) == (0, 0)


def test_boundary_check_attributes_exactly_the_planted_faults():
    w = workloads.make(6, device="cpu", scale="small")
    state = [[t.numpy() for t in x] for x in w.state]
    n_slices = -(-w.numel // w.slice_elems)
    found = set()
    for k in range(n_slices):
        res = adamw.boundary_check(state, k, w.hparams, w.slice_elems)
        loc = res["localize"]
        assert loc["counts"][1] == 0                           # one replica per fault: no undecided
        for u, r in zip(loc["unit"], loc["replica"]):
            found.add((k, int(u), int(r)))
        # the signature vote equals a vote on the raw bytes of the same slices
        off, n = res["offset"], res["n"]
        chunks = [[np.ascontiguousarray(x[r][off:off + n]).view(np.uint8) for x in state] +
                  [o.view(np.uint8) for o in res["outputs"][r]] for r in range(w.R)]
        st, bm, mj = oracle.vote_bytes(chunks)
        assert np.array_equal(st, res["status"]) and np.array_equal(bm, res["bitmap"])
    inputs = {(k, u, r) for (k, u, r) in found if u < 4}
    planted = {(w.fault_slices[i], f.tensor, f.replica) for i, f in enumerate(w.faults)}
    assert inputs == planted
    # every replayed-output outlier belongs to a replica with a faulty input in that slice
    for k, u, r in found - inputs:
        assert any(k == kk and r == rr for kk, _, rr in planted)
    # a corrupted gradient changes the replayed parameter and both moments
    kg, _, rg = next(x for x in planted if x[1] == 1)
    assert {(kg, 4, rg), (kg, 5, rg), (kg, 6, rg)} <= found
