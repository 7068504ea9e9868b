"""Comparison helpers shared by the GPU parity tests (no method arithmetic).

Tolerance for the fp64 sums (GPU vs oracle), derived from the arithmetic:
the GPU sums each lane's elements in plain fp64 (at most a few hundred per
lane), meets lanes in a six-level butterfly and combines waves, tiles and
chunks with TwoSum compensation, so its error is bounded by roughly
(n_lane + 8) u sum|x| <= 1e-13 sqrt(n sumsq) for the chunk sizes here; the
oracle (Neumaier) is within a couple of ulp of the exact sum.  The check is
|gpu - ref| <= max(1e-6 |ref|, 1e-12 sqrt(n_finite * sumsq)): the 1e-6
relative bound of the specification, with an absolute floor for chunks whose
sum cancels (sum|x| <= sqrt(n sumsq)).  sumsq has no cancellation: pure 1e-6
relative.  Everything else (signature, counts, absmax, ids) is bit-exact.
"""
import math

import numpy as np

REL = 1e-6
FLOOR = 1e-12


def sum_ok(g, ref, n_fin, sumsq):
    return abs(g - ref) <= max(REL * abs(ref), FLOOR * math.sqrt(max(n_fin, 0) * max(sumsq, 0.0)))


def sumsq_ok(g, ref):
    return abs(g - ref) <= REL * abs(ref)


def compare_record(gpu, ref, where=""):
    """gpu: numpy record (RECORD_DTYPE row); ref: dict or structured row from the oracle."""
    def f(name_g, name_r=None):
        return gpu[name_g], ref[name_r or name_g]
    assert int(gpu["sig"]) == int(ref["sig"]), f"sig mismatch {where}"
    assert int(gpu["n_elems"]) == int(ref["n_elems"]), f"n_elems {where}"
    assert int(gpu["nan_count"]) == int(ref["nan"]), f"nan {where}"
    assert int(gpu["inf_count"]) == int(ref["inf"]), f"inf {where}"
    assert float(gpu["absmax"]) == float(ref["absmax"]), f"absmax {where}"
    n_fin = int(ref["n_elems"]) - int(ref["nan"]) - int(ref["inf"])
    assert sum_ok(float(gpu["sum"]), float(ref["sum"]), n_fin, float(ref["sumsq"])), \
        f"sum {where}: {gpu['sum']!r} vs {ref['sum']!r}"
    assert sumsq_ok(float(gpu["sumsq"]), float(ref["sumsq"])), \
        f"sumsq {where}: {gpu['sumsq']!r} vs {ref['sumsq']!r}"


def compare_all_records(g, ref):
    """g: [R, C] RECORD_DTYPE array; ref: oracle.signature dict of [R, C] arrays."""
    assert g.shape == ref["sig"].shape
    assert np.array_equal(g["sig"], ref["sig"]), \
        f"signatures differ at {np.argwhere(g['sig'] != ref['sig'])[:5].tolist()}"
    assert np.array_equal(g["n_elems"], ref["n_elems"])
    assert np.array_equal(g["nan_count"], ref["nan"])
    assert np.array_equal(g["inf_count"], ref["inf"])
    assert np.array_equal(g["tensor"], ref["tensor"])
    assert np.array_equal(g["chunk_in_tensor"], ref["chunk"])
    assert np.array_equal(g["absmax"], ref["absmax"])
    n_fin = ref["n_elems"].astype(np.float64) - ref["nan"] - ref["inf"]
    floor = FLOOR * np.sqrt(np.maximum(n_fin, 0) * np.maximum(ref["sumsq"], 0))
    err = np.abs(g["sum"] - ref["sum"])
    bad = err > np.maximum(REL * np.abs(ref["sum"]), floor)
    assert not bad.any(), f"sum outside tolerance at {np.argwhere(bad)[:5].tolist()}"
    bad = np.abs(g["sumsq"] - ref["sumsq"]) > REL * np.abs(ref["sumsq"])
    assert not bad.any(), f"sumsq outside tolerance at {np.argwhere(bad)[:5].tolist()}"
