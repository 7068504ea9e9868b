"""Out-of-band hang localization (Sec. 7), on the CPU.

* the shared-memory progress record: geometry checks, round trips across
  processes, snapshots never torn under a concurrent writer, silence waits;
* fingerprints (C3FP-1, this implementation's construction: parity unpinned
  by the paper) against the oracle's transcription of the specification and
  for sensitivity to every field;
* the classification against the oracle's plain tuple-majority definition,
  by brute force over label vectors, and on the Sec. 7 cases
  (tests/golden/hang_cases.txt);
* end to end: trainer processes in a Gloo training group publish progress
  around real all_reduce calls; one is frozen with SIGSTOP, or publishes a
  different collective, or all stall together; CPU observers in their own
  Gloo group detect the silence, exchange records and must all reach the
  expected verdict.
"""
import ctypes
import itertools
import multiprocessing as mp
import os
import random
import time

import pytest

import oracle
from oracle import oob as ooob

oob = pytest.importorskip("paper_2608_11034_amd.oob")

HERE = os.path.dirname(os.path.abspath(__file__))


def _name(tag):
    return f"/c3test_{tag}_{os.getpid()}_{random.randrange(1 << 30)}"


def test_record_roundtrip_and_geometry():
    name = _name("geom")
    seg = oob.ProgressSegment(name, 4, create=True)
    try:
        assert seg.n_slots == 4
        for s in range(4):
            seg.publish(s, 10 + s, 20 + s, 0xDEADBEEF00 + s, pending=bool(s & 1))
        other = oob.ProgressSegment(name)                   # attach
        for s in range(4):
            p = other.read(s)
            assert (p.step, p.op_id, p.fingerprint) == (10 + s, 20 + s, 0xDEADBEEF00 + s)
            assert p.flags == (s & 1) and p.publishes == 1 and p.pid == os.getpid()
            assert p.publish_ns > 0
        other.close()
        same = oob.ProgressSegment(name, 4, create=True)    # same geometry: reused, not cleared
        assert same.read(3).step == 13
        same.close()
        with pytest.raises(oob.OOBError):
            oob.ProgressSegment(name, 5, create=True)       # other geometry
        with pytest.raises(oob.OOBError):
            seg.read(4)
        with pytest.raises(oob.OOBError):
            seg.publish(-1, 0, 0)
    finally:
        seg.close(unlink=True)
    with pytest.raises(oob.OOBError):
        oob.ProgressSegment(name)                           # gone
    with pytest.raises(oob.OOBError):
        oob.ProgressSegment(name, 0, create=True)
    with pytest.raises(oob.OOBError):
        oob.ProgressSegment(name, 65, create=True)


def _writer(name, slot, seconds):
    from paper_2608_11034_amd import oob as o
    seg = o.ProgressSegment(name)
    t_end = time.monotonic() + seconds
    i = 0
    while time.monotonic() < t_end:
        for _ in range(1000):
            i += 1
            seg.publish(slot, i, 3 * i + 1, (i * 0x9E3779B97F4A7C15) & ((1 << 64) - 1) or 1,
                        pending=bool(i & 1))
    seg.close()


def test_snapshots_are_never_torn_under_a_concurrent_writer():
    name = _name("torn")
    seg = oob.ProgressSegment(name, 2, create=True)
    ctx = mp.get_context("spawn")
    w = ctx.Process(target=_writer, args=(name, 1, 3.0))
    w.start()
    try:
        seen, t_end = 0, time.monotonic() + 20
        while seen < 200000 and time.monotonic() < t_end and (w.is_alive() or seen == 0):
            p = seg.read(1)
            if p.publishes == 0:
                continue
            i = p.step
            assert p.op_id == 3 * i + 1
            assert p.fingerprint == ((i * 0x9E3779B97F4A7C15) & ((1 << 64) - 1) or 1)
            assert p.flags == (i & 1) and p.publishes == i
            seen += 1
        assert seen > 1000
    finally:
        w.join(30)
        if w.is_alive():
            w.kill()
        seg.close(unlink=True)


def test_wait_silence_and_max_wait():
    import threading
    name = _name("silence")
    seg = oob.ProgressSegment(name, 1, create=True)
    try:
        stop = time.monotonic() + 0.3

        def pub():
            i = 0
            while time.monotonic() < stop:
                i += 1
                seg.publish(0, i, 0)
                time.sleep(0.005)

        th = threading.Thread(target=pub)
        t0 = time.monotonic()
        th.start()
        silent, p = seg.wait_silence(0, 0.2, 0.005, 5.0)
        dt = time.monotonic() - t0
        th.join()
        assert silent and 0.45 <= dt < 2.0, dt
        assert p.publishes == p.step and p.step > 10
        t0 = time.monotonic()
        seg.publish(0, 1, 1)
        silent, _ = seg.wait_silence(0, 5.0, 0.01, 0.2)     # max wait first
        assert not silent and time.monotonic() - t0 < 1.0
    finally:
        seg.close(unlink=True)


def _random_coll(rng):
    ranks = rng.sample(range(64), rng.randint(1, 8))
    nd = rng.choice([-1, 0, 1, 2, 3, 8])
    shape = tuple(rng.randint(0, 1 << 40) for _ in range(max(nd, 0)))
    return dict(kind=rng.randint(1, 9), dtype=rng.randint(0, 30), ranks=ranks,
                reduce_op=rng.choice([-1, 0, 1, 2]), root=rng.choice([-1, 0, 3]), shape=shape,
                nd=nd)


def _fp(d):
    return oob.collective_fingerprint(d["kind"], d["ranks"], d["dtype"], d["shape"],
                                      d["reduce_op"], d["root"], rank_dependent_shape=d["nd"] < 0)


def _fp_oracle(d):
    return ooob.fingerprint(d["kind"], d["dtype"], ooob.group_id(d["ranks"]), d["reduce_op"],
                            d["root"], d["shape"], ndim=d["nd"] if d["nd"] < 0 else None)


def test_fingerprint_matches_the_specification():
    rng = random.Random(7)
    for _ in range(300):
        d = _random_coll(rng)
        assert oob.group_id(d["ranks"]) == ooob.group_id(d["ranks"])
        assert _fp(d) == _fp_oracle(d)


def test_fingerprint_sees_every_field():
    base = dict(kind=1, dtype=6, ranks=[0, 1, 2, 3], reduce_op=0, root=-1, shape=(4096, 16), nd=2)
    f0 = _fp(base)
    variants = [dict(kind=2), dict(dtype=7), dict(ranks=[0, 1, 2]), dict(ranks=[1, 0, 2, 3]),
                dict(reduce_op=1), dict(root=0), dict(shape=(4096, 17), nd=2),
                dict(shape=(16, 4096), nd=2), dict(shape=(4096, 16, 1), nd=3),
                dict(shape=(65536,), nd=1), dict(shape=(), nd=0)]
    seen = {f0}
    for v in variants:
        d = dict(base, **v)
        f = _fp(d)
        assert f not in seen, v
        seen.add(f)
    # a rank-dependent shape is left out: any shapes agree
    a = dict(base, nd=-1, shape=(1, 2))
    b = dict(base, nd=-1, shape=(9,))
    assert _fp(a) == _fp(b) and _fp(a) not in seen


def _labels_records(labels, rng):
    """Records whose tuples are equal iff their labels are equal."""
    pool = {}
    out = []
    for lab in labels:
        if lab not in pool:
            pool[lab] = dict(step=rng.randint(0, 3), op_id=rng.randint(0, 3),
                             fingerprint=rng.choice([0, rng.getrandbits(64) or 1]),
                             flags=rng.randint(0, 1))
            while any(pool[lab][k] == q[k] for q in pool.values() if q is not pool[lab]
                      for k in ("fingerprint",)) and pool[lab]["fingerprint"] != 0:
                pool[lab]["fingerprint"] = rng.getrandbits(64) or 1
        out.append(dict(pool[lab], publish_ns=rng.getrandbits(40), publishes=rng.randint(1, 99),
                        pid=rng.randint(1, 1 << 20)))
    # distinct labels must give distinct tuples
    keys = {}
    for lab, r in zip(labels, out):
        keys.setdefault((r["step"], r["op_id"], r["fingerprint"], r["flags"]), set()).add(lab)
    if any(len(v) > 1 for v in keys.values()):
        return None
    return out


@pytest.mark.parametrize("R", [2, 3, 4, 5, 6])
def test_classify_matches_the_tuple_majority_definition(R):
    rng = random.Random(R)
    n = 0
    for labels in itertools.product(range(R), repeat=R):
        recs = _labels_records(labels, rng)
        if recs is None:
            continue
        n += 1
        v = oob.classify(recs)
        cls, maj, outl, reasons = ooob.classify(recs)
        assert v["class"] == cls and v["majority_idx"] == maj
        assert v["outliers"] == outl and v["reasons"] == reasons
        # agreement with the oracle's own exact vote on the evidence values
        ev = [oob.evidence(oob._records_array([r])[0]) for r in recs]
        import numpy as np
        st, bm, mj = oracle.vote_exact(np.array(ev, dtype=np.uint64).reshape(R, 1))
        assert int(bm[0]) == v["bitmap"]
        assert {0: "group_stall", 1: "rank_divergence", 2: "inconclusive"}[int(st[0])] == v["class"]
    assert n > 0


def test_single_rank_is_rejected():
    """Sec. 4: a single rank has no peer to be compared with; the library, its
    binding and the oracle all refuse to classify it."""
    rec = [dict(step=3, op_id=1, fingerprint=0, flags=0)]
    with pytest.raises(oob.OOBError):
        oob.classify(rec)
    with pytest.raises(ValueError):
        ooob.classify(rec)
    v = oob.HangVerdict()
    assert oob.lib().c3_hang_classify(oob._records_array(rec), 1, ctypes.byref(v)) == -1


def _parse_cases():
    cases = []
    for line in open(os.path.join(HERE, "golden", "hang_cases.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, cls, outl, recs = [x.strip() for x in line.split("|")]
        fps = {"0": 0, "F": 0x1111111111111111, "G": 0x2222222222222222}
        records = []
        for r in recs.split():
            st, op, fp, pend = r.split("/")
            records.append(dict(step=int(st), op_id=int(op), fingerprint=fps[fp], flags=int(pend)))
        expect = {} if outl == "-" else {int(a): b for a, b in (x.split(":") for x in outl.split(","))}
        cases.append((name, cls, expect, records))
    return cases


@pytest.mark.parametrize("case", _parse_cases(), ids=lambda c: c[0])
def test_paper_hang_cases(case):
    name, cls, expect, records = case
    c, _, outl, reasons = ooob.classify(records)
    assert c == cls and reasons == expect and outl == sorted(expect)
    v = oob.classify(records)
    assert v["class"] == cls and v["reasons"] == expect


# ---------------------------------------------------------------------------
# end to end: trainers (Gloo training group) and observers (own Gloo group)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("scenario,expect_cls,expect", [
    ("freeze", "rank_divergence", {2: "progress"}),
    ("protocol", "rank_divergence", {1: "protocol"}),
    ("stall", "group_stall", {}),
])
def test_observers_localize_a_hang_end_to_end(scenario, expect_cls, expect):
    from paper_2608_11034_amd import oob_drill
    world = 4
    res = oob_drill.run_drill(scenario, world=world, at_step=5, silence_s=0.5)
    verdicts = res["verdicts"]
    assert len(verdicts) == world, f"verdicts from {sorted(verdicts)}"
    first = verdicts[0]
    for r, v in verdicts.items():
        assert v is not None, f"observer {r} saw no silence"
        assert v["class"] == expect_cls, (r, v)
        assert {int(k): x for k, x in v["reasons"].items()} == expect, (r, v)
        assert v["records"] == first["records"]            # every observer saw the same table
    # the verdict follows the hang by the silence threshold plus the exchange
    assert len(res["latency_s"]) == world
    assert all(0.5 <= t < 30 for t in res["latency_s"].values()), res["latency_s"]
    # the gathered records agree with the oracle's tuple-majority definition
    cls, _, outl, reasons = ooob.classify(first["records"])
    assert cls == expect_cls and reasons == expect


def test_library_exports_every_declared_symbol():
    import ctypes
    import re
    src = open(os.path.join(os.path.dirname(HERE), "include", "c3_oob.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b(c3_\w+)\s*\(", src, flags=re.M))
    assert {"c3_progress_open", "c3_progress_publish", "c3_progress_read", "c3_hang_classify",
            "c3_collective_fingerprint", "c3_progress_wait_silence"} <= names
    L = oob.lib()
    for n in names:
        assert hasattr(L, n), n
    assert ctypes.sizeof(oob.Progress) == 48 and ctypes.sizeof(oob.Collective) == 96
    assert ctypes.sizeof(oob.HangVerdict) == 80


def test_native_progress_path_benchmark_runs_clean():
    import json
    import subprocess
    from paper_2608_11034_amd import build as b
    out = subprocess.run([b.OOB_BENCH, "200000"], check=True, capture_output=True, text=True,
                         timeout=120).stdout
    r = json.loads(out)
    assert r["torn"] == 0 and r["busy"] == 0 and r["publish_ns"] > 0
