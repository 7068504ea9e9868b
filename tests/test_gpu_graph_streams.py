"""Two properties of the C ABI that callers rely on, through the binding:

* HIP graph capture.  After one eager call has staged the plan into the
  workspace, c3_signature with C3_OPT_PLAN_STAGED, c3_consensus and
  c3_localize launch kernels only (no host staging, no memset node), so a
  caller can capture them once and replay.  Every replay, with the replica
  bytes changed in place between replays and the program's own eager work
  in between, must equal the eager result bit for bit.  The same holds for
  c3_timing_consensus (both of its execution paths).
  A vote and localization over a 130-replica group are captured the same
  way.
* Streams.  Calls on different streams with disjoint outputs and
  workspaces may run concurrently: two signature + vote + localize passes
  over different replica sets, enqueued alternately on two streams, give
  the results each gives alone.
"""
import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu

c3 = pytest.importorskip("paper_2608_11034_amd.c3")
DEV = "cuda"


def _case(*a):
    print("CASE", *a, flush=True)


class _Pipe:
    """Preallocated outputs of signature -> consensus -> localize."""

    def __init__(self, replicas, chunk_bytes):
        self.plan = c3.SignaturePlan(replicas, chunk_bytes)
        self.rec = self.plan.new_records()
        self.ws = self.plan.new_workspace()
        C = self.rec.shape[1]
        R = self.rec.shape[0]
        self.vote = (torch.empty(C, dtype=torch.uint8, device=DEV),
                     torch.empty(C, dtype=torch.int64, device=DEV),
                     torch.empty(C, dtype=torch.int32, device=DEV))
        self.lists = (torch.zeros((C * R, 80), dtype=torch.uint8, device=DEV),
                      torch.zeros(C, dtype=torch.int64, device=DEV),
                      torch.zeros(3, dtype=torch.int64, device=DEV))
        self.lws = torch.empty(max(c3.localize_workspace_size(C), 256), dtype=torch.uint8,
                               device=DEV)

    def run(self, staged=False, stream=None):
        self.plan.run(self.rec, self.ws, stream=stream, plan_staged=staged)
        c3.consensus(self.rec, c3.EXACT, stream=stream, out=self.vote)
        c3.localize(*self.vote, self.rec, stream=stream, out=self.lists, workspace=self.lws)

    def snapshot(self):
        """Records, votes, counts, and the lists up to their counts (entries
        past a count are not written)."""
        counts = self.lists[2].cpu().numpy().copy()
        no, nu = int(counts[0]), int(counts[1])
        return ([t.cpu().numpy().copy() for t in (self.rec,) + self.vote]
                + [self.lists[0][:no].cpu().numpy().copy(), self.lists[1][:nu].cpu().numpy().copy(),
                   counts])


def _equal(a, b, where):
    for i, (x, y) in enumerate(zip(a, b)):
        if x.tobytes() != y.tobytes():
            bad = np.nonzero(x.reshape(-1) != y.reshape(-1))[0]
            raise AssertionError(f"{where} output {i}: {bad.size} differing values, first at "
                                 f"{bad[:8].tolist()}: got {x.reshape(-1)[bad[:8]].tolist()} "
                                 f"want {y.reshape(-1)[bad[:8]].tolist()}; counts got "
                                 f"{a[-1].tolist()} want {b[-1].tolist()}")


@pytest.mark.parametrize("k", [1, 3])
def test_graph_replays_equal_eager(k):
    _case("graph replay", k)
    w = workloads.make(k, device=DEV, scale="small")
    pipe = _Pipe(w.replicas, w.chunk_bytes)
    ref_pipe = _Pipe(w.replicas, w.chunk_bytes)
    pipe.run()                                   # eager: stages the plan
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        pipe.run(staged=True)
    gen = torch.Generator(device="cpu")
    gen.manual_seed(k)
    flat = [t.view(-1).view(torch.uint8) for t in w.replicas[1]]
    for step in range(5):
        # change replica 1 in place (a byte of some tensor), then replay
        t = int(torch.randint(0, len(flat), (1,), generator=gen))
        i = int(torch.randint(0, flat[t].numel(), (1,), generator=gen))
        flat[t][i] ^= 0x10
        g.replay()
        torch.cuda.synchronize()
        got = pipe.snapshot()
        ref_pipe.run()
        torch.cuda.synchronize()
        _equal(got, ref_pipe.snapshot(), ("replay", step))


@pytest.mark.parametrize("G,per_unit", [(64, True), (64, False), (4096, False)])
def test_graph_replays_timing_consensus(G, per_unit):
    """G = 4096 without per-unit results takes the single-pass kernel, the
    others the clear + votes + confirmation launches."""
    _case("graph timing", G, per_unit)
    R, T = 8, 40
    rng = np.random.default_rng(G)
    fp = torch.from_numpy(np.repeat(rng.integers(-(2 ** 63), 2 ** 63 - 1, size=(T, G, 1),
                                                 dtype=np.int64), R, axis=2)).to(DEV)
    tau = torch.from_numpy(np.exp(rng.normal(0, 0.02, size=(T, G, R))).astype(np.float32)).to(DEV)
    U = T * G

    def outs():
        ver = torch.empty((R * G, 24), dtype=torch.uint8, device=DEV)
        if not per_unit:
            return ver, None, None
        mk = lambda: (torch.empty(U, dtype=torch.uint8, device=DEV),  # noqa: E731
                      torch.empty(U, dtype=torch.int64, device=DEV),
                      torch.empty(U, dtype=torch.int32, device=DEV))
        return ver, mk(), mk()

    ws = torch.empty(c3.timing_consensus_workspace_size(R, G, T, 16), dtype=torch.uint8, device=DEV)
    o = outs()
    c3.timing_consensus(fp, tau, window=16, out=o, workspace=ws)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        c3.timing_consensus(fp, tau, window=16, out=o, workspace=ws)
    ref_ws = torch.empty_like(ws)
    for step in range(4):
        # a slower rank and a divergent fingerprint, different each replay
        tau[:, step, step] *= 1.5
        fp[step * 3:, step + 1, (step + 2) % R] ^= 12345
        g.replay()
        torch.cuda.synchronize()
        got = [o[0].cpu().numpy().copy()]
        if per_unit:
            got += [x.cpu().numpy().copy() for x in o[1] + o[2]]
        r = outs()
        c3.timing_consensus(fp, tau, window=16, out=r, workspace=ref_ws)
        torch.cuda.synchronize()
        want = [r[0].cpu().numpy()]
        if per_unit:
            want += [x.cpu().numpy() for x in r[1] + r[2]]
        _equal(got, want, ("timing replay", step))


@pytest.mark.parametrize("mode", ["exact", "statistical"])
def test_graph_replays_wide_group(mode):
    """A 130-replica vote (three bitmap words per unit) and its localization
    captured once; every replay, with the evidence changed in place, equals
    the eager result."""
    _case("graph wide", mode)
    R, U = 130, 3000
    rng = np.random.default_rng(130)
    if mode == "exact":
        ev = torch.from_numpy(np.repeat(rng.integers(-(2 ** 62), 2 ** 62, size=(U, 1)), R,
                                        axis=1)).to(DEV)
        m = c3.EXACT
    else:
        ev = torch.from_numpy(np.exp(rng.normal(0, 0.02, size=(U, R)))).to(DEV)
        m = c3.STATISTICAL
    W = c3.bitmap_words(R)
    vote = (torch.empty(U, dtype=torch.uint8, device=DEV),
            torch.empty((U, W), dtype=torch.int64, device=DEV),
            torch.empty(U, dtype=torch.int32, device=DEV))
    lists = (torch.zeros((U * 4, 80), dtype=torch.uint8, device=DEV),
             torch.zeros(U, dtype=torch.int64, device=DEV),
             torch.zeros(3, dtype=torch.int64, device=DEV))
    lws = torch.empty(max(c3.localize_workspace_size(U), 256), dtype=torch.uint8, device=DEV)

    def run(out_v, out_l, ws):
        c3.consensus(ev, m, out=out_v)
        c3.localize(*out_v, None, R=R, out_cap=U * 4, out=out_l, workspace=ws)

    def snap(v, lo):
        n_o, n_u = int(lo[2][0]), int(lo[2][1])
        return [x.cpu().numpy().copy() for x in v] + [lo[0][:n_o].cpu().numpy().copy(),
                                                      lo[1][:n_u].cpu().numpy().copy(),
                                                      lo[2].cpu().numpy().copy()]

    run(vote, lists, lws)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        run(vote, lists, lws)
    ref_v = tuple(torch.empty_like(x) for x in vote)
    ref_l = tuple(torch.zeros_like(x) for x in lists)
    ref_ws = torch.empty_like(lws)
    for step in range(4):
        # a different replica in a different word diverges at a few units
        r = (37 * step + 60) % R
        if mode == "exact":
            ev[step::50, r] ^= 1 << step
        else:
            ev[step::50, r] *= 1.5
        g.replay()
        torch.cuda.synchronize()
        got = snap(vote, lists)
        run(ref_v, ref_l, ref_ws)
        torch.cuda.synchronize()
        _equal(got, snap(ref_v, ref_l), ("wide replay", mode, step))
        assert int(lists[2][0]) > 0


def test_two_streams_concurrently():
    _case("two streams")
    a = workloads.make(3, device=DEV, scale="small")
    b = workloads.make(2, device=DEV, scale="small")
    pa, pb = _Pipe(a.replicas, a.chunk_bytes), _Pipe(b.replicas, b.chunk_bytes)
    pa.run()
    pb.run()
    torch.cuda.synchronize()
    want_a, want_b = pa.snapshot(), pb.snapshot()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    for it in range(20):                        # more calls than staging slots
        for pipe in (pa, pb):
            for t in (pipe.rec,) + pipe.vote + pipe.lists:
                t.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(sa):
            pa.run()
        with torch.cuda.stream(sb):
            pb.run()
        torch.cuda.synchronize()
        _equal(pa.snapshot(), want_a, ("stream a", it))
        _equal(pb.snapshot(), want_b, ("stream b", it))
