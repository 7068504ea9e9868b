"""Hang drill for out-of-band hang localization (Sec. 7), CPU only.

Starts ``world`` trainer processes in a Gloo training group that publish
their progress around real ``all_reduce`` calls, and one observer process per
rank in a separate Gloo group.  At step ``at_step`` the scenario makes the
job hang:

* ``freeze``   -- rank 2 stops itself with SIGSTOP after finishing the step
                  (a rank-local stall: the others wait in the next all_reduce);
* ``protocol`` -- rank 1 announces a collective with another shape and
                  never enters it (a collective-protocol mismatch);
* ``stall``    -- every rank announces the same collective and never
                  returns from it (a group-scoped stall).

The hang is triggered once every observer is connected and watching; the
observers detect the silence, exchange records and classify the hang.
``run_drill`` returns every observer's verdict and the hang-to-verdict
latencies, then kills the trainers.  Used by the tests and the benchmark;
also a quick check that a node's observer path works.
"""
from __future__ import annotations

import multiprocessing as mp
import os
import random
import signal
import socket
import time

from . import oob


def _free_port():
    s = socket.socket()
    s.bind(("127.0.0.1", 0))
    port = s.getsockname()[1]
    s.close()
    return port


def _quiet_stdout():
    # Gloo reports connections on stdout; keep stdout for the caller's output
    os.dup2(2, 1)


def _mark_hang(hang):
    t = time.monotonic()
    with hang.get_lock():
        if hang.value == 0.0 or t < hang.value:
            hang.value = t


def _trainer(seg, rank, world, port, scenario, at_step, hang, armed):
    _quiet_stdout()
    import torch
    import torch.distributed as dist
    dist.init_process_group("gloo", init_method=f"tcp://127.0.0.1:{port}", rank=rank,
                            world_size=world)
    pub = oob.ProgressPublisher(seg, rank, world)
    ranks = list(range(world))
    x = torch.ones(16)
    for step in range(10 ** 7):
        if step == at_step:
            armed.wait(120)          # every observer is connected and watching
        if scenario == "protocol" and rank == 1 and step == at_step:
            with pub.collective("all_reduce", ranks, dtype=6, shape=(17,), reduce_op=0):
                _mark_hang(hang)
                time.sleep(3600)
        if scenario == "stall" and step == at_step:
            with pub.collective("all_reduce", ranks, dtype=6, shape=(16,), reduce_op=0):
                _mark_hang(hang)
                time.sleep(3600)
        with pub.collective("all_reduce", ranks, dtype=6, shape=(16,), reduce_op=0):
            dist.all_reduce(x)
        pub.step_done()
        if scenario == "freeze" and rank == 2 and step == at_step:
            _mark_hang(hang)
            os.kill(os.getpid(), signal.SIGSTOP)
        time.sleep(0.002)


def _observer(seg, rank, world, port, silence_s, q):
    _quiet_stdout()
    obs = oob.Observer(seg, rank, rank, world, f"tcp://127.0.0.1:{port}", exchange_timeout_s=60)
    q.put(("ready", rank))
    v = obs.watch(silence_s=silence_s, poll_s=0.005, max_wait_s=120)
    q.put(("verdict", rank, time.monotonic(), v))
    obs.close()


def run_drill(scenario: str, world: int = 4, at_step: int = 5, silence_s: float = 0.5,
              timeout_s: float = 150.0) -> dict:
    if scenario not in ("freeze", "protocol", "stall"):
        raise ValueError(scenario)
    if scenario == "freeze" and world < 3:
        raise ValueError("the freeze scenario stops rank 2")
    seg_name = f"/c3drill_{scenario}_{os.getpid()}_{random.randrange(1 << 30)}"
    seg = oob.ProgressSegment(seg_name, world, create=True)
    ctx = mp.get_context("spawn")
    q = ctx.Queue()
    hang = ctx.Value("d", 0.0)
    armed = ctx.Event()
    tport, oport = _free_port(), _free_port()
    trainers = [ctx.Process(target=_trainer, args=(seg_name, r, world, tport, scenario, at_step,
                                                   hang, armed))
                for r in range(world)]
    observers = [ctx.Process(target=_observer, args=(seg_name, r, world, oport, silence_s, q))
                 for r in range(world)]
    procs = trainers + observers
    for p in procs:
        p.start()
    verdicts, v_time, ready = {}, {}, set()
    try:
        t_end = time.monotonic() + timeout_s
        while len(verdicts) < world and time.monotonic() < t_end:
            try:
                msg = q.get(timeout=1.0)
            except Exception:
                continue
            if msg[0] == "ready":
                ready.add(msg[1])
                if len(ready) == world:
                    armed.set()
            elif msg[0] == "verdict":
                verdicts[msg[1]] = msg[3]
                v_time[msg[1]] = msg[2]
    finally:
        for p in trainers:
            if p.is_alive():
                os.kill(p.pid, signal.SIGKILL)      # also ends a stopped process
        for p in procs:
            p.join(30)
            if p.is_alive():
                os.kill(p.pid, signal.SIGKILL)
                p.join(5)
        seg.close(unlink=True)
    hang_time = hang.value
    lat = {r: t - hang_time for r, t in v_time.items()} if hang_time > 0.0 else {}
    return {"scenario": scenario, "world": world, "silence_s": silence_s, "verdicts": verdicts,
            "latency_s": lat}
