"""Checkpoint certification (Sec. 8, Algorithm 3): libc3's state machine
against the oracle's transcription of the algorithm and the paper's
two-recipe recovery scenario.  Host-only: no GPU needed."""
import os

import numpy as np
import pytest

from oracle import ckpt as ockpt

c3 = pytest.importorskip("paper_2608_11034_amd.c3")
GOLD = os.path.join(os.path.dirname(__file__), "golden", "checkpoint_two_recipe.txt")
CODE = {"OK": 0, "STRAGGLER": 1, "SDC": 2, "HANG": 3}


def _rows():
    for ln in open(GOLD):
        if ln.strip() and not ln.startswith("#"):
            yield [x.strip() for x in ln.split("|")]


def test_paper_two_recipe_scenario_oracle():
    p = ockpt.CheckpointProtocol(K=2)
    for step, outcome, cand, ver, got in _rows():
        act = p.save(outcome, int(step))
        assert (p.candidate if p.candidate is not None else -1) == int(cand), step
        assert (p.verified if p.verified is not None else -1) == int(ver), step
        if got != "-":
            assert act["retrieve"] == int(got)


def test_paper_two_recipe_scenario_library():
    g = c3.CheckpointGate(K=2)
    for step, outcome, cand, ver, got in _rows():
        act = g.save(CODE[outcome], int(step))
        assert g.state.candidate == int(cand) and g.state.verified == int(ver), step
        if got != "-":
            assert act.retrieve == 1 and act.retrieve_id == int(got)
        else:
            assert act.retrieve == 0 and act.captured == 1


@pytest.mark.parametrize("K", [1, 2, 3, 5])
def test_library_matches_oracle_on_random_sequences(K):
    rng = np.random.default_rng(K)
    names = ["OK", "OK", "OK", "STRAGGLER", "SDC", "HANG"]
    for trial in range(50):
        p, g = ockpt.CheckpointProtocol(K), c3.CheckpointGate(K)
        for step in range(40):
            outcome = names[int(rng.integers(0, len(names)))]
            acc = bool(rng.random() < 0.8)
            cat = bool(rng.random() < 0.3)
            a = p.save(outcome, step, acc, cat)
            b = g.save(CODE[outcome], step, acc, cat)
            assert (g.state.q, g.state.latest, g.state.candidate, g.state.verified) == \
                (p.q, -1 if p.latest is None else p.latest, -1 if p.candidate is None else p.candidate,
                 -1 if p.verified is None else p.verified), (trial, step)
            if "retrieve" in a:
                assert b.retrieve == 1
                assert b.retrieve_id == (-1 if a["retrieve"] is None else a["retrieve"])
            else:
                assert b.retrieve == 0 and b.captured == 1
                assert b.persisted_id == a.get("persisted", -1)
                assert b.promoted == (1 if "promoted" in a else 0)
            for o in CODE:
                want = p.retrieve(o, acc, cat)
                assert g.retrieve(CODE[o], acc, cat) == (-1 if want is None else want)


@pytest.mark.parametrize("K", [1, 2, 4])
def test_promotion_needs_two_accepted_cycles(K):
    # a checkpoint persisted at the end of one accepted cycle is verified only
    # at the end of the next (2K checks), and an SDC before that keeps the
    # older verified checkpoint
    g = c3.CheckpointGate(K)
    for step in range(1, 2 * K + 1):
        g.save(c3.OUTCOME_OK, step)
    assert g.state.candidate == 2 * K and g.state.verified == K
    for step in range(2 * K + 1, 3 * K):
        g.save(c3.OUTCOME_OK, step)
    act = g.save(c3.OUTCOME_SDC, 3 * K)
    assert act.retrieve_id == K
    assert g.retrieve(c3.OUTCOME_STRAGGLER) == (3 * K - 1 if K > 1 else 2 * K)


def test_retrieval_rules():
    g = c3.CheckpointGate(1)
    g.save(c3.OUTCOME_OK, 10)
    g.save(c3.OUTCOME_OK, 11)          # 10 verified, 11 candidate and latest
    assert g.retrieve(c3.OUTCOME_SDC) == 10
    assert g.retrieve(c3.OUTCOME_STRAGGLER) == 11
    assert g.retrieve(c3.OUTCOME_HANG) == 11
    assert g.retrieve(c3.OUTCOME_HANG, full_catalog_sdc=True) == 10
    assert g.retrieve(c3.OUTCOME_STRAGGLER, machines_accessible=False) == 10
    assert c3.CheckpointGate(3).retrieve(c3.OUTCOME_SDC) == -1   # nothing verified yet


def test_job_outcome_precedence():
    for s in (0, 3):
        for h in (0, 1):
            for t in (0, 2):
                assert c3.job_outcome(s, h, t) == CODE[ockpt.job_outcome(s, h, t)]
    with pytest.raises(c3.C3Error):
        c3.job_outcome(-1, 0, 0)


def test_invalid_arguments():
    with pytest.raises(c3.C3Error):
        c3.CheckpointGate(0)
    g = c3.CheckpointGate(2)
    with pytest.raises(c3.C3Error):
        g.save(7, 1)
    with pytest.raises(c3.C3Error):
        g.save(c3.OUTCOME_OK, -5)
