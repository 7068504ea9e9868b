"""Checkpoint saving and retrieval, Sec. 8, Algorithm 3 -- oracle.

TEST INFRASTRUCTURE ONLY (see the package docstring).  A plain transcription
of the algorithm's state: q accepted recipes of a K-recipe catalog, and the
latest, candidate and verified checkpoints (None = no checkpoint).

Outcomes: "OK" and "STRAGGLER" are accepted checks (the straggler is
reported separately; slowness is not numerical divergence); "SDC" and "HANG"
invoke retrieval.
"""


class CheckpointProtocol:
    def __init__(self, K: int):
        assert K >= 1
        self.K = K
        self.q = 0
        self.latest = None
        self.candidate = None
        self.verified = None

    def save(self, outcome: str, checkpoint, machines_accessible=True, full_catalog_sdc=False):
        """CheckpointSave.  Returns a dict of what happened."""
        if outcome in ("SDC", "HANG"):
            return {"retrieve": self.retrieve(outcome, machines_accessible, full_catalog_sdc)}
        self.latest = checkpoint                 # newly captured in-memory checkpoint
        self.q += 1
        act = {"captured": checkpoint}
        if self.q == self.K:                     # a complete accepted cycle
            self.q = 0
            if self.candidate is not None:
                act["promoted"] = self.candidate
            self.verified = self.candidate       # the previous candidate is now trusted
            act["persisted"] = self.latest       # persist latest as the new candidate
            self.candidate = self.latest
        return act

    def retrieve(self, outcome: str, machines_accessible=True, full_catalog_sdc=False):
        """CheckpointRetrieval."""
        if outcome == "SDC" or not machines_accessible:
            return self.verified
        if outcome == "STRAGGLER":
            return self.latest
        if full_catalog_sdc:                     # ReplayFullCatalog found SDC
            return self.verified
        return self.latest


def job_outcome(sdc_units: int, hang_signals: int, stragglers: int) -> str:
    """Most severe evidence of one boundary first."""
    if sdc_units > 0:
        return "SDC"
    if hang_signals > 0:
        return "HANG"
    if stragglers > 0:
        return "STRAGGLER"
    return "OK"
