"""Oracle of out-of-band hang localization (Sec. 7).

TEST INFRASTRUCTURE ONLY, like the rest of this package.

Sec. 7: each rank publishes a progress coordinate (optimizer step, operation
id) and, before a collective that may block, a fingerprint of what healthy
callers of that collective share (process group, type, shape, dtype,
reduction, root).  After a silence, observers compare the records with exact
C3: a minority of differing records localizes the ranks (a different
coordinate: a lagging or diverged rank; the same coordinate with another
collective: a protocol mismatch); agreement of all ranks is a group-scoped
stall.

The classification here is the plain definition: strict majority of equal
(step, op_id, fingerprint, pending) tuples, compared as tuples.  The
fingerprint and group-id constructions (C3FP-1) are this implementation's
definitions, written from their specification with the oracle's own
fmix64; their exact bits are parity unpinned by the paper and pinned by
sensitivity properties in the tests.
"""
from . import fmix64

M64 = (1 << 64) - 1
TAG_GROUP = 0x4333475250000001
TAG_COLL = 0x4333465000000001
PENDING = 1


def group_id(ranks):
    h = fmix64(TAG_GROUP ^ (len(ranks) & 0xFFFFFFFF))
    for r in ranks:
        h = fmix64(h ^ (r & 0xFFFFFFFF))
    return h


def fingerprint(kind, dtype, process_group, reduce_op=-1, root=-1, shape=(), ndim=None):
    """C3FP-1; ndim = -1 leaves a rank-dependent shape out."""
    nd = len(shape) if ndim is None else ndim
    h = fmix64(TAG_COLL ^ ((kind & 0xFFFFFFFF) << 32) ^ (dtype & 0xFFFFFFFF))
    h = fmix64(h ^ process_group)
    h = fmix64(h ^ (((reduce_op & 0xFFFFFFFF) << 32) | (root & 0xFFFFFFFF)))
    h = fmix64(h ^ (nd & M64))
    for d in range(max(nd, 0)):
        h = fmix64(h ^ (shape[d] & M64))
    return h if h else 1


def classify(records):
    """records: list of dicts with step, op_id, fingerprint, flags.
    Returns (class, majority_idx, outliers, reasons)."""
    R = len(records)
    if R < 2:
        raise ValueError("a single rank has no peer to compare with (Sec. 4)")
    key = [(r["step"], r["op_id"], r["fingerprint"], r["flags"] & PENDING) for r in records]
    counts = [sum(1 for k in key if k == key[i]) for i in range(R)]
    best = max(range(R), key=lambda i: (counts[i], -i))
    if 2 * counts[best] <= R:
        return "inconclusive", -1, [], {}
    outliers = [i for i in range(R) if key[i] != key[best]]
    reasons = {i: ("protocol" if key[i][:2] == key[best][:2] else "progress") for i in outliers}
    return ("rank_divergence" if outliers else "group_stall"), best, outliers, reasons
