// Checkpoint certification of C3 (Sec. 8, Algorithm 3): a host-side state
// machine fed by the job-wide outcome of each replay boundary.
//
// States: latest (newest in-memory checkpoint), candidate (persisted,
// awaiting a full accepted cycle), verified (numerically trusted).  An
// accepted check (healthy or straggler) captures a new latest checkpoint and
// counts one recipe; after K accepted recipes the previous candidate becomes
// verified and the latest is persisted as the new candidate, so promotion
// needs two consecutive accepted cycles (2K checks).  An SDC or a hang
// invokes retrieval instead: SDC or an unreachable machine -> verified;
// straggler -> latest; anything else -> latest unless a full-catalog replay
// finds SDC.
#include <string.h>

#include "c3_internal.h"

namespace {

bool valid_outcome(int f) {
    return f == C3_OUTCOME_OK || f == C3_OUTCOME_STRAGGLER || f == C3_OUTCOME_SDC ||
           f == C3_OUTCOME_HANG;
}

int64_t retrieval(const c3_ckpt_state_t* st, int f, int machines_accessible,
                  int full_catalog_sdc) {
    if (f == C3_OUTCOME_SDC || !machines_accessible) return st->verified;
    if (f == C3_OUTCOME_STRAGGLER) return st->latest;
    if (full_catalog_sdc) return st->verified;
    return st->latest;
}

}  // namespace

extern "C" {

int c3_job_outcome(int64_t sdc_units, int64_t hang_signals, int64_t stragglers) {
    if (sdc_units < 0 || hang_signals < 0 || stragglers < 0) return C3_E_INVAL;
    if (sdc_units > 0) return C3_OUTCOME_SDC;
    if (hang_signals > 0) return C3_OUTCOME_HANG;
    if (stragglers > 0) return C3_OUTCOME_STRAGGLER;
    return C3_OUTCOME_OK;
}

int c3_ckpt_init(c3_ckpt_state_t* st, int K) {
    if (st == nullptr || K < 1) return C3_E_INVAL;
    memset(st, 0, sizeof(*st));
    st->K = K;
    st->q = 0;
    st->latest = -1;
    st->candidate = -1;
    st->verified = -1;
    return C3_OK;
}

int c3_ckpt_save(c3_ckpt_state_t* st, int outcome, int64_t checkpoint_id, int machines_accessible,
                 int full_catalog_sdc, c3_ckpt_action_t* act) {
    if (st == nullptr || act == nullptr || !valid_outcome(outcome) || st->K < 1 ||
        st->q < 0 || st->q >= st->K || checkpoint_id < 0)
        return C3_E_INVAL;
    memset(act, 0, sizeof(*act));
    act->persisted_id = -1;
    act->retrieve_id = -1;
    if (outcome == C3_OUTCOME_SDC || outcome == C3_OUTCOME_HANG) {
        act->retrieve = 1;
        act->retrieve_id = retrieval(st, outcome, machines_accessible, full_catalog_sdc);
        return C3_OK;
    }
    st->latest = checkpoint_id;
    act->captured = 1;
    st->q += 1;
    if (st->q == st->K) {
        st->q = 0;
        act->promoted = st->candidate >= 0 ? 1 : 0;
        st->verified = st->candidate;
        act->persisted_id = st->latest;
        st->candidate = st->latest;
    }
    return C3_OK;
}

int c3_ckpt_retrieve(const c3_ckpt_state_t* st, int outcome, int machines_accessible,
                     int full_catalog_sdc, int64_t* checkpoint_id) {
    if (st == nullptr || checkpoint_id == nullptr || !valid_outcome(outcome)) return C3_E_INVAL;
    *checkpoint_id = retrieval(st, outcome, machines_accessible, full_catalog_sdc);
    return C3_OK;
}

}  // extern "C"
