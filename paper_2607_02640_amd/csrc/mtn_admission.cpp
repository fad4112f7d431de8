// Deadline-aware admission (Metronome §4.2): an AIMD loop on the measured
// per-frame latency.  The admission cap drops multiplicatively when a tick's
// latency reaches the target, rises additively when there is headroom and
// demand presses against it, and arrivals beyond the cap are rejected cleanly
// instead of degrading every admitted session.  Host-only; no device work.
#include "mtn.h"

#include <cmath>
#include <new>

struct mtn_admission {
    mtn_admission_config cfg;
    int32_t cap = 0;
    int32_t admitted = 0;
    int32_t hold = 0;        // observations left before the next decision
    bool pressed = false;    // demand reached the cap since the last observation
    int64_t offered = 0, rejected = 0, ticks = 0, decreases = 0, increases = 0;
};

extern "C" {

mtn_status mtn_admission_create(const mtn_admission_config *cfg, mtn_admission **out) {
    if (!cfg || !out) return MTN_ERR_INVALID_ARG;
    if (!(cfg->target_ms > 0.0) || !std::isfinite(cfg->target_ms)) return MTN_ERR_INVALID_ARG;
    if (!(cfg->backoff > 0.0 && cfg->backoff < 1.0)) return MTN_ERR_INVALID_ARG;
    if (cfg->increase < 1 || cfg->min_cap < 1 || cfg->initial_cap < cfg->min_cap ||
        cfg->max_cap < cfg->initial_cap || cfg->hold_ticks < 0)
        return MTN_ERR_INVALID_ARG;
    mtn_admission *a = new (std::nothrow) mtn_admission;
    if (!a) return MTN_ERR_HOST_MEMORY;
    a->cfg = *cfg;
    a->cap = cfg->initial_cap;
    *out = a;
    return MTN_OK;
}

void mtn_admission_destroy(mtn_admission *a) { delete a; }

mtn_status mtn_admission_offer(mtn_admission *a, int32_t *admitted) {
    if (!a || !admitted) return MTN_ERR_INVALID_ARG;
    ++a->offered;
    if (a->admitted < a->cap) {
        ++a->admitted;
        if (a->admitted == a->cap) a->pressed = true;
        *admitted = 1;
    } else {
        ++a->rejected;
        a->pressed = true;
        *admitted = 0;
    }
    return MTN_OK;
}

mtn_status mtn_admission_release(mtn_admission *a) {
    if (!a) return MTN_ERR_INVALID_ARG;
    if (a->admitted == 0) return MTN_ERR_BAD_STATE;
    --a->admitted;
    return MTN_OK;
}

mtn_status mtn_admission_observe(mtn_admission *a, double tick_ms) {
    if (!a || !(tick_ms >= 0.0) || !std::isfinite(tick_ms)) return MTN_ERR_INVALID_ARG;
    ++a->ticks;
    const bool pressed = a->pressed;
    a->pressed = false;
    if (a->hold > 0) {  // the last cut has not reached the signal yet
        --a->hold;
        return MTN_OK;
    }
    if (tick_ms >= a->cfg.target_ms) {
        // multiplicative decrease, relative to the load that produced the
        // latency; never raises the cap, never evicts admitted sessions
        const int32_t cut = (int32_t)std::floor(a->cfg.backoff * (double)a->admitted);
        int32_t c = cut < a->cap ? cut : a->cap;
        a->cap = c < a->cfg.min_cap ? a->cfg.min_cap : c;
        a->hold = a->cfg.hold_ticks;
        ++a->decreases;
    } else if (pressed) {
        // additive increase: probe for headroom only while demand is capped
        const int64_t c = (int64_t)a->cap + a->cfg.increase;
        a->cap = (int32_t)(c > a->cfg.max_cap ? a->cfg.max_cap : c);
        ++a->increases;
    }
    return MTN_OK;
}

mtn_status mtn_admission_get(const mtn_admission *a, mtn_admission_state *out) {
    if (!a || !out) return MTN_ERR_INVALID_ARG;
    out->cap = a->cap;
    out->admitted = a->admitted;
    out->hold = a->hold;
    out->offered = a->offered;
    out->rejected = a->rejected;
    out->ticks = a->ticks;
    out->decreases = a->decreases;
    out->increases = a->increases;
    return MTN_OK;
}

}  // extern "C"
