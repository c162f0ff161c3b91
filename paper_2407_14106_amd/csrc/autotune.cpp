// The Auto Tuner of the transfer threshold (§3.4, hyperparameter modeling):
// a running loss F_t = 0.9 F_{t-1} + 0.1 L_t (F_0 = L_0), the loss descent
// rate LDR_t = (F_t - F_{t-1}) / et_t, and a walk over the threshold ladder
// {0, bG, 1.5 bG, 5 bG, 7 bG, 10 bG, 1} (bG = nnz / n^2, each capped at 1)
// starting at bG.  A decision is taken at epoch t once LDR_{t-delta} exists and
// delta epochs have passed since the last change: LDR_t >= LDR_{t-delta} moves
// one step up, otherwise one step down, clamped at both ends.
//
// Host code only; every operation is a separate IEEE double operation (no
// contraction), so the walk is reproducible bit for bit.
#include <math.h>

#include "common.h"

#pragma clang fp contract(off)

namespace {

void set_rung(gt_autotuner* st, int i, uint64_t num, uint64_t den) {
    if (num >= den) num = den = 1;  // capped at 1
    st->num[i] = num;
    st->den[i] = den;
}

}  // namespace

extern "C" gt_status gt_autotuner_init(gt_autotuner* st, int64_t n, int64_t nnz, int32_t delta) {
    if (!st) return gt::fail(GT_ERR_INVALID_ARG, "gt_autotuner_init: null state");
    if (n < 1 || n >= (int64_t(1) << 31) || nnz < 0 || nnz >= (int64_t(1) << 32))
        return gt::fail(GT_ERR_INVALID_ARG, "gt_autotuner_init: n or nnz out of range");
    if (delta < 1 || delta >= GT_AUTOTUNER_HISTORY)
        return gt::fail(GT_ERR_INVALID_ARG, "gt_autotuner_init: delta must be in [1, GT_AUTOTUNER_HISTORY)");
    const uint64_t nn = uint64_t(n) * uint64_t(n), e = uint64_t(nnz);
    set_rung(st, 0, 0, 1);
    set_rung(st, 1, e, nn);
    set_rung(st, 2, 3 * e, 2 * nn);
    set_rung(st, 3, 5 * e, nn);
    set_rung(st, 4, 7 * e, nn);
    set_rung(st, 5, 10 * e, nn);
    set_rung(st, 6, 1, 1);
    st->F = 0.0;
    for (int i = 0; i < GT_AUTOTUNER_HISTORY; ++i) st->ldr[i] = 0.0;
    st->t = -1;
    st->last_change = 0;
    st->level = 1;
    st->delta = delta;
    return GT_OK;
}

extern "C" gt_status gt_autotuner_step(gt_autotuner* st, double loss, double epoch_seconds, int32_t* level,
                                       uint64_t* num, uint64_t* den) {
    if (!st) return gt::fail(GT_ERR_INVALID_ARG, "gt_autotuner_step: null state");
    if (!(epoch_seconds > 0.0) || !isfinite(loss))
        return gt::fail(GT_ERR_INVALID_ARG, "gt_autotuner_step: epoch time must be positive and the loss finite");
    if (st->delta < 1 || st->delta >= GT_AUTOTUNER_HISTORY || st->level < 0 || st->level >= GT_AUTOTUNER_RUNGS)
        return gt::fail(GT_ERR_INVALID_ARG, "gt_autotuner_step: state not initialised");
    const int64_t t = ++st->t;
    if (t == 0) {
        st->F = loss;
    } else {
        const double prev = st->F;
        const double a = 0.9 * prev;
        const double b = 0.1 * loss;
        st->F = a + b;
        const double ldr = (st->F - prev) / epoch_seconds;
        st->ldr[t % GT_AUTOTUNER_HISTORY] = ldr;
        if (t - st->delta >= 1 && t - st->last_change >= st->delta) {
            const double then = st->ldr[(t - st->delta) % GT_AUTOTUNER_HISTORY];
            int32_t nl = ldr >= then ? st->level + 1 : st->level - 1;
            if (nl < 0) nl = 0;
            if (nl > GT_AUTOTUNER_RUNGS - 1) nl = GT_AUTOTUNER_RUNGS - 1;
            if (nl != st->level) {
                st->level = nl;
                st->last_change = t;
            }
        }
    }
    if (level) *level = st->level;
    if (num) *num = st->num[st->level];
    if (den) *den = st->den[st->level];
    return GT_OK;
}
