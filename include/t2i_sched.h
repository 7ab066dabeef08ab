/*
 * t2i_sched.h -- vTime fair scheduler for model-function invocations.
 *
 * The control-plane algorithm of ServerlessT2I (Sec. 6, "Ensure Fairness in
 * Multi-tenant Serving", Alg. 1) as a host library that decides which ready
 * invocation -- e.g. one t2i_dit_step of some tenant's workflow -- runs next on
 * an idle executor:
 *   - vTime accounting: the owner is charged the estimated execution time at
 *     dispatch, corrected by (measured - estimated) on completion;
 *   - vTime lift: a tenant with ready work that had none ready or running
 *     (new or returning) starts at the minimum vTime of the active tenants;
 *   - layer 1: only tenants within `delta` of the smallest vTime among
 *     tenants with ready work are candidates;
 *   - layer 2: among their ready invocations the highest normalised score
 *     w/max(w) - r/max(r) - e/max(e) wins (w: waiting time, r: remaining
 *     critical-path time of the workflow, e: estimated execution time; each
 *     term 0 when its maximum is 0), ties to the earlier ready time, then the
 *     smaller id.
 * For two tenants that always have ready work over an interval, the service
 * they receive differs by at most 2 (delta + L_max), L_max the largest
 * single charge.
 *
 * Host-only; no GPU calls.  Times are in any consistent unit (double).  A
 * handle is not thread-safe: one caller at a time.  Errors come back as
 * t2i_status (t2i_dit.h) and never abort.
 */
#ifndef T2I_SCHED_H
#define T2I_SCHED_H

#include <stdint.h>
#include "t2i_dit.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct t2i_sched t2i_sched;

/* delta >= 0 (finite or +inf). */
t2i_status t2i_sched_create(double delta, t2i_sched** out);
void t2i_sched_destroy(t2i_sched* s);

/* Invocation fn_id (unique among ready and running ones) of `tenant` becomes
 * ready at time `now`; est > 0 and remaining >= 0 finite. */
t2i_status t2i_sched_submit(t2i_sched* s, int32_t tenant, int64_t fn_id, double est,
                            double remaining, double now);

/* Alg. 1 Schedule at time `now`: *picked = 1 and the chosen invocation, its
 * tenant and the charged estimate; *picked = 0 when nothing is ready. */
t2i_status t2i_sched_schedule(t2i_sched* s, double now, int32_t* picked, int64_t* fn_id,
                              int32_t* tenant, double* charged);

/* Alg. 1 OnComplete: a running invocation finished after `measured` time. */
t2i_status t2i_sched_complete(t2i_sched* s, int64_t fn_id, double measured);

/* Current vTime of a tenant (0 for a tenant never seen). */
t2i_status t2i_sched_vtime(const t2i_sched* s, int32_t tenant, double* v);

#ifdef __cplusplus
}
#endif
#endif /* T2I_SCHED_H */
