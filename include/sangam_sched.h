/*
 * sangam_sched.h - host-side admission of whole prefills into a microbatch of
 * in-flight block decodes: the deficit token-budget rule of the Sangam paper
 * (Sec. 4.1, Alg. 1), which composes the mixed batches that
 * sangam_attn_forward serves.
 *
 * Host only, no device work, no allocation; thread safe (no global state).
 */
#ifndef SANGAM_SCHED_H
#define SANGAM_SCHED_H

#include <stdint.h>

#include "sangam_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * One iteration of deficit token-budget admission (Sec. 4.1, Alg. 1).
 *
 * tau            per-iteration token budget (>= 0)
 * decode_tokens  tokens of the in-flight decodes, which are all seated and
 *                never displaced (>= 0; a block decode counts its block size)
 * num_decodes    number of in-flight decodes (>= 0); with none, the
 *                microbatch starts empty
 * waiting        tokens of each waiting prefill, in arrival-time order
 *                (host array of num_waiting entries, each >= 1; may be NULL
 *                when num_waiting is 0). A prefill is indivisible.
 * deficit        in: unspent budget carried from the previous iteration
 *                (>= 0); out: the budget carried to the next one
 * num_admitted   out: how many prefills, from the head of the queue, join
 *                this iteration's microbatch
 *
 * Rule: with no prefill waiting the iteration is decode-only and the deficit
 * is cleared. Otherwise budget = tau - decode_tokens + deficit, and the head
 * prefill is admitted while it fits the budget (which it then reduces), or
 * unconditionally while the microbatch is still empty (the idle rule, for
 * liveness of prefills larger than tau); the first that does not fit stops
 * the scan. The carried deficit is max(budget, 0).
 *
 * Errors: SANGAM_ERR_INVALID_ARG for a negative argument, a non-positive
 * prefill size, or a NULL output (nothing is written then).
 */
sangam_status sangam_deficit_admit(int64_t tau, int64_t decode_tokens, int32_t num_decodes,
                                   const int64_t *waiting, int32_t num_waiting, int64_t *deficit,
                                   int32_t *num_admitted);

#ifdef __cplusplus
}
#endif

#endif /* SANGAM_SCHED_H */
