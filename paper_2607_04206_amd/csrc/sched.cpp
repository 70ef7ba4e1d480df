// Deficit token-budget admission of whole prefills (Sangam paper, Sec. 4.1,
// Alg. 1): the host-side rule that composes the mixed microbatches of block
// decodes and indivisible prefills that the attention call serves.
#include <string>

#include "../../include/sangam_sched.h"

namespace sangam {
void set_error(const std::string& msg);
void clear_error();
}  // namespace sangam

extern "C" sangam_status sangam_deficit_admit(int64_t tau, int64_t decode_tokens, int32_t num_decodes,
                                              const int64_t* waiting, int32_t num_waiting, int64_t* deficit,
                                              int32_t* num_admitted) {
    sangam::clear_error();
    if (!deficit || !num_admitted || (num_waiting > 0 && !waiting)) {
        sangam::set_error("deficit and num_admitted must not be NULL, nor waiting when num_waiting > 0");
        return SANGAM_ERR_INVALID_ARG;
    }
    if (tau < 0 || decode_tokens < 0 || num_decodes < 0 || num_waiting < 0 || *deficit < 0) {
        sangam::set_error("tau, decode_tokens, num_decodes, num_waiting and the deficit must be >= 0");
        return SANGAM_ERR_INVALID_ARG;
    }
    for (int32_t k = 0; k < num_waiting; ++k)
        if (waiting[k] < 1) {
            sangam::set_error("prefill " + std::to_string(k) + " has no tokens");
            return SANGAM_ERR_INVALID_ARG;
        }
    if (num_waiting == 0) {  // decode-only iteration: nothing to carry the budget for
        *deficit = 0;
        *num_admitted = 0;
        return SANGAM_OK;
    }
    // the decodes are seated first; what they leave, plus the carry, is the
    // prefill budget (it may start negative when the decodes exceed tau)
    int64_t budget = tau - decode_tokens + *deficit;
    int32_t admitted = 0;
    while (admitted < num_waiting) {
        const bool empty = num_decodes == 0 && admitted == 0;
        const int64_t need = waiting[admitted];
        if (need > budget && !empty) break;  // indivisible: it waits for more budget
        budget -= need;
        ++admitted;
    }
    *deficit = budget > 0 ? budget : 0;
    *num_admitted = admitted;
    return SANGAM_OK;
}
