/* Test hooks of libarplan.so; not part of the public ABI (include/ar_plan.h). */
#ifndef AR_DEBUG_H
#define AR_DEBUG_H
#include "../../include/ar_plan.h"
#ifdef __cplusplus
extern "C" {
#endif
/* Host-only check of the launch tiling the executor would use for `plan`
 * (vecok != 0: all buffers 16-byte aligned).  Walks every wave tile of every
 * launch with the kernel's own index helpers and checks that each step range
 * is covered exactly once, in bounds, with aligned vector parts.  AR_OK, or
 * AR_ERR_INTERNAL with the first problem in `msg` (msglen bytes). */
ar_status ar_debug_check_tiling(ar_plan* plan, int32_t vecok, char* msg,
                                int64_t msglen);
#ifdef __cplusplus
}
#endif
#endif
