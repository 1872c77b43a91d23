/* Test hooks, exported only by the test build of the library
 * (lib/libarplan_check.so); not part of the public ABI (include/ar_plan.h). */
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

/* The executed steps of `plan` under its current options (after the
 * executor's rewrites), in executed-phase order: step i folds its nsrc[i]
 * sources over [begin[i], end[i]) and stores the result into its ndst[i]
 * destinations; its sources and then its destinations are the next
 * nsrc[i] + ndst[i] entries of idx.  *count / *idx_count receive the totals;
 * entries are written while they fit in step_cap / idx_cap (any array may be
 * NULL to query the totals).  Host only. */
ar_status ar_debug_exec_steps(ar_plan* plan, int64_t step_cap, int32_t* phase,
                              int64_t* begin, int64_t* end, int32_t* nsrc,
                              int32_t* ndst, int64_t idx_cap, int32_t* idx,
                              int64_t* count, int64_t* idx_count);

/* The tables of launch `stage` (as in ar_plan_launch_info) when it is a
 * resident or streamed sliced launch: info[0..4] = first executed phase,
 * number of phases, number of units (workgroups), words of the program, LDS
 * slots (0: a resident launch, one row per buffer); units[7 i .. 7 i + 6] =
 * first element of unit i's tile, rows to load (bit b = buffer b), rows to
 * store, 16-byte vectors in the tile, first word and number of words of its
 * step records, first word of its alias table (-1: none; masks 0 and no
 * alias table for a streamed launch); prog the program words (the resident
 * or streamed kernel's encoding).  Call with NULL arrays to read info
 * first.  AR_ERR_INVALID_ARG when the launch is neither.  Host only. */
ar_status ar_debug_resident(ar_plan* plan, int32_t stage, int64_t* info,
                            int64_t* units, uint32_t* prog);

/* How phase launch `stage` (as in ar_plan_launch_info) runs: out[0] = its
 * kernel's template source count (0: read at run time), out[1] = cache mode
 * (bit 0: nontemporal loads, bit 1: nontemporal stores), out[2] = wave tile
 * in elements, out[3] = wave tiles, out[4] = wavefronts per block, out[5] =
 * 1 when the tiles come from a table, out[6] = sources whose loads the
 * runtime-source-count kernel keeps in flight together, out[7] = waves per
 * tile (1, or the wavefronts per block in a split launch), out[8] = 1 when
 * the tile table places tiles on XCDs by position, out[9] = 1 when the launch
 * runs a wide instance (2-source, or 8-source of 4-byte elements; out has room
 * for 10).
 * AR_ERR_INVALID_ARG for a sliced launch.  Host only. */
ar_status ar_debug_launch_desc(ar_plan* plan, int32_t stage, int64_t* out);
#ifdef __cplusplus
}
#endif
#endif
