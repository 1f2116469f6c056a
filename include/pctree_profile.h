/*
 * pctree_profile.h -- event timing of the tree builder's dominant kernel, and
 * diagnostic overrides of its launch for tests.
 *
 * For measurement tools (a benchmark that prices the head-stream kernel
 * against the HBM roofline): when enabled, the library brackets every launch
 * of its dominant kernel with hipEvents recorded on the caller's stream.
 * Recording adds two event markers per launch, so leave it disabled in the
 * region whose wall time is reported.  Not thread-safe against concurrent
 * enable/read calls from several threads; a process-wide setting.
 */
#ifndef PCTREE_PROFILE_H
#define PCTREE_PROFILE_H

#include <stdint.h>

#include "pctree.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Start (enable != 0) or stop recording; starting discards earlier records. */
pctree_status pctree_profile_enable(int32_t enable);

/* Wait for the recorded events, then report the summed duration in
 * milliseconds and the number of launches recorded since enabling, and the
 * kernel's name (static string).  Clears the records.  PCTREE_ERR_HIP if an
 * event query fails. */
pctree_status pctree_profile_read(double* total_ms, int64_t* launches, const char** kernel);

/* Diagnostic overrides of how pctree_build_tree and pctree_chain_decode
 * launch a round, for tests of properties that must hold under any launch
 * (the tree does not depend on how the vocabulary is sliced, Alg. 1) and of
 * the abandoned-round path.  Process-wide; set them only while no call is
 * being enqueued.  The defaults (all fields as after pctree_debug_set(NULL))
 * are what every other caller gets. */
typedef struct pctree_debug_config {
  int64_t wait_ticks;        /* < 0 (default): every bounded cross-workgroup wait
                                of the single-launch round gives up after 2 s of
                                device wall clock; >= 0: after this many ticks of
                                the device wall clock (0: at the first poll that
                                finds its words missing), which abandons the
                                round: count = -1 and padded rows, see
                                pctree_build_tree                                */
  int32_t force_multilaunch; /* nonzero: build every round with per-stage
                                launches, also where one persistent launch
                                would serve                                      */
  int32_t round_slices;      /* > 0: at most this many vocabulary slices in the
                                single-launch round (default 0: one per compute
                                unit but one, at most 256)                       */
  int32_t wide_unbounded;    /* nonzero: stages with more than 16 frontier rows
                                ignore each row's lower bound of its k'-th best
                                logit, so every logit is a candidate and every
                                (row, slice) takes the exact per-slice path      */
} pctree_debug_config;

/* Install `cfg` (NULL restores the defaults).  PCTREE_ERR_INVALID_ARGUMENT if
 * round_slices is negative. */
pctree_status pctree_debug_set(const pctree_debug_config* cfg);

/* Stage timeline, for measurement tools that break a round into its steps.
 * A diagnostic build of the library (libpctree_timeline.so, compiled with
 * -DPCTREE_TIMELINE) stamps the device wall clock from thread 0 of a few
 * workgroups at the steps of every stage into a device array
 * [PCTREE_TIMELINE_WHO][PCTREE_TIMELINE_STAGES][PCTREE_TIMELINE_EVENTS] of
 * int64 ticks (0: not stamped; the clock runs at a fixed rate and is common
 * to the whole device).  Each stamp is one global store; the tree is the
 * same as the default build's.  The default library (libpctree.so) has no
 * stamps.  Rows of the array (who), stage d:
 *   0  keeper of the single-launch round: 0 merge starts, 1 every slice
 *      record seen and the rows merged, 2 stage selected (frontier
 *      published); stage PCTREE_TIMELINE_STAGES - 1: 0 stages done,
 *      1 emission done
 *   1  first streaming workgroup of the single-launch round, 2 the last
 *      one: 0 frontier wait begins, 1 head input built, 2 stream done,
 *      3 slice records published
 *   3  per-stage launches, a stage of the wide form (every stage of a round
 *      whose frontier can exceed 16 rows): workgroup 0 of the head kernel:
 *      0 start, 1 stream done, 2 end
 *   4  the same stage's merge-and-select workgroup of request 0: 0 start,
 *      1 rows merged, 2 end (selection, next head input and row bounds)
 * Every stage has its row (B <= PCTREE_MAX_BLOCK < PCTREE_TIMELINE_STAGES - 1). */
#define PCTREE_TIMELINE_WHO 5
#define PCTREE_TIMELINE_STAGES 65
#define PCTREE_TIMELINE_EVENTS 8

/* 1 in the timeline build, 0 in the default build. */
int32_t pctree_timeline_available(void);

/* Copy the stamps (PCTREE_TIMELINE_WHO * PCTREE_TIMELINE_STAGES *
 * PCTREE_TIMELINE_EVENTS entries, row-major) into `out` and the clock's rate
 * in ticks per microsecond into `ticks_per_us`, then zero the stamps.  A
 * blocking copy from the current device: call it once the rounds to read
 * have finished (and once before them, to start from zero).
 * PCTREE_ERR_UNSUPPORTED in the default build, PCTREE_ERR_INVALID_ARGUMENT
 * for a null pointer, PCTREE_ERR_HIP if a copy or the rate query fails. */
pctree_status pctree_timeline_read(int64_t* out, double* ticks_per_us);

#ifdef __cplusplus
}
#endif

#endif /* PCTREE_PROFILE_H */
