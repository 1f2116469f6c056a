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

#ifdef __cplusplus
}
#endif

#endif /* PCTREE_PROFILE_H */
