/*
 * pctree_profile.h -- event timing of the tree builder's dominant kernel.
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

#ifdef __cplusplus
}
#endif

#endif /* PCTREE_PROFILE_H */
