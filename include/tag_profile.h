/*
 * tag_profile.h -- optional per-kernel timing for libtag.so.
 *
 * While a profile is active, the library records a pair of HIP events on the
 * launch stream around every launch of one kernel stage, so a caller can
 * measure that kernel's average duration inside a timed region without an
 * external profiler.  The state is process-wide and not thread-safe: use it
 * from one host thread, with no other library calls in flight on other
 * threads.  Event handles are host objects; no device memory is allocated.
 */
#ifndef TAG_PROFILE_H
#define TAG_PROFILE_H

#include <stdint.h>

#include "tag.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Kernel stages that can be timed (one kernel per stage and launch, except
 * where noted). */
enum {
    TAG_STAGE_GRAPH_BUILD = 0,    /* all kernels of tag_graph_build (one pair per call)      */
    TAG_STAGE_ENCODE = 1,         /* node encoders (op and device launches, one pair)        */
    TAG_STAGE_TRANSFORM = 2,      /* relation transforms W^h h, op and device rows (1/layer) */
    TAG_STAGE_AGG_OP_OP = 3,      /* op <- op aggregation (1/layer); on the path for heads   */
                                  /* narrower than 16 channels this also covers op <- dev    */
    TAG_STAGE_AGG_OP_DEV = 4,     /* op <- dev aggregation + combine (1/layer)               */
    TAG_STAGE_AGG_DEV_OP = 5,     /* dev <- op partial records (1/layer)                     */
    TAG_STAGE_AGG_DEV_MERGE = 6,  /* dev <- op merge + dev <- dev (1/layer)                  */
    TAG_STAGE_DEV_PREP = 7,       /* device message table (1/layer)                          */
    TAG_STAGE_DECIDE = 8,         /* all kernels of tag_gnn_decide (one pair per call)       */
    /* tag_train_step (include/tag_train.h); its forward pass records the   */
    /* stages above                                                         */
    TAG_STAGE_BWD_DECODER = 9,    /* decoder loss + backward kernels (one pair per call)     */
    TAG_STAGE_BWD_SCORES = 10,    /* per-entry scores, one launch per bucket (4/layer)       */
    TAG_STAGE_BWD_SOFTMAX = 11,   /* per-destination softmax backward (4/layer)              */
    TAG_STAGE_BWD_MESSAGES = 12,  /* per-source message backward (4/layer)                   */
    TAG_STAGE_BWD_DH = 13,        /* dH = dY W GEMMs, op and device rows (2/layer)           */
    TAG_STAGE_BWD_DW = 14,        /* split-K dW^h = dY^T H GEMMs (2/layer)                   */
    TAG_STAGE_COUNT = 15
};

/* Start recording event pairs around launches of `stage`, for at most
 * `capacity` launches (later launches are not recorded).  Replaces any
 * active profile. */
tag_status tag_profile_begin(int32_t stage, int32_t capacity);

/* Synchronise the recorded events, return the summed elapsed time of the
 * recorded launches (ms) and their count, and end the profile. */
tag_status tag_profile_end(double *total_ms, int32_t *n_launches);

#ifdef __cplusplus
}
#endif
#endif /* TAG_PROFILE_H */
