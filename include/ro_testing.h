/*
 * ro_testing.h -- test aids of the ro library (include/ro.h).  Not part of
 * the operations' interface: tests use them to reach rarely taken paths
 * within a few calls.
 */
#ifndef RO_TESTING_H
#define RO_TESTING_H

#include "ro.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Test aid: move epochs forward so that their wrap-around paths run after a
 * few calls instead of about 2^30 or 2^32.  The context's next gathers use
 * canonical epochs up to the last one and then wrap after canon_left - 1 of
 * them; the stream s (may be NULL) wraps its slot epoch after run_left
 * resets and its group-failure epoch after gf_left reports; the Grain set g
 * (may be NULL) wraps its fence epoch after fence_left commits.  A value
 * below 1, or one that would move an epoch backwards, leaves that epoch as
 * it is.  Results are unchanged by design: every wrap clears what an old
 * epoch could be confused with. */
int ro_debug_epochs(ro_ctx *ctx, ro_stream *s, ro_grains *g, int64_t canon_left, int64_t run_left,
                    int64_t gf_left, int64_t fence_left);

#ifdef __cplusplus
}
#endif

#endif /* RO_TESTING_H */
