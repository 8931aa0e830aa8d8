/*
 * turnkl_testing.h -- measurement and test hooks of libturnkl.so.
 *
 * Not part of the product interface of turnkl.h: these entry points exist so
 * that benchmarks can time the row kernel on its own stream and tests can
 * reach tilings and error paths that production inputs do not.  Each hook
 * holds its setting per host thread and applies to the calls that thread
 * makes afterwards; turnkl_workspace_bytes never depends on them.
 */
#ifndef TURNKL_TESTING_H_
#define TURNKL_TESTING_H_

#include "turnkl.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Profiling hook: while both events are non-NULL, every turnkl_fwd_bwd (and
 * turnkl_fwd_bwd_noalloc) call made by this thread records `before`
 * immediately before and `after` immediately after its row kernel (the kernel
 * that reads the logits and writes the gradient), on the call's stream; a
 * turnkl_fwd_bwd_topk call brackets its support and dense-gradient kernels.
 * Pass NULL, NULL to stop.  The events must outlive the calls that record
 * them.  Returns TURNKL_OK.
 */
int turnkl_profile_row_kernel(hipEvent_t before, hipEvent_t after);

/*
 * Tiling override.  The row kernel splits each row of V logits into
 * ceil(V / (256 * e * n)) chunks, one workgroup of 256 threads per chunk,
 * where e is the number of elements in a 16-byte vector (8 bf16, 4 fp32) and
 * n = vectors_per_thread is the most vectors a thread holds (1 to 25; default
 * 25).  Smaller n means more, smaller chunks per row, hence more exchange
 * slots: size the workspace with turnkl_testing_workspace_bytes for the same
 * n.  0 restores the default.  Results agree up to floating-point summation
 * order.  Returns TURNKL_ERR_INVALID_ARG for values outside 0..25.
 */
int turnkl_set_row_tiling(int vectors_per_thread);

/* turnkl_workspace_bytes for a call made under turnkl_set_row_tiling(n)
 * (n = 0: the default tiling, the same value as turnkl_workspace_bytes);
 * 0 for invalid arguments or n outside 0..25. */
size_t turnkl_testing_workspace_bytes(int64_t n_tokens, int64_t vocab, int dtype,
                                      int32_t max_turns, int aligned_rows,
                                      int vectors_per_thread);

/*
 * Bound on the row kernel's wait for the partials of a row's other chunks: a
 * workgroup gives up after this many polls that find a partial missing,
 * records TURNKL_ERR_SYNC_TIMEOUT in the workspace and exits; the other
 * workgroups that wait give up within 256 polls of their own wait, and the
 * later kernels of the call see the error and skip their work.  0
 * restores the default (2^22 polls).  A bound of 1 makes a batch of
 * multi-chunk rows time out at once while every kernel still exits normally,
 * which is how the tests reach that error path.  Returns
 * TURNKL_ERR_INVALID_ARG for a negative value.
 */
int turnkl_set_spin_limit(int polls);

#ifdef __cplusplus
}
#endif

#endif /* TURNKL_TESTING_H_ */
