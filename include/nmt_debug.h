/*
 * nmt_debug.h -- a test hook of libnmt, not an operation of the paper.
 *
 * Lets a test make the library's device allocations fail, to check that
 * every call that allocates reports NMT_ENOMEM and releases what it had
 * allocated when an allocation fails part-way, and choose which of the two
 * bf16 GRU kernel forms a call takes, so that both are checked at sizes the
 * reference implementation finishes quickly.
 */
#ifndef NMT_DEBUG_H
#define NMT_DEBUG_H

#include "nmt.h"

#ifdef __cplusplus
extern "C" {
#endif

/* fail_after >= 0: the next fail_after device allocations of the library
 * succeed and every one after them fails as out of memory, until the next
 * call; fail_after < 0: no injected failures (the default).  Process-wide,
 * not thread-safe against concurrent library calls.  Returns the number of
 * the library's device allocations alive at the time of the call. */
int64_t nmt_debug_alloc_hook(int32_t fail_after);

/* The kernel form of the bf16 GRUs of Section 5.1's decoder step: 0 (the
 * default) streams the weights from L2 into registers where the operand
 * shape allows it (H a multiple of 128; for the first GRU, an embedding
 * width padded to a multiple of 128) and the batch gives every compute unit
 * a block; 1 streams wherever the shape allows it, whatever the batch, and
 * skips the split over K that small batches otherwise take; 2 always stages
 * both operands through LDS.  Both forms accumulate the same bf16 products
 * 16 at a time in increasing k, so where neither splits K they give the same
 * states.  Process-wide.  Returns the previous form, or -1 (and changes
 * nothing) for a form outside 0..2. */
int32_t nmt_debug_gru_form(int32_t form);

/* How many GRU launches of the process took the weight-streaming form, so a
 * test can tell which form ran. */
int64_t nmt_debug_gru_streamed(void);

#ifdef __cplusplus
}
#endif
#endif /* NMT_DEBUG_H */
