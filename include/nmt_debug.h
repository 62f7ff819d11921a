/*
 * nmt_debug.h -- a test hook of libnmt, not an operation of the paper.
 *
 * Lets a test make the library's device allocations fail, to check that
 * every call that allocates reports NMT_ENOMEM and releases what it had
 * allocated when an allocation fails part-way, and choose which of the two
 * kernel forms the bf16 products of a step take, so that both are checked
 * at sizes the reference implementation finishes quickly, and whether fp32
 * models precompute the products of the previous word and of the context.
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

/* The kernel form of the bf16 products of Section 5.1's decoder step (the
 * two GRUs, the attention query and the readout): 0 (the default) streams
 * the weights from L2 into registers where the operand shapes allow it (H a
 * multiple of 128; every A segment a whole number of 128-column chunks) and
 * the batch gives every compute unit a block; 1 streams wherever the shapes
 * allow it, whatever the batch, and skips the split over K that small
 * batches otherwise take; 2 always stages both operands through LDS; 3 and 4
 * are form 1 with the query's and readout's split of each chunk's k steps
 * between two wave groups forced off (3) or on (4).  Where neither form
 * splits K both accumulate the same bf16 products 16 at a time in
 * increasing k and give the same values.  Process-wide.  Returns the
 * previous form, or -1 (and changes nothing) for a form outside 0..4. */
int32_t nmt_debug_gemm_form(int32_t form);

/* How many launches of the process took a weight-streaming form (GRU or
 * plain product), so a test can tell which form ran. */
int64_t nmt_debug_gemm_streamed(void);

/* Whether fp32 models created from now on take the previous word's and the
 * context's products from per-word tables and per-position projections
 * (1, the default) or compute them in each step's GEMMs (0), so a test can
 * compare the two on the same weights.  Models keep the form they were
 * created with (an average takes its first member's).  Process-wide.
 * Returns the previous setting, or -1 (and changes nothing) for a value
 * other than 0 or 1. */
int32_t nmt_debug_precompute(int32_t on);

#ifdef __cplusplus
}
#endif
#endif /* NMT_DEBUG_H */
