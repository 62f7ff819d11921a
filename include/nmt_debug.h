/*
 * nmt_debug.h -- a test hook of libnmt, not an operation of the paper.
 *
 * Lets a test make the library's device allocations fail, to check that
 * every call that allocates reports NMT_ENOMEM and releases what it had
 * allocated when an allocation fails part-way.
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

#ifdef __cplusplus
}
#endif
#endif /* NMT_DEBUG_H */
