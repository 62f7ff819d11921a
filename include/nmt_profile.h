/*
 * nmt_profile.h -- instrumentation of libnmt's batched decoder step.
 *
 * Not an operation of the paper: these calls let a benchmark time each
 * kernel of nmt_score_batch with HIP events recorded on the caller's stream,
 * between the kernels of the step, while the step runs as usual.
 */
#ifndef NMT_PROFILE_H
#define NMT_PROFILE_H

#include "nmt.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Phases of one step, in launch order. */
enum {
  NMT_PHASE_GRU1 = 0,      /* first GRU (with the embedding gather) */
  NMT_PHASE_QUERY = 1,     /* attention query projection */
  NMT_PHASE_ATTENTION = 2, /* masked attention and context */
  NMT_PHASE_GRU2 = 3,      /* second GRU (new states) */
  NMT_PHASE_READOUT = 4,   /* tanh readout */
  NMT_PHASE_VOCAB = 5,     /* vocabulary projection with per-tile log-sum-exp */
  NMT_PHASE_COMBINE = 6,   /* partial merge, requested-word score, id checks */
  NMT_NUM_PHASES = 7
};

typedef struct {
  int32_t steps;               /* steps timed */
  double ms[NMT_NUM_PHASES];   /* summed milliseconds per phase over those steps */
} nmt_timing;

/* Start timing the next `max_steps` calls of nmt_score_batch(_debug) on
 * model `m` (events are created here; synchronous).  Calls beyond
 * max_steps run untimed.  Errors: NMT_EINVAL, NMT_ENOMEM, NMT_EDEVICE. */
nmt_status nmt_profile_begin(nmt_model* m, int32_t max_steps);

/* Wait for `stream`, sum the recorded phase times into *out and stop
 * timing.  Errors: NMT_EINVAL (no profile running), NMT_EDEVICE. */
nmt_status nmt_profile_end(nmt_model* m, void* stream, nmt_timing* out);

#ifdef __cplusplus
}
#endif
#endif /* NMT_PROFILE_H */
