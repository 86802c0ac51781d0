/*
 * cleanba_profile.h -- per-kernel timing of the learner-update library (benchmarking aid).
 *
 * While a profile is open, every kernel launch the library makes (or, with `only_key`, every
 * launch whose key equals it) is bracketed by a pair of HIP events recorded on the stream the
 * kernel is launched on. Keys name the kernel family, precision and shape, for example
 * "conv_fwd/bf16/16x16/42x42" or "wgrad/bf16/4x16/84x84". Closing the profile waits for the
 * recorded events and aggregates elapsed time per key.
 *
 * Process-global and not thread-safe: open, run, and close from one host thread. The events
 * are created when the profile opens, so the timed launches allocate nothing.
 */
#ifndef CLEANBA_PROFILE_H
#define CLEANBA_PROFILE_H

#include <stddef.h>
#include <stdint.h>

#include "cleanba_learner.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Open a profile recording up to max_launches launches (older ones are kept, later ones are
 * dropped and counted). only_key: NULL records every launch. */
impala_status_t impala_profile_begin(const char* only_key, int32_t max_launches);

/* Close the profile (synchronizes the recorded events); returns the number of distinct keys,
 * or a negative status. */
int impala_profile_end(void);

/* Result i of the last closed profile: key (NUL-terminated, truncated to key_cap), total
 * milliseconds and launch count. Returns IMPALA_EINVAL when i is out of range. */
impala_status_t impala_profile_key(int32_t i, char* key, size_t key_cap, double* total_ms,
                                   int32_t* launches);

/* Launches that were not recorded because max_launches was reached in the last profile. */
int32_t impala_profile_dropped(void);

#ifdef __cplusplus
}
#endif
#endif /* CLEANBA_PROFILE_H */
