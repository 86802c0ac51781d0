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

/* The achievable matrix-core rate, for reporting kernels against it beside the published
 * dense peak: `blocks` workgroups of 4 waves, each wave `iters` rounds of 8 independent
 * v_mfma_f32_16x16x32_bf16 on operands held in registers (no memory traffic in the loop).
 * sink: device float32 [blocks * 256], written with one checksum per thread. *flop receives
 * the matrix-core flop of the launch (2 per multiply-add). 1 <= blocks <= 65536,
 * 1 <= iters <= 1<<20; the caller times the launch (for example with HIP events). */
impala_status_t impala_probe_mfma_bf16(int32_t blocks, int32_t iters, float* sink, int64_t* flop,
                                       hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* CLEANBA_PROFILE_H */
