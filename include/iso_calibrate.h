/*
 * iso_calibrate.h -- C ABI of libiso_calibrate.so, the streaming calibration used to state the
 * achievable bandwidth of the fused single-read merge (not part of the merge path itself).
 *
 * iso_calibrate_stream: reads n_in (1..8) device arrays of n_vec 16-byte vectors once each
 * (nontemporal loads, two vectors per thread, 256-thread workgroups: the launch shape of the
 * fused pass) and, when `write` is nonzero, writes their XOR once to `out` (n_vec vectors);
 * with write == 0 only out[0] may be written, and only for data no calibration uses.  Arrays
 * are caller-owned device memory, 16-byte aligned.  Queued asynchronously on `stream`.
 * Returns 0 on success, 1 on bad arguments (nothing queued), 2 on a HIP launch error.
 */
#ifndef ISO_CALIBRATE_H
#define ISO_CALIBRATE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int iso_calibrate_stream(const void* const* in, int n_in, void* out, int64_t n_vec, int write, void* stream);

#ifdef __cplusplus
}
#endif

#endif
