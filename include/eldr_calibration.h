/*
 * eldr_calibration.h -- a measurement aid, not part of the MoE path.
 *
 * The layer's figure of merit is achieved HBM bandwidth against the MI355X
 * peak of about 8 TB/s.  moe_stream_read_probe reads a device buffer once,
 * as a plain streaming kernel with no other work, so that the achievable
 * read bandwidth on the same device can be reported beside that peak.
 */
#ifndef ELDR_CALIBRATION_H_
#define ELDR_CALIBRATION_H_

#include <stddef.h>
#include <stdint.h>

#include "eldr_moe.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * moe_stream_read_probe -- read `bytes` bytes at `buf` (device memory,
 * 16-byte aligned, bytes a multiple of 16) exactly once: 2048 workgroups of
 * 256 threads, each workgroup a contiguous stretch, non-temporal 16-byte
 * loads (the hint the expert FFN's weight loads carry) with eight per thread
 * in flight.  The loaded words are folded into a checksum that is
 * stored to sink[0] (one uint32 on the device) only if it equals a fixed
 * constant, so the loads cannot be optimised away and nothing else is
 * written.  Asynchronous on `stream`; returns MOE_OK or a negative code.
 */
int moe_stream_read_probe(const void* buf, size_t bytes, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif  /* ELDR_CALIBRATION_H_ */
