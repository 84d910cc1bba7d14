/*
 * mosaic_probe.h -- measurement aid of libmosaic (not a step of the
 * protocol): the throughput ceiling of the 8-bit matrix instruction the ring
 * product runs on, with operands held in registers.
 */
#ifndef MOSAIC_PROBE_H
#define MOSAIC_PROBE_H

#include <stdint.h>

#include "mosaic.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Launches 2 workgroups per compute unit, each of 4 waves running ``iters``
 * rounds of 8 independent v_mfma_i32_32x32x32_i8 on register operands:
 * mode 0 zero operands, 1 constant operands, 2 uniformly random operands
 * that change from one instruction to the next (the data the ring product
 * sees, since masked operands are uniform). ``out`` is a device int32 that
 * the launch adds to (its value has no meaning); ``ops`` (host) receives the
 * number of int8 operations launched (2 per multiply-accumulate), to be
 * divided by the time the caller measures on ``stream``. iters >= 1,
 * mode in {0, 1, 2}; otherwise MOSAIC_ERR_INVALID_ARG. */
mosaic_status mosaic_probe_mfma_i8(int32_t mode, int64_t iters, int32_t* out, int64_t* ops, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MOSAIC_PROBE_H */
