/*
 * tbn_tuning.h -- test and tuning hook of libtbn (not part of the compute path).
 *
 * Callers: the parity tests, which run every kernel variant the library can choose (each
 * tile shape, reduction split and stage layout) against the oracle, and offline tuning
 * sweeps.  Production callers never need it: with every knob unset (-1, the state at load)
 * the library picks kernels from the layer geometry alone, and nothing else -- no
 * environment variable -- changes that choice.
 *
 * The knobs are process-wide and stored atomically, so setting one never races with a
 * call in flight on another thread; a call reads each knob once, so its workspace query
 * and its launch agree only if the knob does not change between them.
 */
#ifndef TBN_TUNING_H
#define TBN_TUNING_H

#include <stdint.h>

#include "tbn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum tbn_knob {
    /* forward / backward-data GEMM family and tile shape: 0-1 register-staged fallback,
     * 10-19 LDS-DMA tile shapes, 20 thin-input kernel, 30 weight streaming */
    TBN_KNOB_CONV_TILE = 0,
    /* forward / backward-data reduction split (>= 1) */
    TBN_KNOB_CONV_SPLITS = 1,
    /* weight-gradient stage layout: 0 segment-major, 1 pixel-major */
    TBN_KNOB_WGRAD_CFG = 2,
    /* pixel-major weight gradient: pixels per stage (32, 48 or 64) */
    TBN_KNOB_WGRAD_PIX = 3,
    /* weight gradient: L2 prefetch this many stages ahead (0 = off) */
    TBN_KNOB_WGRAD_PF = 4,
    /* int8-activation forward tile: 1 128x256, 2 128x128, 3 128x64, 4 64x128 */
    TBN_KNOB_I8_TILE = 5,
    /* weight-streaming forward: 0-7 select (16-byte code loads per buffer, buffers in flight
     * per wave, groups of four waves per block) = (2,4,1) (4,2,1) (8,2,1) (4,3,1) (2,4,2)
     * (4,2,2) (2,2,4) (2,3,2) */
    TBN_KNOB_FC_VARIANT = 6,
    /* fp8-activation forward tile: 1 128x256, 2 128x128, 3 128x64, 4 64x128 */
    TBN_KNOB_FP8_TILE = 7,
    TBN_KNOB_COUNT = 8
} tbn_knob;

/* Set a knob (value -1 restores the built-in choice).  TBN_ERR_SHAPE for an unknown knob. */
tbn_status tbn_tuning_set(tbn_knob knob, int32_t value);

/* Current value of a knob (-1 = unset, also for an unknown knob). */
int32_t tbn_tuning_get(tbn_knob knob);

#ifdef __cplusplus
}
#endif

#endif /* TBN_TUNING_H */
