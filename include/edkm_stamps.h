/*
 * edkm_stamps.h — block timeline of the diagnostics build of the eDKM library.
 *
 * Not part of the product ABI.  The same sources compiled with
 * -DEDKM_BLOCK_STAMPS (libedkm_stamps.so, next to libedkm.so) export every
 * entry point of edkm.h unchanged plus the three calls below; the product
 * library libedkm.so exports none of them and records nothing.  The extra cost
 * of the diagnostics build is a few global stores per block, so its launch
 * times are close to, but not the same as, the product's.
 *
 * What is recorded.  Every kernel launch made by the library after the last
 * edkm_stamps_reset() gets the next launch index q (enqueue order, counted on
 * the host, over all plans and streams of the process).  For the first
 * EDKM_STAMP_LAUNCHES launches and the first EDKM_STAMP_BLOCKS blocks of each
 * (linear block index x + gx (y + gy z)), the block writes one record of
 * EDKM_STAMP_WORDS 64-bit words at
 *     stamps[(q * EDKM_STAMP_BLOCKS + block) * EDKM_STAMP_WORDS + word]:
 *   word 0  wall clock when the block started (its thread 0),
 *   word 1  wall clock when its last wave left,
 *   words 2..6  phase marks of the block's thread 0, where a kernel has them
 *           (0 = not reached or not instrumented),
 *   word 7  the XCC (accelerator complex die) the block ran on.
 * Records of blocks that did not run (or of launches beyond the limit) stay 0.
 * The wall clock is the GPU's constant-rate counter; edkm_stamps_clock_khz()
 * gives its rate.  The record lives in one device array per process of
 * EDKM_STAMP_LAUNCHES * EDKM_STAMP_BLOCKS * EDKM_STAMP_WORDS * 8 bytes (24 MiB),
 * on the device that was current when the library was loaded.  Concurrent
 * launches from several host threads number their launches in an unspecified
 * order; use one thread.
 */
#ifndef EDKM_STAMPS_H
#define EDKM_STAMPS_H

#include "edkm.h"

#ifdef __cplusplus
extern "C" {
#endif

enum { EDKM_STAMP_LAUNCHES = 96, EDKM_STAMP_BLOCKS = 4096, EDKM_STAMP_WORDS = 8 };

/* Clears the record (synchronously, with the whole device) and restarts the
 * launch count at 0.  Returns 0 or a hipError_t code. */
int edkm_stamps_reset(void);

/* Waits for the device, then copies the whole record to the host array
 * `stamps` (EDKM_STAMP_LAUNCHES * EDKM_STAMP_BLOCKS * EDKM_STAMP_WORDS words,
 * caller-owned) and the launch names to `names` (EDKM_STAMP_LAUNCHES entries
 * of 32 bytes, NUL-terminated: the kernel name as the library's error
 * messages give it).  Returns the number of launches made since the last
 * reset (records exist for the first EDKM_STAMP_LAUNCHES of them), or -1 if a
 * HIP call failed. */
int edkm_stamps_dump(unsigned long long* stamps, char* names);

/* Rate of the stamp clock of the current device in kHz, or 0 on error. */
int edkm_stamps_clock_khz(void);

#ifdef __cplusplus
}
#endif

#endif /* EDKM_STAMPS_H */
