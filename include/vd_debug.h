/*
 * vd_debug.h -- the debug build of the library (libvd_debug.so, built with
 * VD_DEBUG=1).  It has the calls of vd.h, and in its kernels every index into
 * a dynamically planned LDS region (the keys and the second selection
 * histogram, the move lists, the staged rows, the fp64 reduction scratch, the
 * FastCAOTE row buffer) is checked against the extent the host planned for
 * it.  A violation sets one bit of a device error word per failing site (bit
 * 0 keys, 1 histograms, 2 evicted list, 3 mover list, 4 staged rows, 5 fp64
 * reduction scratch, 6 FastCAOTE rows, 7 the standalone compaction's lists)
 * and the access goes to index 0 of its region instead, so a violation
 * neither faults nor touches memory past the region.  A checking tool, not
 * part of the method: the release library has no such checks and no such
 * entry point.
 */
#ifndef VD_DEBUG_H
#define VD_DEBUG_H

#include "vd.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Waits for the current device to finish its work, then stores the error
 * word in *word and clears it.  VD_ERR_INVALID_ARG for a null word,
 * VD_ERR_HIP if the device or the copy fails.  Exported by libvd_debug.so
 * only. */
vd_status vd_debug_take_error_word(uint32_t *word);

#ifdef __cplusplus
}
#endif

#endif /* VD_DEBUG_H */
