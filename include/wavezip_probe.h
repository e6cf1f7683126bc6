/*
 * wavezip_probe.h -- measurement aid shipped with the WaveZip library: a plain
 * streaming read of a device buffer, the achievable HBM read rate that the
 * condensation pass's one read of the frames is compared with (beside the
 * device's nominal peak).  Not part of the condensation pass.
 */
#ifndef WAVEZIP_PROBE_H
#define WAVEZIP_PROBE_H

#include <stddef.h>
#include <stdint.h>

#include "wavezip.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Reads `bytes` bytes (a multiple of 16) of device memory at `data` (16-byte
 * aligned) once, in 16-byte vectors spread over the whole device, and writes
 * nothing except possibly one word of `sink` (a device array of at least
 * 4096 uint32 values, needed so that the reads cannot be skipped).  One
 * kernel launch on `stream` (a hipStream_t as void*, NULL = default).
 * Returns WZ_ERR_NULL / WZ_ERR_ALIGN / WZ_ERR_SHAPE for a bad argument
 * (nothing enqueued), WZ_ERR_DEVICE if the launch fails, else WZ_OK.        */
wz_status wz_probe_stream_read(const void* data, size_t bytes, uint32_t* sink,
                               void* stream);

#ifdef __cplusplus
}
#endif

#endif /* WAVEZIP_PROBE_H */
