/*
 * svprobe.h -- measurement probe shipped beside libspecverify (libsvprobe.so).
 * Not part of the verify round: it gives the streaming-read bandwidth that a plain
 * kernel reaches on the device, the practical ceiling against which the HBM-bound
 * kernels' algorithmic GB/s are read (the published 8 TB/s is the nominal peak).
 */
#ifndef SVPROBE_H
#define SVPROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * svprobe_stream_read -- read `bytes` of device memory at `buf` once: one workgroup per
 * 32 KB chunk, every 16-byte non-temporal load of a chunk issued before any use, the
 * values folded into a checksum that is stored to sink[0] only if it equals one
 * fixed pattern (so the loads cannot be dropped; sink's content is meaningless). buf 16-byte aligned, bytes a
 * multiple of 32768 and > 0; sink device memory of one uint32. Asynchronous on
 * `stream`. Returns 0, or -1 for an invalid argument (nothing enqueued), or the HIP
 * error code of the launch.
 */
int32_t svprobe_stream_read(const void* buf, size_t bytes, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif
