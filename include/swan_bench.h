/*
 * swan_bench.h -- measurement support shipped beside libswan (libswanbench.so).
 * Not part of the SWAN decode path.
 */
#ifndef SWAN_BENCH_H
#define SWAN_BENCH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Streaming-read ceiling.  Reads the first floor(bytes / 1024) * 1024 bytes of
 * `buf` (device, 16-byte aligned) once, with the load form of the decode
 * attention kernels' page stream (16-byte nontemporal loads, 1 KiB contiguous
 * per wave load, `loads_in_flight` (4, 8 or 16) per wave, wave w reading the
 * w-th of `waves` contiguous slices), and writes one word per wave to
 * sink[0..waves) (device),
 * a fold of what it read, so that no load is dropped.  Enqueued on `stream`
 * (a hipStream_t, NULL = the null stream); the caller times it.  Returns 0, 1
 * for a bad argument (nothing enqueued) or 5 if the launch failed.
 */
int32_t swan_stream_read(const void* buf, size_t bytes, int32_t waves, int32_t loads_in_flight,
                         uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SWAN_BENCH_H */
