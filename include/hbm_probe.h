/*
 * hbm_probe.h -- HBM bandwidth probes for one MI355X (gfx950), built into
 * libhbmprobe.so.
 *
 * Measurement only, not part of the lossy step: each call enqueues one
 * kernel that moves bytes in the access forms the step uses (16-byte vector
 * loads, 16-byte non-temporal stores, one 256-thread workgroup per
 * contiguous piece), so that the step's rate can be compared with what the
 * HBM gives for plain streams and for the step's many-row shape.  The caller
 * times the call (events on `stream`) and divides the bytes by the time.
 *
 * Conventions: device pointers, 16-byte aligned; sizes in bytes, multiples of
 * 16; `stream` is a hipStream_t (NULL = default stream); nothing is
 * allocated and nothing synchronises.  `sink` is a device buffer of at least
 * HBM_PROBE_SINK_BYTES that read-only probes may write to (in practice never:
 * it keeps the compiler from dropping loads whose values are otherwise
 * unused).  Return codes: HBM_PROBE_OK, HBM_PROBE_EINVAL for a NULL or
 * misaligned pointer, a size that is not a multiple of 16 or a grid that
 * would exceed the launch limit, HBM_PROBE_EHIP when the launch fails.
 */
#ifndef HBM_PROBE_H
#define HBM_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define HBM_PROBE_API __attribute__((visibility("default")))
#else
#define HBM_PROBE_API
#endif

enum { HBM_PROBE_OK = 0, HBM_PROBE_EINVAL = -1, HBM_PROBE_EHIP = -3 };
enum { HBM_PROBE_SINK_BYTES = 4096 };

/* Copy `bytes` from src to dst (one 16-byte load and one non-temporal
 * 16-byte store per thread, 4 KiB per workgroup).  Traffic: 2 * bytes. */
HBM_PROBE_API int hbm_probe_copy(const void* src, void* dst, size_t bytes, void* stream);

/* Read `bytes` from src (one 16-byte load per thread).  Traffic: bytes. */
HBM_PROBE_API int hbm_probe_read(const void* src, size_t bytes, void* sink, void* stream);

/* Write `bytes` of a constant to dst (one non-temporal 16-byte store per
 * thread).  Traffic: bytes. */
HBM_PROBE_API int hbm_probe_write(void* dst, size_t bytes, void* stream);

/* The step's many-row shape without its arithmetic: rows of row_bytes bytes,
 * ld_bytes apart.  Workgroup t takes 4 KiB at offset 4096 t of each of the
 * n_read rows of src (4 rows in flight per thread), then stores their XOR at
 * the same offset of each of the n_write rows of dst.  Traffic:
 * (n_read + n_write) * row_bytes. */
HBM_PROBE_API int hbm_probe_rows(const void* src, int32_t n_read, void* dst, int32_t n_write,
                                 int64_t row_bytes, int64_t ld_bytes, void* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HBM_PROBE_H */
