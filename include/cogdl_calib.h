/*
 * cogdl_calib.h -- kernels of known memory traffic, used to calibrate the
 * hardware counters (rocprofv3 FETCH_SIZE / WRITE_SIZE) against which the
 * roofline of the operators of cogdl.h is measured.  Not part of the paper's
 * method: each call moves a number of bytes fixed by its arguments, so the
 * ratio of what a counter reports to those bytes is the counter's scale for
 * that access pattern (streaming reads, streaming writes, whole-line random
 * gathers, sub-line random gathers).
 *
 * Every pointer is a device pointer owned by the caller; calls are
 * asynchronous on `stream`; arguments are checked on the host and a bad one
 * returns 1 without launching anything (0 on success, 5 when a launch fails:
 * the codes of cogdl_status).  Library: libcogdl_calib.so.
 */
#ifndef COGDL_CALIB_H
#define COGDL_CALIB_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reads `bytes` (a multiple of 16, src 16-byte aligned) once, front to
 * back; writes one 32-bit checksum per workgroup to sink (at least 4096
 * entries): bytes read, 16 KiB at most written. */
int cogdl_calib_read(const void *src, int64_t bytes, uint32_t *sink, hipStream_t stream);

/* dst[0, bytes) = src[0, bytes) with 16-byte loads and stores (bytes a
 * multiple of 16, both 16-byte aligned): bytes read, bytes written. */
int cogdl_calib_copy(const void *src, void *dst, int64_t bytes, hipStream_t stream);

/* For i in [0, n): out[i] = checksum of the row_bytes bytes at
 * table + idx[i] * stride (row_bytes 16, 32, 64 or 128, stride a multiple of 128 and
 * at least row_bytes, table 128-byte aligned): reads idx (4 n bytes), the n
 * gathered rows (n * row_bytes bytes of data, each row inside one 128-byte
 * line, so n distinct indices touch n distinct lines) and writes 4 n bytes. */
int cogdl_calib_gather(const void *table, int64_t stride, int32_t row_bytes, const int32_t *idx,
                       int64_t n, uint32_t *out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* COGDL_CALIB_H */
