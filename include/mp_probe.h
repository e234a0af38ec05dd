/*
 * mp_probe.h -- bandwidth probes of libmp.so.
 *
 * Measurement kernels, not part of the message-passing path: the simplest
 * kernels with the aggregation's memory traffic, timed next to it to state
 * what the device actually delivers for that traffic (the achievable
 * ceiling), beside the published HBM peak.  Conventions as in mp.h: device
 * pointers owned by the caller, no allocation, asynchronous on `stream`,
 * argument errors (MP_ERR_NULL, MP_ERR_SIZE, MP_ERR_ALIGN) returned before
 * anything is enqueued.
 */
#ifndef MP_PROBE_H_
#define MP_PROBE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Device uint32 words a probe's sink must hold (one word per wavefront). */
#define MP_PROBE_SINK_WORDS 65536

/* Streaming read of `bytes` bytes at p (16-byte loads, every word folded into
 * an XOR stored to sink, so no load is dead).  p 16-byte aligned, bytes a
 * multiple of 16. */
int mp_probe_read(const void* p, int64_t bytes, uint32_t* sink, void* stream);

/* Streaming copy of `bytes` bytes from in to out (16-byte loads and stores;
 * both 16-byte aligned, bytes a multiple of 16, no overlap). */
int mp_probe_copy(const void* in, void* out, int64_t bytes, void* stream);

/* Row gather in the order of an index stream: for p in [0, n), read the
 * row_bytes bytes of row idx[p] of a table whose rows are stride_bytes apart
 * -- the aggregation's gather of x[col[p]] with no reduction and no output
 * rows (traffic: 4 + row_bytes per index).  Loads are 16 bytes, one slot of
 * row_bytes / 16 lanes per row, 8 rows per slot in flight, as in the
 * aggregation.  idx values must lie in [0, rows of the table) (not checked).
 * table and stride_bytes 16-byte aligned; row_bytes a multiple of 16 in
 * [16, 1024] and <= stride_bytes; 0 <= n <= INT32_MAX. */
int mp_probe_gather(const int32_t* idx, int64_t n, const void* table, int64_t stride_bytes,
                    int64_t row_bytes, uint32_t* sink, void* stream);

/* Scatter in the order of a destination stream: out[dest[i]] = in[i] for i
 * in [0, n), with elements of elem_bytes (4 or 8) bytes -- a radix pass's
 * data movement (reads in order, writes in the digit runs its stable order
 * makes) with no ranking (traffic: elem_bytes + 4 read and elem_bytes written
 * per element).  dest must be a permutation of [0, n) (not checked).  in and
 * out aligned to elem_bytes, dest to 4, no overlap; 0 <= n <= INT32_MAX. */
int mp_probe_scatter(const void* in, const int32_t* dest, int64_t n, int64_t elem_bytes,
                     void* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MP_PROBE_H_ */
