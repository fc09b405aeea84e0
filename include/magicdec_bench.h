/*
 * magicdec_bench.h -- measurement helpers exported by libmagicdec.so for the
 * benchmark harness.  They are not part of the attention method; they give
 * the numbers its roofline is judged against.
 *
 * All pointers are device pointers, 16-byte aligned; sizes are multiples of
 * 16 bytes.  Calls are asynchronous on `stream` (hipStream_t as void*) and
 * return an md_status (MD_ERR_INVALID_ARG for NULL or misaligned arguments,
 * MD_ERR_HIP for a launch failure).
 */
#ifndef MAGICDEC_BENCH_H_
#define MAGICDEC_BENCH_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` of `buf` once with 16-byte loads from every compute unit: the
 * achievable HBM read bandwidth with the attention kernel's access width.
 * `sink` (one float) is written only in an astronomically unlikely case that
 * keeps the loads from being optimised away. */
int md_bench_stream_read(const void* buf, size_t bytes, float* sink, void* stream);

/* dst[0:bytes] = src[0:bytes]: a plain copy of known size, used to calibrate
 * the HBM byte counters (FETCH_SIZE, WRITE_SIZE). */
int md_bench_copy(void* dst, const void* src, size_t bytes, void* stream);

/* Fill `bytes` of `buf` with the 32-bit `value`; writing a buffer larger than
 * the last-level caches evicts the KV cache before a cold-cache timing. */
int md_bench_fill(void* buf, size_t bytes, uint32_t value, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MAGICDEC_BENCH_H_ */
