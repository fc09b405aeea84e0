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

#include "magicdec.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` of `buf` once with 16-byte loads from every compute unit: the
 * achievable HBM read bandwidth with the attention kernel's access width.
 * `sink` (one float) is written only in an astronomically unlikely case that
 * keeps the loads from being optimised away. */
int md_bench_stream_read(const void* buf, size_t bytes, float* sink, void* stream);

/* Read `bytes` of `buf` once with ordinary (cache-allocating) 16-byte loads:
 * reading a buffer larger than the L2s and the last-level cache evicts them
 * before a cold-cache timing and, unlike md_bench_fill, leaves no dirty lines
 * for the timed call to write back.  `sink` as for md_bench_stream_read. */
int md_bench_evict(const void* buf, size_t bytes, float* sink, void* stream);

/* dst[0:bytes] = src[0:bytes]: a plain copy of known size, used to calibrate
 * the HBM byte counters (FETCH_SIZE, WRITE_SIZE). */
int md_bench_copy(void* dst, const void* src, size_t bytes, void* stream);

/* Fill `bytes` of `buf` with the 32-bit `value`; writing a buffer larger than
 * the last-level caches evicts the KV cache before a cold-cache timing. */
int md_bench_fill(void* buf, size_t bytes, uint32_t value, void* stream);

/* md_verify_attn (mode 0) or md_draft_attn (mode 1) on `a`, with each
 * workgroup of the attention launch recording four readings of the GPU's
 * constant-rate wall clock (100 MHz on MI355X) into stamps[4 w .. 4 w + 3]:
 * its start, the end of its first K/V tile, the end of its main loop and its
 * end (after the split-KV merge, when it is the workgroup that merges).
 * `*n_workgroups` receives the launch's workgroup count (also on
 * MD_ERR_INVALID_ARG for a short `stamps`, so a caller can size it; a
 * longest-first launch's surplus workgroups leave their entries unwritten).
 * stamps: device uint64 [stamps_len], 8-byte aligned.  Errors as the
 * attention call, and MD_ERR_INVALID_ARG for NULL n_workgroups, a bad mode
 * or stamps_len < 4 * workgroups. */
int md_bench_attn_stamps(const md_attn_args* a, int32_t mode, int32_t n_sink, int32_t window,
                         uint64_t* stamps, int64_t stamps_len, int64_t* n_workgroups,
                         void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MAGICDEC_BENCH_H_ */
