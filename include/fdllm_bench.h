/*
 * fdllm_bench.h -- C ABI of libfdllm_bench.so, the bandwidth reference used
 * when reporting the commit selector's throughput on MI355X (gfx950).
 *
 * The vocabulary pass of the selector (arXiv 2606.02955, Alg. 1, per-position
 * confidence) must read every logit of a candidate row once, so its ceiling is
 * the rate at which HBM can be read.  fdllm_stream_read measures that rate
 * with the same access pattern and no arithmetic beyond what keeps the loads
 * alive: the buffer is cut into 256 KiB chunks (about one bf16 logits row at
 * V = 126464) that at most 768 persistent 64-lane wavefronts take
 * round-robin, the same number each; a
 * wavefront streams a chunk with 16-byte non-temporal loads, lane l reading
 * vectors l, l+64, ..., two batches of eight loads in flight per lane.
 *
 *   src     device memory, 16-byte aligned, `bytes` readable bytes (in);
 *           `bytes` must be a multiple of 16.
 *   sink    device memory, one uint32 (in/out): receives an XOR of the data
 *           (its value has no meaning; it only keeps the loads from being
 *           removed).  The caller owns both buffers.
 *   stream  HIP stream (NULL = null stream); the call only enqueues.
 * Returns 0, -1 for a null pointer, misalignment or a size that is not a
 * multiple of 16, -5 when the launch is rejected.  bytes == 0 is a no-op.
 */
#ifndef FDLLM_BENCH_H
#define FDLLM_BENCH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* fdllm_bench_stream;

int fdllm_stream_read(const void* src, size_t bytes, uint32_t* sink, fdllm_bench_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* FDLLM_BENCH_H */
