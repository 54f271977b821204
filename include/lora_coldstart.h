/*
 * Adapter cold start (Section 2.3 C1; Section 4.1 "CPU LoRA" and CPU
 * assistance; Section 4.2): moving a cold adapter to the GPU on a side stream
 * while the adapted rows run on the CPU, and the stream-ordered hand-offs
 * between the two.
 *
 * Host flags are uint32 words in pinned host memory (hipHostMalloc); the GPU
 * writes them with a system-scope release store from a one-wave kernel queued
 * after the work it announces, so no host thread waits on the stream (the
 * asynchronous copy and signal of Section 4.2, [F2', F3']).  Values are
 * sequence numbers: a waiter waits for the flag to reach a value.
 *
 * Return codes are the LORA_* codes of lora.h; nothing is enqueued on an
 * argument error.  A capturing stream is allowed: every call enqueues only
 * copies and kernels (no host memory is reused behind the caller's back; the
 * caller owns host_x, the flag and the delta buffers and keeps them alive and
 * unchanged until the signal has been seen).
 */
#ifndef LORA_COLDSTART_H
#define LORA_COLDSTART_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Sync-free hand-off of a layer's input to the CPU (Section 4.2): enqueues
 * on `stream` a copy of x [n_rows, h] (16-bit elements, row stride ldx >= h
 * elements, device memory) into host_x [n_rows, ld_host] (pinned host, ld_host
 * >= h), then a store of `value` into *host_flag once the copy has completed.
 * Returns at once (no host synchronisation); the data in host_x is valid for
 * a reader that has seen *host_flag >= value (lora_flag_wait).  n_rows may be
 * 0 (only the signal).
 */
int lora_handoff_x(const void* x, int64_t ldx, int32_t n_rows, int32_t h, void* host_x, int64_t ld_host,
                   uint32_t* host_flag, uint32_t value, void* stream);

/*
 * Asynchronous load of a cold adapter (Section 2.3 C1; Section 4.1): copies
 * `bytes` from pinned host memory src_host into device memory dst_dev on
 * `stream` (meant to be a side stream, so that the serving stream keeps
 * running), then stores `value` into *host_flag (pinned host).  A caller
 * switches the adapter's rows to the GPU once the flag shows the value, and
 * orders its GPU use after the copy (same stream, or an event).
 */
int lora_adapter_load_async(void* dst_dev, const void* src_host, size_t bytes, uint32_t* host_flag, uint32_t value,
                            void* stream);

/* Pinned, coherent host memory for flags, hand-off buffers and adapters in
 * host memory (hipHostMalloc, fine-grained: the CPU sees the GPU's signal
 * stores without a cache flush).  *out is 256-byte aligned; lora_host_free of
 * NULL does nothing. */
int lora_host_alloc(size_t bytes, void** out);
int lora_host_free(void* p);

/* The signal alone: *host_flag = value after the work queued before it on
 * `stream`. */
int lora_signal(uint32_t* host_flag, uint32_t value, void* stream);

/*
 * CPU side: waits until *host_flag >= value (acquire), spinning, for at most
 * timeout_ns nanoseconds (< 0: no limit).  LORA_OK, or LORA_E_SYNC on timeout.
 * LORA_E_ARG for a NULL flag.
 */
int lora_flag_wait(const uint32_t* host_flag, uint32_t value, int64_t timeout_ns);

/* Non-blocking probe: 1 when *host_flag >= value (acquire), else 0; -1 for a
 * NULL flag. */
int lora_flag_test(const uint32_t* host_flag, uint32_t value);

/*
 * CPU LoRA (Section 4.1 "CPU LoRA"; Section 4.2 "Profiling-guided LoRA
 * parallelization"): the adapter delta of rows [0, n_rows) of a prompt,
 *
 *     delta[t, :] = s ((x[t, :] . A) . B)       (float32, Eq. 1's x A B)
 *
 * with x [n_rows, ldx] 16-bit (dtype LORA_F16 / LORA_BF16 of lora.h), A
 * [h_in, rank] and B [rank, h_out] row-major 16-bit, all in host memory, and
 * delta [n_rows, ld_delta] float32 host memory.  Accumulation in float32
 * (x . A per rank, then the sum over ranks per output).  The rows are split
 * into slices of tokens_per_thread rows, one thread each, up to max_threads
 * threads (tokens_per_thread <= 0: n_rows / max_threads rounded up): the
 * ceil(L / c) cores of one request that a per-core profile of c tokens asks
 * for.  Synchronous; returns when every slice is done.  h_in, h_out >= 1,
 * rank in [1, 256].
 */
int lora_cpu_delta(const void* x, int64_t ldx, int32_t n_rows, int32_t h_in, int32_t h_out, int32_t dtype,
                   const void* A, const void* B, int32_t rank, float scale, float* delta, int64_t ld_delta,
                   int32_t tokens_per_thread, int32_t max_threads);

/*
 * Merge of a CPU-computed delta (Eq. 1: the base output adapted by x A B):
 * y[t, :] = round(y[t, :] + delta[t, :]) for rows [0, n_rows), y [n_rows, ldy]
 * 16-bit device memory (dtype as above), delta [n_rows, ld_delta] float32
 * device memory.  One HBM-bound kernel on `stream`.  h_out, ldy and ld_delta
 * multiples of 4, y 8-byte and delta 16-byte aligned.
 */
int lora_add_delta(const float* delta, int64_t ld_delta, void* y, int64_t ldy, int32_t n_rows, int32_t h_out,
                   int32_t dtype, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LORA_COLDSTART_H */
