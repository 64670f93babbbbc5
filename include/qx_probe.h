/*
 * qx_probe.h -- measurement helpers shipped next to libqx (libqxprobe.so).
 *
 * Two kernels that do nothing but what every libqx kernel must also do: stream
 * bytes from HBM once, and launch and retire a grid. Timing them on the same
 * device gives the floor against which the GEMV kernels are judged: a GEMV
 * cannot be faster than a plain coalesced read of its packed bytes in one
 * launch of similar shape. They are not part of the libqx interface.
 *
 * Return values: 0 on success, -1 for a bad argument (null or misaligned
 * pointer, size out of range), -4 if the launch failed. Both calls are
 * asynchronous on `stream` and allocate nothing.
 */
#ifndef QX_PROBE_H
#define QX_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hipStream_t;

/* Reads `bytes` bytes at device address `src` once, one 16-byte nontemporal
 * load per thread, 256 threads per block. `src` must be 16-byte aligned and
 * `bytes` a positive multiple of 16 below 2^40. `sink` (device, one uint32_t)
 * is written only when the XOR of a thread's 16 bytes equals 0x9E3779B9, which
 * keeps the loads from being optimized away; its content is meaningless. */
int qxp_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream);

/* Launches `blocks` blocks of 256 threads that do no work (1 <= blocks <= 2^20);
 * `sink` (device, one uint32_t) is never written for blocks < 2^20. */
int qxp_empty(int32_t blocks, uint32_t* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* QX_PROBE_H */
