/* HBM read-bandwidth probe: the practical ceiling the verify-step kernels'
 * bandwidth is compared with (a measurement aid beside the three calls of
 * the verify step, not part of it).
 *
 * specrouter_hbm_read_probe
 *   Streams `bytes` bytes of device memory at `buf` through the GPU once:
 *   eight workgroups per CU each read one contiguous block with independent
 *   16-byte loads, eight in flight per lane, and fold the words into a value
 *   that is stored to
 *   `*sink` only if it equals a fixed constant (so the loads cannot be
 *   dropped; in practice nothing is written). The time of the launch, taken
 *   by the caller with events on `stream`, gives the read bandwidth.
 *
 *   buf    device pointer, 16-byte aligned; read only
 *   bytes  a multiple of 16, > 0
 *   sink   device pointer to one uint32 (caller-owned), or NULL
 *   stream hipStream_t as void* (NULL = the default stream); the call only
 *          enqueues the kernel
 *
 *   Returns SR_OK, SR_EINVAL (NULL or unaligned buf, bytes 0 or not a
 *   multiple of 16) or SR_ELAUNCH.
 */
#ifndef SPECROUTER_PROBE_H
#define SPECROUTER_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int specrouter_hbm_read_probe(const void* buf, size_t bytes, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif
