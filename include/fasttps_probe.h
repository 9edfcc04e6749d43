/*
 * fasttps_probe.h -- measurement aid shipped next to the FastTPS layer library
 * (libfasttps_probe.so): a streaming read of device memory with 16-byte
 * loads, plain or non-temporal, which gives the HBM read rate this GPU
 * sustains in the same process.
 * The layer's roofline is reported against both the published HBM peak and
 * this measured rate. It is not part of the decode step.
 */
#ifndef FASTTPS_PROBE_H
#define FASTTPS_PROBE_H

#include <stddef.h>

#if defined(__GNUC__) || defined(__clang__)
#define FASTTPS_PROBE_API __attribute__((visibility("default")))
#else
#define FASTTPS_PROBE_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Read `bytes` of device memory at `src` once with 16-byte vector loads
 * (grid-stride over `blocks` workgroups of 256 threads, `unroll` loads in
 * flight per thread), and time that one launch with HIP events on `stream`.
 *   src    device, 16-byte aligned, `bytes` a positive multiple of 16;
 *          only read.
 *   sink   device, at least 1 KiB; written only in the practically
 *          impossible case that the folded data equals a fixed constant
 *          (it keeps the loads from being removed).
 *   blocks 1 .. 65536; unroll one of 1, 2, 4, 8.
 *   nontemporal
 *          0: plain loads; 1: loads with the non-temporal cache policy
 *          (global_load ... nt), the policy of the layer's weight streams.
 *   ms     host; receives the launch's duration in milliseconds.
 * The call synchronizes with `stream` (it waits for the stop event).
 * Returns 0, or -1 for an invalid argument, -6 for a HIP error.
 */
FASTTPS_PROBE_API int fasttps_probe_stream_read(const void* src, size_t bytes, void* sink, int blocks, int unroll,
                                                int nontemporal, void* stream, float* ms);

#ifdef __cplusplus
}
#endif

#endif /* FASTTPS_PROBE_H */
