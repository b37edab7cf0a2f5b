/*
 * dlfp_probe.h -- achievable-ceiling probes of one MI355X (libdlfp_probe.so).
 *
 * Measurement tools, not part of the hot path: they give the HBM bandwidth
 * and bf16 matrix-core rate the device delivers to access patterns like the
 * hot path's, so that its roofline fractions can be read against them as
 * well as against the vendor peaks (8 TB/s, 2.5 PFLOP/s dense bf16).
 * Return value: 0, or -1 for a bad argument (nothing launched), -4 when the
 * launch failed.  Asynchronous on `stream`; time them with HIP events.
 */
#ifndef DLFP_PROBE_H
#define DLFP_PROBE_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* `waves` wavefronts (a multiple of 4; 256-thread workgroups) each read
 * `per_wave` pieces of `piece_bytes` bytes (1024..8192, a multiple of 1024)
 * of the device buffer `buf` (`buf_bytes` bytes): wavefront w reads pieces
 * pieces[w * per_wave + p] (device int32, piece indices, clamped into the
 * buffer), `inflight` (1, 2 or 4) pieces outstanding at a time, with 16-byte
 * loads, marked non-temporal when `nontemporal` is 1 (0: default caching).
 * sink: device uint32 [waves * 64], one folded word per lane. */
int dlfp_probe_hbm_read(const void* buf, int64_t buf_bytes, const int32_t* pieces, int32_t waves,
                        int32_t per_wave, int32_t piece_bytes, int32_t inflight,
                        int32_t nontemporal, uint32_t* sink, hipStream_t stream);

/* `workgroups` 256-thread workgroups, each wavefront issuing `iters` x 4
 * independent v_mfma_f32_32x32x16_bf16 (32768 flop each).  sink: device
 * float [workgroups * 256]. */
int dlfp_probe_mfma(int32_t workgroups, int32_t iters, float* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DLFP_PROBE_H */
