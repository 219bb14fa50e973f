/* Peak probes of the machine the library runs on (libtorpor_probe.so): the figures the
 * benchmark sets its rooflines and bounds against, measured instead of assumed. Not part
 * of the serving path and independent of libtorpor.so; every call allocates what it uses
 * on the current HIP device and frees it before returning, and synchronises the device.
 * Return value: 0 on success, else a hipError_t code (the outputs are then unspecified). */
#ifndef TORPOR_PROBE_H
#define TORPOR_PROBE_H
#include <stdint.h>

#ifndef TPP_API
#define TPP_API __attribute__((visibility("default")))
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Dense bf16 matrix-core throughput: `wgs` workgroups of 4 waves, each wave issuing
 * `iters` rounds of 8 independent v_mfma_f32_16x16x32_bf16 (16,384 FLOPs each), timed
 * with HIP events; best of `reps` launches. *tflops = FLOPs / time. *clock_ghz is the
 * shader clock during the launch: the cycle counter's advance over the 100 MHz real-time
 * counter's, read by the first wave (0 if unavailable). */
TPP_API int tpp_mfma_bf16(int wgs, int iters, int reps, double* tflops, double* clock_ghz);

/* Streaming HBM read: `bytes` (a multiple of 16) of device memory read once per launch
 * with 16-byte non-temporal loads by `wgs` workgroups of 256 threads, best of `reps`
 * launches; *gbs = bytes / time. Use a buffer well above the 256 MB last-level cache. */
TPP_API int tpp_hbm_read(uint64_t bytes, int wgs, int reps, double* gbs);

/* Host-to-device copy by a kernel reading pinned, device-mapped host memory (the gather
 * method of the swap engine) with 16-byte loads: `bytes` (a multiple of 16) by `wgs`
 * workgroups of 256 threads, best of `reps`; *gbs = bytes / time. */
TPP_API int tpp_gather_h2d(uint64_t bytes, int wgs, int reps, double* gbs);

#ifdef __cplusplus
}
#endif
#endif /* TORPOR_PROBE_H */
