/*
 * ugbs_probe.h -- matrix-core ceilings of the device, measured by a tight
 * loop of matrix instructions (libugbs_probe.so).  Measurement support for
 * the benchmark's roofline context; not part of the method's path.
 */
#ifndef UGBS_PROBE_H
#define UGBS_PROBE_H

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__) || defined(__clang__)
#define UGBS_PROBE_API __attribute__((visibility("default")))
#else
#define UGBS_PROBE_API
#endif

#define UGBS_PROBE_MFMA_BF16 0   /* v_mfma_f32_16x16x32_bf16 (dense) */
#define UGBS_PROBE_SMFMAC_BF16 1 /* v_smfmac_f32_16x16x64_bf16 (2:4 sparse, counted dense-equivalent) */

/* Enqueue n_workgroups workgroups of 256 threads, each wave issuing
 * 16 * iters matrix instructions of the given kind on eight independent
 * accumulators; writes one float per thread to out (device memory of
 * ugbs_probe_out_floats(n_workgroups) floats, caller-owned).  Returns 0, 1
 * for invalid arguments (nothing enqueued), 2 for a failed launch. */
UGBS_PROBE_API int ugbs_probe_mfma(int kind, int n_workgroups, int iters, float* out, void* stream);

/* Dense-equivalent FLOP of one ugbs_probe_mfma call with these arguments. */
UGBS_PROBE_API double ugbs_probe_flop(int kind, int n_workgroups, int iters);

/* Floats written to `out` by ugbs_probe_mfma. */
UGBS_PROBE_API int ugbs_probe_out_floats(int n_workgroups);

#ifdef __cplusplus
}
#endif

#endif /* UGBS_PROBE_H */
