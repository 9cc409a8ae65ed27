/*
 * ugbs_probe.h -- matrix-core and LDS-fill ceilings of the device, measured
 * by tight loops (libugbs_probe.so).  Measurement support for
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

/* Floats written to `out` by ugbs_probe_mfma and ugbs_probe_fill. */
UGBS_PROBE_API int ugbs_probe_out_floats(int n_workgroups);

/* Fill rate of the attention kernel's staging path: n_workgroups
 * workgroups of 128 threads each stream `iters` 16 KiB tiles, chosen at
 * random among the n_tiles tiles of `src` (device memory of n_tiles * 16
 * KiB, caller-owned), into LDS with direct loads, at most `depth` (1 or 2)
 * tiles in flight per workgroup.  clk (device, 2 x uint64) receives the
 * shader-clock and the 100 MHz constant-clock ticks of workgroup 0's run;
 * out (device, ugbs_probe_out_floats(n_workgroups) floats; the first 128
 * per workgroup are written) keeps the LDS contents live.  Returns 0, 1 for invalid arguments (nothing enqueued), 2
 * for a failed launch. */
UGBS_PROBE_API int ugbs_probe_fill(int depth, const void* src, unsigned n_tiles, int n_workgroups,
                                   int iters, unsigned long long* clk, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* UGBS_PROBE_H */
