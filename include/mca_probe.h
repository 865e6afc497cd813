/* Issue-cost probes for gfx950 (libmca_probe.so): measurement support for the roofline
 * reasoning about the attention kernels, not part of the Monte-Carlo attention path.
 * Each wave of the probe kernel runs `rounds` rounds of a fixed block of independent
 * instructions between two pairs of clock stamps (shader clock, constant 100 MHz clock).
 */
#ifndef MCA_PROBE_H
#define MCA_PROBE_H

#ifdef __cplusplus
extern "C" {
#endif

/* Runs one probe on the current HIP device, synchronously.
 *   kind            0: 64 v_fma_f32 per round (eight independent chains)
 *                   1: 64 v_exp_f32 per round (eight independent chains)
 *                   2: 16 v_mfma_f32_16x16x32_bf16 per round (eight independent accumulators)
 *                   3: kinds 0 and 2 in one wave
 *                   4: waves 0..3 of each workgroup run kind 0, waves 4..7 kind 2
 *                   5: kinds 1 and 2 in one wave
 *                   6: waves 0..3 of each workgroup run kind 1, waves 4..7 kind 2
 *                   7: 64 v_max3_f32 per round (eight independent chains)
 *                   8: kind 1 and 64 v_fma_f32 (eight more chains) in one wave
 *   waves_per_simd  1, 2 or 4 (kinds 4 and 6: 2); the grid has one workgroup per CU of
 *                   256 * waves_per_simd threads
 *   rounds          1 .. 2^20
 *   stamps          host buffer of 4 * max_waves values; on success wave i leaves
 *                   (shader clock before, after, 100 MHz clock before, after) at 4 i
 *   nwaves          out: the number of waves, CUs * 4 * waves_per_simd
 * The call allocates and frees its own device buffers. Returns 0; -1 for an invalid
 * argument or max_waves < *nwaves (checked before any device work, except the CU count);
 * otherwise the HIP error code.
 */
int mca_issue_probe(int kind, int waves_per_simd, int rounds, long long* stamps, int max_waves, int* nwaves);

#ifdef __cplusplus
}
#endif

#endif /* MCA_PROBE_H */
