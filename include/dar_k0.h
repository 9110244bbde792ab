/*
 * dar_k0.h — machine microbenchmarks for the rooflines that bound the DAR
 * kernels on one MI355X (gfx950). Exported by libdar_k0.so, which holds no
 * part of the attention path.
 *
 * The prefill's distant region (Eq. 3, lifted branch, attended in d_down
 * space) issues 4 * d_down matrix-core flops per score but one exponential
 * (the softmax of Eq. 4), so the exponential rate, not the matrix cores, is
 * its ceiling; the decode streams the split cache once per step, so it is
 * bound by HBM reads. These figures are measured here rather than taken from
 * data sheets:
 *   - bf16 matrix-core rate of v_mfma_f32_32x32x16_bf16 (independent
 *     accumulators, 1, 2 and 4 waves per SIMD);
 *   - v_exp_f32 rate (independent chains), in lanes per clock per compute
 *     unit at the clock measured during the same kernel;
 *   - both in one wavefront's instruction stream (8 matrix ops and 16
 *     exponentials per iteration), to see how far the two pipes overlap,
 *     and the same with 16 plain fp32 FMAs in place of the exponentials;
 *   - streaming HBM reads (16-byte loads, grid-stride) and writes over a
 *     caller-provided buffer larger than the caches;
 *   - the shader clock under load: the ratio of the shader cycle counter to
 *     the 100 MHz constant clock over the run, read by the first wavefront.
 *
 * dar_k0_measure runs every benchmark, synchronously, on `stream` and fills
 * `out`. buf: device buffer of buf_bytes bytes (at least 1 GiB, 16-byte
 * aligned; caller-owned, overwritten). Returns 0 on success, 1 on a bad
 * argument, 5 when the HIP runtime refuses a launch or an event.
 */
#ifndef DAR_K0_H
#define DAR_K0_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int n_cu;                      /* compute units of the device            */
    double mfma_bf16_tflops[3];    /* 1, 2, 4 waves per SIMD                 */
    double mfma_clock_mhz;         /* shader clock during the 2-wave run     */
    double exp_lanes_per_clk_cu;   /* v_exp_f32 results per clock per CU     */
    double exp_per_s;              /* device total, at exp_clock_mhz         */
    double exp_clock_mhz;
    double mix_cycles_per_iter;    /* SIMD cycles per wave-iteration of 8 MFMA + 16 exp, 2 waves/SIMD */
    double mfma_only_cycles_per_iter;  /* the 8 MFMA alone, same shape       */
    double exp_only_cycles_per_iter;   /* the 16 exp alone, same shape       */
    double fma_only_cycles_per_iter;   /* 16 v_fma_f32 alone, same shape     */
    double mix_fma_cycles_per_iter;    /* 8 MFMA + 16 v_fma_f32 in one stream */
    double hbm_read_gbs;           /* best of the grid sizes tried           */
    double hbm_write_gbs;
} dar_k0_result;

int dar_k0_measure(void* buf, size_t buf_bytes, dar_k0_result* out, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* DAR_K0_H */
