/*
 * peaks.h — achievable-peak probes of MI355X (gfx950) for the rooflines of
 * the attention kernels in attn.h.
 *
 * The paper profiles its kernels against the hardware with rocprofv3 (Section
 * "Experimental Methodology") and notes that long compute-bound kernels make
 * the GPU lower its clock (appendix throughput figures).  The published peaks
 * (8 TB/s HBM3E, 2.5 PFLOP/s dense fp16/bf16 MFMA at 2.4 GHz) are what the
 * attention rooflines are quoted against; these two probes measure what one
 * MI355X reaches with the same instruction mix under the same conditions, and
 * the shader clock it holds meanwhile:
 *
 *   peaks_hbm_read   a streaming read of a device buffer (16-byte loads, every
 *                    byte read once), the bound of the decode kernels;
 *   peaks_mfma       back-to-back v_mfma_f32_32x32x16 (fp16 or bf16) on
 *                    operands that change every instruction (random data, as
 *                    in attention, so that the power draw and the clock are
 *                    those of real operands), the bound of the prefill kernel.
 *
 * All pointers are device pointers; calls are asynchronous on `stream`.
 * Return value: 0, or -2 for bad sizes / NULL pointers (nothing launched), or
 * -5 if a launch failed (see attn_last_hip_error in attn.h).
 */
#ifndef PEAKS_H
#define PEAKS_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Read `bytes` (a multiple of 16, >= 16) of `buf` once and write one partial
 * sum per workgroup to `sink` (float[peaks_hbm_read_sink_floats()]), so that
 * no load is dead.  `buf` is 16-byte aligned.
 */
int peaks_hbm_read(const void* buf, size_t bytes, float* sink, hipStream_t stream);

/* Floats that `sink` of peaks_hbm_read must hold. */
int peaks_hbm_read_sink_floats(void);

/*
 * Every wave of a persistent grid (two 4-wave workgroups per compute unit)
 * issues `iters` x 16 MFMAs of 32x32x16 (dtype 0 = fp16, 1 = bf16) with fp32
 * accumulation: 16 operand fragments per lane are read once from `operands`
 * (peaks_mfma_operand_bytes() bytes of random data) and rotated so that each
 * MFMA takes a different pair.  Each wave writes its accumulator sum to
 * `sink` (float[peaks_mfma_waves()]).  `clocks` (unsigned long long[2]) gets
 * the shader-clock and the 100 MHz reference-clock ticks that the first wave
 * measured over its loop: shader clock = clocks[0] / clocks[1] * 100 MHz.
 * Flops of one call: peaks_mfma_waves() * iters * 16 * 32768.
 */
int peaks_mfma(int dtype, int iters, const void* operands, float* sink, unsigned long long* clocks,
               hipStream_t stream);

/* Waves that peaks_mfma runs (on the current device), and its operand bytes. */
int peaks_mfma_waves(void);
size_t peaks_mfma_operand_bytes(void);

#ifdef __cplusplus
}
#endif

#endif /* PEAKS_H */
