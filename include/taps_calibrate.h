/* taps_calibrate.h -- measured VALU issue ceilings of the GPU.
 *
 * Measurement support for the benchmark (the roofline of the edge-table
 * kernel, whose limit is VALU issue), not part of the cost-table path:
 * libtaps_calibrate.so, built beside libtaps.so.
 */
#pragma once
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Number of instruction kinds taps_calibrate_valu times (0 .. count - 1). */
int taps_calibrate_valu_kinds(void);

/* The instruction(s) of a kind, a static string; NULL for a kind out of range. */
const char *taps_calibrate_valu_name(int kind);

/* Times a kernel of 8 independent dependency chains of one 32-bit integer
 * VALU instruction class per thread, at 8 wavefronts per SIMD on every CU of
 * the current device, `iters` loop iterations of 128 instructions each (the
 * best of three launches on the null stream; the call synchronises).
 *   kind  0: v_add_u32 / v_xor_b32 on vector operands (the highest-rate class
 *            on gfx950); 1: v_bfe_u32 / v_lshl_or_b32 (3-operand and
 *            bit-field operations); 2 and up: one instruction each
 *            (taps_calibrate_valu_name), the classes the edge kernels'
 *            choice of instructions rests on.
 *   ms                 out: the launch's duration in milliseconds.
 *   wave_instructions  out: wavefront instructions the launch issued.
 *   simds              out: SIMDs of the device (4 per CU).
 * Returns 0, or nonzero for a bad argument (1) or a HIP error (2-6); the
 * outputs are then not written.  Allocates and frees a small buffer. */
int taps_calibrate_valu(int kind, uint32_t iters, float *ms, double *wave_instructions,
                        uint32_t *simds);

#ifdef __cplusplus
}
#endif
