/* Matrix-core ceiling probe (measurement only; not part of the blockwise transformer).
 *
 * Loops of bf16 32x32x16 matrix-core instructions on register or LDS operands, with no
 * global-memory traffic inside the loop. Timed over long launches it gives the rate
 * that the chip sustains for pure matrix work under its own clock and power management,
 * the practical ceiling against which the layer's kernels can be read beside the nominal
 * 2.5 PFLOP/s. Built into libbpt_probe.so, separate from libbpt.so. */
#ifndef BPT_PROBE_H
#define BPT_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Launch `workgroups` workgroups of 256 threads (4 waves). Each wave runs `iters`
 * iterations of 4 independent 32x32x16 bf16 products accumulated in fp32 registers, so
 * one launch performs workgroups * 4 * iters * 4 * 32768 floating-point operations.
 * Where the A operands come from, and the occupancy (set by the LDS each workgroup
 * reserves: 64 KiB lets two workgroups share a CU, two waves per SIMD; 96 KiB leaves one,
 * one wave per SIMD):
 *   mode 0: every product uses the same register operand pair (no LDS);
 *   mode 1: four different register pairs in turn (no LDS);
 *   mode 2: one 1 KiB LDS fragment per product, read at the start of each iteration
 *           (16 fragments per wave, row reads), two waves per SIMD: the fragment traffic
 *           and occupancy of the layer's attention kernels;
 *   mode 3: as 2, the fragments read one iteration ahead into a second register set;
 *   mode 4: one fragment per two products (each meets two B operands), read ahead, two
 *           waves per SIMD;
 *   mode 5: as 3 at one wave per SIMD;
 *   mode 6: as 4 at one wave per SIMD;
 *   mode 7: as 1 at one wave per SIMD.
 * seed: 4096 device floats (operand values); out: workgroups * 256 device floats (one sum
 * per thread, written once so the loop is not removed). Both caller-owned. stream: a
 * hipStream_t (null = default stream). Asynchronous.
 * Returns 0 on success, 1 for an invalid argument (workgroups outside 1..2^24, iters < 1,
 * mode outside 0..7, a null pointer), 4 if the launch failed. */
int32_t bpt_probe_mfma_loop(int64_t workgroups, int32_t iters, int32_t mode, const float* seed,
                            float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BPT_PROBE_H */
