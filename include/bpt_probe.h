/* Matrix-core ceiling probe (measurement only; not part of the blockwise transformer).
 *
 * A loop of bf16 32x32x16 matrix-core instructions on register operands, with no LDS and
 * no global-memory traffic inside the loop. Timed over long launches it gives the rate
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
 * mode 0: every product uses the same register operand pair; 1: four different register
 * pairs in turn; 2: the A operand of every product is a 1 KiB fragment read from LDS
 * (16 fragments per wave, row reads, 64 KiB of LDS per workgroup, so at most two
 * workgroups share a CU): the rate of a kernel that reads one LDS fragment per product.
 * seed: 4096 device floats (operand values); out: workgroups * 256 device floats (one sum
 * per thread, written once so the loop is not removed). Both caller-owned. stream: a
 * hipStream_t (null = default stream). Asynchronous.
 * Returns 0 on success, 1 for an invalid argument (workgroups outside 1..2^24, iters < 1,
 * mode outside 0..2, a null pointer), 4 if the launch failed. */
int32_t bpt_probe_mfma_loop(int64_t workgroups, int32_t iters, int32_t mode, const float* seed,
                            float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BPT_PROBE_H */
