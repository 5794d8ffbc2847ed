/*
 * evo_probe.h -- unit-rate probe of the MI355X (gfx950) library.
 *
 * Measures how many lane operations per second the vector ALU of the whole
 * GPU retires for the operations the softmax of the attention is made of
 * (the exponential and the fused multiply-add), so that the throughput
 * bounds quoted for the attention kernels can be reproduced on the machine
 * at hand.  Not part of the attention computation itself.
 */
#ifndef EVO_PROBE_H
#define EVO_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum evo_probe_op {
    EVO_PROBE_EXP2 = 0, /* v_exp_f32: base-2 exponential, fp32 */
    EVO_PROBE_FMA = 1   /* v_fma_f32: fused multiply-add, fp32 */
};

/*
 * Enqueue one probe launch on `stream`: `n_blocks` workgroups of 256 threads,
 * each thread running 8 independent chains of `iters` operations of kind
 * `op`, one instruction per chain step (so the launch retires
 * n_blocks * 256 * 8 * iters lane operations of that instruction alone).
 * `sink` is caller-owned device memory of at least n_blocks * 256 floats; one
 * result per thread is written there so the work cannot be optimised away.
 * Returns 0, 1 (invalid argument: unknown op, n_blocks < 1, iters < 1, NULL
 * sink) or 5 (launch failed).  Time it with events on `stream`.
 */
int evo_probe_rate(int op, int n_blocks, int iters, float *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* EVO_PROBE_H */
