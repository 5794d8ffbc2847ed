// evo_probe.hip -- unit-rate probe (include/evo_probe.h): chains of base-2
// exponentials or fused multiply-adds, eight independent chains per lane so
// that issue, not dependency latency, bounds the rate.  Each chain step is one
// instruction: v_exp_f32 (its input negated and made absolute by operand
// modifiers, so the chain stays in (0, 1]) or the three-operand v_fma_f32 with
// all operands in vector registers, the form of the attention kernels'
// exponent arguments.
#include <hip/hip_runtime.h>

#include "evo_probe.h"

namespace {

template <int OP>
__global__ void __launch_bounds__(256) probe_kernel(float *sink, int iters, float seed) {
    float x[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = seed * (float)(threadIdx.x + 1) - 0.125f * (float)c;  // in [-1.2, 0]
    // per-lane multiplier and addend (vector registers, as in the kernels)
    const float m = 0.999f - 1e-7f * (float)threadIdx.x, b = 1e-3f + 1e-9f * (float)threadIdx.x;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            if constexpr (OP == EVO_PROBE_EXP2) {
                // exp2 of a value in [-1.2, 0] lies in (0.4, 1]: the chain stays there
                x[c] = __builtin_amdgcn_exp2f(-fabsf(x[c]));
            } else {
                x[c] = __builtin_fmaf(x[c], m, b);
            }
        }
    }
    float acc = 0.0f;
#pragma unroll
    for (int c = 0; c < 8; ++c) acc += x[c];
    sink[blockIdx.x * 256 + threadIdx.x] = acc;
}

}  // namespace

extern "C" int evo_probe_rate(int op, int n_blocks, int iters, float *sink, void *stream) {
    if ((op != EVO_PROBE_EXP2 && op != EVO_PROBE_FMA) || n_blocks < 1 || iters < 1 || !sink) return 1;
    hipStream_t s = (hipStream_t)stream;
    if (op == EVO_PROBE_EXP2)
        hipLaunchKernelGGL(probe_kernel<EVO_PROBE_EXP2>, dim3(n_blocks), dim3(256), 0, s, sink, iters, -1e-3f);
    else
        hipLaunchKernelGGL(probe_kernel<EVO_PROBE_FMA>, dim3(n_blocks), dim3(256), 0, s, sink, iters, 1e-3f);
    return hipGetLastError() == hipSuccess ? 0 : 5;
}
