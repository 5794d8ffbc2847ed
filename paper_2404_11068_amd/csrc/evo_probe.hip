// evo_probe.hip -- unit-rate probe (include/evo_probe.h): chains of base-2
// exponentials or fused multiply-adds, eight independent chains per lane so
// that issue, not dependency latency, bounds the rate.
#include <hip/hip_runtime.h>

#include "evo_probe.h"

namespace {

template <int OP>
__global__ void __launch_bounds__(256) probe_kernel(float *sink, int iters, float seed) {
    float x[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = seed * (float)(threadIdx.x + 1) - 0.125f * (float)c;  // in [-1.2, 0]
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            if constexpr (OP == EVO_PROBE_EXP2) {
                // stays in (-1, 0]: exp2 of a value in [-1, 0] lies in [0.5, 1]
                x[c] = __builtin_amdgcn_exp2f(x[c]) - 1.0f;
            } else {
                x[c] = __builtin_fmaf(x[c], 0.999f, 1e-3f);
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
