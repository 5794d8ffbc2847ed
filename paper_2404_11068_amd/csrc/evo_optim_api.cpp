// evo_optim_api.cpp -- the C ABI declared in include/evo_optim.h: host-side
// chunk tables, validation (before any HIP call) and dispatch.
#include "evo_optim.h"

#include <hip/hip_runtime.h>
#include <math.h>

#include "evo_kernels.h"

extern "C" {

int64_t evo_mt_chunk_count(const int64_t *numels, int32_t n_tensors) {
    if (n_tensors < 0 || (n_tensors > 0 && !numels)) return -1;
    int64_t total = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        if (numels[i] < 0) return -1;
        const int64_t c = (numels[i] + EVO_MT_CHUNK - 1) / EVO_MT_CHUNK;
        if (c > 0x7fffffffLL) return -1;
        total += c;
        if (total > 0x7fffffffLL) return -1;
    }
    return total;
}

int64_t evo_mt_build_chunks(const int64_t *numels, int32_t n_tensors, evo_mt_chunk *out, int64_t capacity) {
    const int64_t n = evo_mt_chunk_count(numels, n_tensors);
    if (n < 0 || n > capacity || (n > 0 && !out)) return -1;
    int64_t k = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        const int64_t c = (numels[i] + EVO_MT_CHUNK - 1) / EVO_MT_CHUNK;
        for (int64_t j = 0; j < c; ++j) {
            out[k].tensor = i;
            out[k].index = (int32_t)j;
            ++k;
        }
    }
    return k;
}

int evo_grad_clip_scale(const evo_mt_tensor *tensors, int32_t n_tensors, const evo_mt_chunk *chunks, int32_t n_chunks,
                        float max_norm, float *workspace, float *norm_out, float *scale_out, void *stream) {
    if (n_tensors < 0 || n_chunks < 0 || !(max_norm > 0.0f) || !isfinite(max_norm)) return EVO_ERR_INVALID_ARG;
    if (n_chunks > 0 && (!tensors || !chunks || !workspace)) return EVO_ERR_INVALID_ARG;
    if (!norm_out && !scale_out) return EVO_OK;
    if (((uintptr_t)tensors & 7u) || ((uintptr_t)chunks & 7u) || ((uintptr_t)workspace & 3u) ||
        ((uintptr_t)norm_out & 3u) || ((uintptr_t)scale_out & 3u))
        return EVO_ERR_ALIGNMENT;
    return evo::launch_clip_scale(tensors, n_tensors, chunks, n_chunks, max_norm, workspace, norm_out, scale_out,
                                  (hipStream_t)stream) == hipSuccess
               ? EVO_OK
               : EVO_ERR_HIP;
}

int evo_adam_swa_step(const evo_adam_swa_hparams *hp, const evo_mt_tensor *tensors, int32_t n_tensors,
                      const evo_mt_chunk *chunks, int32_t n_chunks, const float *grad_scale, void *stream) {
    if (!hp || n_tensors < 0 || n_chunks < 0) return EVO_ERR_INVALID_ARG;
    const double f[] = {hp->lr, hp->beta1, hp->beta2, hp->eps, hp->weight_decay, hp->swa_decay};
    for (double x : f)
        if (!isfinite(x)) return EVO_ERR_INVALID_ARG;
    if (hp->step < 1 || hp->beta1 < 0.0 || hp->beta1 >= 1.0 || hp->beta2 < 0.0 || hp->beta2 >= 1.0 || hp->eps < 0.0 ||
        hp->swa_decay < 0.0 || hp->swa_decay > 1.0)
        return EVO_ERR_INVALID_ARG;
    if (n_chunks == 0) return EVO_OK;
    if (!tensors || !chunks) return EVO_ERR_INVALID_ARG;
    if (((uintptr_t)tensors & 7u) || ((uintptr_t)chunks & 7u) || ((uintptr_t)grad_scale & 3u)) return EVO_ERR_ALIGNMENT;
    return evo::launch_adam_swa(*hp, tensors, n_tensors, chunks, n_chunks, grad_scale, (hipStream_t)stream) ==
                   hipSuccess
               ? EVO_OK
               : EVO_ERR_HIP;
}

}  // extern "C"
