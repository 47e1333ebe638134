/*
 * synth_dev.hip -- device build of the synthetic-input generator.
 *
 * Fills HBM buffers with the value kinds of synth_rng.h.  Compiled with
 * -ffp-contract=off so that every value has the same bits as the host build
 * (synth_host.c) produces for the same (seed, stream, index).
 */
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SYNTH_FN __device__ static inline
#include "synth_rng.h"

__global__ void __launch_bounds__(256)
synth_fill_kernel(synth_spec sp, int64_t i0, int64_t n, void* out) {
  const uint64_t k1 = synth_stream_key(sp.seed, sp.stream);
  const uint64_t k2 = synth_stream_key(sp.seed, sp.stream2);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += stride) {
    const uint64_t i = (uint64_t)(i0 + j);
    switch (sp.kind) {
      case SYN_NORMAL_F32:
        ((float*)out)[j] = (float)(sp.mean + sp.std * synth_normal(k1, i, 0));
        break;
      case SYN_NORMAL_BF16:
        ((uint16_t*)out)[j] = synth_bf16((float)(sp.mean + sp.std * synth_normal(k1, i, 0)));
        break;
      case SYN_DRIFT_F32:
        ((float*)out)[j] = synth_drift_f32(&sp, k1, k2, i);
        break;
      case SYN_DRIFT_BF16:
        ((uint16_t*)out)[j] = synth_bf16(synth_drift_f32(&sp, k1, k2, i));
        break;
      case SYN_STUDENT3_BF16:
        ((uint16_t*)out)[j] = synth_bf16(synth_student3(&sp, k1, i));
        break;
      default:
        break;
    }
  }
}

/* Fill out[0..n) (device memory; float for f32 kinds, uint16 for bf16 kinds)
 * with the values at indices i0..i0+n-1, enqueued on `stream`.
 * Returns 0, -1 on a bad argument, -2 on a launch error. */
extern "C" int synth_dev_fill(const synth_spec* sp, int64_t i0, int64_t n, void* out,
                              void* stream) {
  if (!sp || sp->kind < SYN_NORMAL_F32 || sp->kind > SYN_STUDENT3_BF16 || n < 0 || i0 < 0)
    return -1;
  if (n == 0) return 0;
  if (!out) return -1;
  const int64_t threads = 256;
  int64_t blocks = (n + threads - 1) / threads;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(synth_fill_kernel, dim3((unsigned)blocks), dim3((unsigned)threads), 0,
                     (hipStream_t)stream, *sp, i0, n, out);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
