// The library's device code as one translation unit, hence one code object.
//
// Why one: the batch-1 step is a chain of short kernels (a few microseconds
// each), so every launch starts by fetching its code into the instruction
// cache, which a pair of CUs share (64 KiB).  With the kernels in three code
// objects the step's hot code (~53 KiB) landed at offsets that the rest of
// the code decided: adding 8.5 KiB of unrelated batched-kernel code ahead of
// the small-M GEMMs slowed the batch-1 step by 1.4% (same-machine, identical
// kernel code), shifting them by a further 64 KiB restored it, and the same
// offsets with the old code reproduced the loss.  Here the kernels of that
// step are instantiated first, in launch order, so they sit contiguously at
// the start of the code and, being smaller than the cache, cannot evict each
// other whatever the load address (same-machine: 0.7065 -> 0.7048 ms per step,
// independent of the code that follows).
//
// The set is the batch-1 step of the 1024-wide expert with 256-wide heads:
// time embedding, time-MLP in and out, then per layer QKV, split-KV
// attention and its merge, O and down (one instance), gate/up + GeGLU, and
// the final projection with the Euler update.
#include "uad_internal.h"

namespace uad {

template <int R>
__global__ __launch_bounds__(256) void temb_kernel(const float *__restrict__ x, const float *__restrict__ t, int M,
                                                    int Da, int d, const float *__restrict__ w_in,
                                                    const float *__restrict__ b_in,
                                                    const float *__restrict__ freqs, op_t *__restrict__ te,
                                                    unsigned *status, const int32_t *env_map, int chunk);
template <int EPI, int T, int KPW, bool DUAL, bool PIPE>
__global__ __launch_bounds__(512) void gemm_kernel(GemmArgs g);
template <int HD, int NB, bool LOWREG, int NW>
__global__ __launch_bounds__(64 * NW) void attn_kernel(AttnArgs a);
template <int SMAX, int W>
__global__ __launch_bounds__(64 * W) void attn_combine_kernel(AttnArgs a, int hd);
template <int NC>
__global__ __launch_bounds__(256) void final_kernel(FinalArgs f);

template __global__ void temb_kernel<1>(const float *__restrict__, const float *__restrict__, int, int, int,
                                        const float *__restrict__, const float *__restrict__,
                                        const float *__restrict__, op_t *__restrict__, unsigned *, const int32_t *,
                                        int);
template __global__ void gemm_kernel<EPI_BIAS_SILU, 1, 4, false, true>(GemmArgs);
template __global__ void gemm_kernel<EPI_RESID_F32, 1, 4, false, false>(GemmArgs);
template __global__ void gemm_kernel<EPI_QKV, 1, 4, false, false>(GemmArgs);
template __global__ void attn_kernel<256, 2, false, 4>(AttnArgs);
template __global__ void attn_combine_kernel<16, 4>(AttnArgs, int);
template __global__ void gemm_kernel<EPI_RESID_F32, 1, 4, false, true>(GemmArgs);
template __global__ void gemm_kernel<EPI_GEGLU, 2, 4, false, false>(GemmArgs);
template __global__ void final_kernel<4>(FinalArgs);

}  // namespace uad

#include "k_misc.inl"
#include "k_attn.inl"
#include "k_gemm.inl"
