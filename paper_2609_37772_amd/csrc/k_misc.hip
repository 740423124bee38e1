// Small per-token kernels of the step: the per-token time embedding and
// action input projection, RMSNorm to bf16 GEMM operands, and the final
// norm + action projection fused with the masked per-token Euler update.
#include "uad_internal.h"

namespace uad {

// Sum over a 256-thread block in a fixed order (wave shuffles, then 4 partials).
__device__ __forceinline__ float block_sum_256(float v, float *scratch) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) scratch[wave] = v;
  __syncthreads();
  return (scratch[0] + scratch[1]) + (scratch[2] + scratch[3]);
}

// te[m] = [ x_m W_in^T + b_in ; sin(w t_m) ; cos(w t_m) ] as split bf16 planes
// (per-token flow-time conditioning before the action MLP)
__global__ __launch_bounds__(256) void temb_kernel(const float *__restrict__ x, const float *__restrict__ t,
                                                    int Da, int d, const float *__restrict__ w_in,
                                                    const float *__restrict__ b_in,
                                                    const float *__restrict__ freqs, __bf16 *__restrict__ te,
                                                    size_t plane) {
  __shared__ float xs[64];
  const int m = blockIdx.x;
  if (threadIdx.x < Da) xs[threadIdx.x] = x[(size_t)m * Da + threadIdx.x];
  __syncthreads();
  __bf16 *row = te + (size_t)m * 2 * d;
  for (int n = threadIdx.x; n < d; n += blockDim.x) {
    float acc = b_in[n];
    const float *w = w_in + (size_t)n * Da;
    for (int j = 0; j < Da; ++j) acc += xs[j] * w[j];
    store_split(row + n, plane, acc);
  }
  const float tm = t[m];
  const int half = d >> 1;
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    const float arg = freqs[j] * tm;
    store_split(row + d + j, plane, sinf(arg));
    store_split(row + d + half + j, plane, cosf(arg));
  }
}

// out[m] = h[m] / sqrt(mean(h[m]^2) + eps) * gain, as split bf16 planes
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float *__restrict__ h, const float *__restrict__ gain,
                                                       float eps, int d, __bf16 *__restrict__ out,
                                                       size_t plane) {
  __shared__ float scratch[4];
  const int m = blockIdx.x;
  const float *hr = h + (size_t)m * d;
  float ss = 0.f;
  for (int k = threadIdx.x; k < d; k += blockDim.x) ss += hr[k] * hr[k];
  ss = block_sum_256(ss, scratch);
  const float rstd = 1.0f / sqrtf(ss / (float)d + eps);
  __bf16 *orow = out + (size_t)m * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) store_split(orow + k, plane, hr[k] * rstd * gain[k]);
}

// v = RMSNorm(h) W_out^T + b_out, then x <- x + dt v unless frozen (mask or
// dt == 0: copy, so frozen tokens are bit-identical whatever v holds).
__global__ __launch_bounds__(256) void final_kernel(FinalArgs f) {
  __shared__ float scratch[4];
  __shared__ float vs[64];
  const int m = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (f.debug_field) {
    if (threadIdx.x < f.Da) vs[threadIdx.x] = f.dbg_alpha * f.x[(size_t)m * f.Da + threadIdx.x] + f.dbg_beta;
  } else {
    const float *hr = f.h + (size_t)m * f.d;
    float ss = 0.f;
    for (int k = threadIdx.x; k < f.d; k += blockDim.x) ss += hr[k] * hr[k];
    ss = block_sum_256(ss, scratch);
    const float rstd = 1.0f / sqrtf(ss / (float)f.d + f.eps);
    for (int a = wave; a < f.Da; a += 4) {
      const float *w = f.w_out + (size_t)a * f.d;
      float acc = 0.f;
      for (int k = lane; k < f.d; k += 64) acc += (hr[k] * rstd * f.gain[k]) * w[k];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
      if (lane == 0) vs[a] = acc + f.b_out[a];
    }
  }
  __syncthreads();
  if (threadIdx.x < f.Da) {
    const int a = threadIdx.x;
    const size_t idx = (size_t)m * f.Da + a;
    const float v = vs[a];
    const float dtm = f.dt[m];
    const bool frozen = (f.mask[m] != 0) || (dtm == 0.0f);
    const float xo = f.x[idx];
    const float xn = frozen ? xo : xo + dtm * v;
    f.x[idx] = xn;
    if (f.v_out) f.v_out[idx] = v;
    const bool releasing = !frozen && (f.is_last_step || (f.next_mask && f.next_mask[m] != 0));
    if (releasing) {
      if (f.released) f.released[idx] = xn;
      if (f.release_step && a == 0) f.release_step[m] = f.step;
    }
  }
}

__global__ void stamp_kernel(uint64_t *dst) {
  if (threadIdx.x == 0) {
    const uint64_t now = __builtin_amdgcn_s_memrealtime();
    __hip_atomic_store(dst, now, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

hipError_t launch_temb(const float *x, const float *t, int M, int Da, int d, const float *w_in,
                       const float *b_in, const float *freqs, __bf16 *te, size_t plane, hipStream_t s) {
  hipLaunchKernelGGL(temb_kernel, dim3(M), dim3(256), 0, s, x, t, Da, d, w_in, b_in, freqs, te, plane);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const float *h, const float *gain, float eps, int M, int d, __bf16 *out,
                          size_t plane, hipStream_t s) {
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(M), dim3(256), 0, s, h, gain, eps, d, out, plane);
  return hipGetLastError();
}

hipError_t launch_final(const FinalArgs &f, hipStream_t s) {
  hipLaunchKernelGGL(final_kernel, dim3(f.M), dim3(256), 0, s, f);
  return hipGetLastError();
}

hipError_t launch_stamp(uint64_t *dst, hipStream_t s) {
  hipLaunchKernelGGL(stamp_kernel, dim3(1), dim3(64), 0, s, dst);
  return hipGetLastError();
}

}  // namespace uad
