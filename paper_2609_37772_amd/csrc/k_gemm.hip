// Projection GEMMs of the action expert: C[M][N] = A[M][K] * W[N][K]^T with
// bf16 operands on the gfx950 MFMA units (v_mfma_f32_16x16x32_bf16), fp32
// accumulation, and the epilogue of the layer fused in.
//
// Shape of the work: M is the token count (B*H: 16..3200), N and K are the
// projection sizes (256..8192).  At batch 1 the step streams ~0.6 GB of weights
// for ~50 tokens, so this kernel is organised around the weight stream:
//   * a workgroup owns NT 16-column weight tiles and a 64-token row block;
//   * its waves split K, each streaming a contiguous slice of the packed tiles
//     with 16-byte loads (one MFMA operand per lane per load);
//   * the activation fragments (64 rows x 32 k per step) come from L2;
//   * the per-wave partial tiles are reduced through LDS in a fixed order
//     (deterministic, no atomics) and the epilogue writes the result.
#include "uad_internal.h"

namespace uad {

__device__ __forceinline__ float bf2f(__bf16 v) { return (float)v; }
__device__ __forceinline__ __bf16 f2bf(float v) { return (__bf16)v; }

__device__ __forceinline__ float gelu_tanh(float z) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  return 0.5f * z * (1.0f + tanhf(c * (z + 0.044715f * z * z * z)));
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

template <int EPI, int NT>
__global__ __launch_bounds__(1024) void gemm_skinny_kernel(GemmArgs g) {
  extern __shared__ float red[];  // [waves][NT*16 values/lane-slot][64 lanes]
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int waves = blockDim.x >> 6;
  const int tile0 = blockIdx.x * NT;  // first 16-column tile
  const int m0 = blockIdx.y * 64;
  const int KB = g.K / kTileK;
  const int kb0 = (wave * KB) / waves;
  const int kb1 = ((wave + 1) * KB) / waves;

  f32x4 acc[4][NT];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const __bf16 *arow = g.A + (size_t)(m0 + (lane & 15)) * g.lda + (lane >> 4) * 8;
  const __bf16 *wt = g.W + (size_t)tile0 * KB * kBlockElems + lane * 8;

#pragma unroll 4
  for (int kb = kb0; kb < kb1; ++kb) {
    bf16x8 a[4], al[4], b[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      b[nt] = *(const bf16x8 *)(wt + ((size_t)nt * KB + kb) * kBlockElems);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const __bf16 *ap = arow + (size_t)mt * 16 * g.lda + kb * kTileK;
      a[mt] = *(const bf16x8 *)ap;
      al[mt] = *(const bf16x8 *)(ap + g.a_plane);
    }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], b[nt], acc[mt][nt], 0, 0, 0);
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[mt], b[nt], acc[mt][nt], 0, 0, 0);
      }
  }

  // Cross-wave reduction through LDS, fixed order over waves.
  constexpr int SLOTS = 16 * NT;  // (mt, nt, r) triples per lane
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((wave * SLOTS) + (mt * NT + nt) * 4 + r) * 64 + lane] = acc[mt][nt][r];
  __syncthreads();

  // element e = slot*64 + lane; slot = (mt*NT + nt)*4 + r
  const int n_out = (EPI == EPI_GEGLU_BF16) ? 1024 : 1024 * NT;
  for (int e = threadIdx.x; e < n_out; e += blockDim.x) {
    const int ln = e & 63;
    int slot = e >> 6;
    int mt, nt, r;
    if (EPI == EPI_GEGLU_BF16) {  // slot enumerates (mt, r); gate is nt=0, up nt=1
      mt = slot >> 2;
      r = slot & 3;
      nt = 0;
    } else {
      r = slot & 3;
      nt = (slot >> 2) % NT;
      mt = (slot >> 2) / NT;
    }
    const int row = m0 + mt * 16 + (ln >> 4) * 4 + r;
    if (row >= g.M) continue;
    const int s0 = (mt * NT + nt) * 4 + r;
    float v = 0.f;
    for (int w = 0; w < waves; ++w) v += red[(w * SLOTS + s0) * 64 + ln];
    if (EPI == EPI_GEGLU_BF16) {
      const int s1 = (mt * NT + 1) * 4 + r;
      float u = 0.f;
      for (int w = 0; w < waves; ++w) u += red[(w * SLOTS + s1) * 64 + ln];
      const int col = (tile0 >> 1) * 16 + (ln & 15);
      store_split((__bf16 *)g.out + (size_t)row * g.ldo + col, g.out_plane, gelu_tanh(v) * u);
    } else {
      const int col = (tile0 + nt) * 16 + (ln & 15);
      if (EPI == EPI_BIAS_SILU_BF16) {
        store_split((__bf16 *)g.out + (size_t)row * g.ldo + col, g.out_plane, silu(v + g.bias[col]));
      } else if (EPI == EPI_BIAS_F32) {
        ((float *)g.out)[(size_t)row * g.ldo + col] = v + g.bias[col];
      } else if (EPI == EPI_RESID_F32) {
        float *o = (float *)g.out + (size_t)row * g.ldo + col;
        *o = *o + v;
      } else if (EPI == EPI_QKV) {
        if (col < g.q_dim) {
          ((__bf16 *)g.out)[(size_t)row * g.ldo + col] = f2bf(v);
        } else {
          const int b = row / g.chunk, i = row - b * g.chunk;
          const int kvd = g.n_kv_heads * g.head_dim;
          const int c2 = col - g.q_dim;
          const bool is_v = c2 >= kvd;
          const int c3 = is_v ? c2 - kvd : c2;
          const int kvh = c3 / g.head_dim, c = c3 - kvh * g.head_dim;
          const size_t env_head = (size_t)b * g.n_kv_heads + kvh;
          const int s = g.prefix + i;
          if (!is_v)
            g.kc[(env_head * g.s_alloc + s) * g.head_dim + c] = f2bf(v);
          else
            g.vtc[(env_head * g.head_dim + c) * g.s_alloc + s] = f2bf(v);
        }
      }
    }
  }
}

template <int EPI, int NT>
static hipError_t launch_t(const GemmArgs &g, hipStream_t s) {
  const int KB = g.K / kTileK;
  int waves = KB / 4;  // about four 32-deep k blocks per wave
  const int maxw = 16 / NT;
  if (waves > maxw) waves = maxw;
  if (waves < 1) waves = 1;
  dim3 grid(g.N / kTileN / NT, (g.M + 63) / 64);
  const size_t lds = (size_t)waves * 16 * NT * 64 * sizeof(float);
  hipLaunchKernelGGL((gemm_skinny_kernel<EPI, NT>), grid, dim3(waves * 64), lds, s, g);
  return hipGetLastError();
}

hipError_t launch_gemm(int epi, const GemmArgs &g, hipStream_t s) {
  switch (epi) {
    case EPI_BIAS_SILU_BF16: return launch_t<EPI_BIAS_SILU_BF16, 1>(g, s);
    case EPI_BIAS_F32: return launch_t<EPI_BIAS_F32, 1>(g, s);
    case EPI_RESID_F32: return launch_t<EPI_RESID_F32, 1>(g, s);
    case EPI_GEGLU_BF16: return launch_t<EPI_GEGLU_BF16, 2>(g, s);
    case EPI_QKV: return launch_t<EPI_QKV, 1>(g, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace uad
