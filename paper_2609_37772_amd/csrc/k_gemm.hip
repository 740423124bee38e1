// Projection GEMMs of the action expert: C[M][N] = A[M][K] * W[N][K]^T on the
// gfx950 MFMA units (v_mfma_f32_16x16x32_bf16), fp32 accumulation, with the
// epilogue of the layer fused in.
//
// Shape of the work: M is the token count (B*H: 16..3200), N and K are the
// projection sizes (256..8192).  At batch 1 a step streams ~0.6 GB of weights
// for ~50 tokens, so the kernel is organised around the weight stream:
//   * a workgroup owns T 16-column weight tiles, one 64-row block and one
//     K split; its waves cut that K range into runs of KPW 32-deep blocks and
//     issue all loads of a run (weights and activations) before its first
//     MFMA, so each wave keeps KPW*(T + 2*4) 16-byte loads in flight;
//   * weights and activations are both stored in MFMA fragment order, so each
//     operand load is one aligned 16-byte load per lane and 1 KiB contiguous
//     per wave;
//   * activations are hi/lo bf16 planes: every weight fragment feeds two
//     MFMAs (the MFMA units idle at batch 1, HBM does not);
//   * rows past M are neither loaded nor multiplied;
//   * per-wave partial tiles are reduced through LDS in fixed wave order
//     (deterministic, no atomics); with a K split the workgroup writes an fp32
//     partial and a separate reduce kernel sums the splits in fixed order.
#include "uad_internal.h"

namespace uad {

__device__ __forceinline__ float gelu_tanh(float z) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  return 0.5f * z * (1.0f + tanhf(c * (z + 0.044715f * z * z * z)));
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

template <int EPI, int T, int KPW>
__global__ __launch_bounds__(512) void gemm_kernel(GemmArgs g) {
  extern __shared__ float red[];  // [waves][4*T*4 slots][64 lanes]
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int waves = blockDim.x >> 6;
  const int tile0 = blockIdx.x * T;  // first 16-column weight tile
  const int split = blockIdx.y;
  const int m0 = blockIdx.z * 64;
  const int KB = g.K / kTileK;
  const int kb_split = KB / gridDim.y;
  const int passes = kb_split / (KPW * waves);
  const int mt_valid = min(4, (g.M - m0 + 15) >> 4);  // wave-uniform

  f32x4 acc[4][T];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int t = 0; t < T; ++t) acc[mt][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int pass = 0; pass < passes; ++pass) {
    const int kb0 = split * kb_split + (pass * waves + wave) * KPW;
    bf16x8 w[KPW][T], ah[KPW][4], al[KPW][4];
    const __bf16 *wp = g.W + ((size_t)tile0 * KB + kb0) * kBlockElems + lane * 8;
#pragma unroll
    for (int j = 0; j < KPW; ++j)
#pragma unroll
      for (int t = 0; t < T; ++t) w[j][t] = *(const bf16x8 *)(wp + ((size_t)t * KB + j) * kBlockElems);
    const __bf16 *ap = g.A + ((size_t)(m0 >> 4) * KB + kb0) * kBlockElems + lane * 8;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const bool ok = mt < mt_valid && (m0 + mt * 16 + (lane & 15)) < g.M;
#pragma unroll
      for (int j = 0; j < KPW; ++j) {
        if (ok) {
          const __bf16 *p = ap + ((size_t)mt * KB + j) * kBlockElems;
          ah[j][mt] = *(const bf16x8 *)p;
          al[j][mt] = *(const bf16x8 *)(p + g.a_plane);
        } else {
          ah[j][mt] = bf16x8{};
          al[j][mt] = bf16x8{};
        }
      }
    }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      if (mt >= mt_valid) break;
#pragma unroll
      for (int j = 0; j < KPW; ++j)
#pragma unroll
        for (int t = 0; t < T; ++t) {
          acc[mt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[j][mt], w[j][t], acc[mt][t], 0, 0, 0);
          acc[mt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[j][mt], w[j][t], acc[mt][t], 0, 0, 0);
        }
    }
  }

  // Cross-wave reduction through LDS, fixed order over waves.
  constexpr int SLOTS = 16 * T;  // (mt, t, r) triples per lane
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((wave * SLOTS) + (mt * T + t) * 4 + r) * 64 + lane] = acc[mt][t][r];
  __syncthreads();

  // element e = slot*64 + lane, slot = (mt*T + t)*4 + r; the D fragment of a
  // 16x16 MFMA holds row 4*(lane>>4)+r, column lane&15 in each lane.
  const int n_out = (EPI == EPI_GEGLU_BF16) ? 1024 * (T / 2) : 1024 * T;
  for (int e = threadIdx.x; e < n_out; e += blockDim.x) {
    const int ln = e & 63;
    const int slot = e >> 6;
    int mt, t, r;
    if (EPI == EPI_GEGLU_BF16) {  // slot = (mt*(T/2) + pair)*4 + r; gate tile 2*pair, up tile 2*pair+1
      r = slot & 3;
      const int q = slot >> 2;
      t = 2 * (q % (T / 2));
      mt = q / (T / 2);
    } else {
      r = slot & 3;
      t = (slot >> 2) % T;
      mt = (slot >> 2) / T;
    }
    const int row = m0 + mt * 16 + (ln >> 4) * 4 + r;
    if (row >= g.M) continue;
    const int s0 = (mt * T + t) * 4 + r;
    float v = 0.f;
    for (int w2 = 0; w2 < waves; ++w2) v += red[(w2 * SLOTS + s0) * 64 + ln];
    if (EPI == EPI_GEGLU_BF16) {
      const int s1 = (mt * T + t + 1) * 4 + r;
      float u = 0.f;
      for (int w2 = 0; w2 < waves; ++w2) u += red[(w2 * SLOTS + s1) * 64 + ln];
      const int col = ((tile0 + t) >> 1) * 16 + (ln & 15);
      store_split((__bf16 *)g.out + afrag_index(row, col, g.ldo / kTileK), g.out_plane, gelu_tanh(v) * u);
    } else {
      const int col = (tile0 + t) * 16 + (ln & 15);
      if (EPI == EPI_BIAS_SILU_BF16) {
        store_split((__bf16 *)g.out + afrag_index(row, col, g.ldo / kTileK), g.out_plane, silu(v + g.bias[col]));
      } else if (EPI == EPI_PARTIAL_F32) {
        ((float *)g.out)[((size_t)split * g.part_rows + row) * g.ldo + col] = v;
      } else if (EPI == EPI_QKV) {
        if (col < g.q_dim) {
          ((__bf16 *)g.out)[(size_t)row * g.ldo + col] = (__bf16)v;
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
            g.kc[(env_head * g.s_alloc + s) * g.head_dim + c] = (__bf16)v;
          else
            g.vtc[(env_head * g.head_dim + c) * g.s_alloc + s] = (__bf16)v;
        }
      }
    }
  }
}

template <int EPI, int T, int KPW>
static hipError_t launch_t(const GemmArgs &g, const GemmPlan &p, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  dim3 grid(g.N / kTileN / T, p.splits, (g.M + 63) / 64);
  const uint32_t lds = (uint32_t)(p.waves * 16 * T * 64 * sizeof(float));
  UAD_LAUNCH((gemm_kernel<EPI, T, KPW>), grid, dim3(p.waves * 64), lds, s, ev0, ev1, g);
  return hipGetLastError();
}

// Launch shape: T tiles per workgroup (2 = a gate/up pair), a power-of-two K
// split (partial-output GEMMs only) until the grid has >= 256 workgroups while
// each split keeps >= 4 k-blocks, KPW = 4 k-blocks per wave and pass, <= 8
// waves, and as many passes as the split's K range needs.
GemmPlan plan_gemm(int epi, int M, int N, int K, int max_splits) {
  GemmPlan p{};
  const int KB = K / kTileK;
  p.T = (epi == EPI_GEGLU_BF16) ? 2 : 1;
  const int groups = (N / kTileN / p.T) * ((M + 63) / 64);
  p.splits = 1;
  if (epi == EPI_PARTIAL_F32)
    while (p.splits * 2 <= max_splits && groups * p.splits < 256 && KB % (p.splits * 2) == 0 &&
           KB / (p.splits * 2) >= 4)
      p.splits *= 2;
  const int kb_split = KB / p.splits;
  p.kpw = (kb_split % 4 == 0) ? 4 : (kb_split % 2 == 0 ? 2 : 1);
  p.waves = kb_split / p.kpw < 8 ? kb_split / p.kpw : 8;
  while (p.waves > 1 && kb_split % (p.kpw * p.waves) != 0) --p.waves;
  p.passes = kb_split / (p.kpw * p.waves);
  p.ok = KB >= 1 && N % (kTileN * p.T) == 0 && p.waves >= 1 && kb_split == p.passes * p.kpw * p.waves;
  return p;
}

#define UAD_GEMM_KPW_CASES(EPI, T)                            \
  switch (p.kpw) {                                            \
    case 1: return launch_t<EPI, T, 1>(g, p, s, ev0, ev1);    \
    case 2: return launch_t<EPI, T, 2>(g, p, s, ev0, ev1);    \
    case 4: return launch_t<EPI, T, 4>(g, p, s, ev0, ev1);    \
  }                                                           \
  return hipErrorInvalidValue;

hipError_t launch_gemm(int epi, const GemmArgs &g, const GemmPlan &p, hipStream_t s, hipEvent_t ev0,
                       hipEvent_t ev1) {
  if (!p.ok) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_BIAS_SILU_BF16: UAD_GEMM_KPW_CASES(EPI_BIAS_SILU_BF16, 1)
    case EPI_PARTIAL_F32: UAD_GEMM_KPW_CASES(EPI_PARTIAL_F32, 1)
    case EPI_GEGLU_BF16: UAD_GEMM_KPW_CASES(EPI_GEGLU_BF16, 2)
    case EPI_QKV: UAD_GEMM_KPW_CASES(EPI_QKV, 1)
  }
  return hipErrorInvalidValue;
}

}  // namespace uad
