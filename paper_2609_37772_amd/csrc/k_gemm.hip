// Projection GEMMs of the action expert: C[M][N] = A[M][K] * W[N][K]^T on the
// gfx950 MFMA units (v_mfma_f32_16x16x32_f16), fp32 accumulation, with the
// epilogue of the layer fused in.
//
// Shape of the work: M is the token count (B*H: 16..3200), N and K are the
// projection sizes (256..8192).  At batch 1 a step streams ~0.6 GB of weights
// for ~50 tokens, and each CU's vector-memory pipe (not HBM) is what a
// workgroup waits on, so the work is cut to balance the bytes per workgroup:
//   * a workgroup owns T 16-column weight tiles over the full K and a group of
//     up to four 16-row tiles (batch 1: the ~50 rows are split over 2-3
//     workgroups, which re-read the weight tile from L2 instead of every
//     workgroup reading all rows of the activations);
//   * its waves cut K into runs of KPW 32-deep blocks and issue all loads of
//     a run (weights and activations) before its first MFMA;
//   * weights and activations are both stored in MFMA fragment order, so each
//     operand load is one aligned 16-byte load per lane, 1 KiB per wave;
//   * per-wave partial tiles are reduced through LDS in fixed wave order
//     (deterministic, no atomics).
// RMSNorm is folded into the GEMMs: the residual GEMMs (time-MLP out, O, down)
// update h for their columns, write the per-16-column sum of squares of every
// row and the next operand fp16(h * gain_next); the GEMMs that consume a
// normalised input (QKV, gate/up) scale their accumulators by
// rstd[row] = (sum of those sums / d + eps)^-1/2, since
// RMSNorm(h) W^T = rstd * ((h * gain) W^T).
#include "uad_internal.h"

namespace uad {

__device__ __forceinline__ float gelu_tanh(float z) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  return 0.5f * z * (1.0f + tanhf(c * (z + 0.044715f * z * z * z)));
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

constexpr int kMaxTilesPerGroup = 4;
constexpr int kMaxSsqTiles = 2048 / 16;  // d_model <= 2048

template <int EPI, int T, int KPW, bool DUAL>
__global__ __launch_bounds__(512) void gemm_kernel(GemmArgs g) {
  extern __shared__ float red[];  // [waves][4*T*4 slots][64 lanes]
  constexpr bool kRstd = (EPI == EPI_QKV || EPI == EPI_GEGLU);
  __shared__ float ssq_s[kRstd ? kMaxSsqTiles : 1][64];  // this group's rows' per-tile sums of squares
  __shared__ float rstd_s[64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int waves = blockDim.x >> 6;
  const int tile0 = blockIdx.x * T;  // first 16-column weight tile
  const int MT = (g.M + 15) >> 4;
  const int mt0 = (blockIdx.z * MT) / gridDim.z;
  const int nmt = ((blockIdx.z + 1) * MT) / gridDim.z - mt0;  // 1..4, uniform
  const int m0 = mt0 * 16;
  const int KB = g.K / kTileK;
  const int passes = KB / (KPW * waves);

  f32x4 acc[kMaxTilesPerGroup][T], acc2[kMaxTilesPerGroup][DUAL ? T : 1];
#pragma unroll
  for (int mt = 0; mt < kMaxTilesPerGroup; ++mt) {
#pragma unroll
    for (int t = 0; t < T; ++t) acc[mt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < (DUAL ? T : 1); ++t) acc2[mt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Operand loads of one pass (a run of KPW k-blocks per wave) and its MFMAs.
  f16x8 w[KPW][T], a[KPW][kMaxTilesPerGroup], a2[KPW][DUAL ? kMaxTilesPerGroup : 1];
  auto load_pass = [&](int pass) {
    const int kb0 = (pass * waves + wave) * KPW;
    const op_t *wp = g.W + ((size_t)tile0 * KB + kb0) * kBlockElems + lane * 8;
#pragma unroll
    for (int j = 0; j < KPW; ++j)
#pragma unroll
      for (int t = 0; t < T; ++t) w[j][t] = *(const f16x8 *)(wp + ((size_t)t * KB + j) * kBlockElems);
    const op_t *ap = g.A + ((size_t)mt0 * KB + kb0) * kBlockElems + lane * 8;
#pragma unroll
    for (int mt = 0; mt < kMaxTilesPerGroup; ++mt) {
      const bool ok = mt < nmt && (m0 + mt * 16 + (lane & 15)) < g.M;
#pragma unroll
      for (int j = 0; j < KPW; ++j) a[j][mt] = ok ? *(const f16x8 *)(ap + ((size_t)mt * KB + j) * kBlockElems) : f16x8{};
      if (DUAL) {
        const op_t *ap2 = g.A2 + ((size_t)mt0 * KB + kb0) * kBlockElems + lane * 8;
#pragma unroll
        for (int j = 0; j < KPW; ++j)
          a2[j][mt] = ok ? *(const f16x8 *)(ap2 + ((size_t)mt * KB + j) * kBlockElems) : f16x8{};
      }
    }
  };
  auto mma_pass = [&]() {
#pragma unroll
    for (int mt = 0; mt < kMaxTilesPerGroup; ++mt) {
      if (mt >= nmt) break;
#pragma unroll
      for (int j = 0; j < KPW; ++j)
#pragma unroll
        for (int t = 0; t < T; ++t) {
          acc[mt][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[j][mt], w[j][t], acc[mt][t], 0, 0, 0);
          if (DUAL)
            acc2[mt][DUAL ? t : 0] =
                __builtin_amdgcn_mfma_f32_16x16x32_f16(a2[j][mt], w[j][t], acc2[mt][DUAL ? t : 0], 0, 0, 0);
        }
    }
  };

  // The first pass's operand loads go out first: any wait for the loads
  // issued after them (norm statistics, epilogue operands) covers them too,
  // so the kernel pays one memory round trip before its first MFMA.
  load_pass(0);
  // Every global load the kernel needs is issued before the first use so a
  // launch costs one memory round trip:
  //  * rstd of this group's rows comes from the residual GEMM's per-tile sums
  //    of squares; they go straight to LDS (LDS-direct loads, 64 rows of one
  //    tile per wave instruction), so they hold no registers and nothing waits
  //    on them before the main loop is done;
  //  * the residual epilogue's h, gain / modulation and gate values of this
  //    thread's first kEpiPrefetch output elements.
  if (kRstd && g.use_rstd) {
    const int srow = min(m0 + lane, g.M - 1);
    for (int j = wave; j < g.ssq_tiles; j += waves)
      __builtin_amdgcn_global_load_lds((const void *)(g.ssq + (size_t)j * g.m_alloc + srow),
                                       (__attribute__((address_space(3))) void *)&ssq_s[j][0], 4, 0, 0);
  }
  const int n_out_all = (EPI == EPI_GEGLU) ? nmt * 256 * (T / 2) : nmt * 256 * T;
  constexpr int kEpiPrefetch = 2;
  float pre_h[kEpiPrefetch], pre_s[kEpiPrefetch], pre_g[kEpiPrefetch];
  if (EPI == EPI_RESID_F32) {
    // branch-free: every load is unconditional from a valid address (h itself
    // stands in for an absent operand) and the value is selected afterwards
    const bool has_mod = g.mod_scale_next != nullptr, has_gain = g.gain_next != nullptr;
    const bool has_gate = g.mod_gate != nullptr;
#pragma unroll
    for (int it = 0; it < kEpiPrefetch; ++it) {
      const int e = it * (int)blockDim.x + threadIdx.x;
      const int ln = e & 63, slot = e >> 6;
      const int r = slot & 3, t = (slot >> 2) % T, mt = min((slot >> 2) / T, kMaxTilesPerGroup - 1);
      const int row = min(m0 + mt * 16 + (ln >> 4) * 4 + r, g.M - 1);
      const int col = min((tile0 + t) * 16 + (ln & 15), g.N - 1);
      const float *hp = (const float *)g.out + (size_t)row * g.ldo + col;
      const size_t ro = (size_t)row * g.mod_ld + col;
      const float *sp = has_mod ? g.mod_scale_next + ro : (has_gain ? g.gain_next + col : hp);
      const float *gp = has_gate ? g.mod_gate + ro : hp;
      const float hv = *hp, sv = *sp, gv = *gp;
      pre_h[it] = hv;
      pre_s[it] = has_mod ? 1.0f + sv : (has_gain ? sv : 0.f);
      pre_g[it] = has_gate ? gv : 1.0f;
    }
  }

  for (int pass = 0; pass < passes; ++pass) {
    if (pass > 0) load_pass(pass);
    mma_pass();
  }

  if (kRstd && g.use_rstd) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the LDS-direct sums landed

  // Dual operand (normalised input = rstd * A + A2): fold rstd into each
  // wave's partial tile before the cross-wave reduction (it is linear).
  if (DUAL) {
    __syncthreads();  // ssq_s complete
    if (threadIdx.x < 64) {
      float ss = 0.f;
      for (int j = 0; j < g.ssq_tiles; ++j) ss += ssq_s[j][threadIdx.x];
      rstd_s[threadIdx.x] = 1.0f / sqrtf(ss / (float)(g.ssq_tiles * kTileN) + g.eps);
    }
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < kMaxTilesPerGroup; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float rs = rstd_s[mt * 16 + (lane >> 4) * 4 + r];
#pragma unroll
        for (int t = 0; t < T; ++t) acc[mt][t][r] = rs * acc[mt][t][r] + acc2[mt][DUAL ? t : 0][r];
      }
  }

  // Cross-wave reduction through LDS, fixed order over waves.
  constexpr int SLOTS = kMaxTilesPerGroup * T * 4;  // (mt, t, r) triples per lane
#pragma unroll
  for (int mt = 0; mt < kMaxTilesPerGroup; ++mt)
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((wave * SLOTS) + (mt * T + t) * 4 + r) * 64 + lane] = acc[mt][t][r];
  __syncthreads();
  if (!DUAL && kRstd && g.use_rstd && threadIdx.x < 64) {
    float ss = 0.f;
    for (int j = 0; j < g.ssq_tiles; ++j) ss += ssq_s[j][threadIdx.x];
    rstd_s[threadIdx.x] = 1.0f / sqrtf(ss / (float)(g.ssq_tiles * kTileN) + g.eps);
  }
  __syncthreads();

  // Epilogue. Element e = slot*64 + lane with slot = (mt*T + t)*4 + r (for
  // GeGLU slot = (mt*(T/2) + pair)*4 + r); the D fragment of a 16x16 MFMA holds
  // row 4*(lane>>4)+r, column lane&15.  The per-wave trip count is uniform and
  // the 16 lanes holding one row are always active together.
  const int n_out = n_out_all;
  for (int e0 = 0, it = 0; e0 < n_out; e0 += blockDim.x, ++it) {
    const int e = e0 + threadIdx.x;
    if (e >= n_out) continue;  // whole waves only (n_out and blockDim are multiples of 64)
    const int ln = e & 63;
    const int slot = e >> 6;
    int mt, t, r;
    if (EPI == EPI_GEGLU) {
      r = slot & 3;
      const int q = slot >> 2;
      t = 2 * (q % (T / 2));
      mt = q / (T / 2);
    } else {
      r = slot & 3;
      t = (slot >> 2) % T;
      mt = (slot >> 2) / T;
    }
    const int rl = mt * 16 + (ln >> 4) * 4 + r;  // row within the group
    const int row = m0 + rl;
    const bool row_ok = row < g.M;
    const int s0 = (mt * T + t) * 4 + r;
    float v = 0.f;
    for (int w2 = 0; w2 < waves; ++w2) v += red[(w2 * SLOTS + s0) * 64 + ln];
    if (EPI == EPI_MOD) {
      // column c: layer c / 6d, part (c % 6d) / d (0..5 = a, b, g of the
      // attention norm, then of the MLP norm), index c % d; the final norm's
      // (a, b) follow the layers
      const int col = (tile0 + t) * 16 + (ln & 15);
      if (row_ok) {
        const float mv = v + g.bias[col];
        ((float *)g.out)[(size_t)row * g.ldo + col] = mv;
        const int per_layer = 6 * g.d_model;
        const int l = col / per_layer;
        if (l < g.n_layers) {
          const int r6 = col - l * per_layer;
          const int part = r6 / g.d_model, j = r6 - part * g.d_model;
          const int KBd = g.d_model / kTileK;
          if (part == 1 || part == 4)
            store_op(g.mod_shift_ops + (size_t)(2 * l + (part == 4)) * g.shift_stride + afrag_index(row, j, KBd), mv);
          else if (part == 0 && l == 0)
            store_op(g.next + afrag_index(row, j, KBd), g.h_in[(size_t)row * g.d_model + j] * (1.0f + mv));
        }
      }
      continue;
    }
    if (EPI == EPI_RESID_F32) {
      const int col = (tile0 + t) * 16 + (ln & 15);
      float hv = 0.f;
      const bool pf = it < kEpiPrefetch;
      float hv0 = 0.f, sc = 0.f, gt = 1.f;
#pragma unroll
      for (int k = 0; k < kEpiPrefetch; ++k)
        if (it == k) { hv0 = pre_h[k]; sc = pre_s[k]; gt = pre_g[k]; }
      if (row_ok) {
        float *hp = (float *)g.out + (size_t)row * g.ldo + col;
        const size_t ro = (size_t)row * g.mod_ld + col;
        if (!pf) {
          hv0 = g.bias ? 0.f : *hp;
          sc = g.mod_scale_next ? 1.0f + g.mod_scale_next[ro] : (g.gain_next ? g.gain_next[col] : 0.f);
          gt = g.mod_gate ? g.mod_gate[ro] : 1.0f;
        }
        hv = (g.bias ? g.bias[col] : hv0) + gt * v;
        *hp = hv;
      }
      float sq = hv * hv;  // sum over the 16 columns of this row (lanes sharing ln>>4)
#pragma unroll
      for (int off = 8; off >= 1; off >>= 1) sq += __shfl_xor(sq, off, 16);
      if (row_ok) {
        if ((ln & 15) == 0) g.ssq[(size_t)(tile0 + t) * g.m_alloc + row] = sq;
        if (g.mod_scale_next || g.gain_next) store_op(g.next + afrag_index(row, col, g.N / kTileK), hv * sc);
      }
      continue;
    }
    if (!row_ok) continue;
    const float rs = (!DUAL && (EPI == EPI_QKV || EPI == EPI_GEGLU) && g.use_rstd) ? rstd_s[rl] : 1.0f;
    if (EPI == EPI_GEGLU) {
      const int s1 = (mt * T + t + 1) * 4 + r;
      float u = 0.f;
      for (int w2 = 0; w2 < waves; ++w2) u += red[(w2 * SLOTS + s1) * 64 + ln];
      const int col = ((tile0 + t) >> 1) * 16 + (ln & 15);
      store_op((op_t *)g.out + afrag_index(row, col, g.ldo / kTileK), gelu_tanh(v * rs) * (u * rs));
    } else {
      const int col = (tile0 + t) * 16 + (ln & 15);
      if (EPI == EPI_BIAS_SILU) {
        store_op((op_t *)g.out + afrag_index(row, col, g.ldo / kTileK), silu(v + g.bias[col]));
      } else if (EPI == EPI_QKV) {
        v *= rs;
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
            g.vtc[vt_index(env_head, s, c, g.head_dim, g.s_alloc)] = (__bf16)v;
        }
      }
    }
  }
}

template <int EPI, int T, int KPW>
static hipError_t launch_t(const GemmArgs &g, const GemmPlan &p, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  dim3 grid(g.N / kTileN / T, 1, p.mgroups);
  const uint32_t lds = (uint32_t)(p.waves * kMaxTilesPerGroup * T * 4 * 64 * sizeof(float));
  if constexpr (EPI == EPI_QKV || EPI == EPI_GEGLU) {
    if (g.A2) {
      if (!g.use_rstd) return hipErrorInvalidValue;
      UAD_LAUNCH((gemm_kernel<EPI, T, KPW, true>), grid, dim3(p.waves * 64), lds, s, ev0, ev1, g);
      return hipGetLastError();
    }
  }
  UAD_LAUNCH((gemm_kernel<EPI, T, KPW, false>), grid, dim3(p.waves * 64), lds, s, ev0, ev1, g);
  return hipGetLastError();
}

// Launch shape.  Row groups: up to four 16-row tiles each; when the rows fit
// in four tiles they are spread over more groups (see below).  K: runs of
// KPW = 4 k-blocks per wave, <= 8 waves, as many passes as needed.
GemmPlan plan_gemm(int epi, int M, int N, int K) {
  GemmPlan p{};
  const int KB = K / kTileK;
  p.T = (epi == EPI_GEGLU || epi == EPI_MOD) ? 2 : 1;
  const int ngroups = N / kTileN / p.T;
  const int MT = (M + 15) / 16;
  if (MT > kMaxTilesPerGroup) {
    p.mgroups = (MT + kMaxTilesPerGroup - 1) / kMaxTilesPerGroup;
  } else {
    // small M: spread the row tiles over up to ~1.5 workgroups per CU (each
    // extra group re-reads the weight tile from L2 but halves the activation
    // rows per workgroup; measured best at batch 1: O and down 4 groups,
    // QKV 2-3, gate/up 1)
    const int want = 384 / ngroups;
    p.mgroups = want < MT ? want : MT;
    if (p.mgroups < 1) p.mgroups = 1;
  }
  p.kpw = (KB % 4 == 0) ? 4 : (KB % 2 == 0 ? 2 : 1);
  p.waves = KB / p.kpw < 8 ? KB / p.kpw : 8;
  while (p.waves > 1 && KB % (p.kpw * p.waves) != 0) --p.waves;
  p.passes = KB / (p.kpw * p.waves);
  // every row group must hold 1..4 tiles
  const int max_tiles = (MT + p.mgroups - 1) / p.mgroups;
  p.ok = KB >= 1 && N % (kTileN * p.T) == 0 && p.waves >= 1 && KB == p.passes * p.kpw * p.waves &&
         max_tiles <= kMaxTilesPerGroup && p.mgroups <= MT;
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
    case EPI_BIAS_SILU: UAD_GEMM_KPW_CASES(EPI_BIAS_SILU, 1)
    case EPI_RESID_F32: UAD_GEMM_KPW_CASES(EPI_RESID_F32, 1)
    case EPI_GEGLU: UAD_GEMM_KPW_CASES(EPI_GEGLU, 2)
    case EPI_QKV: UAD_GEMM_KPW_CASES(EPI_QKV, 1)
    case EPI_MOD: UAD_GEMM_KPW_CASES(EPI_MOD, 2)
  }
  return hipErrorInvalidValue;
}

}  // namespace uad
