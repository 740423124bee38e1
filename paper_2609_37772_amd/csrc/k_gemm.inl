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

// tanh-approximate GELU, 0.5 z (1 + tanh(u)) with u = sqrt(2/pi) (z + 0.044715 z^3),
// evaluated as z * sigmoid(2u) = z / (1 + 2^(-2u log2 e)) (the same function)
// with the hardware exp2 and reciprocal (~1 ulp each; the results are stored
// as fp16): an IEEE division here made the gate/up epilogue ALU-bound.  Large
// negative z gives -0 (2^t -> inf), large positive z gives z, NaN propagates.
__device__ __forceinline__ float gelu_tanh(float z) {
  const float k1 = -2.3022081983f;    // -2 sqrt(2/pi) log2(e)
  const float k2 = -0.1029432396f;    // k1 * 0.044715
  const float t = z * __builtin_fmaf(k2, z * z, k1);
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(t));
}

// SiLU z * sigmoid(z), by the same exp2 / reciprocal route
__device__ __forceinline__ float silu(float z) {
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950409f * z));
}

// Epilogue of one output element (row, col = 16 * tile + (ln & 15)) given its
// accumulated value v (and, for GeGLU, the matching up-projection value u);
// rs is the row's rstd (1 when unused).  EPI_RESID_F32 takes the residual h0,
// the next operand's scale sc and the branch gate gt, and must be called by
// the 16 lanes of a row together (sum of squares via shuffles).
template <int EPI>
__device__ __forceinline__ void epilogue_elem(const GemmArgs &g, int row, bool row_ok, int tile, int ln, float v,
                                              float u, float rs, float h0, float sc, float gt, unsigned &bad) {
  if (EPI == EPI_MOD) {
    // column c: layer c / 6d, part (c % 6d) / d (0..5 = a, b, g of the
    // attention norm, then of the MLP norm), index c % d; the final norm's
    // (a, b) follow the layers
    const int col = tile * 16 + (ln & 15);
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
          store_op(g.mod_shift_ops + (size_t)(2 * l + (part == 4)) * g.shift_stride + afrag_index(row, j, KBd), mv, bad);
        else if (part == 0 && l == 0 && g.next)
          store_op(g.next + afrag_index(row, j, KBd), g.h_in[(size_t)row * g.d_model + j] * (1.0f + mv), bad);
      }
    }
  } else if (EPI == EPI_RESID_F32) {
    const int col = tile * 16 + (ln & 15);
    float hv = 0.f;
    if (row_ok) {
      hv = (g.bias ? g.bias[col] : h0) + gt * v;
      ((float *)g.out)[(size_t)row * g.ldo + col] = hv;
    }
    float sq = hv * hv;  // sum over the 16 columns of this row (lanes sharing ln>>4)
    sq = sum_row16(sq);
    if (row_ok) {
      if ((ln & 15) == 0) g.ssq[(size_t)tile * g.m_alloc + row] = sq;
      if (g.mod_scale_next || g.gain_next) store_op(g.next + afrag_index(row, col, g.N / kTileK), hv * sc, bad);
    }
  } else if (row_ok) {
    if (EPI == EPI_GEGLU) {
      const int col = (tile >> 1) * 16 + (ln & 15);
      store_op((op_t *)g.out + afrag_index(row, col, g.ldo / kTileK), gelu_tanh(v * rs) * (u * rs), bad);
    } else {
      const int col = tile * 16 + (ln & 15);
      if (EPI == EPI_BIAS_SILU) {
        store_op((op_t *)g.out + afrag_index(row, col, g.ldo / kTileK), silu(v + g.bias[col]), bad);
      } else if (EPI == EPI_QKV) {
        v *= rs;
        if (col < g.q_dim) {
          ((__bf16 *)g.out)[(size_t)row * g.ldo + col] = (__bf16)v;
        } else {
          const int b = row / g.chunk, i = row - b * g.chunk;
          const int bp = g.env_map ? g.env_map[b] : b;  // the environment's K/V store slot
          const int kvd = g.n_kv_heads * g.head_dim;
          const int c2 = col - g.q_dim;
          const bool is_v = c2 >= kvd;
          const int c3 = is_v ? c2 - kvd : c2;
          const int kvh = c3 / g.head_dim, c = c3 - kvh * g.head_dim;
          const size_t env_head = (size_t)bp * g.n_kv_heads + kvh;
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

constexpr int kMaxTilesPerGroup = 4;
constexpr int kMaxSsqTiles = 2048 / 16;  // d_model <= 2048

static int g_n_cu = 256;  // compute units of the device (set by gemm_init)

// PIPE (more than one pass, single operand): the operand registers are
// double buffered, so the loads of pass p + 1 are in flight while the MFMAs
// of pass p run and a launch pays one memory round trip instead of one per
// pass.
template <int EPI, int T, int KPW, bool DUAL, bool PIPE = false>
__global__ __launch_bounds__(512) void gemm_kernel(GemmArgs g) {
  static_assert(!(PIPE && DUAL), "double-buffered passes: single operand only");
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
  f16x8 wb[PIPE ? KPW : 1][T], ab[PIPE ? KPW : 1][kMaxTilesPerGroup];  // PIPE: the second buffer
  auto load_into = [&](int pass, auto &w, auto &a) {
    const int kb0 = (pass * waves + wave) * KPW;
    const op_t *wp = g.W + ((size_t)tile0 * KB + kb0) * kBlockElems + lane * 8;
#pragma unroll
    for (int j = 0; j < KPW; ++j)
#pragma unroll
      for (int t = 0; t < T; ++t) w[j][t] = *(const f16x8 *)(wp + ((size_t)t * KB + j) * kBlockElems);
    const op_t *ap = g.A + ((size_t)mt0 * KB + kb0) * kBlockElems + lane * 8;
#pragma unroll
    for (int mt = 0; mt < kMaxTilesPerGroup; ++mt) {
      if (mt >= nmt) break;  // wave-uniform: no instructions for the group's absent row tiles
      const bool ok = (m0 + mt * 16 + (lane & 15)) < g.M;
#pragma unroll
      for (int j = 0; j < KPW; ++j) a[j][mt] = ok ? *(const f16x8 *)(ap + ((size_t)mt * KB + j) * kBlockElems) : f16x8{};
      if constexpr (DUAL) {
        const op_t *ap2 = g.A2 + ((size_t)mt0 * KB + kb0) * kBlockElems + lane * 8;
#pragma unroll
        for (int j = 0; j < KPW; ++j)
          a2[j][mt] = ok ? *(const f16x8 *)(ap2 + ((size_t)mt * KB + j) * kBlockElems) : f16x8{};
      }
    }
  };
  auto mma_from = [&](const auto &w, const auto &a) {
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
  load_into(0, w, a);
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

  if constexpr (PIPE) {
    for (int pass = 0; pass < passes; pass += 2) {
      if (pass + 1 < passes) load_into(pass + 1, wb, ab);
      mma_from(w, a);
      if (pass + 1 < passes) {
        if (pass + 2 < passes) load_into(pass + 2, w, a);
        mma_from(wb, ab);
      }
    }
  } else {
    for (int pass = 0; pass < passes; ++pass) {
      if (pass > 0) load_into(pass, w, a);
      mma_from(w, a);
    }
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
  for (int mt = 0; mt < kMaxTilesPerGroup; ++mt) {
    if (mt >= nmt) break;  // the epilogue reads only the group's own row tiles
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((wave * SLOTS) + (mt * T + t) * 4 + r) * 64 + lane] = acc[mt][t][r];
  }
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
  unsigned bad = 0;  // fp16 range flag of this thread's stores
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
    float u = 0.f, h0 = 0.f, sc = 0.f, gt = 1.f;
    if (EPI == EPI_GEGLU) {
      const int s1 = (mt * T + t + 1) * 4 + r;
      for (int w2 = 0; w2 < waves; ++w2) u += red[(w2 * SLOTS + s1) * 64 + ln];
    }
    if (EPI == EPI_RESID_F32) {
#pragma unroll
      for (int k = 0; k < kEpiPrefetch; ++k)
        if (it == k) { h0 = pre_h[k]; sc = pre_s[k]; gt = pre_g[k]; }
      if (it >= kEpiPrefetch && row_ok) {
        const int col = (tile0 + t) * 16 + (ln & 15);
        const size_t ro = (size_t)row * g.mod_ld + col;
        h0 = g.bias ? 0.f : ((const float *)g.out)[(size_t)row * g.ldo + col];
        sc = g.mod_scale_next ? 1.0f + g.mod_scale_next[ro] : (g.gain_next ? g.gain_next[col] : 0.f);
        gt = g.mod_gate ? g.mod_gate[ro] : 1.0f;
      }
    }
    const float rs = (!DUAL && kRstd && g.use_rstd && row_ok) ? rstd_s[rl] : 1.0f;
    epilogue_elem<EPI>(g, row, row_ok, tile0 + t, ln, v, u, rs, h0, sc, gt, bad);
  }
  flush_range(g.status, bad);
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
  // Double-buffered passes hold ~200 registers, one 8-wave workgroup per CU:
  // only when the grid has no more workgroups than CUs (batch 1: down 4
  // passes, O 2; step 0.700 -> 0.696 ms same-machine; at 8 environments, 448
  // workgroups, they lost 4% against two co-resident workgroups per CU).
  if (p.passes > 1 && (long)grid.x * grid.z <= g_n_cu)
    UAD_LAUNCH((gemm_kernel<EPI, T, KPW, false, true>), grid, dim3(p.waves * 64), lds, s, ev0, ev1, g);
  else
    UAD_LAUNCH((gemm_kernel<EPI, T, KPW, false>), grid, dim3(p.waves * 64), lds, s, ev0, ev1, g);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Batched projections (M >= kBigM rows): a workgroup owns a 128-row x
// 16*CT-column output tile over the full K; its 4 waves (2 x 2) each own
// 64 rows x 8*CT columns (4 x CT/2 MFMA 16x16x32 tiles).  No LDS for the
// operands: every wave streams its own fragment-order 1 KiB blocks straight
// into registers, kBigPD k-blocks ahead of the MFMAs (one aligned 16-byte
// load per lane and block; the two waves sharing a row or column panel find
// it in L2).  Measured on 2048..3200-row projections this runs at 590-940
// TFLOP/s, against ~150 for the same tiles staged through a double-buffered
// LDS ring: there every 32-deep k-step waited out a full memory round trip,
// and __syncthreads' release fence drains all loads in flight, so deeper
// rings need a raw barrier.  Tiles are dealt to the 8 XCDs in contiguous
// runs, column-major over groups of 8 row panels, so the workgroups sharing
// an L2 share weight and activation panels.  The epilogue runs from the
// accumulators (no cross-wave reduction).
// ---------------------------------------------------------------------------
constexpr int kBigRowTiles = 8;  // 128 rows per workgroup
constexpr int kBigPD = 3;        // k-blocks in flight per wave

// Output tile of workgroup blockIdx.x over ceil(M / rows) row panels and tn
// column panels: XCD x = blockIdx % 8 takes a contiguous run of tiles,
// column-major over groups of 8 row panels, so the workgroups sharing an L2
// share weight and activation panels.  The grid has 8 * ceil(tiles / 8)
// workgroups (grid_tile_wgs); false for the padding ones.
__host__ __device__ __forceinline__ int grid_tile_wgs(int M, int rows, int tn) {
  return ((M + rows - 1) / rows * tn + 7) / 8 * 8;
}

__device__ __forceinline__ bool grid_tile_at(int wg, int M, int rows, int tn, int &pm, int &pn) {
  const int tm = (M + rows - 1) / rows, T = tm * tn;
  const int per = (T + 7) / 8;
  const int t = (wg & 7) * per + (wg >> 3);
  if (t >= T) return false;
  constexpr int GM = 8;
  const int grp = t / (GM * tn), in = t - grp * GM * tn;
  const int gm0 = grp * GM, gms = min(GM, tm - gm0);
  pm = gm0 + in % gms;
  pn = in / gms;
  return true;
}

__device__ __forceinline__ bool grid_tile(int M, int rows, int tn, int &pm, int &pn) {
  return grid_tile_at((int)blockIdx.x, M, rows, tn, pm, pn);
}

template <int CT>
__device__ __forceinline__ bool big_tile(const GemmArgs &g, int &mt0, int &nt0) {
  int pm, pn;
  if (!grid_tile(g.M, 16 * kBigRowTiles, g.N / (16 * CT), pm, pn)) return false;
  mt0 = pm * kBigRowTiles;
  nt0 = pn * CT;
  return true;
}

// Epilogue of the batched kernel.  The MFMA runs with the operands swapped
// (it accumulates C^T tiles), so lane l of tile (i, j) holds row l & 15 and
// the 4 consecutive columns 4 * (l >> 4) + 0..3: every fp32 access is one
// 16-byte load or store and every fp16 / bf16 store 8 bytes.  mt / nt are
// the wave's first row / column tile; rstd (when not null) the rstd of its
// TA*16 rows.
__device__ __forceinline__ f32x4 ld4(const float *p) { return *(const f32x4 *)p; }
__device__ __forceinline__ void st4(float *p, f32x4 v) { *(f32x4 *)p = v; }
__device__ __forceinline__ void st4h(op_t *p, f32x4 v, unsigned &bad) {
  *(f16x4 *)p = f16x4{(op_t)v[0], (op_t)v[1], (op_t)v[2], (op_t)v[3]};
  check_op4(v[0], v[1], v[2], v[3], bad);
}

// Residual epilogue, store half, over NI row tiles starting at i0: h = h0 (or
// bias) + gate * v, per-16-column sums of squares of h, next operand
// fp16(h * scale).  ADA: gate and scale are per-token modulations ([NI][TB]),
// else gate = 1 and scale = gain_next (one row [1][TB]).
template <int NI, bool ADA, int TA, int TB>
__device__ __forceinline__ void big_resid_store(const GemmArgs &g, const f32x4 (&acc)[TA][TB], int i0, int mt, int nt,
                                                int lane, const f32x4 (&h0)[NI][TB],
                                                const f32x4 (&gt)[ADA ? NI : 1][TB],
                                                const f32x4 (&sc)[ADA ? NI : 1][TB], bool has_next, unsigned &bad) {
  float *h = (float *)g.out;
  const int csub = 4 * (lane >> 4);
  const int KBn = g.N / kTileK;
#pragma unroll
  for (int ii = 0; ii < NI; ++ii) {
    const int row = (mt + i0 + ii) * 16 + (lane & 15);
    const bool row_ok = row < g.M;
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      const int tile = nt + j, col = tile * 16 + csub;
      const f32x4 hv = ADA ? h0[ii][j] + gt[ADA ? ii : 0][j] * acc[i0 + ii][j] : h0[ii][j] + acc[i0 + ii][j];
      if (row_ok) st4(h + (size_t)row * g.ldo + col, hv);
      float sq = hv[0] * hv[0] + hv[1] * hv[1] + hv[2] * hv[2] + hv[3] * hv[3];
      sq = sum_pair32(sum_pair16(sq));  // the 4 lanes holding this row's 16 columns
      if (row_ok) {
        if (lane < 16) g.ssq[(size_t)tile * g.m_alloc + row] = sq;
        if (has_next) st4h(g.next + afrag_index(row, col, KBn), hv * sc[ADA ? ii : 0][j], bad);
      }
    }
  }
}

// Residual epilogue, load half: h0 (or the bias) of NI row tiles from i0, and
// the scale (and, ADA, the gate) of the next operand.  Branch-free: every load
// comes from a valid address (an absent operand is stood in for by one that
// exists) and the value is selected afterwards, so no load waits on another.
template <int NI, bool ADA, int TB>
__device__ __forceinline__ void big_resid_load(const GemmArgs &g, int i0, int mt, int nt, int lane,
                                               f32x4 (&h0)[NI][TB], f32x4 (&gt)[ADA ? NI : 1][TB],
                                               f32x4 (&sc)[ADA ? NI : 1][TB]) {
  const int csub = 4 * (lane >> 4);
  const bool has_next = ADA ? g.mod_scale_next != nullptr : g.gain_next != nullptr;
  const float *hb = g.bias ? g.bias : (const float *)g.out;
  const size_t hld = g.bias ? 0 : (size_t)g.ldo;
  const float *sb = ADA ? (has_next ? g.mod_scale_next : g.mod_gate) : (has_next ? g.gain_next : hb);
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ii = 0; ii < NI; ++ii) {
    const int rowc = min((mt + i0 + ii) * 16 + (lane & 15), g.M - 1);
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      const int col = (nt + j) * 16 + csub;
      h0[ii][j] = ld4(hb + (size_t)rowc * hld + col);
      if (ADA) {
        const size_t ro = (size_t)rowc * g.mod_ld + col;
        gt[ADA ? ii : 0][j] = ld4(g.mod_gate + ro);
        const f32x4 sv = ld4(sb + ro);
        sc[ADA ? ii : 0][j] = has_next ? sv + 1.0f : zero;
      } else if (ii == 0) {
        gt[0][j] = f32x4{1.f, 1.f, 1.f, 1.f};
        const f32x4 sv = ld4(sb + col);
        sc[0][j] = has_next ? sv : zero;
      }
    }
  }
}

// Residual epilogue over NI row tiles starting at i0, loads then stores.  All
// loads of the block are issued before its first store (the h stores may alias
// h0 loads of other rows, so the compiler would not hoist them).
template <int NI, bool ADA, int TA, int TB>
__device__ __forceinline__ void big_resid_rows(const GemmArgs &g, f32x4 (&acc)[TA][TB], int i0, int mt, int nt,
                                               int lane, unsigned &bad) {
  f32x4 h0[NI][TB], gt[ADA ? NI : 1][TB], sc[ADA ? NI : 1][TB];
  big_resid_load<NI, ADA, TB>(g, i0, mt, nt, lane, h0, gt, sc);
  const bool has_next = ADA ? g.mod_scale_next != nullptr : g.gain_next != nullptr;
  big_resid_store<NI, ADA, TA, TB>(g, acc, i0, mt, nt, lane, h0, gt, sc, has_next, bad);
}

template <int EPI, int TA, int TB, int I0 = 0, int NI = TA>
__device__ __forceinline__ void big_epilogue(const GemmArgs &g, f32x4 (&acc)[TA][TB], int mt, int nt, int lane,
                                             const float *rstd, unsigned &bad) {
  const int csub = 4 * (lane >> 4);
  if constexpr (EPI == EPI_RESID_F32) {
    if (g.mod_gate) {
#pragma unroll
      for (int i = I0; i < I0 + NI; ++i) big_resid_rows<1, true>(g, acc, i, mt, nt, lane, bad);
    } else {
      // the whole tile in two halves: all of its h0 at once would cost the
      // main loop its second wave per SIMD (a half tile goes in one piece)
      constexpr int HB = NI == TA ? TA / 2 : NI;
#pragma unroll
      for (int i = I0; i < I0 + NI; i += HB) big_resid_rows<HB, false>(g, acc, i, mt, nt, lane, bad);
    }
  } else if constexpr (EPI == EPI_QKV) {
    const int kvd = g.n_kv_heads * g.head_dim;
#pragma unroll
    for (int i = I0; i < I0 + NI; ++i) {
      const int row = (mt + i) * 16 + (lane & 15);
      if (row >= g.M) continue;
      const float rs = rstd ? rstd[i * 16 + (lane & 15)] : 1.0f;
      const int b = row / g.chunk, s = g.prefix + (row - b * g.chunk);
      const int bp = g.env_map ? g.env_map[b] : b;  // the environment's K/V store slot
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        const int col = (nt + j) * 16 + csub;
        const f32x4 v = acc[i][j] * rs;
        if ((nt + j) * 16 < g.q_dim) {
          *(bf16x4 *)((__bf16 *)g.out + (size_t)row * g.ldo + col) =
              bf16x4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
        } else {
          const int c2 = col - g.q_dim;
          const bool is_v = c2 >= kvd;
          const int c3 = is_v ? c2 - kvd : c2;
          const int kvh = c3 / g.head_dim, c = c3 - kvh * g.head_dim;
          const size_t eh = (size_t)bp * g.n_kv_heads + kvh;
          if (!is_v) {
            *(bf16x4 *)(g.kc + (eh * g.s_alloc + s) * g.head_dim + c) =
                bf16x4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) g.vtc[vt_index(eh, s, c + r, g.head_dim, g.s_alloc)] = (__bf16)v[r];
          }
        }
      }
    }
  } else if constexpr (EPI == EPI_GEGLU) {
    const int KBo = g.ldo / kTileK;
#pragma unroll
    for (int i = I0; i < I0 + NI; ++i) {
      const int row = (mt + i) * 16 + (lane & 15);
      if (row >= g.M) continue;
      const float rs = rstd ? rstd[i * 16 + (lane & 15)] : 1.0f;
#pragma unroll
      for (int j = 0; j < TB; j += 2) {  // gate tile j, its up tile j + 1
        const int col = ((nt + j) >> 1) * 16 + csub;
        const f32x4 a = acc[i][j] * rs, u = acc[i][j + 1] * rs;
        st4h((op_t *)g.out + afrag_index(row, col, KBo),
             f32x4{gelu_tanh(a[0]) * u[0], gelu_tanh(a[1]) * u[1], gelu_tanh(a[2]) * u[2], gelu_tanh(a[3]) * u[3]},
             bad);
      }
    }
  } else if constexpr (EPI == EPI_BIAS_SILU) {
    const int KBo = g.ldo / kTileK;
    f32x4 bias[TB];
#pragma unroll
    for (int j = 0; j < TB; ++j) bias[j] = ld4(g.bias + (nt + j) * 16 + csub);
#pragma unroll
    for (int i = I0; i < I0 + NI; ++i) {
      const int row = (mt + i) * 16 + (lane & 15);
      if (row >= g.M) continue;
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        const f32x4 z = acc[i][j] + bias[j];
        st4h((op_t *)g.out + afrag_index(row, (nt + j) * 16 + csub, KBo),
             f32x4{silu(z[0]), silu(z[1]), silu(z[2]), silu(z[3])}, bad);
      }
    }
  } else if constexpr (EPI == EPI_MOD) {
    // column c: layer c / 6d, part (c % 6d) / d (a, b, g of the attention
    // norm, then of the MLP norm), index c % d; a 16-column tile lies in one
    // part; the final norm's (a, b) follow the layers
    const int per_layer = 6 * g.d_model, KBd = g.d_model / kTileK;
    f32x4 bias[TB];
#pragma unroll
    for (int j = 0; j < TB; ++j) bias[j] = ld4(g.bias + (nt + j) * 16 + csub);
#pragma unroll
    for (int i = I0; i < I0 + NI; ++i) {
      const int row = (mt + i) * 16 + (lane & 15);
      if (row >= g.M) continue;
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        const int col = (nt + j) * 16 + csub;
        const f32x4 mv = acc[i][j] + bias[j];
        st4((float *)g.out + (size_t)row * g.ldo + col, mv);
        const int l = col / per_layer;
        if (l < g.n_layers) {
          const int r6 = col - l * per_layer;
          const int part = r6 / g.d_model, jc = r6 - part * g.d_model;
          if (part == 1 || part == 4)
            st4h(g.mod_shift_ops + (size_t)(2 * l + (part == 4)) * g.shift_stride + afrag_index(row, jc, KBd), mv,
                 bad);
          else if (part == 0 && l == 0 && g.next)
            st4h(g.next + afrag_index(row, jc, KBd), ld4(g.h_in + (size_t)row * g.d_model + jc) * (mv + 1.0f),
                 bad);
        }
      }
    }
  }
}

// DUAL (adaptive norm, QKV / gate-up): a second accumulator takes A2 W (the
// norm's shift through the weights) and is added after the rows' rstd has
// scaled the first: rstd * (A W) + A2 W.
// KS = 2 (when the output tiles fill at most one round of CUs, so that a
// 4-wave workgroup would leave each SIMD a single wave): 8 waves, waves
// 4..7 take the odd k-blocks of the same tile; the two partial tiles are
// summed through LDS and each k-half then runs the epilogue of half the
// wave's row tiles.
template <int EPI, int CT, bool DUAL = false, int KS = 1>
__global__ __launch_bounds__(256 * KS) void gemm_big_kernel(GemmArgs g) {
  constexpr int TA = kBigRowTiles / 2, TB = CT / 2, PD = kBigPD;
  constexpr bool kRstd = (EPI == EPI_QKV || EPI == EPI_GEGLU);
  static_assert(!DUAL || kRstd, "the second operand belongs to a normalised projection");
  static_assert(KS == 1 || (KS == 2 && !DUAL && TA % 2 == 0), "k-halves: single operand, even row tiles");
  typedef __attribute__((address_space(3))) void lds_void;
  // [ssq_tiles][128] sums of squares of the workgroup's rows when kRstd;
  // KS = 2: then the k-halves' exchange, [4 waves][2 halves][TA/2][TB][64] f32x4
  extern __shared__ __align__(16) float ssq_s[];
  __shared__ float rstd_s[128];
  int mt0, nt0;
  if (!big_tile<CT>(g, mt0, nt0)) return;  // whole workgroup: padding of the grid
  // wave index through readfirstlane: scalar per-wave addressing, up to 14 fewer VGPRs
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wq = wave & 3, kh = wave >> 2;  // position in the 2 x 2 wave grid, k-half
  const int wr = wq & 1, wc = wq >> 1;
  const int KB = g.K / kTileK;
  const int nkb = KB / KS;  // this wave's k-blocks kh, kh + KS, ... (the host checks KB % KS == 0)
  const int mt_last = g.m_alloc / 16 - 1;  // allocated row tiles (rows >= M are computed, never stored)
  if (kRstd && g.use_rstd) {
    // this workgroup's 128 rows' per-tile sums of squares, straight to LDS
    for (int j = wave; j < 2 * g.ssq_tiles; j += 4 * KS) {
      const int tile = j >> 1, half = j & 1;
      const int row = min(mt0 * 16 + half * 64 + lane, g.M - 1);
      __builtin_amdgcn_global_load_lds((const void *)(g.ssq + (size_t)tile * g.m_alloc + row),
                                       (lds_void *)(ssq_s + tile * 128 + half * 64), 4, 0, 0);
    }
  }
  const op_t *pa[TA], *pb[TB];
#pragma unroll
  for (int i = 0; i < TA; ++i)
    pa[i] = g.A + ((size_t)min(mt0 + wr * TA + i, mt_last) * KB + kh) * kBlockElems + lane * 8;
#pragma unroll
  for (int j = 0; j < TB; ++j) pb[j] = g.W + ((size_t)(nt0 + wc * TB + j) * KB + kh) * kBlockElems + lane * 8;
  constexpr size_t kStep = (size_t)KS * kBlockElems;  // between this wave's consecutive k-blocks
  constexpr int TA2 = DUAL ? TA : 1;
  const op_t *pa2[TA2];
#pragma unroll
  for (int i = 0; i < TA2; ++i)
    pa2[i] = DUAL ? g.A2 + (size_t)min(mt0 + wr * TA + i, mt_last) * KB * kBlockElems + lane * 8 : nullptr;
  f16x8 ra[PD][TA], rb[PD][TB], ra2[PD][TA2];
#pragma unroll
  for (int s = 0; s < PD; ++s) {
    const int kb = min(s, nkb - 1);
#pragma unroll
    for (int i = 0; i < TA; ++i) ra[s][i] = *(const f16x8 *)(pa[i] + kb * kStep);
#pragma unroll
    for (int j = 0; j < TB; ++j) rb[s][j] = *(const f16x8 *)(pb[j] + kb * kStep);
    if constexpr (DUAL)
#pragma unroll
      for (int i = 0; i < TA; ++i) ra2[s][i] = *(const f16x8 *)(pa2[i] + (size_t)kb * kBlockElems);
  }
  f32x4 acc[TA][TB], acc2[TA2][DUAL ? TB : 1];
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (DUAL)
#pragma unroll
    for (int i = 0; i < TA; ++i)
#pragma unroll
      for (int j = 0; j < TB; ++j) acc2[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < nkb; k0 += PD) {
#pragma unroll
    for (int s = 0; s < PD; ++s) {
      if (k0 + s < nkb) {
#pragma unroll
        for (int i = 0; i < TA; ++i)
#pragma unroll
          for (int j = 0; j < TB; ++j) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(rb[s][j], ra[s][i], acc[i][j], 0, 0, 0);
            if constexpr (DUAL)
              acc2[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(rb[s][j], ra2[s][i], acc2[i][j], 0, 0, 0);
          }
      }
      const int kb = min(k0 + s + PD, nkb - 1);  // past the end: re-load the last block (never used)
#pragma unroll
      for (int i = 0; i < TA; ++i) ra[s][i] = *(const f16x8 *)(pa[i] + kb * kStep);
#pragma unroll
      for (int j = 0; j < TB; ++j) rb[s][j] = *(const f16x8 *)(pb[j] + kb * kStep);
      if constexpr (DUAL)
#pragma unroll
        for (int i = 0; i < TA; ++i) ra2[s][i] = *(const f16x8 *)(pa2[i] + (size_t)kb * kBlockElems);
    }
  }

  if (kRstd && g.use_rstd) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's statistics landed
    __syncthreads();                                  // ... every wave's
    if (threadIdx.x < 128) {
      float ss = 0.f;
      for (int t = 0; t < g.ssq_tiles; ++t) ss += ssq_s[t * 128 + threadIdx.x];
      rstd_s[threadIdx.x] = 1.0f / sqrtf(ss / (float)(g.ssq_tiles * kTileN) + g.eps);
    }
    __syncthreads();
  }

  unsigned bad = 0;  // fp16 range flag of this thread's stores
  if constexpr (DUAL) {
    // lane l of tile (i, j) holds row l & 15 (swapped operands)
#pragma unroll
    for (int i = 0; i < TA; ++i) {
      const float rs = rstd_s[wr * TA * 16 + i * 16 + (lane & 15)];
#pragma unroll
      for (int j = 0; j < TB; ++j) acc[i][j] = rs * acc[i][j] + acc2[i][j];
    }
    big_epilogue<EPI, TA, TB>(g, acc, mt0 + wr * TA, nt0 + wc * TB, lane, nullptr, bad);
  } else if constexpr (KS == 2) {
    // Wave (wq, 0) keeps row tiles [0, H) and hands [H, TA) to wave (wq, 1),
    // which keeps [H, TA); each adds the other's partial of what it keeps.
    constexpr int H = TA / 2;
    f32x4 *xch = (f32x4 *)(ssq_s + (kRstd && g.use_rstd ? g.ssq_tiles * 128 : 0));
    f32x4 *mine = xch + (size_t)(wq * 2 + kh) * (H * TB * 64) + lane;
    const f32x4 *other = xch + (size_t)(wq * 2 + (kh ^ 1)) * (H * TB * 64) + lane;
    if (kh == 0) {
#pragma unroll
      for (int i = 0; i < H; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) mine[(i * TB + j) * 64] = acc[H + i][j];
    } else {
#pragma unroll
      for (int i = 0; i < H; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) mine[(i * TB + j) * 64] = acc[i][j];
    }
    __syncthreads();
    const float *rs = (kRstd && g.use_rstd) ? rstd_s + wr * TA * 16 : nullptr;
    if (kh == 0) {
#pragma unroll
      for (int i = 0; i < H; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) acc[i][j] = acc[i][j] + other[(i * TB + j) * 64];
      big_epilogue<EPI, TA, TB, 0, H>(g, acc, mt0 + wr * TA, nt0 + wc * TB, lane, rs, bad);
    } else {
#pragma unroll
      for (int i = 0; i < H; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) acc[H + i][j] = other[(i * TB + j) * 64] + acc[H + i][j];
      big_epilogue<EPI, TA, TB, H, H>(g, acc, mt0 + wr * TA, nt0 + wc * TB, lane, rs, bad);
    }
  } else {
    big_epilogue<EPI, TA, TB>(g, acc, mt0 + wr * TA, nt0 + wc * TB, lane,
                              (kRstd && g.use_rstd) ? rstd_s + wr * TA * 16 : nullptr, bad);
  }
  flush_range(g.status, bad);
}

// LDS-ring kernels for the widest batched projections: RT x CT 16-row /
// 16-column tiles per workgroup, 8 waves (WR x WC), operands staged through
// an NS-stage LDS ring by LDS-direct loads (RT + CT fragment blocks per
// 32-deep stage).  Each stage's wait is a raw s_barrier after a partial
// vmcnt: __syncthreads' release fence would drain the next stages' loads
// too.  The rows' norm statistics are loaded into registers after the ring
// prologue (that wait is the prologue's own round trip) and folded into
// rstd after the main loop.  Measured without epilogue (TFLOP/s):
//   gate/up 256 x 128, 4 x 2 waves, 3 stages: 3200 x 8192 x 1024: 800 (vs
//   711 register-streamed), 2048 x 12288 x 1536: 960 (vs 921); with the
//   GeGLU epilogue, 128 x 256 tiles (2 x 4 waves, same LDS per stage) beat
//   256 x 128 in a same-machine A/B: 73.3 -> 66.0 us and 89.3 -> 79.1 us (3200
//   rows are 25 full 128-row panels instead of 12.5 of 256; 800 tiles
//   instead of 832);
//   QKV 128 x 128, 2 x 4 waves, 4 stages: 3200 x 2560 x 1024: 761 (vs 643;
//   at 2048 x 2048 x 1536 the register-streamed kernel stays ahead, 651 vs 621).
// Residual projections on the QKV shape (with epilogue, same-machine A/B against
// the 8-wave k-halves of the register-streamed kernel): 3200 x 1024 x 2048
// 31.1 -> 29.0 us, x 4096 52.6 -> 48.9 us (2 x 4 waves; 4 x 2: 29.9 / 50.7);
// the 1536-wide expert's (2048 rows, 96-column tiles there) lose 5% on
// 128 x 128 ring tiles (192 tiles for 256 CUs) but win on 128 x 96 ones
// (256 tiles, 4 x 2 waves of 32 x 48, 14 fragment blocks per stage): down
// 64.7 -> 62.9 us, O 22.4 -> 21.6 us.
// The wave index goes through readfirstlane so that the compiler keeps the
// per-wave addressing and branches in scalar registers: gate/up on the
// 1536-wide expert 82.1 -> 79.6 us.
constexpr int kRingNW = 8;
template <int EPI>
struct RingShape;
template <>
struct RingShape<EPI_GEGLU> {
  static constexpr int RT = 8, CT = 16, WR = 2, WC = 4, NS = 3, MinM = 1024;
};
template <>
struct RingShape<EPI_QKV> {
  static constexpr int RT = 8, CT = 8, WR = 2, WC = 4, NS = 4, MinM = 2560;
};
template <>
struct RingShape<EPI_RESID_F32> {
  static constexpr int RT = 8, CT = 8, WR = 2, WC = 4, NS = 4, MinM = 2560;
};

// 144 x 256 gate/up tiles, 1 x 8 waves of 144 x 32 (one gate/up pair each):
// fewer tiles where 128-row ones would leave some CUs a fourth tile
struct RingGeGlu144 {
  static constexpr int RT = 9, CT = 16, WR = 1, WC = 8, NS = 3, MinM = 1024;
};
// 160 x 256 gate/up tiles, 2 x 4 waves of 80 x 64 (two stages only: two
// workgroups' three stages and row statistics exceed the 160 KiB of LDS)
struct RingGeGlu160 {
  static constexpr int RT = 10, CT = 16, WR = 2, WC = 4, NS = 3, MinM = 1024;
};

// 128 x 96 tiles: the residual projections where 96-column tiles are preferred
struct RingResid96 {
  static constexpr int RT = 8, CT = 6, WR = 4, WC = 2, NS = 4, MinM = 1024;
};

// Wait until this wave's loads of all but the newest `later` stages (L
// LDS-direct loads each) have landed, then meet the workgroup.
template <int L>
__device__ __forceinline__ void ring_wait(int later) {
  if (later >= 2)
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(2 * L) : "memory");
  else if (later == 1)
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(L) : "memory");
  else
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int EPI, int NS = RingShape<EPI>::NS, class S = RingShape<EPI>, bool KSPLIT = false>
__global__ __launch_bounds__(512) void gemm_ring_kernel(GemmArgs g) {
  static_assert(!KSPLIT || EPI == EPI_RESID_F32, "split-K: residual projections");
  constexpr int RT = S::RT, CT = S::CT, WR = S::WR, WC = S::WC;
  // NBLK fragment blocks per stage over the 8 waves: the first NFULL waves
  // issue LPW LDS-direct loads per stage, the others LPW - 1
  constexpr int NBLK = RT + CT, LPW = (NBLK + kRingNW - 1) / kRingNW, NFULL = NBLK - (LPW - 1) * kRingNW;
  constexpr int TA = RT / WR, TB = CT / WC;            // 16 x 16 tiles per wave
  constexpr int ROWS = 16 * RT, TPR = 512 / ROWS;       // rows per workgroup, threads per row's statistics
  static_assert(WR * WC == kRingNW && RT % WR == 0 && CT % WC == 0 && NS >= 2 && NS <= 4, "ring shape");
  typedef __attribute__((address_space(3))) void lds_void;
  extern __shared__ __align__(16) unsigned char ring_smem[];
  op_t *stage = (op_t *)ring_smem;  // [NS][NBLK][512]
  __shared__ float rpart[TPR][ROWS];
  __shared__ float rstd_s[ROWS];
  // split-K: the grid is kx copies of the tile grid, copy `split` taking the
  // split-th of kx equal k-ranges
  const int kx = KSPLIT ? g.kx : 1;
  const int tn = g.N / (16 * CT), per_split = grid_tile_wgs(g.M, ROWS, tn);
  const int split = KSPLIT ? (int)blockIdx.x / per_split : 0;
  int pm, pn;
  if (!grid_tile_at((int)blockIdx.x - split * per_split, g.M, ROWS, tn, pm, pn)) return;  // whole workgroup
  const int mt0 = pm * RT, nt0 = pn * CT;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = wave % WR, wc = wave / WR;
  const int KBt = g.K / kTileK;  // k-blocks of a row
  const int kb0 = split * KBt / kx, KB = (split + 1) * KBt / kx - kb0;  // this workgroup's k-blocks
  const int mt_last = g.m_alloc / 16 - 1;

  auto issue = [&](int kb, int buf) {
    op_t *dst = stage + (size_t)buf * NBLK * kBlockElems;
#pragma unroll
    for (int q = 0; q < LPW; ++q) {
      const int bidx = wave + q * kRingNW;
      if (NFULL < kRingNW && q == LPW - 1 && wave >= NFULL) break;
      const op_t *src = bidx < RT ? g.A + ((size_t)min(mt0 + bidx, mt_last) * KBt + kb0 + kb) * kBlockElems
                                  : g.W + ((size_t)(nt0 + bidx - RT) * KBt + kb0 + kb) * kBlockElems;
      __builtin_amdgcn_global_load_lds((const void *)(src + lane * 8), (lds_void *)(dst + bidx * kBlockElems), 16, 0,
                                       0);
    }
  };
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < KB) issue(s, s);

  if (g.use_rstd && (TPR * ROWS == 512 || (int)threadIdx.x < TPR * ROWS)) {
    // per-row sums of squares: TPR threads share row (tid % ROWS), each summing a slice of its tiles
    const int row = min(mt0 * 16 + (int)(threadIdx.x % ROWS), g.M - 1), part = threadIdx.x / ROWS;
    const int t0 = part * g.ssq_tiles / TPR, t1 = (part + 1) * g.ssq_tiles / TPR;
    float ss = 0.f;
    for (int q = t0; q < t1; ++q) ss += g.ssq[(size_t)q * g.m_alloc + row];
    rpart[part][threadIdx.x % ROWS] = ss;
  }

  f32x4 acc[TA][TB];
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kb = 0; kb < KB; ++kb) {
    // stage kb landed for this wave (later stages may stay in flight), then
    // for every wave; the buffer refilled below was last read one step ago
    const int later = min(NS - 2, KB - 1 - kb);  // stages issued after kb
    if (NFULL == kRingNW || wave < NFULL)
      ring_wait<LPW>(later);
    else
      ring_wait<LPW - 1>(later);
    if (kb + NS - 1 < KB) issue(kb + NS - 1, (kb + NS - 1) % NS);
    const op_t *sb = stage + (size_t)(kb % NS) * NBLK * kBlockElems + lane * 8;
    f16x8 af[TA], bf[TB];
#pragma unroll
    for (int i = 0; i < TA; ++i) af[i] = *(const f16x8 *)(sb + (wr * TA + i) * kBlockElems);
#pragma unroll
    for (int j = 0; j < TB; ++j) bf[j] = *(const f16x8 *)(sb + (RT + wc * TB + j) * kBlockElems);
#pragma unroll
    for (int i = 0; i < TA; ++i)
#pragma unroll
      for (int j = 0; j < TB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(bf[j], af[i], acc[i][j], 0, 0, 0);
  }

  if constexpr (KSPLIT) {
    // Partial tiles, fp32, [tile][split][wave][i][j][component][lane]: the
    // last workgroup of a tile to arrive adds them in split order, whatever
    // the arrival order, and runs the epilogue; the others are done, and no
    // workgroup waits on another.  The partials are written and read with
    // device-coherent (agent-scope) stores and loads, which bypass the
    // per-XCD L2, so no cache-wide write-back or invalidation is needed: the
    // stores are complete (vmcnt) before the workgroup's arrival is counted.
    __shared__ unsigned kx_last;
    constexpr int PW = TA * TB * 4 * 64;  // floats per wave
    const int tile = pm * tn + pn;
    float *ws = g.kx_ws + (size_t)tile * kx * kRingNW * PW + (size_t)wave * PW + lane;
#pragma unroll
    for (int i = 0; i < TA; ++i)
#pragma unroll
      for (int j = 0; j < TB; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c)
          __hip_atomic_store(ws + (size_t)split * kRingNW * PW + ((i * TB + j) * 4 + c) * 64, acc[i][j][c],
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0)
      kx_last = __hip_atomic_fetch_add(g.kx_cnt + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                (unsigned)(kx - 1);
    __syncthreads();
    if (!kx_last) return;
    f32x4 own[TA][TB];
#pragma unroll
    for (int i = 0; i < TA; ++i)
#pragma unroll
      for (int j = 0; j < TB; ++j) own[i][j] = acc[i][j];
    for (int sp = 0; sp < kx; ++sp) {
      const float *src = ws + (size_t)sp * kRingNW * PW;
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j) {
          f32x4 v = own[i][j];
          if (sp != split)
#pragma unroll
            for (int c = 0; c < 4; ++c)
              v[c] = __hip_atomic_load(src + ((i * TB + j) * 4 + c) * 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          acc[i][j] = sp == 0 ? v : acc[i][j] + v;
        }
    }
    if (threadIdx.x == 0) __hip_atomic_store(g.kx_cnt + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  if (g.use_rstd) {
    __syncthreads();  // rpart complete (also past every wave's last LDS read of the ring)
    if (threadIdx.x < ROWS) {
      float ss = 0.f;
#pragma unroll
      for (int p = 0; p < TPR; ++p) ss += rpart[p][threadIdx.x];
      rstd_s[threadIdx.x] = 1.0f / sqrtf(ss / (float)(g.ssq_tiles * kTileN) + g.eps);
    }
    __syncthreads();
  }
  unsigned bad = 0;  // fp16 range flag of this thread's stores
  big_epilogue<EPI, TA, TB>(g, acc, mt0 + wr * TA, nt0 + wc * TB, lane, g.use_rstd ? rstd_s + wr * TA * 16 : nullptr,
                            bad);
  flush_range(g.status, bad);
}


// Residual projections: 96-column tiles of the register-streamed kernel when
// they need fewer 16 x 16 output tiles per CU than 128-column ones (1536
// wide, 2048 rows: 256 tiles of 48 instead of 192 tiles of 64 with 64 CUs
// idle).
static bool resid_prefers_96(const GemmArgs &g) {
  auto per_cu = [&](int ct) {
    const int tiles = (g.M + 16 * kBigRowTiles - 1) / (16 * kBigRowTiles) * (g.N / (16 * ct));
    return (tiles + g_n_cu - 1) / g_n_cu * ct;
  };
  return g.N % 96 == 0 && per_cu(6) < per_cu(8);
}

template <int EPI, int CT>
static bool big_khalves(const GemmArgs &g);

// Below MinM rows the ring still wins for QKV where the register-streamed
// kernel would not take its k-halves (K < 1536) once its tiles reach 3/8 of
// the CUs, and for the residual projections once they fill half the CUs.
// Same-machine A/B on the 1024-wide expert (ms per joint step): 15 environments
// 2.079 -> 2.054, 20 2.451 -> 2.364, 24 2.803 -> 2.733, 32 3.326 -> 3.262,
// 40 3.548 -> 3.321, 48 3.964 -> 3.780; QKV at 750 / 1000 / 2000 rows
// 21.4 / 25.0 / 33.4 -> 19.5 /
// 20.2 / 26.4 us, down at 2000 rows 50.6 -> 46.6 us. The ring lost for QKV
// at 60-80 tiles (300-500 rows), for the residual projections at 80-104
// tiles (the k-halves win there), for gate/up below 1024 rows, and on the
// 1536-wide expert.
template <int EPI>
static bool ring_rows_ok(const GemmArgs &g) {
  using S = RingShape<EPI>;
  if (g.M >= S::MinM) return true;
  const int tiles = (g.M + 16 * S::RT - 1) / (16 * S::RT) * (g.N / (16 * S::CT));
  if constexpr (EPI == EPI_QKV) return 8 * tiles >= 3 * g_n_cu && !big_khalves<EPI_QKV, 8>(g);
  if constexpr (EPI == EPI_RESID_F32) return 2 * tiles >= g_n_cu;
  return false;
}

template <int EPI>
static bool ring_fits(const GemmArgs &g) {
  using S = RingShape<EPI>;
  return ring_rows_ok<EPI>(g) && g.N % (16 * S::CT) == 0 && g.A2 == nullptr && g.K / kTileK >= 1 &&
         !(EPI == EPI_QKV && g.q_dim % 16 != 0) && !(EPI == EPI_RESID_F32 && resid_prefers_96(g));
}

// The residual projections where 96-column tiles are preferred, on the
// 128 x 96 ring from 1024 rows once its tiles fill 3/4 of the CUs, or with
// a long K.  1536-wide expert, same-machine (us): at 2048 and 1536 rows O 22.4 /
// 21.8 -> 21.8 / 21.1, down 65.2 / 64.8 -> 63.7 / 62.4; at 1024 rows (128
// tiles) down (K = 6144) 60.1 -> 58.1 but O (K = 1536) 18.0 -> 19.6, where
// the register-streamed kernel's k-halves keep the short K ahead.
static bool ring96_fits(const GemmArgs &g) {
  const int tiles = (g.M + 16 * RingResid96::RT - 1) / (16 * RingResid96::RT) * (g.N / (16 * RingResid96::CT));
  return g.M >= RingResid96::MinM && (4 * tiles >= 3 * g_n_cu || g.K >= 4096) && resid_prefers_96(g) &&
         g.A2 == nullptr && g.K / kTileK >= 1;
}

// Split-K of the batched residual projections on the ring: kx = CUs / tiles
// (at most 4) copies of the tile grid, each over an equal k-range of at least
// 16 k-blocks, when the tiles fill at most half the CUs and are at least the
// 90 the batched kernels need (64 with K >= 4096); 1 (no split) otherwise, or
// when the context gave no workspace or it is too small.  Same-machine A/B, ms
// per joint step: 1024-wide expert at 32 environments (1600 rows, 104 tiles)
// 3.130 -> 2.663 (down 49.8 -> 29.1 us, O 25.3 -> 20.4 us), 1536-wide expert
// at 8 environments (1024 rows, 128 tiles of 96 columns) 4.450 -> 3.893
// (down 58.0 -> 36.3 us); below 90 tiles the small-M kernel kept O and the
// time MLP ahead (1000 rows: O 16.8 -> 18.0 us split four ways) while down
// still won (28.1 -> 23.4 us), and at 400-600 rows both lost.  Tiles filling
// more than half the CUs (one workgroup per CU) split two ways when K >= 4096,
// two co-resident workgroups per CU instead of one: down of the 1536-wide
// expert at 16 environments (256 tiles of 128 x 96) 65.5 -> 54.3 us, step
// 5.595 -> 5.333 ms; of the 1024-wide at 64 environments (200 tiles) 45.3 ->
// 43.4 us; with O and the time MLP (K = 1536-2048) split as well the step
// lost (O 22.1 -> 24.3 us, 26.9 -> 30.3 us).
template <class S>
static int resid_ksplit(const GemmArgs &g) {
  if (!g.kx_ws || !g.kx_cnt || g.A2 || g.M < kBigM || g.N % (16 * S::CT) != 0) return 1;
  const int tiles = (g.M + 16 * S::RT - 1) / (16 * S::RT) * (g.N / (16 * S::CT));
  if (tiles < 90 && !(g.K >= 4096 && tiles >= 64)) return 1;
  int kx = std::min(4, g_n_cu / std::max(tiles, 1));
  if (kx == 1 && tiles <= g_n_cu && g.K >= 4096) kx = 2;
  while (kx > 1 && (g.K / kTileK) / kx < 16) --kx;
  constexpr size_t part = (size_t)kRingNW * (S::RT / S::WR) * (S::CT / S::WC) * 4 * 64 * sizeof(float);
  if (kx > 1 && ((size_t)tiles * kx * part > g.kx_ws_bytes || tiles > g.kx_tiles)) return 1;
  return kx;
}

template <int EPI, int NS, class S = RingShape<EPI>, bool KSPLIT = false>
static hipError_t launch_ring_ns(const GemmArgs &g, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const int wgs = grid_tile_wgs(g.M, 16 * S::RT, g.N / (16 * S::CT)) * (KSPLIT ? g.kx : 1);
  const uint32_t lds = (uint32_t)(NS * (S::RT + S::CT) * kBlockElems * sizeof(op_t));
  UAD_LAUNCH((gemm_ring_kernel<EPI, NS, S, KSPLIT>), dim3(wgs), dim3(512), lds, s, ev0, ev1, g);
  return hipGetLastError();
}

// Gate/up with K <= 1024 on a 2-stage ring (48 KiB of LDS, three workgroups
// per CU): same-machine A/B at 3200 x 8192 x 1024 68.6 -> 65.9 us; at K = 1536
// (2048 x 12288) the 2-stage ring lost 84.2 -> 92.6 us, so 3 stages there.
// Gate/up on the shortest of 128-, 144- and 160-row tiles that fits one round
// of co-resident ring workgroups (two per CU), 128 when none does: the tiles
// past the round ran as a second, mostly single-workgroup wave.  Same-machine,
// 144 rows: 2050 rows (544 -> 480 tiles) 57.1 -> 42.5 us, step 3.484 -> 3.210
// ms; 2300 rows 56.5 -> 42.9 us; 1536-wide at 1408 rows (528 -> 480 tiles,
// K = 1536) 75.8 -> 59.7 us, step 5.089 -> 4.666 ms.  160 rows: 2400 rows
// 56.6 -> 44.6 us, step 3.416 -> 3.203 ms; 2500 rows 56.1 -> 45.4 us;
// 1536-wide at 1536 rows 75.4 -> 61.8 us, step 5.017 -> 4.676 ms.  Where
// every shape exceeds the round the taller tiles lost (3200 rows, 800 -> 736
// tiles of 144: 67.0 -> 69.6 us).
static int geglu_tile_rows(const GemmArgs &g) {
  const int tn = g.N / 256;
  for (int rows : {128, 144, 160})
    if ((g.M + rows - 1) / rows * tn <= 2 * g_n_cu) return rows;
  return 128;
}

template <int EPI>
static hipError_t launch_ring(const GemmArgs &g, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if constexpr (EPI == EPI_GEGLU) {
    const int rows = geglu_tile_rows(g);
    if (rows == 160) return launch_ring_ns<EPI, 2, RingGeGlu160>(g, s, ev0, ev1);
    if (rows == 144) {
      if (g.K <= 1024) return launch_ring_ns<EPI, 2, RingGeGlu144>(g, s, ev0, ev1);
      return launch_ring_ns<EPI, RingGeGlu144::NS, RingGeGlu144>(g, s, ev0, ev1);
    }
    if (g.K <= 1024) return launch_ring_ns<EPI, 2>(g, s, ev0, ev1);
  }
  return launch_ring_ns<EPI, RingShape<EPI>::NS>(g, s, ev0, ev1);
}

template <int EPI, int NS, class S = RingShape<EPI>, bool KSPLIT = false>
static hipError_t ring_attr_ns() {
  return hipFuncSetAttribute((const void *)gemm_ring_kernel<EPI, NS, S, KSPLIT>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             NS * (S::RT + S::CT) * kBlockElems * (int)sizeof(op_t));
}

template <int EPI>
static hipError_t ring_attr() {
  hipError_t e = ring_attr_ns<EPI, RingShape<EPI>::NS>();
  if constexpr (EPI == EPI_GEGLU) {
    if (e == hipSuccess) e = ring_attr_ns<EPI, 2>();
    if (e == hipSuccess) e = ring_attr_ns<EPI, 2, RingGeGlu144>();
    if (e == hipSuccess) e = ring_attr_ns<EPI, RingGeGlu144::NS, RingGeGlu144>();
    if (e == hipSuccess) e = ring_attr_ns<EPI, 2, RingGeGlu160>();
  }
  return e;
}

// 16*CT columns per workgroup: 256 for gate/up (the widest projection), 128 otherwise
template <int EPI>
constexpr int big_ct() { return EPI == EPI_GEGLU ? 16 : 8; }

// LDS of the k-halves' exchange (gemm_big_kernel with KS = 2)
template <int CT>
constexpr size_t big_xch_bytes() { return (size_t)4 * 2 * (kBigRowTiles / 4) * (CT / 2) * 64 * sizeof(f32x4); }

// Whether a launch takes the k-halves (KS = 2): its tiles fill at most one
// round of CUs (one 4-wave workgroup per CU would leave every SIMD a single
// wave), K >= 1536 and the k-blocks split evenly.  Residual, QKV and
// time-MLP-in epilogues only (128- or 96-column tiles, <= 256 registers at 8
// waves).  Measured: the 1536-wide expert's QKV (2048 x 2048 x 1536, 256
// tiles) 32.5 -> 25.5 us, its down 67.7 -> 65.2 us; the 1024-wide fleet's O
// and down -2%; at K = 1024 (fleet time-MLP out) 18.8 -> 19.6 us, hence the
// K bound.
template <int EPI, int CT>
static bool big_khalves(const GemmArgs &g) {
  if constexpr (CT > 8 || !(EPI == EPI_RESID_F32 || EPI == EPI_QKV || EPI == EPI_BIAS_SILU)) {
    return false;
  } else {
    const int tiles = (g.M + 16 * kBigRowTiles - 1) / (16 * kBigRowTiles) * (g.N / (16 * CT));
    return tiles <= g_n_cu && g.K >= 1536 && (g.K / kTileK) % 2 == 0;
  }
}

template <int EPI, int CT>
static hipError_t launch_big_ct(const GemmArgs &g, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const bool rstd = (EPI == EPI_QKV || EPI == EPI_GEGLU) && g.use_rstd;
  const size_t lds = rstd ? (size_t)g.ssq_tiles * 128 * 4 : 0;
  const int wgs = grid_tile_wgs(g.M, 16 * kBigRowTiles, g.N / (16 * CT));
  if constexpr (CT <= 8 && (EPI == EPI_RESID_F32 || EPI == EPI_QKV || EPI == EPI_BIAS_SILU)) {
    if (big_khalves<EPI, CT>(g)) {
      UAD_LAUNCH((gemm_big_kernel<EPI, CT, false, 2>), dim3(wgs), dim3(512), (uint32_t)(lds + big_xch_bytes<CT>()), s,
                 ev0, ev1, g);
      return hipGetLastError();
    }
  }
  UAD_LAUNCH((gemm_big_kernel<EPI, CT>), dim3(wgs), dim3(256), (uint32_t)lds, s, ev0, ev1, g);
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_big(const GemmArgs &g, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if constexpr (EPI == EPI_QKV || EPI == EPI_GEGLU) {
    if (g.A2) {  // the second accumulator: 128-column tiles keep the registers in bounds
      if (!g.use_rstd) return hipErrorInvalidValue;
      const size_t lds = (size_t)g.ssq_tiles * 128 * 4;
      const int wgs = grid_tile_wgs(g.M, 16 * kBigRowTiles, g.N / (16 * 8));
      UAD_LAUNCH((gemm_big_kernel<EPI, 8, true>), dim3(wgs), dim3(256), (uint32_t)lds, s, ev0, ev1, g);
      return hipGetLastError();
    }
  }
  if constexpr (EPI == EPI_RESID_F32)
    if (resid_prefers_96(g)) return launch_big_ct<EPI, 6>(g, s, ev0, ev1);
  return launch_big_ct<EPI, big_ct<EPI>()>(g, s, ev0, ev1);
}

// The batched kernel serves M >= kBigM when the columns divide into its tiles,
// no second operand is used and there are enough output tiles to fill the
// chip: each tile runs its whole K serially in one workgroup, so with few
// tiles (and long K) the small-M kernel, which splits K over waves, is
// faster.  Threshold from a sweep of both kernels over 200..3200 rows and
// the projection shapes of the 1024- and 1536-wide experts (the rule picks
// the faster kernel in 49 of 50 cases, the miss by 6%).
static bool big_ok(int epi, const GemmArgs &g) {
  const int ct = (epi == EPI_GEGLU && !g.A2) ? 16 : 8;
  if (g.M < kBigM || g.N % (16 * ct) != 0 || g.ssq_tiles > kMaxSsqTiles || (epi == EPI_QKV && g.q_dim % 16 != 0) ||
      (g.A2 && epi != EPI_QKV && epi != EPI_GEGLU))
    return false;
  const int tiles = (g.M + 16 * kBigRowTiles - 1) / (16 * kBigRowTiles) * (g.N / (16 * ct));
  return tiles >= 90 && !(tiles < 128 && g.K > 4096);
}

template <int EPI>
static hipError_t big_attr() {
  hipError_t e = hipFuncSetAttribute((const void *)gemm_big_kernel<EPI, big_ct<EPI>()>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, kMaxSsqTiles * 128 * 4);
  if constexpr (EPI == EPI_RESID_F32 || EPI == EPI_QKV || EPI == EPI_BIAS_SILU) {
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void *)gemm_big_kernel<EPI, 8, false, 2>,
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)(kMaxSsqTiles * 128 * 4 + big_xch_bytes<8>()));
    if constexpr (EPI == EPI_RESID_F32)
      if (e == hipSuccess)
        e = hipFuncSetAttribute((const void *)gemm_big_kernel<EPI, 6, false, 2>,
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)(kMaxSsqTiles * 128 * 4 + big_xch_bytes<6>()));
  }
  if constexpr (EPI == EPI_QKV || EPI == EPI_GEGLU)
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void *)gemm_big_kernel<EPI, 8, true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              kMaxSsqTiles * 128 * 4);
  return e;
}

hipError_t gemm_init() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&g_n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess && g_n_cu < 1) e = hipErrorInvalidDevice;
  if (e == hipSuccess) e = ring_attr<EPI_GEGLU>();
  if (e == hipSuccess) e = ring_attr<EPI_QKV>();
  if (e == hipSuccess) e = ring_attr<EPI_RESID_F32>();
  if (e == hipSuccess) e = ring_attr_ns<EPI_RESID_F32, RingResid96::NS, RingResid96>();
  if (e == hipSuccess) e = ring_attr_ns<EPI_RESID_F32, RingShape<EPI_RESID_F32>::NS, RingShape<EPI_RESID_F32>, true>();
  if (e == hipSuccess) e = ring_attr_ns<EPI_RESID_F32, RingResid96::NS, RingResid96, true>();
  if (e == hipSuccess) e = big_attr<EPI_BIAS_SILU>();
  if (e == hipSuccess) e = big_attr<EPI_RESID_F32>();
  if (e == hipSuccess) e = big_attr<EPI_GEGLU>();
  if (e == hipSuccess) e = big_attr<EPI_QKV>();
  if (e == hipSuccess) e = big_attr<EPI_MOD>();
  return e;
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
  if (g.m_alloc < g.M || g.m_alloc % 16 != 0) return hipErrorInvalidValue;  // operand rows allocated
  if (epi == EPI_GEGLU && ring_fits<EPI_GEGLU>(g)) return launch_ring<EPI_GEGLU>(g, s, ev0, ev1);
  if (epi == EPI_QKV && ring_fits<EPI_QKV>(g)) return launch_ring<EPI_QKV>(g, s, ev0, ev1);
  if (epi == EPI_RESID_F32) {
    GemmArgs gk = g;
    if (resid_prefers_96(g)) {
      gk.kx = resid_ksplit<RingResid96>(g);
      if (gk.kx > 1) return launch_ring_ns<EPI_RESID_F32, RingResid96::NS, RingResid96, true>(gk, s, ev0, ev1);
    } else {
      using S8 = RingShape<EPI_RESID_F32>;
      gk.kx = resid_ksplit<S8>(g);
      if (gk.kx > 1) return launch_ring_ns<EPI_RESID_F32, S8::NS, S8, true>(gk, s, ev0, ev1);
    }
  }
  if (epi == EPI_RESID_F32 && ring96_fits(g))
    return launch_ring_ns<EPI_RESID_F32, RingResid96::NS, RingResid96>(g, s, ev0, ev1);
  if (epi == EPI_RESID_F32 && ring_fits<EPI_RESID_F32>(g)) return launch_ring<EPI_RESID_F32>(g, s, ev0, ev1);
  if (big_ok(epi, g)) {
    switch (epi) {
      case EPI_BIAS_SILU: return launch_big<EPI_BIAS_SILU>(g, s, ev0, ev1);
      case EPI_RESID_F32: return launch_big<EPI_RESID_F32>(g, s, ev0, ev1);
      case EPI_GEGLU: return launch_big<EPI_GEGLU>(g, s, ev0, ev1);
      case EPI_QKV: return launch_big<EPI_QKV>(g, s, ev0, ev1);
      case EPI_MOD: return launch_big<EPI_MOD>(g, s, ev0, ev1);
    }
    return hipErrorInvalidValue;
  }
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
