// Per-token kernels of the step: the per-token time embedding and action
// input projection, and the final norm + action projection fused with the
// masked per-token Euler update.
#include "uad_internal.h"

namespace uad {


// Sum over a 256-thread block in a fixed order (wave shuffles, then 4 partials).
__device__ __forceinline__ float block_sum_256(float v, float *scratch) {
  v = sum_wave64(v);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) scratch[wave] = v;
  __syncthreads();
  return (scratch[0] + scratch[1]) + (scratch[2] + scratch[3]);
}

// Rows per workgroup of the embedding kernels: R tokens share one read of
// their columns' W_in rows (R = 16 when batched: with one token per
// workgroup the 3,200-token fleet re-read W_in 3,200 times from L2).
// Token m of a compacted step is token env_map[m / chunk] * chunk + m % chunk
// of the caller's arrays (null map: token m).
__device__ __forceinline__ int phys_token(const int32_t *env_map, int chunk, int m) {
  if (!env_map) return m;
  const int b = m / chunk;
  return env_map[b] * chunk + (m - b * chunk);
}

template <int R>
__device__ __forceinline__ int load_action_rows(const float *__restrict__ x, int M, int Da, float (*xs)[64],
                                                const int32_t *env_map = nullptr, int chunk = 1) {
  const int m0 = blockIdx.x * R;
  const int rows = min(R, M - m0);
  for (int i = threadIdx.x; i < rows * Da; i += blockDim.x) {
    const int r = i / Da, j = i - r * Da;
    xs[r][j] = x[(size_t)phys_token(env_map, chunk, m0 + r) * Da + j];
  }
  __syncthreads();
  return rows;
}

// acc[r] += sum_j xs[r][j] w[j] over one W_in row (this thread's output
// column), in j order.  16-byte loads when the row allows: each of a wave's
// load instructions then touches every lane's 128-byte row once, where
// 4-byte loads touched 64 rows per instruction 32 times over.
template <int R>
__device__ __forceinline__ void action_row_dot(const float *__restrict__ w, int Da, const float (*xs)[64],
                                               float (&acc)[R]) {
  if ((Da & 3) == 0 && ((uintptr_t)w & 15) == 0) {
    for (int j = 0; j < Da; j += 4) {
      const f32x4 w4 = *(const f32x4 *)(w + j);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] += xs[r][j + e] * w4[e];  // rows past the end: never stored
    }
  } else {
    for (int j = 0; j < Da; ++j) {
      const float wj = w[j];
#pragma unroll
      for (int r = 0; r < R; ++r) acc[r] += xs[r][j] * wj;
    }
  }
}

// te[m] = [ x_m W_in^T + b_in ; sin(w t_m) ; cos(w t_m) ] as the fp16 operand
// of the time MLP in fragment order (K = 2d): the per-token flow-time
// conditioning placed before the action MLP.  Workgroup (g, y): tokens
// g R .. g R + R - 1, columns y * blockDim.x + tid of the action projection
// and the same indices of the sinusoids.
template <int R>
__global__ __launch_bounds__(256) void temb_kernel(const float *__restrict__ x, const float *__restrict__ t, int M,
                                                    int Da, int d, const float *__restrict__ w_in,
                                                    const float *__restrict__ b_in,
                                                    const float *__restrict__ freqs, op_t *__restrict__ te,
                                                    unsigned *status, const int32_t *env_map, int chunk) {
  __shared__ float xs[R][64];
  const int m0 = blockIdx.x * R;
  const int rows = load_action_rows<R>(x, M, Da, xs, env_map, chunk);
  const int KB = 2 * d / kTileK;
  unsigned bad = 0;  // fp16 range flag of this thread's stores
  const int n = blockIdx.y * blockDim.x + threadIdx.x;
  if (n < d) {
    float acc[R];
    const float bn = b_in[n];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = bn;
    action_row_dot<R>(w_in + (size_t)n * Da, Da, xs, acc);
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (r < rows) store_op(te + afrag_index(m0 + r, n, KB), acc[r], bad);
  }
  const int half = d >> 1;
  if (n < half)
    for (int r = 0; r < rows; ++r) {
      const float arg = freqs[n] * t[phys_token(env_map, chunk, m0 + r)];
      float sv, cv;
      sincosf(arg, &sv, &cv);  // one range reduction for both
      store_op(te + afrag_index(m0 + r, d + n, KB), sv, bad);
      store_op(te + afrag_index(m0 + r, d + half + n, KB), cv, bad);
    }
  flush_range(status, bad);
}

// Adaptive-norm variant: te[m] = e(t_m) alone (K = d) as the time MLP's fp16
// operand; the action token itself starts the residual stream,
// h[m] = x_m W_in^T + b_in (fp32), with its per-16-column sums of squares.
// t null: no time features (the schedule computed its time conditioning up
// front); mod_a0 not null: also the first attention norm's operand
// next = fp16(h_0 (1 + a)) with a the token's layer-0 scale, row stride mod_ld.
template <int R>
__global__ __launch_bounds__(256) void temb_ada_kernel(const float *__restrict__ x, const float *__restrict__ t,
                                                        int M, int Da, int d, const float *__restrict__ w_in,
                                                        const float *__restrict__ b_in,
                                                        const float *__restrict__ freqs, op_t *__restrict__ te,
                                                        float *__restrict__ h, float *__restrict__ ssq,
                                                        int m_alloc, const float *__restrict__ mod_a0, int mod_ld,
                                                        op_t *__restrict__ next, unsigned *status) {
  __shared__ float xs[R][64];
  const int m0 = blockIdx.x * R;
  const int rows = load_action_rows<R>(x, M, Da, xs);
  const int KB = d / kTileK;
  unsigned bad = 0;  // fp16 range flag of this thread's stores
  // d is a multiple of 32, so the 16 lanes of a 16-column tile are active together
  const int n = blockIdx.y * blockDim.x + threadIdx.x;
  if (n < d) {
    float acc[R];
    const float bn = b_in[n];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = bn;
    action_row_dot<R>(w_in + (size_t)n * Da, Da, xs, acc);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (r < rows) {  // uniform over the workgroup
        const int m = m0 + r;
        h[(size_t)m * d + n] = acc[r];
        float sq = acc[r] * acc[r];
        sq = sum_row16(sq);
        if ((n & 15) == 0) ssq[(size_t)(n >> 4) * m_alloc + m] = sq;
        if (mod_a0) store_op(next + afrag_index(m, n, KB), acc[r] * (1.0f + mod_a0[(size_t)m * mod_ld + n]), bad);
      }
    }
  }
  const int half = d >> 1;
  if (t && n < half)
    for (int r = 0; r < rows; ++r) {
      const float arg = freqs[n] * t[m0 + r];
      float sv, cv;
      sincosf(arg, &sv, &cv);  // one range reduction for both
      store_op(te + afrag_index(m0 + r, n, KB), sv, bad);
      store_op(te + afrag_index(m0 + r, half + n, KB), cv, bad);
    }
  flush_range(status, bad);
}

// v = RMSNorm(h) W_out^T + b_out, then x <- x + dt v unless frozen (mask or
// dt == 0: copy, so frozen tokens are bit-identical whatever v holds).
// Workgroup = (token m, group of up to 8 action dims); thread t owns columns
// t + 256 i of the row for all 8 dims, loads unconditional as above.
constexpr int kFinalOuts = 8;

// Masked Euler update of token m, action dim a with velocity v (a copy when
// frozen), the velocity outputs and the release bookkeeping.
__device__ __forceinline__ void euler_out(const FinalArgs &f, int mc, int a, float v) {
  const int m = phys_token(f.env_map, f.chunk, mc);  // the caller's token of step row mc
  const size_t idx = (size_t)m * f.Da + a;
  const float dtm = f.dt[m];
  const bool frozen = (f.mask[m] != 0) || (dtm == 0.0f);
  const float xo = f.x[idx];
  const float xn = frozen ? xo : xo + dtm * v;
  f.x[idx] = xn;
  if (f.v_out) f.v_out[idx] = v;
  if (f.vsum && (m % f.chunk) < f.vsum_tokens) f.vsum[idx] += v;
  const bool releasing = !frozen && (f.is_last_step || (f.next_mask && f.next_mask[m] != 0));
  if (releasing) {
    if (f.released) f.released[idx] = xn;
    if (f.release_step && a == 0) f.release_step[m] = f.step;
  }
}

template <int NC>
__global__ __launch_bounds__(256) void final_kernel(FinalArgs f) {
  __shared__ float scratch[4];
  __shared__ float wsum[4][kFinalOuts];
  __shared__ float vs[kFinalOuts];
  const int m = blockIdx.x;
  const int a0 = blockIdx.y * kFinalOuts;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int d = f.d;
  if (f.debug_field) {
    if (threadIdx.x < kFinalOuts && a0 + threadIdx.x < f.Da)
      vs[threadIdx.x] = f.dbg_alpha * f.x[(size_t)phys_token(f.env_map, f.chunk, m) * f.Da + a0 + threadIdx.x] +
                        f.dbg_beta;
  } else {
    const float *__restrict__ hr = f.h + (size_t)m * d;
    float hv[NC], gv[NC], sv[NC], wv[kFinalOuts][NC];
    const bool ada = f.mod_scale != nullptr;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = min(threadIdx.x + 256 * i, d - 1);
      hv[i] = hr[c];
      // adaptive norm: per-token scale (1 + a) and shift b; else the gain
      gv[i] = ada ? 1.0f + f.mod_scale[(size_t)m * f.mod_ld + c] : f.gain[c];
      sv[i] = ada ? f.mod_shift[(size_t)m * f.mod_ld + c] : 0.f;
#pragma unroll
      for (int o = 0; o < kFinalOuts; ++o) wv[o][i] = f.w_out[(size_t)min(a0 + o, f.Da - 1) * d + c];
    }
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      if (threadIdx.x + 256 * i >= d) hv[i] = sv[i] = 0.f;  // clamped duplicate columns contribute nothing
      ss += hv[i] * hv[i];
    }
    ss = block_sum_256(ss, scratch);
    const float rstd = 1.0f / sqrtf(ss / (float)d + f.eps);
    float acc[kFinalOuts];
#pragma unroll
    for (int o = 0; o < kFinalOuts; ++o) {
      acc[o] = 0.f;
#pragma unroll
      for (int i = 0; i < NC; ++i) acc[o] += (hv[i] * rstd * gv[i] + sv[i]) * wv[o][i];
      acc[o] = sum_wave64(acc[o]);
    }
    if (lane == 0)
#pragma unroll
      for (int o = 0; o < kFinalOuts; ++o) wsum[wave][o] = acc[o];
    __syncthreads();
    if (threadIdx.x < kFinalOuts && a0 + threadIdx.x < f.Da) {
      const int o = threadIdx.x;
      vs[o] = ((wsum[0][o] + wsum[1][o]) + (wsum[2][o] + wsum[3][o])) + f.b_out[a0 + o];
    }
  }
  __syncthreads();
  if (threadIdx.x < kFinalOuts && a0 + threadIdx.x < f.Da) euler_out(f, m, a0 + threadIdx.x, vs[threadIdx.x]);
}

// Batched steps (many tokens, no adaptive norm, no debug field): the
// projection as a product on the fp32 MFMA (v_mfma_f32_16x16x4_f32), 16
// tokens x all Da outputs per workgroup, the d columns split over its 4
// waves: v = rstd * ((h * gain) W_out^T) + b_out.  The row-blocked form it
// replaces spent its time in 72 wave reductions per wave (one per token and
// output) and re-read h once per group of 8 outputs.  Within a wave, k-step
// (q, e) of lane group kq = lane / 16 covers column c0 + 16 q + 4 kq + e, so
// each lane reads 16-byte runs of h, gain and W_out and feeds the same
// column to both operands.  The k-groups run in batches of 8 (uniform trip
// count: the loop bound does not depend on kq), loads first.
template <int NT>
__global__ __launch_bounds__(256) void final_mfma_kernel(FinalArgs f) {
  __shared__ f32x4 part[4][NT][64];  // per wave and output tile: each lane's accumulators
  __shared__ float ssq[4][64];       // per wave and lane: partial sum of squares of the lane's row
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m0 = blockIdx.x * 16, kq = lane >> 4;
  const float *__restrict__ hr = f.h + (size_t)min(m0 + (lane & 15), f.M - 1) * f.d;  // rows past M: never stored
  const float *__restrict__ wr[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) wr[t] = f.w_out + (size_t)min(16 * t + (lane & 15), f.Da - 1) * f.d;
  const int cpw = f.d >> 2;  // columns per wave (d % 512 == 0: whole batches)
  f32x4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float ss = 0.f;
  // batches of 8 k-groups of 16 columns: all their loads go out before the first MFMA
  for (int b = 0; b < cpw; b += 128) {
    const int cb = wave * cpw + 4 * kq + b;
    f32x4 hv[8], gv[8], wv[8][NT];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      hv[u] = *(const f32x4 *)(hr + cb + 16 * u);
      gv[u] = *(const f32x4 *)(f.gain + cb + 16 * u);
#pragma unroll
      for (int t = 0; t < NT; ++t) wv[u][t] = *(const f32x4 *)(wr[t] + cb + 16 * u);
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the batch's loads ahead of its MFMAs
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ss += hv[u][e] * hv[u][e];
        const float a = hv[u][e] * gv[u][e];
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, wv[u][t][e], acc[t], 0, 0, 0);
      }
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) part[wave][t][lane] = acc[t];
  ssq[wave][lane] = ss;
  __syncthreads();
  // thread (i, j): token m0 + i, outputs 16 t + j; D[i][j] of a tile sits in
  // lane j + 16 (i / 4), component i % 4
  const int i = threadIdx.x >> 4, j = threadIdx.x & 15, m = m0 + i;
  if (m >= f.M) return;
  float s2 = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w)
#pragma unroll
    for (int q = 0; q < 4; ++q) s2 += ssq[w][i + 16 * q];
  const float rstd = 1.0f / sqrtf(s2 / (float)f.d + f.eps);
  const int src = j + 16 * (i >> 2), cmp = i & 3;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int a = 16 * t + j;
    if (a < f.Da) {
      const float v = (part[0][t][src][cmp] + part[1][t][src][cmp]) + (part[2][t][src][cmp] + part[3][t][src][cmp]);
      euler_out(f, m, a, rstd * v + f.b_out[a]);
    }
  }
}

// Trajectory Reconciliation set-up: keep the initial noise x_0 and clear the
// velocity sums of the urgent tokens.
__global__ __launch_bounds__(256) void tr_init_kernel(TrArgs a) {
  const int n = a.B * a.H * a.Da;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    a.x0[i] = a.x[i];
    a.vsum[i] = 0.f;
  }
}

// Release after step K (Sec. 4.2): the urgent actions a^i = x_K^i, i < U, are
// copied out; with Trajectory Reconciliation (Sec. 4.3, Eq. 6) their internal
// states are then re-integrated under the canonical step,
// x'_K = x_0 + (1/N*) sum_k v_k, written in the flow-time convention of the
// integrator (dt* = -1/N*) and in the same form as its Euler update, so that
// with K = 1 the reconciled state equals the uniform schedule's x_1 bit for bit.
__global__ __launch_bounds__(256) void tr_release_kernel(TrArgs a) {
  const int n = a.B * a.U * a.Da;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const int c = i % a.Da;
    const int bu = i / a.Da;
    const int b = bu / a.U, u = bu - b * a.U;
    const size_t idx = ((size_t)b * a.H + u) * a.Da + c;
    const float v = a.x[idx];
    a.urgent[i] = v;
    if (a.urgent_host) a.urgent_host[i] = v;  // straight to the controller's pinned buffer
    if (a.reconcile) a.x[idx] = a.x0[idx] + a.dt_star * a.vsum[idx];
  }
  if (a.urgent_host) __threadfence_system();
}

// Ghost Action Correction (Sec. 4.4): E = sum_{i<U} (a'^i - a^i) over the ghost
// actions a'^i = x'^i_{N*} and released a^i (Eq. 8, summed in token order),
// then a^i = x^i_{N*} + E / (S - U) for i = U .. S-1 on the corrected
// dimensions (Eq. 9); executed[0..U) are the released actions unchanged.
__global__ __launch_bounds__(64) void gac_kernel(TrArgs a) {
  const int b = blockIdx.x;
  const int c = threadIdx.x;
  if (c >= a.Da) return;
  const float *xb = a.x + (size_t)b * a.H * a.Da;
  const float *ub = a.urgent + (size_t)b * a.U * a.Da;
  float *eb = a.executed + (size_t)b * a.S * a.Da;
  float E = 0.f;
  for (int i = 0; i < a.U; ++i) E += xb[(size_t)i * a.Da + c] - ub[(size_t)i * a.Da + c];
  const float shift = (a.gac_mask == nullptr || a.gac_mask[c] != 0) ? E / (float)(a.S - a.U) : 0.f;
  for (int i = 0; i < a.U; ++i) eb[(size_t)i * a.Da + c] = ub[(size_t)i * a.Da + c];
  for (int i = a.U; i < a.S; ++i) eb[(size_t)i * a.Da + c] = xb[(size_t)i * a.Da + c] + shift;
}

__global__ void stamp_kernel(uint64_t *dst) {
  if (threadIdx.x == 0) {
    const uint64_t now = __builtin_amdgcn_s_memrealtime();
    __hip_atomic_store(dst, now, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

hipError_t launch_temb(const float *x, const float *t, int M, int Da, int d, const float *w_in,
                       const float *b_in, const float *freqs, op_t *te, unsigned *status, hipStream_t s,
                       hipEvent_t ev0, hipEvent_t ev1, const int32_t *env_map, int chunk) {
  if (env_map && chunk < 1) return hipErrorInvalidValue;
  if (M >= 1024)
    UAD_LAUNCH(temb_kernel<16>, dim3((M + 15) / 16, (d + 255) / 256), dim3(256), 0, s, ev0, ev1, x, t, M, Da, d, w_in,
               b_in, freqs, te, status, env_map, chunk);
  else
    UAD_LAUNCH(temb_kernel<1>, dim3(M, (d + 255) / 256), dim3(256), 0, s, ev0, ev1, x, t, M, Da, d, w_in, b_in, freqs,
               te, status, env_map, chunk);
  return hipGetLastError();
}

hipError_t launch_temb_ada(const float *x, const float *t, int M, int Da, int d, const float *w_in,
                           const float *b_in, const float *freqs, op_t *te, float *h, float *ssq, int m_alloc,
                           unsigned *status, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1, const float *mod_a0,
                           int mod_ld, op_t *next) {
  if (mod_a0 && !next) return hipErrorInvalidValue;
  if (M >= 1024)
    UAD_LAUNCH(temb_ada_kernel<16>, dim3((M + 15) / 16, (d + 255) / 256), dim3(256), 0, s, ev0, ev1, x, t, M, Da, d,
               w_in, b_in, freqs, te, h, ssq, m_alloc, mod_a0, mod_ld, next, status);
  else
    UAD_LAUNCH(temb_ada_kernel<1>, dim3(M, (d + 255) / 256), dim3(256), 0, s, ev0, ev1, x, t, M, Da, d, w_in, b_in,
               freqs, te, h, ssq, m_alloc, mod_a0, mod_ld, next, status);
  return hipGetLastError();
}

// Time features of a whole schedule: row r = step * m_alloc + i takes the
// flow time t[step * M + i] (i < M), padding rows time 0.
__global__ __launch_bounds__(256) void time_feat_kernel(const float *__restrict__ t, int M, int m_alloc, int rows,
                                                         int d, const float *__restrict__ freqs,
                                                         op_t *__restrict__ te, unsigned *status) {
  const int r = blockIdx.x;
  const int n = blockIdx.y * blockDim.x + threadIdx.x;
  const int half = d >> 1;
  if (r >= rows || n >= half) return;
  const int st = r / m_alloc, i = r - st * m_alloc;
  const float tv = i < M ? t[(size_t)st * M + i] : 0.f;
  const float arg = freqs[n] * tv;
  const int KB = d / kTileK;
  float sv, cv;
  sincosf(arg, &sv, &cv);  // one range reduction for both
  unsigned bad = 0;
  store_op(te + afrag_index(r, n, KB), sv, bad);
  store_op(te + afrag_index(r, half + n, KB), cv, bad);
  flush_range(status, bad);
}

hipError_t launch_time_features(const float *t, int M, int m_alloc, int n_steps, int d, const float *freqs,
                                op_t *te, unsigned *status, hipStream_t s) {
  if (M < 1 || m_alloc < M || m_alloc % 16 != 0 || n_steps < 1 || d % 64 != 0) return hipErrorInvalidValue;
  const int rows = n_steps * m_alloc;
  hipLaunchKernelGGL(time_feat_kernel, dim3(rows, (d / 2 + 255) / 256), dim3(256), 0, s, t, M, m_alloc, rows, d,
                     freqs, te, status);
  return hipGetLastError();
}

hipError_t launch_final(const FinalArgs &f, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (f.M >= 1024 && !f.debug_field && !f.mod_scale && f.d % 512 == 0 && f.Da <= 64) {
    const dim3 gr((f.M + 15) / 16);
    switch ((f.Da + 15) / 16) {
      case 1: UAD_LAUNCH(final_mfma_kernel<1>, gr, dim3(256), 0, s, ev0, ev1, f); return hipGetLastError();
      case 2: UAD_LAUNCH(final_mfma_kernel<2>, gr, dim3(256), 0, s, ev0, ev1, f); return hipGetLastError();
      case 3: UAD_LAUNCH(final_mfma_kernel<3>, gr, dim3(256), 0, s, ev0, ev1, f); return hipGetLastError();
      case 4: UAD_LAUNCH(final_mfma_kernel<4>, gr, dim3(256), 0, s, ev0, ev1, f); return hipGetLastError();
    }
  }
  const dim3 grid(f.M, (f.Da + kFinalOuts - 1) / kFinalOuts);
  switch ((f.d + 255) / 256) {
    case 1: UAD_LAUNCH(final_kernel<1>, grid, dim3(256), 0, s, ev0, ev1, f); break;
    case 2: UAD_LAUNCH(final_kernel<2>, grid, dim3(256), 0, s, ev0, ev1, f); break;
    case 3: UAD_LAUNCH(final_kernel<3>, grid, dim3(256), 0, s, ev0, ev1, f); break;
    case 4: UAD_LAUNCH(final_kernel<4>, grid, dim3(256), 0, s, ev0, ev1, f); break;
    case 5: UAD_LAUNCH(final_kernel<5>, grid, dim3(256), 0, s, ev0, ev1, f); break;
    case 6: UAD_LAUNCH(final_kernel<6>, grid, dim3(256), 0, s, ev0, ev1, f); break;
    case 7: UAD_LAUNCH(final_kernel<7>, grid, dim3(256), 0, s, ev0, ev1, f); break;
    case 8: UAD_LAUNCH(final_kernel<8>, grid, dim3(256), 0, s, ev0, ev1, f); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_tr_init(const TrArgs &a, hipStream_t s) {
  const int n = a.B * a.H * a.Da;
  hipLaunchKernelGGL(tr_init_kernel, dim3((n + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_tr_release(const TrArgs &a, hipStream_t s) {
  const int n = a.B * a.U * a.Da;
  hipLaunchKernelGGL(tr_release_kernel, dim3((n + 255) / 256), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gac(const TrArgs &a, hipStream_t s) {
  if (a.Da > 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gac_kernel, dim3(a.B), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_stamp(uint64_t *dst, hipStream_t s) {
  hipLaunchKernelGGL(stamp_kernel, dim3(1), dim3(64), 0, s, dst);
  return hipGetLastError();
}

}  // namespace uad
