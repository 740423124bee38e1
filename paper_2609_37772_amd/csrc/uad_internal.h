// Internal declarations shared by the translation units of libuad.
// Not part of the public ABI (see include/uad.h).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/uad.h"

namespace uad {

// Kernel launch; with events (measurement hook) the start/stop timestamps are
// taken from the dispatch packet itself, so they time exactly the kernel.
#define UAD_LAUNCH(kernel, grid, block, shmem, stream, ev0, ev1, ...)                                  \
  do {                                                                                               \
    if ((ev0) || (ev1))                                                                              \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ev0, ev1, 0, __VA_ARGS__);           \
    else                                                                                             \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                           \
  } while (0)

// ---------------------------------------------------------------------------
// Vector types for the gfx950 MFMA builtins
// ---------------------------------------------------------------------------
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 f16x4;

// Projection operands (weights and activations) are fp16.  The model's
// weights are bf16 values and fp16 holds every bf16 value of magnitude in
// [2^-14, 65504] exactly (8 significant bits fit in 11), so the weight stream
// is the bf16 model itself; smaller magnitudes round to the nearest fp16
// subnormal (absolute error <= 2^-25) and larger ones are rejected at load.
// Activations keep 11 significant bits instead of bf16's 8, which keeps the
// rounding accumulated over the layer stack and the Euler steps well inside
// the velocity tolerance while each activation costs 2 bytes to stream.
typedef _Float16 op_t;

// Packed weight layout used by every MFMA GEMM ("fragment order"):
// a row-major W[N][K] (PyTorch [out][in]) is cut into 16x32 blocks; block
// (nt, kb) holds 64 lanes x 8 consecutive-k fp16 values, lane l carrying
// W[16*nt + (l & 15)][32*kb + 8*(l >> 4) + e], e = 0..7.  Blocks are stored
// n-tile major, so one 16-column tile's whole K stream is contiguous and each
// lane's operand is one aligned 16-byte load.
constexpr int kMaxTrSteps = 64;  // longest canonical schedule N* of the release path
// fp32 elements of one split-K partial tile (a 128 x 128 output tile); the
// context holds two per CU
constexpr size_t kKxPartialFloats = 128 * 128;
constexpr int kTileN = 16;
constexpr int kTileK = 32;
// token rows from which the projections run on the batched (128-row tile)
// kernels rather than the small-M weight-streaming one
constexpr int kBigM = 256;
constexpr int kBlockElems = kTileN * kTileK;  // 512 fp16 = 1 KiB

// Device status word of a context (bits, cleared and reported by
// uad_synchronize): an fp16 operand that was not finite after rounding, and an
// in-kernel wait that gave up.
constexpr unsigned kStatusRange = 1u;
constexpr unsigned kStatusTimeout = 2u;

__device__ __forceinline__ void raise_status(unsigned *status, unsigned bit) {
  __hip_atomic_fetch_or(status, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Every fp16 operand store checks its value: fp16 holds magnitudes below
// 65520 (which round to at most 65504); anything larger becomes inf and a NaN
// stays NaN.  The check is branch-free: a thread collects a flag over its
// stores (`bad`) and raises the context's range bit once, at the end of its
// kernel (flush_range), so the stores are issued as before.
__device__ __forceinline__ void store_op(op_t *p, float v, unsigned &bad) {
  *p = (op_t)v;
  bad |= (unsigned)!(__builtin_fabsf(v) < 65520.0f);
}
__device__ __forceinline__ void check_op4(float a, float b, float c, float d, unsigned &bad) {
  const float T = 65520.0f;
  bad |= (unsigned)(!(__builtin_fabsf(a) < T) | !(__builtin_fabsf(b) < T) | !(__builtin_fabsf(c) < T) |
                    !(__builtin_fabsf(d) < T));
}
__device__ __forceinline__ void flush_range(unsigned *status, unsigned bad) {
  if (bad) raise_status(status, kStatusRange);
}

// ---------------------------------------------------------------------------
// Cross-lane reductions without the LDS crossbar (ds_bpermute): DPP within a
// row of 16 lanes (quad permutes for lane ^ 1 and lane ^ 2, then the half-row
// and row mirrors, which pair the remaining groups), and the gfx950 lane-swap
// instructions across rows (swapping a value with itself leaves each lane its
// own value and that of lane ^ 16 / lane ^ 32).  Every lane of the group ends
// with the same (bitwise) result.  Lane layouts checked by in-bounds probes.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float sum_row16(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1,0,3,2]: lane ^ 1
  v += dpp_f<0x4E>(v);   // quad_perm [2,3,0,1]: lane ^ 2
  v += dpp_f<0x141>(v);  // row_half_mirror: the other quad of the 8
  v += dpp_f<0x140>(v);  // row_mirror: the other 8 of the 16
  return v;
}
__device__ __forceinline__ float sum_pair16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_pair32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float max_pair16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_pair32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_wave64(float v) { return sum_pair32(sum_pair16(sum_row16(v))); }

// Activation operands use the same fragment order as the weights: a
// [rows][K] matrix (rows padded to 16) is stored as [rows/16][K/32][64][8],
// element (r, c) at lane (r & 15) + 16 * ((c & 31) >> 3), slot c & 7, so a
// wave loads one 16x32 A fragment as 1 KiB contiguous.
__host__ __device__ __forceinline__ size_t afrag_index(int r, int c, int KB) {
  return ((size_t)((r >> 4) * KB + (c >> 5)) * 64 + (r & 15) + 16 * ((c & 31) >> 3)) * 8 + (c & 7);
}

// K/V store layout per (layer, environment, KV head) with key slots padded to
// s_alloc (a multiple of 32): K as [s_alloc][hd]; V transposed in 32-key
// blocks, [s_alloc/32][hd][32], so one block's V^T tile is 32*hd contiguous
// values.  Within a block the 32 keys of a V^T row are stored permuted: key
// 16h + 4g + r (h < 2, g < 4, r < 4) at position 8g + 4h + r, the order in
// which the attention kernel's P V operand consumes them (8 contiguous keys
// per lane).  Index of V(key s, column c) of environment-head eh:
__host__ __device__ __forceinline__ int vt_key_pos(int k) { return ((k >> 2) & 3) * 8 + (k >> 4) * 4 + (k & 3); }
__host__ __device__ __forceinline__ size_t vt_index(size_t eh, int s, int c, int hd, int s_alloc) {
  return eh * (size_t)hd * s_alloc + ((size_t)(s >> 5) * hd + c) * 32 + vt_key_pos(s & 31);
}

// ---------------------------------------------------------------------------
// Kernel argument blocks
// ---------------------------------------------------------------------------
enum Epilogue : int {
  EPI_BIAS_SILU = 0,   // out = fp16 silu(acc + bias), fragment order
  EPI_RESID_F32 = 1,   // h = (bias | h) + acc; per-tile sum of squares; next operand fp16(h * gain_next)
  EPI_GEGLU = 3,       // out = fp16 gelu_tanh(rstd*acc_gate) * rstd*acc_up (interleaved gate/up)
  EPI_QKV = 4,         // rstd*acc: q -> bf16 q buffer; k, v -> per-layer K / V^T store
  EPI_MOD = 5,         // adaptive-norm modulations of every norm site (see uad_ctx::mod)
};

struct GemmPlan {
  int T;        // 16-column weight tiles per workgroup
  int mgroups;  // row groups (grid.z); group z owns 16-row tiles [z*MT/mgroups, (z+1)*MT/mgroups)
  int kpw;      // 32-deep k-blocks per wave and pass
  int waves;    // waves per workgroup
  int passes;   // runs of kpw blocks per wave
  bool ok;
};

struct GemmArgs {
  const op_t *A;    // activations, fragment order [rows/16][K/32][64][8]
  // RMSNorm folded into the GEMMs: a residual GEMM writes ssq[tile][row] (sum of
  // squares of h over its 16 columns) and the next operand fp16(h * gain_next);
  // a consuming GEMM scales its accumulator by rstd[row] from those sums.
  float *ssq;             // [d/16][m_alloc]
  int ssq_tiles;
  int m_alloc;            // rows allocated in every operand / output buffer (>= M, multiple of 16)
  float eps;
  const float *gain_next; // EPI_RESID_F32: gain of the following RMSNorm (nullptr: none)
  op_t *next;             // EPI_RESID_F32: next operand, fragment order (K = N)
  int use_rstd;           // EPI_QKV / EPI_GEGLU: scale by rstd from ssq
  // adaptive-norm conditioning
  const op_t *A2;         // EPI_QKV / EPI_GEGLU: second operand (the norm's shift), result rstd*(A W) + A2 W
  const float *mod_gate;  // EPI_RESID_F32: h += gate[row * mod_ld + col] * acc (nullptr: gate 1)
  const float *mod_scale_next;  // EPI_RESID_F32: next operand fp16(h * (1 + scale[row * mod_ld + col]))
  int mod_ld;
  // EPI_MOD destinations: fp32 [M][N] row-major (out), the shifts as fp16
  // operands, and the first attention norm's operand fp16(h * (1 + scale))
  op_t *mod_shift_ops;    // [L][2][m_alloc*d] fragment order
  const float *h_in;      // [M][d] residual stream
  int d_model, n_layers;
  size_t shift_stride;    // elements per shift operand
  const op_t *W;    // packed weights, N/16 tiles x K/32 blocks
  int M, N, K;      // N counts packed output columns (2F for gate/up)
  void *out;        // epilogue destination
  int ldo;          // its row length (= K of the consuming GEMM for fragment-order outputs)
  const float *bias;
  // EPI_QKV destinations
  __bf16 *kc;   // layer K store [B][Hkv][S_alloc][hd]
  __bf16 *vtc;  // layer V^T store, 32-key blocks (vt_index)
  int chunk, prefix, s_alloc, n_kv_heads, head_dim, q_dim;
  unsigned *status;  // context status word (range bit of the fp16 operand stores)
  // compacted steps: environment j of this step is environment env_map[j] of
  // the caller's batch (its K/V store slot); null when every environment runs
  const int32_t *env_map;
  // Split-K of the batched residual projections when their tiles leave most
  // CUs idle (null workspace: never).  kx_ws holds the fp32 partial tiles
  // (kx_ws_bytes), kx_cnt one arrival counter per output tile, zero between
  // launches (the last workgroup of a tile to arrive resets it); kx is the
  // split count of the launch, set by the launcher.
  float *kx_ws;
  unsigned *kx_cnt;
  size_t kx_ws_bytes;
  int kx_tiles;  // counters available
  int kx;
};

// Up to two byte ranges (weights of the next projections) that otherwise idle
// workgroups of a latency-bound launch read ahead of their use, so that the
// projections find them in the memory-side cache instead of HBM.
struct Prefetch {
  const char *p[2];
  uint32_t bytes[2];  // multiples of 16
  int wgs;            // workgroups given to it (0: no prefetch)
};

struct AttnArgs {
  const __bf16 *q;  // [M][ldq] bf16, query head j at columns j*hd
  int ldq;
  const __bf16 *kc;  // layer K store
  const __bf16 *vtc; // layer V^T store
  int s_alloc;
  int n_keys;        // prefix + chunk
  int chunk, n_heads, n_kv_heads, group, rows, rows_pad;
  int splits, blocks_per_split;
  int qblocks, n_eh;  // 64-row query blocks per environment-head; environment-heads (B * Hkv)
  float scale_log2;  // log2(e) / sqrt(hd)
  op_t *o;           // O-projection operand, fragment order, K = ldo
  int ldo;
  op_t *opart;       // split partials o_s / l_s, fp16 (splits > 1), accumulator layout
  float *mlpart;     // [splits][B*Hkv][rows_pad][2] (max, sum) per row
  Prefetch pre_attn;  // read by extra workgroups of the attention kernel
  Prefetch pre_comb;  // read by an extra slice of the split-merge grid (wgs: nonzero = on)
  unsigned *pf_sink;  // one word the prefetch may write (keeps its loads alive)
  unsigned *status;   // context status word (range bit of the fp16 stores)
  const int32_t *env_map;  // compacted steps: K/V store environment of each environment of the step, or null
};

struct FinalArgs {
  const float *h;       // [M][d]
  const float *gain;    // final_norm [d]
  const float *w_out;   // [Da][d] fp32
  const float *b_out;   // [Da]
  float eps;
  int M, d, Da;
  float *x;             // [M][Da] in/out
  const float *t, *dt;  // [M]
  const uint8_t *mask;  // [M]
  const uint8_t *next_mask;  // [M] or null (schedule: mask of the next step)
  int is_last_step;
  int step;
  float *v_out;         // [M][Da] or null
  float *released;      // [M][Da] or null
  int32_t *release_step;// [M] or null
  int debug_field;
  float dbg_alpha, dbg_beta;
  // adaptive-norm conditioning of the final norm: RMS(h) * (1 + scale) + shift
  const float *mod_scale, *mod_shift;  // [M][mod_ld] or null (then the gain applies)
  int mod_ld;
  // Trajectory Reconciliation: vsum[m] += v for tokens (m % chunk) < vsum_tokens
  float *vsum;          // [M][Da] or null
  int vsum_tokens, chunk;
  // compacted steps: token m of the step (h row m) is token
  // env_map[m / chunk] * chunk + m % chunk of x, t, dt, masks and outputs
  const int32_t *env_map;
};

// Urgency-aware release with Trajectory Reconciliation and Ghost Action
// Correction over a batch of chunks (x [B][H][Da]).
struct TrArgs {
  float *x;              // live states
  float *x0;             // initial noise (copy)
  float *vsum;           // sum of the urgent tokens' velocities over steps < K
  float *urgent;         // [B][U][Da] released urgent actions x_K
  float *executed;       // [B][S][Da] urgent actions then GAC-corrected tail, or null
  const uint8_t *gac_mask;  // [Da] 1 = additive dimension corrected, or null (all)
  float *urgent_host;    // device address of pinned host [B][U][Da] that also receives them, or null
  int B, H, Da, U, S;
  float dt_star;         // -(1/N*), the canonical step
  int reconcile;         // 1: TR (ghosts continue), 0: plain early release (urgent frozen)
};

// ---------------------------------------------------------------------------
// Launchers (defined in the .hip translation units)
// ---------------------------------------------------------------------------
GemmPlan plan_gemm(int epi, int M, int N, int K);
// ev0 / ev1: optional events recorded at the start / end of the launched
// kernel(s) (nullptr for none).
hipError_t launch_gemm(int epi, const GemmArgs &g, const GemmPlan &p, hipStream_t s, hipEvent_t ev0 = nullptr,
                       hipEvent_t ev1 = nullptr);
hipError_t launch_attention(const AttnArgs &a, int batch, int head_dim, hipStream_t s, hipEvent_t ev0 = nullptr,
                            hipEvent_t ev1 = nullptr);
hipError_t attention_init();             // once per context: raise the kernels' LDS limit
hipError_t gemm_init();                  // once per context: raise the batched GEMM's LDS limit
int attention_chunk_blocks(int head_dim);  // 32-key blocks loaded per round trip
int attention_max_splits(int head_dim);    // split-KV partials the combine accepts
// env_map (compacted steps): token m of the step reads x and t of token
// env_map[m / chunk] * chunk + m % chunk (null: token m)
hipError_t launch_temb(const float *x, const float *t, int M, int Da, int d, const float *w_in,
                       const float *b_in, const float *freqs, op_t *te, unsigned *status, hipStream_t s,
                       hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr, const int32_t *env_map = nullptr,
                       int chunk = 1);
// adaptive-norm variant: te <- e(t) (K = d); h <- W_in x + b_in with its
// per-16-column sums of squares ssq[d/16][m_alloc]
hipError_t launch_temb_ada(const float *x, const float *t, int M, int Da, int d, const float *w_in,
                           const float *b_in, const float *freqs, op_t *te, float *h, float *ssq, int m_alloc,
                           unsigned *status, hipStream_t s, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr,
                           const float *mod_a0 = nullptr, int mod_ld = 0, op_t *next = nullptr);
// sinusoidal time features of n_steps x m_alloc rows (rows past M in a step: time 0)
hipError_t launch_time_features(const float *t, int M, int m_alloc, int n_steps, int d, const float *freqs,
                                op_t *te, unsigned *status, hipStream_t s);
hipError_t launch_final(const FinalArgs &f, hipStream_t s, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
hipError_t launch_stamp(uint64_t *dst, hipStream_t s);
hipError_t launch_tr_init(const TrArgs &a, hipStream_t s);     // x0 <- x, vsum <- 0
hipError_t launch_tr_release(const TrArgs &a, hipStream_t s);  // urgent <- x_K; TR: x_K <- x0 + dt* vsum
hipError_t launch_gac(const TrArgs &a, hipStream_t s);         // E and the corrected executed actions

// Host-side helpers (schedule.cpp)
bool build_schedule_host(const int32_t *budgets, int batch, int chunk, int max_steps, int32_t *n_steps,
                         float *t, float *dt, uint8_t *mask, std::string *err);

}  // namespace uad

// ---------------------------------------------------------------------------
// Context
// ---------------------------------------------------------------------------
// Everything a captured step/schedule graph depends on.
struct GraphKey {
  int kind;  // 0: step / schedule; 1, 2: urgency-aware release phases before / after the release;
             // 3: schedule from budgets with finished environments compacted away
  bool is_schedule;
  float *x;
  const float *t, *dt;
  const uint8_t *mask;
  float *v_out, *released;
  int32_t *release_step;
  uint64_t *step_ticks;
  int n_steps, B, H, prefix_len, prefix_batch;
  // release phases
  int U, Kr, Nstar, S, reconcile;
  float *urgent, *executed;
  const uint8_t *gac_mask;
  float *urgent_host;  // device address of the pinned host copy written by the release kernel, or null
  // kind 3: environments evaluated at each step (their list is device data the graph reads)
  uint16_t active[uad::kMaxTrSteps];
  bool operator==(const GraphKey &o) const {
    for (int i = 0; i < uad::kMaxTrSteps; ++i)
      if (active[i] != o.active[i]) return false;
    return kind == o.kind && U == o.U && Kr == o.Kr && Nstar == o.Nstar && S == o.S && reconcile == o.reconcile &&
           urgent == o.urgent && executed == o.executed && gac_mask == o.gac_mask && urgent_host == o.urgent_host &&
           is_schedule == o.is_schedule && x == o.x && t == o.t && dt == o.dt && mask == o.mask &&
           v_out == o.v_out && released == o.released && release_step == o.release_step &&
           step_ticks == o.step_ticks && n_steps == o.n_steps && B == o.B && H == o.H &&
           prefix_len == o.prefix_len && prefix_batch == o.prefix_batch;
  }
};

struct uad_layer_ptrs {
  const uad::op_t *wqkv, *wo, *wgu, *wdown;
  const float *attn_norm, *mlp_norm;  // input conditioning only
};

struct uad_ctx {
  uad_model_config cfg{};
  int device = 0;
  hipStream_t stream = nullptr;  // the caller's stream (null: the device's null stream)
  std::string err;

  int d = 0, L = 0, Hq = 0, Hkv = 0, hd = 0, F = 0, Da = 0;
  int q_dim = 0, kv_dim = 0, n_qkv = 0;
  int m_alloc = 0;   // activation rows, multiple of 64
  int s_alloc = 0;   // key slots per (layer, env, kv head), multiple of 32

  // weights
  void *wbuf = nullptr;
  size_t wbytes = 0;
  float *action_in_w = nullptr, *action_in_b = nullptr, *t1_b = nullptr, *t2_b = nullptr;
  float *final_norm = nullptr, *action_out_w = nullptr, *action_out_b = nullptr, *freqs = nullptr;
  uad::op_t *t1_w = nullptr, *t2_w = nullptr;
  std::vector<uad_layer_ptrs> layers;
  bool weights_loaded = false;

  // prefix / chunk K,V store
  __bf16 *kcache = nullptr, *vtcache = nullptr;
  size_t kv_layer_elems = 0;  // elements per layer in each store
  int prefix_len = 0, prefix_batch = 0;
  bool prefix_set = false;

  // activation workspace
  float *h = nullptr;
  uad::op_t *a_te = nullptr, *a_z = nullptr, *a_n = nullptr, *a_o = nullptr, *a_g = nullptr;
  __bf16 *q = nullptr;
  uad::op_t *attn_opart = nullptr;
  float *attn_ml = nullptr;
  unsigned *pf_sink = nullptr;
  int n_cu = 0;  // compute units of the device
  size_t attn_part_elems = 0;
  float *ssq = nullptr;   // per-tile sums of squares of h [d/16][m_alloc]
  float *kx_ws = nullptr;     // split-K partial tiles of the batched residual projections
  unsigned *kx_cnt = nullptr; // their per-tile arrival counters (zeroed at creation)
  size_t kx_ws_bytes = 0;
  void *abuf = nullptr;

  // adaptive-norm conditioning (flag UAD_FLAG_ADARMS)
  bool ada = false;
  int n_mod = 0;                      // L*6d + 2d modulation columns
  uad::op_t *w_mod = nullptr;         // packed [n_mod][d]
  float *b_mod = nullptr;             // [n_mod]
  float *mod = nullptr;               // [m_alloc][n_mod] per token: per layer (a,b,g)_attn (a,b,g)_mlp, then (a,b)_final
  uad::op_t *mod_shift_ops = nullptr; // [L][2][m_alloc*d] shifts as fp16 operands
  // schedule-level conditioning (small batches): the modulations depend on the
  // flow time only, so a schedule computes them for all its steps at once,
  // n_steps x m_alloc rows, and each step reads its slice
  void *pre_buf = nullptr;
  size_t pre_rows = 0;                // rows the buffers hold
  float *pre_mod = nullptr;           // [rows][n_mod]
  uad::op_t *pre_shift = nullptr;     // [L][2][rows*d] fragment order
  uad::op_t *pre_te = nullptr, *pre_z = nullptr;  // [rows][d] time MLP operands

  // urgency-aware release with Trajectory Reconciliation
  float *tr_x0 = nullptr, *tr_vsum = nullptr;  // [m_alloc][Da]
  float *tr_t = nullptr, *tr_dt = nullptr;     // [kMaxSteps][m_alloc] step tables of the last configuration
  uint8_t *tr_mask = nullptr;
  int tr_key[6] = {0, 0, 0, 0, 0, -1};         // B, H, U, K, N*, reconcile of the tables
  // schedules from budgets (uad_denoise_budgets): step tables, and per step the
  // ascending list of environments with an active token, for the last budgets
  float *bud_t = nullptr, *bud_dt = nullptr;   // [kMaxTrSteps][m_alloc]
  uint8_t *bud_mask = nullptr;
  int32_t *bud_map = nullptr;                  // [kMaxTrSteps][max_batch]
  std::vector<int32_t> bud_key;                // budgets of the uploaded tables (B, H, then B*H budgets)
  std::vector<uint16_t> bud_active;            // environments per step
  hipStream_t rel_stream = nullptr;            // release copies to pageable host memory
  hipEvent_t ev_rel = nullptr;
  unsigned *status = nullptr;                  // device status word (kStatusRange, kStatusTimeout)

  // captured step / schedule graphs (small LRU cache)
  struct GraphEntry {
    GraphKey key;
    hipGraphExec_t exec;
    uint64_t last_use;
  };
  std::vector<GraphEntry> graphs;
  uint64_t graph_clock = 0;
  hipStream_t cap_stream = nullptr;
  bool graph_broken = false;

  // measurement hook: events around every launch, grouped by kernel class
  struct ProfRec {
    int cls;
    hipEvent_t a, b;
  };
  bool prof_on = false;
  std::vector<ProfRec> prof_pending;
  std::vector<hipEvent_t> ev_pool;
  std::vector<double> prof_ms;
  std::vector<int64_t> prof_n;

  // test hook
  bool dbg = false;
  float dbg_alpha = 0.f, dbg_beta = 0.f;
  double tick_hz = 0.0;
};
