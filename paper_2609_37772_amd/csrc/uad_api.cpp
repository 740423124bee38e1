// C ABI of libuad: context management, argument validation, weight and
// prefix repacking into the kernels' device layouts, and the launch sequence
// of one joint denoising step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "uad_internal.h"

using namespace uad;

namespace {

thread_local std::string g_create_err;

uad_status fail(uad_ctx *c, uad_status st, const std::string &msg) {
  if (c) c->err = msg;
  return st;
}

uad_status hip_fail(uad_ctx *c, hipError_t e, const char *what) {
  return fail(c, UAD_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
int round_up(int x, int m) { return (x + m - 1) / m * m; }

uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x7FFFFFu)) return (uint16_t)((u >> 16) | 0x40);  // quiet NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

float bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// Copy a caller tensor (host or device, f32 or bf16) to a host fp32 vector.
bool fetch_f32(const void *data, int dtype, int on_device, size_t n, std::vector<float> *out, std::string *err) {
  out->resize(n);
  const size_t esz = dtype == UAD_DTYPE_F32 ? 4 : 2;
  std::vector<uint8_t> tmp;
  const void *src = data;
  if (on_device) {
    tmp.resize(n * esz);
    hipError_t e = hipMemcpy(tmp.data(), data, n * esz, hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
      *err = std::string("hipMemcpy(D2H): ") + hipGetErrorString(e);
      return false;
    }
    src = tmp.data();
  }
  if (dtype == UAD_DTYPE_F32) {
    std::memcpy(out->data(), src, n * 4);
  } else {
    const uint16_t *s = (const uint16_t *)src;
    for (size_t i = 0; i < n; ++i) (*out)[i] = bf16_to_f32(s[i]);
  }
  return true;
}

// A projection weight as the kernels hold it: the value rounded once to bf16
// (the model's precision), then stored as fp16, which is exact for bf16
// magnitudes in [2^-14, 65504]; smaller ones round to the nearest fp16
// subnormal.  Returns false for magnitudes beyond the fp16 range (or NaN).
bool weight_to_f16(float w, _Float16 *out) {
  const float b = bf16_to_f32(f32_to_bf16_rne(w));
  if (!(std::fabs(b) <= 65504.0f)) return false;
  *out = (_Float16)b;
  return true;
}

// Pack row-major W[N][K] into the MFMA fragment order (see uad_internal.h),
// writing 16-row tile nt to destination tile (tile_base + nt * tile_step).
bool pack_tiles(const float *W, int N, int K, _Float16 *dst, int tile_base, int tile_step) {
  const int KB = K / kTileK;
  bool ok = true;
  for (int nt = 0; nt < N / kTileN; ++nt) {
    _Float16 *tb = dst + (size_t)(tile_base + nt * tile_step) * KB * kBlockElems;
    for (int kb = 0; kb < KB; ++kb)
      for (int l = 0; l < 64; ++l)
        for (int e = 0; e < 8; ++e)
          ok &= weight_to_f16(W[(size_t)(nt * kTileN + (l & 15)) * K + kb * kTileK + (l >> 4) * 8 + e],
                              &tb[((size_t)kb * 64 + l) * 8 + e]);
  }
  return ok;
}

struct Carve {
  size_t off = 0;
  template <class T>
  size_t take(size_t n) {
    size_t o = off;
    off = align256(off + n * sizeof(T));
    return o;
  }
};

// Kernel classes reported by the measurement hook.
enum KClass { K_TEMB, K_GEMM_TIME_IN, K_GEMM_TIME_OUT, K_GEMM_QKV, K_ATTENTION, K_GEMM_O, K_GEMM_GATEUP,
              K_GEMM_DOWN, K_FINAL, K_GEMM_MOD, K_NCLASS };
const char *kClassNames[K_NCLASS] = {"temb", "gemm_time_in", "gemm_time_out", "gemm_qkv", "attention",
                                     "gemm_o", "gemm_gateup", "gemm_down", "final_euler", "gemm_mod"};

hipEvent_t pool_event(uad_ctx *c) {
  if (!c->ev_pool.empty()) {
    hipEvent_t e = c->ev_pool.back();
    c->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  (void)hipEventCreate(&e);
  return e;
}

// CUs the attention launch has to leave free for the weight read-ahead of its
// extra workgroups (below that the read-ahead is not issued).
constexpr int kReadAheadMinCus = 32;

int attn_splits_nb(const uad_ctx *c, int B, int H, int n_blocks, int *bps) {
  const int rows = (c->Hq / c->Hkv) * H;
  const int qblocks = (rows + 63) / 64;
  const int wgs = qblocks * B * c->Hkv;
  // Split the keys so that the query blocks x splits fill about one round of
  // workgroups (256 CUs): one chunk (one memory round trip) per split when
  // that fits (batch 1), else floor(256 / query blocks) splits (a few
  // environments; measured best at 4 and 8 environments), none when the query
  // blocks alone fill the chip.  Where the projections run on the batched
  // kernels, fewer splits if the grid (its groups padded to a multiple of the
  // 8 XCDs) would leave under kReadAheadMinCus CUs to the weight read-ahead:
  // gate/up then streams its weights from HBM (~28.5 instead of ~22.5 us at
  // 300-850 rows).  Same-machine, ms per joint step, 1024-wide expert: 6
  // environments 1.616 -> 1.588 (6 -> 5 splits), 7 1.679 -> 1.608, 9 1.769 ->
  // 1.695, 11 2.003 -> 1.924, 12 2.053 -> 1.947 (3 -> 2), 17 2.354 -> 2.276
  // (2 -> 1); 1536-wide: 2 environments 2.683 -> 2.581, 5 3.395 -> 3.262.
  // Below 256 rows (5 environments: 7 -> 6 splits, 1.442 -> 1.451 ms) the
  // small-M projections gain less from the read-ahead than the attention
  // loses.
  const int nb = attention_chunk_blocks(c->hd);
  int per = nb;
  if ((long)wgs * ((n_blocks + nb - 1) / nb) > 256) {
    for (int sp = std::max(1, 256 / wgs);; --sp) {
      per = (n_blocks + sp - 1) / sp;
      const int splits = (n_blocks + per - 1) / per;
      if (sp == 1 || B * H < kBigM || 8 * ((B * c->Hkv * splits + 7) / 8) * qblocks <= c->n_cu - kReadAheadMinCus)
        break;
    }
  }
  const int smax = attention_max_splits(c->hd);
  if ((n_blocks + per - 1) / per > smax) per = (n_blocks + smax - 1) / smax;
  if (per > n_blocks) per = n_blocks;
  *bps = per;
  return (n_blocks + per - 1) / per;
}

int attn_splits(const uad_ctx *c, int B, int H, int P, int *bps) { return attn_splits_nb(c, B, H, (P + H + 31) / 32, bps); }

// Split-KV partial rows (x head_dim) that a call with B environments, chunk H
// and prefix P writes.
size_t attn_part_rows(const uad_ctx *c, int B, int H, int P) {
  int bps;
  const int sp = attn_splits(c, B, H, P, &bps);
  if (sp <= 1) return 0;
  const size_t rows_pad = (size_t)((c->Hq / c->Hkv) * H + 63) / 64 * 64;
  return (size_t)sp * B * c->Hkv * rows_pad;
}


// ---------------------------------------------------------------------------
// Scratch of the no-allocation step (uad_denoise_step_static): the split-KV
// partials live in this file-scope device array, one copy per GPU, held until
// the process ends.  Host code never passes the array's name to a kernel (on
// the host it is a stand-in, not a device address): uad_create looks up each
// device's address once, with that device current, and the entry point passes
// that address.  Calls that overlap on one GPU share the array and race.
// ---------------------------------------------------------------------------
constexpr size_t kStaticScratchBytes = (size_t)8 << 20;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];        // device address of `scratch` per device (null: not looked up)
hipError_t g_scratch_err[kMaxDevices];   // result of the failed lookup, reported by the entry point

// Once per device, with that device current: the device address of `scratch`.
hipError_t static_scratch_lookup(int device) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[device]) return hipSuccess;
  void *p = nullptr;
  hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  g_scratch_err[device] = e;
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  g_scratch_ptr[device] = p;
  return hipSuccess;
}

void *static_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  return g_scratch_ptr[device];
}

}  // namespace

extern "C" {

const char *uad_last_error(const uad_ctx *ctx) { return ctx ? ctx->err.c_str() : g_create_err.c_str(); }

uad_status uad_create(const uad_model_config *cfg, int32_t device, void *hip_stream, uad_ctx **out) {
  if (out) *out = nullptr;
  auto cerr = [](uad_status st, const std::string &m) {
    g_create_err = m;
    return st;
  };
  if (!cfg || !out) return cerr(UAD_E_INVALID, "uad_create: null cfg/out");
  const uad_model_config &m = *cfg;
  if (m.n_layers < 1 || m.d_model < 1 || m.n_heads < 1 || m.n_kv_heads < 1 || m.head_dim < 1 || m.d_ff < 1 ||
      m.action_dim < 1 || m.max_batch < 1 || m.max_chunk < 1 || m.max_prefix < 0 || !(m.rms_eps >= 0.f))
    return cerr(UAD_E_INVALID, "uad_create: every dimension must be positive");
  if ((m.flags & ~UAD_FLAG_ADARMS) != 0) return cerr(UAD_E_INVALID, "uad_create: unknown flags");
  if (m.d_model % 32 || m.d_ff % 32) return cerr(UAD_E_UNSUPPORTED, "uad_create: d_model and d_ff must be multiples of 32");
  if (m.head_dim != 64 && m.head_dim != 128 && m.head_dim != 256)
    return cerr(UAD_E_UNSUPPORTED, "uad_create: head_dim must be 64, 128 or 256");
  if (m.n_heads % m.n_kv_heads) return cerr(UAD_E_UNSUPPORTED, "uad_create: n_kv_heads must divide n_heads");
  if (m.action_dim > 64) return cerr(UAD_E_UNSUPPORTED, "uad_create: action_dim must be <= 64");
  if (m.d_model > 2048) return cerr(UAD_E_UNSUPPORTED, "uad_create: d_model must be <= 2048");

  hipError_t e = hipSetDevice(device);
  if (e != hipSuccess) return cerr(UAD_E_HIP, std::string("hipSetDevice: ") + hipGetErrorString(e));

  uad_ctx *c = new uad_ctx();
  c->cfg = m;
  c->device = device;
  e = hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, device);
  if (e != hipSuccess) {
    delete c;
    return cerr(UAD_E_HIP, std::string("hipDeviceGetAttribute: ") + hipGetErrorString(e));
  }
  c->d = m.d_model;
  c->L = m.n_layers;
  c->Hq = m.n_heads;
  c->Hkv = m.n_kv_heads;
  c->hd = m.head_dim;
  c->F = m.d_ff;
  c->Da = m.action_dim;
  c->q_dim = c->Hq * c->hd;
  c->kv_dim = c->Hkv * c->hd;
  c->n_qkv = c->q_dim + 2 * c->kv_dim;
  c->m_alloc = round_up(m.max_batch * m.max_chunk, 64);
  c->ada = (m.flags & UAD_FLAG_ADARMS) != 0;
  c->n_mod = c->ada ? m.n_layers * 6 * m.d_model + 2 * m.d_model : 0;
  c->s_alloc = round_up(m.max_prefix + m.max_chunk, 32);
  c->layers.resize(c->L);

  // the caller's stream; NULL is the device's null stream, so the library's
  // work is ordered with the caller's other work there (a separate stream
  // ordered by events around every call slowed the replayed step graphs by
  // ~14% at batch 1)
  c->stream = (hipStream_t)hip_stream;
  int rate_khz = 0;
  if (hipDeviceGetAttribute(&rate_khz, hipDeviceAttributeWallClockRate, device) == hipSuccess && rate_khz > 0)
    c->tick_hz = rate_khz * 1000.0;
  else
    c->tick_hz = 1e8;

  // weight store
  const int d = c->d, F = c->F, Da = c->Da;
  Carve w;
  size_t o_ain = w.take<float>((size_t)d * Da), o_ainb = w.take<float>(d), o_t1b = w.take<float>(d),
         o_t2b = w.take<float>(d), o_fn = w.take<float>(d), o_aout = w.take<float>((size_t)Da * d),
         o_aoutb = w.take<float>(Da), o_freq = w.take<float>(d / 2),
         o_t1 = w.take<uint16_t>((size_t)d * (c->ada ? d : 2 * d)), o_t2 = w.take<uint16_t>((size_t)d * d),
         o_wmod = w.take<uint16_t>((size_t)c->n_mod * d), o_bmod = w.take<float>(c->n_mod);
  std::vector<size_t> o_l(6 * c->L);
  for (int l = 0; l < c->L; ++l) {
    o_l[6 * l + 0] = w.take<uint16_t>((size_t)c->n_qkv * d);
    o_l[6 * l + 1] = w.take<uint16_t>((size_t)d * c->q_dim);
    o_l[6 * l + 2] = w.take<uint16_t>((size_t)2 * F * d);
    o_l[6 * l + 3] = w.take<uint16_t>((size_t)d * F);
    o_l[6 * l + 4] = w.take<float>(d);
    o_l[6 * l + 5] = w.take<float>(d);
  }
  c->wbytes = w.off;
  e = hipMalloc(&c->wbuf, c->wbytes);
  if (e != hipSuccess) {
    uad_destroy(c);
    return cerr(UAD_E_OOM, std::string("hipMalloc(weights): ") + hipGetErrorString(e));
  }
  char *wb = (char *)c->wbuf;
  c->action_in_w = (float *)(wb + o_ain);
  c->action_in_b = (float *)(wb + o_ainb);
  c->t1_b = (float *)(wb + o_t1b);
  c->t2_b = (float *)(wb + o_t2b);
  c->final_norm = (float *)(wb + o_fn);
  c->action_out_w = (float *)(wb + o_aout);
  c->action_out_b = (float *)(wb + o_aoutb);
  c->freqs = (float *)(wb + o_freq);
  c->t1_w = (op_t *)(wb + o_t1);
  c->t2_w = (op_t *)(wb + o_t2);
  c->w_mod = (op_t *)(wb + o_wmod);
  c->b_mod = (float *)(wb + o_bmod);
  for (int l = 0; l < c->L; ++l) {
    c->layers[l].wqkv = (const op_t *)(wb + o_l[6 * l + 0]);
    c->layers[l].wo = (const op_t *)(wb + o_l[6 * l + 1]);
    c->layers[l].wgu = (const op_t *)(wb + o_l[6 * l + 2]);
    c->layers[l].wdown = (const op_t *)(wb + o_l[6 * l + 3]);
    c->layers[l].attn_norm = (const float *)(wb + o_l[6 * l + 4]);
    c->layers[l].mlp_norm = (const float *)(wb + o_l[6 * l + 5]);
  }
  // time-embedding frequencies w_j = 1000 * 10000^(-j/(d/2)), computed in double
  {
    std::vector<float> fr(d / 2);
    for (int j = 0; j < d / 2; ++j) fr[j] = (float)(1000.0 * std::pow(10000.0, -(double)j / (double)(d / 2)));
    e = hipMemcpy(c->freqs, fr.data(), fr.size() * 4, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      uad_destroy(c);
      return cerr(UAD_E_HIP, std::string("hipMemcpy(freqs): ") + hipGetErrorString(e));
    }
  }

  // K / V^T store: [L][max_batch][Hkv][s_alloc][hd] and [L][max_batch][Hkv][s_alloc/32][hd][32]
  c->kv_layer_elems = (size_t)m.max_batch * c->Hkv * c->s_alloc * c->hd;
  const size_t kv_bytes = c->kv_layer_elems * c->L * 2;
  e = hipMalloc((void **)&c->kcache, kv_bytes);
  if (e == hipSuccess) e = hipMalloc((void **)&c->vtcache, kv_bytes);
  if (e == hipSuccess) e = hipMemset(c->kcache, 0, kv_bytes);
  if (e == hipSuccess) e = hipMemset(c->vtcache, 0, kv_bytes);
  if (e != hipSuccess) {
    uad_destroy(c);
    return cerr(UAD_E_OOM, std::string("hipMalloc(kv store): ") + hipGetErrorString(e));
  }

  // activation workspace (rows padded to 64 and zeroed so padded rows stay finite)
  // The split count is not monotone in the prefix length, so the partials are
  // sized for every (B, H, P) a later call may use; P enters only through the
  // number of 32-key blocks.
  size_t part = 0;
  for (int B = 1; B <= m.max_batch; ++B)
    for (int H = 1; H <= m.max_chunk; ++H)
      for (int nb = (H + 31) / 32; nb <= (m.max_prefix + H + 31) / 32; ++nb) {
        int bps;
        const int sp = attn_splits_nb(c, B, H, nb, &bps);
        if (sp > 1) {
          const size_t rows_pad = (size_t)((c->Hq / c->Hkv) * H + 63) / 64 * 64;
          part = std::max(part, (size_t)sp * B * c->Hkv * rows_pad);
        }
      }
  c->attn_part_elems = part;
  const size_t M = c->m_alloc;
  Carve a;
  // GEMM inputs (te, z, n, o, g) are fp16 in fragment order, M rows each;
  // ssq holds the per-16-column sums of squares of h (RMSNorm folded into the GEMMs)
  size_t o_h = a.take<float>(M * d), o_te = a.take<uint16_t>(M * 2 * d), o_z = a.take<uint16_t>(M * d),
         o_n = a.take<uint16_t>(M * d), o_o = a.take<uint16_t>(M * c->q_dim), o_g = a.take<uint16_t>(M * F),
         o_q = a.take<uint16_t>(M * c->q_dim), o_op = a.take<uint16_t>(std::max<size_t>(part, 1) * c->hd),
         o_ml = a.take<float>(std::max<size_t>(part, 1) * 2), o_ssq = a.take<float>((size_t)(d / 16) * M),
         o_trx0 = a.take<float>(M * Da), o_trv = a.take<float>(M * Da), o_trt = a.take<float>(kMaxTrSteps * M),
         o_trdt = a.take<float>(kMaxTrSteps * M), o_trm = a.take<uint8_t>(kMaxTrSteps * M),
         o_mod = a.take<float>(M * c->n_mod), o_mshift = a.take<uint16_t>(c->ada ? (size_t)2 * c->L * M * d : 0),
         o_pf = a.take<unsigned>(64), o_status = a.take<unsigned>(1),
         o_budt = a.take<float>(kMaxTrSteps * M), o_buddt = a.take<float>(kMaxTrSteps * M),
         o_budm = a.take<uint8_t>(kMaxTrSteps * M), o_budmap = a.take<int32_t>((size_t)kMaxTrSteps * m.max_batch),
         o_kxw = a.take<float>((size_t)2 * c->n_cu * kKxPartialFloats), o_kxc = a.take<unsigned>((size_t)c->n_cu);
  e = hipMalloc(&c->abuf, a.off);
  if (e == hipSuccess) e = hipMemset(c->abuf, 0, a.off);
  if (e != hipSuccess) {
    uad_destroy(c);
    return cerr(UAD_E_OOM, std::string("hipMalloc(workspace): ") + hipGetErrorString(e));
  }
  char *ab = (char *)c->abuf;
  c->h = (float *)(ab + o_h);
  c->a_te = (op_t *)(ab + o_te);
  c->a_z = (op_t *)(ab + o_z);
  c->a_n = (op_t *)(ab + o_n);
  c->a_o = (op_t *)(ab + o_o);
  c->a_g = (op_t *)(ab + o_g);
  c->q = (__bf16 *)(ab + o_q);
  c->attn_opart = (op_t *)(ab + o_op);
  c->attn_ml = (float *)(ab + o_ml);
  c->ssq = (float *)(ab + o_ssq);
  c->tr_x0 = (float *)(ab + o_trx0);
  c->tr_vsum = (float *)(ab + o_trv);
  c->tr_t = (float *)(ab + o_trt);
  c->tr_dt = (float *)(ab + o_trdt);
  c->tr_mask = (uint8_t *)(ab + o_trm);
  c->mod = (float *)(ab + o_mod);
  c->mod_shift_ops = (op_t *)(ab + o_mshift);
  c->pf_sink = (unsigned *)(ab + o_pf);
  c->status = (unsigned *)(ab + o_status);
  c->bud_t = (float *)(ab + o_budt);
  c->bud_dt = (float *)(ab + o_buddt);
  c->bud_mask = (uint8_t *)(ab + o_budm);
  c->bud_map = (int32_t *)(ab + o_budmap);
  c->kx_ws = (float *)(ab + o_kxw);
  c->kx_cnt = (unsigned *)(ab + o_kxc);
  c->kx_ws_bytes = (size_t)2 * c->n_cu * kKxPartialFloats * sizeof(float);
  e = attention_init();
  if (e == hipSuccess) e = gemm_init();
  // the no-allocation step's scratch: its address on this device (a failure is
  // reported by that entry point, the rest of the library does not need it)
  if (e == hipSuccess) (void)static_scratch_lookup(device);
  if (e != hipSuccess) {
    uad_destroy(c);
    return cerr(UAD_E_HIP, std::string("attention kernel set-up: ") + hipGetErrorString(e));
  }
  e = hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->rel_stream, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->ev_rel, hipEventDisableTiming);
  if (e != hipSuccess) {
    uad_destroy(c);
    return cerr(UAD_E_HIP, std::string("hipStreamCreate(capture/release): ") + hipGetErrorString(e));
  }
  *out = c;
  g_create_err.clear();
  return UAD_OK;
}

void uad_destroy(uad_ctx *c) {
  if (!c) return;
  (void)hipSetDevice(c->device);
  if (c->stream) (void)hipStreamSynchronize(c->stream);
  if (c->wbuf) (void)hipFree(c->wbuf);
  if (c->kcache) (void)hipFree(c->kcache);
  if (c->vtcache) (void)hipFree(c->vtcache);
  if (c->abuf) (void)hipFree(c->abuf);
  if (c->pre_buf) (void)hipFree(c->pre_buf);
  for (auto &r : c->prof_pending) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto ev : c->ev_pool) (void)hipEventDestroy(ev);
  for (auto &ge : c->graphs) (void)hipGraphExecDestroy(ge.exec);
  if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  if (c->rel_stream) {
    (void)hipStreamSynchronize(c->rel_stream);
    (void)hipStreamDestroy(c->rel_stream);
  }
  if (c->ev_rel) (void)hipEventDestroy(c->ev_rel);
  delete c;
}

uad_status uad_set_stream(uad_ctx *c, void *hip_stream) {
  if (!c) return UAD_E_INVALID;
  (void)hipSetDevice(c->device);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  c->stream = (hipStream_t)hip_stream;
  return UAD_OK;
}

uad_status uad_load_weights(uad_ctx *c, const uad_tensor *ts, int32_t n) {
  if (!c) return UAD_E_INVALID;
  if (!ts || n < 1) return fail(c, UAD_E_INVALID, "uad_load_weights: no tensors");
  (void)hipSetDevice(c->device);
  // queued steps may still read the weights being replaced
  hipError_t se = hipStreamSynchronize(c->stream);
  if (se != hipSuccess) return hip_fail(c, se, "uad_load_weights: hipStreamSynchronize");
  const int d = c->d, F = c->F, Da = c->Da;
  // required names and shapes
  std::map<std::string, std::vector<int64_t>> need;
  need["action_in.w"] = {d, Da};
  need["action_in.b"] = {d};
  need["time_mlp_in.w"] = {d, c->ada ? d : 2 * d};
  need["time_mlp_in.b"] = {d};
  need["time_mlp_out.w"] = {d, d};
  need["time_mlp_out.b"] = {d};
  if (c->ada) {
    need["final_mod.w"] = {2 * d, d};
    need["final_mod.b"] = {2 * d};
  } else {
    need["final_norm"] = {d};
  }
  need["action_out.w"] = {Da, d};
  need["action_out.b"] = {Da};
  for (int l = 0; l < c->L; ++l) {
    const std::string p = "layers." + std::to_string(l) + ".";
    if (c->ada) {
      need[p + "attn_mod.w"] = {3 * d, d};
      need[p + "attn_mod.b"] = {3 * d};
      need[p + "mlp_mod.w"] = {3 * d, d};
      need[p + "mlp_mod.b"] = {3 * d};
    } else {
      need[p + "attn_norm"] = {d};
      need[p + "mlp_norm"] = {d};
    }
    need[p + "wq"] = {c->q_dim, d};
    need[p + "wk"] = {c->kv_dim, d};
    need[p + "wv"] = {c->kv_dim, d};
    need[p + "wo"] = {d, c->q_dim};
    need[p + "w_gate"] = {F, d};
    need[p + "w_up"] = {F, d};
    need[p + "w_down"] = {d, F};
  }
  std::map<std::string, const uad_tensor *> got;
  for (int i = 0; i < n; ++i) {
    const uad_tensor &t = ts[i];
    if (!t.name || !t.data) return fail(c, UAD_E_INVALID, "uad_load_weights: tensor with null name or data");
    auto it = need.find(t.name);
    if (it == need.end()) return fail(c, UAD_E_MISSING, std::string("uad_load_weights: unknown tensor ") + t.name);
    if (got.count(t.name)) return fail(c, UAD_E_MISSING, std::string("uad_load_weights: duplicated tensor ") + t.name);
    if (t.dtype != UAD_DTYPE_F32 && t.dtype != UAD_DTYPE_BF16)
      return fail(c, UAD_E_INVALID, std::string("uad_load_weights: bad dtype for ") + t.name);
    const auto &shp = it->second;
    bool ok = t.ndim == (int)shp.size();
    for (size_t k = 0; ok && k < shp.size(); ++k) ok = t.shape[k] == shp[k];
    if (!ok) return fail(c, UAD_E_SHAPE, std::string("uad_load_weights: wrong shape for ") + t.name);
    got[t.name] = &t;
  }
  for (auto &kv : need)
    if (!got.count(kv.first)) return fail(c, UAD_E_MISSING, "uad_load_weights: missing tensor " + kv.first);

  std::string err;
  auto host = [&](const std::string &name, std::vector<float> *v) {
    const uad_tensor *t = got[name];
    size_t cnt = 1;
    for (int k = 0; k < t->ndim; ++k) cnt *= (size_t)t->shape[k];
    return fetch_f32(t->data, t->dtype, t->on_device, cnt, v, &err);
  };
  auto up = [&](void *dst, const void *src, size_t bytes) {
    hipError_t e = hipMemcpy(dst, src, bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) err = std::string("hipMemcpy(H2D): ") + hipGetErrorString(e);
    return e == hipSuccess;
  };
  std::vector<float> v1, v2, v3;
  std::vector<_Float16> pk;
  bool range_ok = true;  // every projection weight within the fp16 range
  auto put_f32 = [&](const std::string &name, float *dst) {
    return host(name, &v1) && up(dst, v1.data(), v1.size() * 4);
  };
  bool ok = put_f32("action_in.w", c->action_in_w) && put_f32("action_in.b", c->action_in_b) &&
            put_f32("time_mlp_in.b", c->t1_b) && put_f32("time_mlp_out.b", c->t2_b) &&
            (c->ada || put_f32("final_norm", c->final_norm)) && put_f32("action_out.w", c->action_out_w) &&
            put_f32("action_out.b", c->action_out_b);
  const int k_t1 = c->ada ? d : 2 * d;
  if (ok && (ok = host("time_mlp_in.w", &v1))) {
    pk.assign((size_t)d * k_t1, 0);
    range_ok &= pack_tiles(v1.data(), d, k_t1, pk.data(), 0, 1);
    ok = up(c->t1_w, pk.data(), pk.size() * 2);
  }
  if (ok && (ok = host("time_mlp_out.w", &v1))) {
    pk.assign((size_t)d * d, 0);
    range_ok &= pack_tiles(v1.data(), d, d, pk.data(), 0, 1);
    ok = up(c->t2_w, pk.data(), pk.size() * 2);
  }
  for (int l = 0; ok && l < c->L; ++l) {
    const std::string p = "layers." + std::to_string(l) + ".";
    uad_layer_ptrs &lp = c->layers[l];
    if (!c->ada) {
      ok = put_f32(p + "attn_norm", (float *)lp.attn_norm) && put_f32(p + "mlp_norm", (float *)lp.mlp_norm);
      if (!ok) break;
    }
    // fused QKV: tiles [q | k | v]
    pk.assign((size_t)c->n_qkv * d, 0);
    ok = host(p + "wq", &v1) && host(p + "wk", &v2) && host(p + "wv", &v3);
    if (!ok) break;
    range_ok &= pack_tiles(v1.data(), c->q_dim, d, pk.data(), 0, 1);
    range_ok &= pack_tiles(v2.data(), c->kv_dim, d, pk.data(), c->q_dim / kTileN, 1);
    range_ok &= pack_tiles(v3.data(), c->kv_dim, d, pk.data(), (c->q_dim + c->kv_dim) / kTileN, 1);
    ok = up((void *)lp.wqkv, pk.data(), pk.size() * 2);
    if (!ok) break;
    ok = host(p + "wo", &v1);
    if (!ok) break;
    pk.assign((size_t)d * c->q_dim, 0);
    range_ok &= pack_tiles(v1.data(), d, c->q_dim, pk.data(), 0, 1);
    ok = up((void *)lp.wo, pk.data(), pk.size() * 2);
    if (!ok) break;
    // gate/up interleaved per 16-column tile: tile 2j = gate j, tile 2j+1 = up j
    ok = host(p + "w_gate", &v1) && host(p + "w_up", &v2);
    if (!ok) break;
    pk.assign((size_t)2 * F * d, 0);
    range_ok &= pack_tiles(v1.data(), F, d, pk.data(), 0, 2);
    range_ok &= pack_tiles(v2.data(), F, d, pk.data(), 1, 2);
    ok = up((void *)lp.wgu, pk.data(), pk.size() * 2);
    if (!ok) break;
    ok = host(p + "w_down", &v1);
    if (!ok) break;
    pk.assign((size_t)d * F, 0);
    range_ok &= pack_tiles(v1.data(), d, F, pk.data(), 0, 1);
    ok = up((void *)lp.wdown, pk.data(), pk.size() * 2);
  }
  if (ok && c->ada) {
    // all modulations in one matrix [n_mod][d]: per layer (a, b, g) of the
    // attention norm, (a, b, g) of the MLP norm; then (a, b) of the final norm
    pk.assign((size_t)c->n_mod * d, 0);
    std::vector<float> bm(c->n_mod);
    const int per_layer_tiles = 6 * d / kTileN;
    for (int l = 0; ok && l < c->L; ++l) {
      const std::string p = "layers." + std::to_string(l) + ".";
      ok = host(p + "attn_mod.w", &v1) && host(p + "mlp_mod.w", &v2) && host(p + "attn_mod.b", &v3);
      if (!ok) break;
      range_ok &= pack_tiles(v1.data(), 3 * d, d, pk.data(), l * per_layer_tiles, 1);
      range_ok &= pack_tiles(v2.data(), 3 * d, d, pk.data(), l * per_layer_tiles + 3 * d / kTileN, 1);
      std::copy(v3.begin(), v3.end(), bm.begin() + (size_t)l * 6 * d);
      ok = host(p + "mlp_mod.b", &v3);
      if (!ok) break;
      std::copy(v3.begin(), v3.end(), bm.begin() + (size_t)l * 6 * d + 3 * d);
    }
    if (ok && (ok = host("final_mod.w", &v1) && host("final_mod.b", &v3))) {
      range_ok &= pack_tiles(v1.data(), 2 * d, d, pk.data(), c->L * per_layer_tiles, 1);
      std::copy(v3.begin(), v3.end(), bm.begin() + (size_t)c->L * 6 * d);
      ok = up(c->w_mod, pk.data(), pk.size() * 2) && up(c->b_mod, bm.data(), bm.size() * 4);
    }
  }
  if (!ok) {
    c->weights_loaded = false;
    return fail(c, UAD_E_HIP, "uad_load_weights: " + err);
  }
  if (!range_ok) {
    c->weights_loaded = false;
    return fail(c, UAD_E_INVALID, "uad_load_weights: a projection weight is NaN or beyond the fp16 range (|w| > 65504)");
  }
  c->weights_loaded = true;
  return UAD_OK;
}

uad_status uad_set_prefix_kv(uad_ctx *c, const void *k, const void *v, int32_t dtype, int32_t batch,
                             int32_t prefix_len, int32_t on_device) {
  if (!c) return UAD_E_INVALID;
  if (!k || !v) return fail(c, UAD_E_INVALID, "uad_set_prefix_kv: null k/v");
  if (dtype != UAD_DTYPE_F32 && dtype != UAD_DTYPE_BF16) return fail(c, UAD_E_INVALID, "uad_set_prefix_kv: bad dtype");
  if (batch < 1 || prefix_len < 0) return fail(c, UAD_E_INVALID, "uad_set_prefix_kv: batch must be >= 1, prefix_len >= 0");
  if (batch > c->cfg.max_batch) return fail(c, UAD_E_SHAPE, "uad_set_prefix_kv: batch > max_batch");
  if (prefix_len > c->cfg.max_prefix) return fail(c, UAD_E_SHAPE, "uad_set_prefix_kv: prefix_len > max_prefix");
  (void)hipSetDevice(c->device);
  // queued steps (a release's tail, say) may still read the K/V being replaced
  hipError_t se = hipStreamSynchronize(c->stream);
  if (se != hipSuccess) return hip_fail(c, se, "uad_set_prefix_kv: hipStreamSynchronize");
  const int L = c->L, Hkv = c->Hkv, hd = c->hd, P = prefix_len, S = c->s_alloc;
  const size_t per_layer_in = (size_t)batch * P * Hkv * hd;
  std::string err;
  std::vector<float> kf, vf;
  std::vector<uint16_t> ks((size_t)batch * Hkv * S * hd), vs((size_t)batch * Hkv * hd * S);
  const size_t esz = dtype == UAD_DTYPE_F32 ? 4 : 2;
  for (int l = 0; l < L; ++l) {
    if (!fetch_f32((const char *)k + l * per_layer_in * esz, dtype, on_device, per_layer_in, &kf, &err) ||
        !fetch_f32((const char *)v + l * per_layer_in * esz, dtype, on_device, per_layer_in, &vf, &err))
      return fail(c, UAD_E_HIP, "uad_set_prefix_kv: " + err);
    std::fill(ks.begin(), ks.end(), 0);
    std::fill(vs.begin(), vs.end(), 0);
    for (int b = 0; b < batch; ++b)
      for (int s = 0; s < P; ++s)
        for (int g = 0; g < Hkv; ++g)
          for (int cc = 0; cc < hd; ++cc) {
            const size_t src = (((size_t)b * P + s) * Hkv + g) * hd + cc;
            const size_t eh = (size_t)b * Hkv + g;
            ks[(eh * S + s) * hd + cc] = f32_to_bf16_rne(kf[src]);
            vs[vt_index(eh, s, cc, hd, S)] = f32_to_bf16_rne(vf[src]);
          }
    hipError_t e = hipMemcpy(c->kcache + l * c->kv_layer_elems, ks.data(), ks.size() * 2, hipMemcpyHostToDevice);
    if (e == hipSuccess)
      e = hipMemcpy(c->vtcache + l * c->kv_layer_elems, vs.data(), vs.size() * 2, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(c, e, "uad_set_prefix_kv: hipMemcpy");
  }
  c->prefix_len = P;
  c->prefix_batch = batch;
  c->prefix_set = true;
  return UAD_OK;
}

static uad_status check_step_args(uad_ctx *c, const void *x, const void *t, const void *dt, const void *mask,
                                  int B, int H, const char *fn) {
  if (!x || !t || !dt || !mask) return fail(c, UAD_E_INVALID, std::string(fn) + ": null x/t/dt/mask");
  if (B < 1 || H < 1) return fail(c, UAD_E_INVALID, std::string(fn) + ": batch and chunk must be >= 1");
  if (B > c->cfg.max_batch || H > c->cfg.max_chunk)
    return fail(c, UAD_E_SHAPE, std::string(fn) + ": batch/chunk beyond the context maxima");
  if (!c->dbg) {
    if (!c->weights_loaded) return fail(c, UAD_E_STATE, std::string(fn) + ": weights not loaded");
    if (!c->prefix_set) return fail(c, UAD_E_STATE, std::string(fn) + ": prefix K/V not set");
    if (B > c->prefix_batch) return fail(c, UAD_E_STATE, std::string(fn) + ": prefix set for fewer environments");
  }
  return UAD_OK;
}

// Enqueue one joint step on stream s: F_theta over all B*H tokens, then the
// masked Euler update.  Kernel sequence: temb -> time-MLP in -> time-MLP out
// (+ residual init, RMSNorm sums, next operand) -> per layer [QKV (x rstd) ->
// attention (+ split-KV combine) -> O (+ residual, sums, next operand) ->
// gate/up GeGLU (x rstd) -> down (+ residual, sums, next layer's operand)] ->
// final norm/projection/Euler.
// A step's slice of the schedule-level conditioning (modulations and shift
// operands computed for every step up front), or per-step conditioning when null.
struct AdaSlice {
  const float *mod;        // [m_alloc][n_mod] rows of this step
  const op_t *shift;       // layer 0's attention shift operand of this step
  size_t shift_stride;     // elements from one [layer][norm] shift operand to the next
};

// Split-KV partials of a step in caller-chosen memory instead of the context's
// workspace (the no-allocation entry point), and no measurement events.
struct StepScratch {
  op_t *opart;
  float *mlpart;
};

static uad_status enqueue_step(uad_ctx *c, hipStream_t s, float *x, const float *t, const float *dt,
                               const uint8_t *mask, const uint8_t *next_mask, int is_last, int step, float *v_out,
                               float *released, int32_t *release_step, int B, int H, float *vsum = nullptr,
                               int vsum_tokens = 0, const AdaSlice *pre = nullptr,
                               const StepScratch *scratch = nullptr, const int32_t *env_map = nullptr) {
  const int M = B * H, d = c->d, F = c->F;
  const size_t MA = c->m_alloc;
  const bool prof = c->prof_on && !scratch;
  hipError_t e = hipSuccess;
  // measurement hook: the launch records a start/stop event pair taken from
  // the kernel's own dispatch packet (ea_/eb_ are nullptr when not profiling)
#define UAD_CHECK_CLS(cls, call)                       \
  do {                                                 \
    hipEvent_t ea_ = nullptr, eb_ = nullptr;           \
    if (prof) {                                        \
      ea_ = pool_event(c);                             \
      eb_ = pool_event(c);                             \
    }                                                  \
    e = (call);                                        \
    if (e != hipSuccess) return hip_fail(c, e, #call); \
    if (prof) c->prof_pending.push_back({cls, ea_, eb_}); \
  } while (0)
  if (!c->dbg) {
    // RMSNorm folding: residual GEMMs write ssq and the next operand; consumers scale by rstd
    auto norm_fields = [&](GemmArgs &x) {
      x.ssq = c->ssq; x.ssq_tiles = d / 16; x.m_alloc = (int)MA; x.eps = c->cfg.rms_eps;
      x.kx_ws = c->kx_ws; x.kx_cnt = c->kx_cnt; x.kx_ws_bytes = c->kx_ws_bytes; x.kx_tiles = c->n_cu;
    };
    const int n_mod = c->n_mod;
    if (!c->ada) {
      UAD_CHECK_CLS(K_TEMB, launch_temb(x, t, M, c->Da, d, c->action_in_w, c->action_in_b, c->freqs, c->a_te, c->status, s,
                                        ea_, eb_, env_map, H));
      GemmArgs g{};
      g.status = c->status;
      g.M = M; g.m_alloc = (int)MA;
      g.A = c->a_te; g.W = c->t1_w; g.N = d; g.K = 2 * d;
      g.out = c->a_z; g.ldo = d; g.bias = c->t1_b;
      UAD_CHECK_CLS(K_GEMM_TIME_IN, launch_gemm(EPI_BIAS_SILU, g, plan_gemm(EPI_BIAS_SILU, M, d, 2 * d), s, ea_, eb_));
      GemmArgs g2{};
      g2.status = c->status;
      g2.M = M; g2.A = c->a_z; g2.W = c->t2_w; g2.N = d; g2.K = d;
      g2.out = c->h; g2.ldo = d; g2.bias = c->t2_b; norm_fields(g2);
      g2.gain_next = c->layers[0].attn_norm; g2.next = c->a_n;
      UAD_CHECK_CLS(K_GEMM_TIME_OUT, launch_gemm(EPI_RESID_F32, g2, plan_gemm(EPI_RESID_F32, M, d, d), s, ea_, eb_));
    } else if (pre) {
      // conditioning computed for the whole schedule: h_0 = W_in x + b_in and the
      // first attention norm's operand h_0 (1 + a) from this step's modulations
      UAD_CHECK_CLS(K_TEMB, launch_temb_ada(x, nullptr, M, c->Da, d, c->action_in_w, c->action_in_b, c->freqs,
                                            c->a_te, c->h, c->ssq, (int)MA, c->status, s, ea_, eb_, pre->mod, n_mod,
                                            c->a_n));
    } else {
      // adaptive norms: h_0 = W_in x + b_in, c = SiLU(W2 SiLU(W1 e(t) + b1) + b2), then every
      // modulation (a, b, g per norm site) in one GEMM whose epilogue also forms the
      // first attention norm's operand h_0 * (1 + a)
      UAD_CHECK_CLS(K_TEMB, launch_temb_ada(x, t, M, c->Da, d, c->action_in_w, c->action_in_b, c->freqs, c->a_te,
                                            c->h, c->ssq, (int)MA, c->status, s, ea_, eb_));
      GemmArgs g{};
      g.status = c->status;
      g.M = M; g.m_alloc = (int)MA; g.A = c->a_te; g.W = c->t1_w; g.N = d; g.K = d; g.out = c->a_z; g.ldo = d;
      g.bias = c->t1_b;
      UAD_CHECK_CLS(K_GEMM_TIME_IN, launch_gemm(EPI_BIAS_SILU, g, plan_gemm(EPI_BIAS_SILU, M, d, d), s, ea_, eb_));
      GemmArgs g2{};
      g2.status = c->status;
      g2.M = M; g2.m_alloc = (int)MA; g2.A = c->a_z; g2.W = c->t2_w; g2.N = d; g2.K = d; g2.out = c->a_te;
      g2.ldo = d; g2.bias = c->t2_b;
      UAD_CHECK_CLS(K_GEMM_TIME_OUT, launch_gemm(EPI_BIAS_SILU, g2, plan_gemm(EPI_BIAS_SILU, M, d, d), s, ea_, eb_));
      GemmArgs gm{};
      gm.status = c->status;
      gm.M = M; gm.m_alloc = (int)MA; gm.A = c->a_te; gm.W = c->w_mod; gm.N = n_mod; gm.K = d; gm.out = c->mod; gm.ldo = n_mod;
      gm.bias = c->b_mod; gm.mod_shift_ops = c->mod_shift_ops; gm.shift_stride = MA * d; gm.h_in = c->h;
      gm.d_model = d; gm.n_layers = c->L; gm.next = c->a_n;
      UAD_CHECK_CLS(K_GEMM_MOD, launch_gemm(EPI_MOD, gm, plan_gemm(EPI_MOD, M, n_mod, d), s, ea_, eb_));
    }

    AttnArgs at{};
    at.status = c->status;
    at.env_map = env_map;
    at.q = c->q; at.ldq = c->q_dim; at.s_alloc = c->s_alloc; at.n_keys = c->prefix_len + H;
    at.chunk = H; at.n_heads = c->Hq; at.n_kv_heads = c->Hkv; at.group = c->Hq / c->Hkv;
    at.rows = at.group * H; at.rows_pad = (at.rows + 63) / 64 * 64;
    at.splits = attn_splits(c, B, H, c->prefix_len, &at.blocks_per_split);
    if (!scratch && attn_part_rows(c, B, H, c->prefix_len) > c->attn_part_elems)
      return fail(c, UAD_E_SHAPE, "split-KV partials exceed the workspace sized at uad_create");
    at.qblocks = (at.rows + 63) / 64; at.n_eh = B * c->Hkv;
    at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)c->hd));
    at.o = c->a_o; at.ldo = c->q_dim;
    at.opart = scratch ? scratch->opart : c->attn_opart;
    at.mlpart = scratch ? scratch->mlpart : c->attn_ml;
    at.pf_sink = c->pf_sink;
    // Weight prefetch on otherwise idle CUs: when the attention leaves CUs free
    // (batch 1), its extra workgroups read the layer's O and gate/up weights and
    // the split merge's extra slice reads the down weights and the next
    // layer's QKV weights, so those projections stream them from the
    // memory-side cache instead of HBM.
    const int attn_wgs = 8 * ((at.n_eh * at.splits + 7) / 8) * at.qblocks;
    const int spare_cus = c->n_cu - attn_wgs;

    const GemmPlan pq = plan_gemm(EPI_QKV, M, c->n_qkv, d);
    const GemmPlan po = plan_gemm(EPI_RESID_F32, M, d, c->q_dim);
    const GemmPlan pg = plan_gemm(EPI_GEGLU, M, 2 * F, d);
    const GemmPlan pd = plan_gemm(EPI_RESID_F32, M, d, F);
    for (int l = 0; l < c->L; ++l) {
      const uad_layer_ptrs &lp = c->layers[l];
      __bf16 *kc = c->kcache + l * c->kv_layer_elems;
      __bf16 *vtc = c->vtcache + l * c->kv_layer_elems;
      GemmArgs q{};
      q.status = c->status;
      q.M = M; q.A = c->a_n; q.W = lp.wqkv; q.N = c->n_qkv; q.K = d;
      q.out = c->q; q.ldo = c->q_dim; q.kc = kc; q.vtc = vtc; q.chunk = H; q.prefix = c->prefix_len;
      q.s_alloc = c->s_alloc; q.n_kv_heads = c->Hkv; q.head_dim = c->hd; q.q_dim = c->q_dim;
      q.env_map = env_map;
      norm_fields(q); q.use_rstd = 1;
      const float *mod_base = pre ? pre->mod : c->mod;
      const op_t *shift_base = pre ? pre->shift : c->mod_shift_ops;
      const size_t shift_stride = pre ? pre->shift_stride : MA * d;
      if (c->ada) q.A2 = shift_base + (size_t)(2 * l) * shift_stride;
      UAD_CHECK_CLS(K_GEMM_QKV, launch_gemm(EPI_QKV, q, pq, s, ea_, eb_));
      at.kc = kc; at.vtc = vtc;
      at.pre_attn = Prefetch{};
      at.pre_comb = Prefetch{};
      if (spare_cus >= kReadAheadMinCus) {
        at.pre_attn.p[0] = (const char *)lp.wo;
        at.pre_attn.bytes[0] = (uint32_t)((size_t)d * c->q_dim * sizeof(op_t));
        at.pre_attn.p[1] = (const char *)lp.wgu;
        at.pre_attn.bytes[1] = (uint32_t)((size_t)2 * F * d * sizeof(op_t));
        at.pre_attn.wgs = spare_cus;
        if (at.splits > 1) {
          at.pre_comb.p[0] = (const char *)lp.wdown;
          at.pre_comb.bytes[0] = (uint32_t)((size_t)d * F * sizeof(op_t));
          at.pre_comb.p[1] = (const char *)c->layers[(l + 1) % c->L].wqkv;
          at.pre_comb.bytes[1] = (uint32_t)((size_t)c->n_qkv * d * sizeof(op_t));
          at.pre_comb.wgs = 1;
        }
      }
      UAD_CHECK_CLS(K_ATTENTION, launch_attention(at, B, c->hd, s, ea_, eb_));
      GemmArgs o{};
      o.status = c->status;
      o.M = M; o.A = c->a_o; o.W = lp.wo; o.N = d; o.K = c->q_dim;
      o.out = c->h; o.ldo = d; norm_fields(o);
      o.gain_next = lp.mlp_norm; o.next = c->a_n;
      if (c->ada) {
        const float *ml = mod_base + (size_t)l * 6 * d;
        o.mod_ld = n_mod; o.mod_gate = ml + 2 * d; o.mod_scale_next = ml + 3 * d; o.gain_next = nullptr;
      }
      UAD_CHECK_CLS(K_GEMM_O, launch_gemm(EPI_RESID_F32, o, po, s, ea_, eb_));
      GemmArgs gu{};
      gu.status = c->status;
      gu.M = M; gu.A = c->a_n; gu.W = lp.wgu; gu.N = 2 * F; gu.K = d;
      gu.out = c->a_g; gu.ldo = F; norm_fields(gu); gu.use_rstd = 1;
      if (c->ada) gu.A2 = shift_base + (size_t)(2 * l + 1) * shift_stride;
      UAD_CHECK_CLS(K_GEMM_GATEUP, launch_gemm(EPI_GEGLU, gu, pg, s, ea_, eb_));
      GemmArgs dn{};
      dn.status = c->status;
      dn.M = M; dn.A = c->a_g; dn.W = lp.wdown; dn.N = d; dn.K = F;
      dn.out = c->h; dn.ldo = d; norm_fields(dn);
      dn.gain_next = (l + 1 < c->L) ? c->layers[l + 1].attn_norm : nullptr; dn.next = c->a_n;
      if (c->ada) {
        const float *ml = mod_base + (size_t)l * 6 * d;
        dn.mod_ld = n_mod; dn.mod_gate = ml + 5 * d; dn.gain_next = nullptr;
        dn.mod_scale_next = (l + 1 < c->L) ? ml + 6 * d : nullptr;
      }
      UAD_CHECK_CLS(K_GEMM_DOWN, launch_gemm(EPI_RESID_F32, dn, pd, s, ea_, eb_));
    }
  }
  FinalArgs f{};
  f.h = c->h; f.gain = c->final_norm; f.w_out = c->action_out_w; f.b_out = c->action_out_b; f.eps = c->cfg.rms_eps;
  f.M = M; f.d = d; f.Da = c->Da; f.x = x; f.t = t; f.dt = dt; f.mask = mask; f.next_mask = next_mask;
  f.is_last_step = is_last; f.step = step; f.v_out = v_out; f.released = released; f.release_step = release_step;
  f.debug_field = c->dbg ? 1 : 0; f.dbg_alpha = c->dbg_alpha; f.dbg_beta = c->dbg_beta;
  f.vsum = vsum; f.vsum_tokens = vsum_tokens; f.chunk = H; f.env_map = env_map;
  if (c->ada) {
    f.mod_scale = (pre ? pre->mod : c->mod) + (size_t)c->L * 6 * d; f.mod_shift = f.mod_scale + d;
    f.mod_ld = c->n_mod;
  }
  UAD_CHECK_CLS(K_FINAL, launch_final(f, s, ea_, eb_));
#undef UAD_CHECK_CLS
  return UAD_OK;
}

// Schedule-level conditioning applies to small batches (projections bound by
// the weight stream, where the modulation matrix would be read once per step)
// when the buffers for n_steps x m_alloc rows are in place.
static bool ada_schedule_level(const uad_ctx *c, size_t M, int n_steps) {
  return c->ada && !c->dbg && M <= 256 && (size_t)n_steps * c->m_alloc <= c->pre_rows;
}

// Grow the schedule-level conditioning buffers to `rows` rows (no-op when they
// hold enough, or beyond a 2 GiB budget: the schedule then conditions per step).
// Captured graphs reference the old buffers and are dropped.
static void ensure_ada_rows(uad_ctx *c, size_t rows) {
  if (rows <= c->pre_rows) return;
  // a caller capturing the context stream into a graph of its own: no
  // synchronisation or allocation now (the schedule conditions per step)
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(c->stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
    (void)hipGetLastError();
    return;
  }
  const size_t d = c->d;
  Carve a;
  const size_t o_te = a.take<uint16_t>(rows * d), o_z = a.take<uint16_t>(rows * d),
               o_mod = a.take<float>(rows * c->n_mod), o_sh = a.take<uint16_t>((size_t)2 * c->L * rows * d);
  if (a.off > ((size_t)2 << 30)) return;
  if (hipStreamSynchronize(c->stream) != hipSuccess) return;  // queued work may use the old buffers
  for (auto &ge : c->graphs) (void)hipGraphExecDestroy(ge.exec);
  c->graphs.clear();
  if (c->pre_buf) (void)hipFree(c->pre_buf);
  c->pre_buf = nullptr;
  c->pre_rows = 0;
  if (hipMalloc(&c->pre_buf, a.off) != hipSuccess) {
    (void)hipGetLastError();
    c->pre_buf = nullptr;
    return;
  }
  char *b = (char *)c->pre_buf;
  c->pre_te = (op_t *)(b + o_te);
  c->pre_z = (op_t *)(b + o_z);
  c->pre_mod = (float *)(b + o_mod);
  c->pre_shift = (op_t *)(b + o_sh);
  c->pre_rows = rows;
}

// The time conditioning of every step of a schedule: time features of its
// n_steps x m_alloc rows, time MLP, and all modulations in one GEMM (the first
// attention norm's operand needs h_0 and is formed per step).
static uad_status enqueue_ada_schedule(uad_ctx *c, hipStream_t s, const GraphKey &k) {
  const int d = c->d, rows = k.n_steps * (int)c->m_alloc;
  const int M = k.B * k.H;
  hipError_t e = hipSuccess;
#define UAD_PRE_CLS(cls, call)                         \
  do {                                                 \
    hipEvent_t ea_ = nullptr, eb_ = nullptr;           \
    if (c->prof_on) {                                  \
      ea_ = pool_event(c);                             \
      eb_ = pool_event(c);                             \
    }                                                  \
    e = (call);                                        \
    if (e != hipSuccess) return hip_fail(c, e, #call); \
    if (c->prof_on) c->prof_pending.push_back({cls, ea_, eb_}); \
  } while (0)
  e = launch_time_features(k.t, M, (int)c->m_alloc, k.n_steps, d, c->freqs, c->pre_te, c->status, s);
  if (e != hipSuccess) return hip_fail(c, e, "launch_time_features");
  GemmArgs g{};
  g.status = c->status;
  g.M = rows; g.m_alloc = rows; g.A = c->pre_te; g.W = c->t1_w; g.N = d; g.K = d; g.out = c->pre_z; g.ldo = d;
  g.bias = c->t1_b;
  UAD_PRE_CLS(K_GEMM_TIME_IN, launch_gemm(EPI_BIAS_SILU, g, plan_gemm(EPI_BIAS_SILU, rows, d, d), s, ea_, eb_));
  GemmArgs g2{};
  g2.status = c->status;
  g2.M = rows; g2.m_alloc = rows; g2.A = c->pre_z; g2.W = c->t2_w; g2.N = d; g2.K = d; g2.out = c->pre_te;
  g2.ldo = d; g2.bias = c->t2_b;
  UAD_PRE_CLS(K_GEMM_TIME_OUT, launch_gemm(EPI_BIAS_SILU, g2, plan_gemm(EPI_BIAS_SILU, rows, d, d), s, ea_, eb_));
  GemmArgs gm{};
  gm.status = c->status;
  gm.M = rows; gm.m_alloc = rows; gm.A = c->pre_te; gm.W = c->w_mod; gm.N = c->n_mod; gm.K = d; gm.out = c->pre_mod;
  gm.ldo = c->n_mod; gm.bias = c->b_mod; gm.mod_shift_ops = c->pre_shift; gm.shift_stride = (size_t)rows * d;
  gm.h_in = nullptr; gm.next = nullptr; gm.d_model = d; gm.n_layers = c->L;
  UAD_PRE_CLS(K_GEMM_MOD, launch_gemm(EPI_MOD, gm, plan_gemm(EPI_MOD, rows, c->n_mod, d), s, ea_, eb_));
#undef UAD_PRE_CLS
  return UAD_OK;
}

// Enqueue a whole schedule (or one step when t etc. are single slices) on s.
static uad_status enqueue_schedule(uad_ctx *c, hipStream_t s, const GraphKey &k) {
  const size_t M = (size_t)k.B * k.H;
  if (k.step_ticks) {
    hipError_t e = launch_stamp(k.step_ticks, s);
    if (e != hipSuccess) return hip_fail(c, e, "launch_stamp");
  }
  const bool pre = ada_schedule_level(c, M, k.n_steps);
  if (pre) {
    uad_status rs = enqueue_ada_schedule(c, s, k);
    if (rs != UAD_OK) return rs;
  }
  for (int st = 0; st < k.n_steps; ++st) {
    const bool last = k.is_schedule ? st == k.n_steps - 1 : false;
    const uint8_t *next = (k.is_schedule && !last) ? k.mask + (st + 1) * M : nullptr;
    AdaSlice sl{};
    if (pre) {
      sl.mod = c->pre_mod + (size_t)st * c->m_alloc * c->n_mod;
      sl.shift = c->pre_shift + (size_t)st * c->m_alloc * c->d;
      sl.shift_stride = (size_t)k.n_steps * c->m_alloc * c->d;
    }
    uad_status rs = enqueue_step(c, s, k.x, k.t + st * M, k.dt + st * M, k.mask + st * M, next, last ? 1 : 0, st,
                                 k.v_out, k.released, k.release_step, k.B, k.H, nullptr, 0, pre ? &sl : nullptr);
    if (rs != UAD_OK) return rs;
    if (k.step_ticks) {
      hipError_t e = launch_stamp(k.step_ticks + st + 1, s);
      if (e != hipSuccess) return hip_fail(c, e, "launch_stamp");
    }
  }
  return UAD_OK;
}

// The two phases of an urgency-aware release (Sec. 4.2-4.4) on stream s.
// Phase 1: keep x_0, steps 0 .. K-1 (urgent tokens on step 1/K, velocity sums
// kept for TR), then release the urgent actions and reconcile their states.
// Phase 2: steps K .. N*-1, then Ghost Action Correction of the tail.
static uad_status enqueue_release_phase(uad_ctx *c, hipStream_t s, const GraphKey &k) {
  const size_t M = (size_t)k.B * k.H;
  TrArgs a{};
  a.x = k.x; a.x0 = c->tr_x0; a.vsum = c->tr_vsum; a.urgent = k.urgent; a.executed = k.executed;
  a.gac_mask = k.gac_mask; a.B = k.B; a.H = k.H; a.Da = c->Da; a.U = k.U; a.S = k.S;
  a.urgent_host = k.kind == 1 ? k.urgent_host : nullptr;
  a.dt_star = -(1.0f / (float)k.Nstar); a.reconcile = k.reconcile;
  hipError_t e = hipSuccess;
  const int st0 = k.kind == 1 ? 0 : k.Kr, st1 = k.kind == 1 ? k.Kr : k.Nstar;
  // schedule-level conditioning: phase 1 computes it for all N* steps (the same
  // rows, kernels and values as a uniform N*-step schedule), phase 2 reads it
  const bool pre = ada_schedule_level(c, M, k.Nstar);
  if (k.kind == 1) {
    if (k.step_ticks && (e = launch_stamp(k.step_ticks, s)) != hipSuccess) return hip_fail(c, e, "launch_stamp");
    if ((e = launch_tr_init(a, s)) != hipSuccess) return hip_fail(c, e, "launch_tr_init");
    if (pre) {
      GraphKey kt = k;
      kt.t = c->tr_t;
      kt.n_steps = k.Nstar;
      uad_status rs = enqueue_ada_schedule(c, s, kt);
      if (rs != UAD_OK) return rs;
    }
  }
  for (int st = st0; st < st1; ++st) {
    AdaSlice sl{};
    if (pre) {
      sl.mod = c->pre_mod + (size_t)st * c->m_alloc * c->n_mod;
      sl.shift = c->pre_shift + (size_t)st * c->m_alloc * c->d;
      sl.shift_stride = (size_t)k.Nstar * c->m_alloc * c->d;
    }
    uad_status rs = enqueue_step(c, s, k.x, c->tr_t + st * M, c->tr_dt + st * M, c->tr_mask + st * M, nullptr, 0, st,
                                 nullptr, nullptr, nullptr, k.B, k.H, k.kind == 1 && k.reconcile ? c->tr_vsum : nullptr,
                                 k.U, pre ? &sl : nullptr);
    if (rs != UAD_OK) return rs;
    if (k.step_ticks && (e = launch_stamp(k.step_ticks + st + 1, s)) != hipSuccess)
      return hip_fail(c, e, "launch_stamp");
  }
  if (k.kind == 1 && (e = launch_tr_release(a, s)) != hipSuccess) return hip_fail(c, e, "launch_tr_release");
  if (k.kind == 2 && k.executed && (e = launch_gac(a, s)) != hipSuccess) return hip_fail(c, e, "launch_gac");
  return UAD_OK;
}

// A schedule from budgets (uad_denoise_budgets) on stream s: at step k only
// the k.active[k] environments that still have an active token are evaluated,
// their ascending list at bud_map + k * max_batch; the step tables are the
// library's own (bud_t, bud_dt, bud_mask, [n_steps][B][H]).
static uad_status enqueue_budgets(uad_ctx *c, hipStream_t s, const GraphKey &k) {
  const size_t M = (size_t)k.B * k.H;
  hipError_t e = hipSuccess;
  if (k.step_ticks && (e = launch_stamp(k.step_ticks, s)) != hipSuccess) return hip_fail(c, e, "launch_stamp");
  for (int st = 0; st < k.n_steps; ++st) {
    const bool last = st == k.n_steps - 1;
    const uint8_t *next = last ? nullptr : c->bud_mask + (st + 1) * M;
    const int Bk = k.active[st];
    const int32_t *map = Bk < k.B ? c->bud_map + (size_t)st * c->cfg.max_batch : nullptr;
    uad_status rs = enqueue_step(c, s, k.x, c->bud_t + st * M, c->bud_dt + st * M, c->bud_mask + st * M, next,
                                 last ? 1 : 0, st, nullptr, k.released, k.release_step, Bk, k.H, nullptr, 0, nullptr,
                                 nullptr, map);
    if (rs != UAD_OK) return rs;
    if (k.step_ticks && (e = launch_stamp(k.step_ticks + st + 1, s)) != hipSuccess)
      return hip_fail(c, e, "launch_stamp");
  }
  return UAD_OK;
}

static uad_status enqueue_work(uad_ctx *c, hipStream_t s, const GraphKey &k) {
  if (k.kind == 3) return enqueue_budgets(c, s, k);
  return k.kind == 0 ? enqueue_schedule(c, s, k) : enqueue_release_phase(c, s, k);
}

// Run the work described by k: replay a cached hipGraph of it when possible
// (one graph launch for the whole schedule), else capture one; direct launches
// while profiling or in the synthetic-velocity test mode.
static uad_status run_work(uad_ctx *c, GraphKey k) {
  k.prefix_len = c->prefix_len;
  k.prefix_batch = c->prefix_batch;
  // the measurement hook and the synthetic-velocity test mode launch directly
  if (c->dbg || c->graph_broken || c->prof_on) return enqueue_work(c, c->stream, k);
  ++c->graph_clock;
  uad_ctx::GraphEntry *hit = nullptr;
  for (auto &ge : c->graphs)
    if (ge.key == k) hit = &ge;
  if (!hit) {
    hipError_t e = hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      c->graph_broken = true;
      return enqueue_work(c, c->stream, k);
    }
    uad_status rs = enqueue_work(c, c->cap_stream, k);
    hipGraph_t graph = nullptr;
    e = hipStreamEndCapture(c->cap_stream, &graph);
    if (rs != UAD_OK) {
      if (graph) (void)hipGraphDestroy(graph);
      return rs;
    }
    hipGraphExec_t exec = nullptr;
    if (e == hipSuccess) e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    if (graph) (void)hipGraphDestroy(graph);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      c->graph_broken = true;
      return enqueue_work(c, c->stream, k);
    }
    if (c->graphs.size() >= 8) {  // evict the least recently used graph
      size_t lru = 0;
      for (size_t i = 1; i < c->graphs.size(); ++i)
        if (c->graphs[i].last_use < c->graphs[lru].last_use) lru = i;
      (void)hipGraphExecDestroy(c->graphs[lru].exec);
      c->graphs.erase(c->graphs.begin() + lru);
    }
    c->graphs.push_back({k, exec, c->graph_clock});
    hit = &c->graphs.back();
  }
  hit->last_use = c->graph_clock;
  hipError_t e = hipGraphLaunch(hit->exec, c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipGraphLaunch");
  return UAD_OK;
}

uad_status uad_denoise_step(uad_ctx *c, float *x, const float *t, const float *dt, const uint8_t *mask,
                            float *v_out, int32_t batch, int32_t chunk) {
  if (!c) return UAD_E_INVALID;
  uad_status st = check_step_args(c, x, t, dt, mask, batch, chunk, "uad_denoise_step");
  if (st != UAD_OK) return st;
  (void)hipSetDevice(c->device);
  GraphKey k{};
  k.kind = 0;
  k.is_schedule = false;
  k.x = x; k.t = t; k.dt = dt; k.mask = mask; k.v_out = v_out; k.n_steps = 1; k.B = batch; k.H = chunk;
  return run_work(c, k);
}

uad_status uad_denoise_step_static(uad_ctx *c, float *x, const float *t, const float *dt, const uint8_t *mask,
                                   float *v_out, int32_t batch, int32_t chunk) {
  if (!c) return UAD_E_INVALID;
  const char *fn = "uad_denoise_step_static";
  uad_status st = check_step_args(c, x, t, dt, mask, batch, chunk, fn);
  if (st != UAD_OK) return st;
  (void)hipSetDevice(c->device);
  char *base = (char *)static_scratch(c->device);
  if (!base)
    return fail(c, UAD_E_HIP, std::string(fn) + ": hipGetSymbolAddress(scratch) failed on this device: " +
                                  (c->device < kMaxDevices ? hipGetErrorString(g_scratch_err[c->device])
                                                           : "device index beyond the lookup table"));
  const size_t rows = attn_part_rows(c, batch, chunk, c->prefix_len);
  const size_t o_bytes = align256(rows * c->hd * sizeof(op_t));
  const size_t need = o_bytes + rows * 2 * sizeof(float);
  if (need > kStaticScratchBytes)
    return fail(c, UAD_E_SHAPE, std::string(fn) + ": this batch, chunk and prefix need " + std::to_string(need) +
                                    " bytes of split-KV scratch; the static array holds " +
                                    std::to_string(kStaticScratchBytes));
  const StepScratch sc{(op_t *)base, (float *)(base + o_bytes)};
  // direct launches on the context stream: no graph capture or instantiation
  return enqueue_step(c, c->stream, x, t, dt, mask, nullptr, 0, 0, v_out, nullptr, nullptr, batch, chunk, nullptr, 0,
                      nullptr, &sc);
}

uad_status uad_denoise_schedule(uad_ctx *c, float *x, const float *t_sched, const float *dt_sched,
                                const uint8_t *mask_sched, int32_t n_steps, int32_t batch, int32_t chunk,
                                float *released, int32_t *release_step, uint64_t *step_ticks) {
  if (!c) return UAD_E_INVALID;
  uad_status st = check_step_args(c, x, t_sched, dt_sched, mask_sched, batch, chunk, "uad_denoise_schedule");
  if (st != UAD_OK) return st;
  if (n_steps < 1) return fail(c, UAD_E_INVALID, "uad_denoise_schedule: n_steps must be >= 1");
  (void)hipSetDevice(c->device);
  if (c->ada && !c->dbg && (size_t)batch * chunk <= 256) ensure_ada_rows(c, (size_t)n_steps * c->m_alloc);
  GraphKey k{};
  k.kind = 0;
  k.is_schedule = true;
  k.x = x; k.t = t_sched; k.dt = dt_sched; k.mask = mask_sched; k.n_steps = n_steps; k.B = batch; k.H = chunk;
  k.released = released; k.release_step = release_step; k.step_ticks = step_ticks;
  return run_work(c, k);
}

uad_status uad_denoise_budgets(uad_ctx *c, float *x, const int32_t *budgets, int32_t batch, int32_t chunk,
                               float *released, int32_t *release_step, uint64_t *step_ticks) {
  if (!c) return UAD_E_INVALID;
  const std::string fn = "uad_denoise_budgets";
  if (!x || !budgets) return fail(c, UAD_E_INVALID, fn + ": null x/budgets");
  if (batch < 1 || chunk < 1) return fail(c, UAD_E_INVALID, fn + ": batch and chunk must be >= 1");
  if (batch > c->cfg.max_batch || chunk > c->cfg.max_chunk)
    return fail(c, UAD_E_SHAPE, fn + ": batch/chunk beyond the context maxima");
  if (!c->dbg) {
    if (!c->weights_loaded) return fail(c, UAD_E_STATE, fn + ": weights not loaded");
    if (!c->prefix_set) return fail(c, UAD_E_STATE, fn + ": prefix K/V not set");
    if (batch > c->prefix_batch) return fail(c, UAD_E_STATE, fn + ": prefix set for fewer environments");
  }
  (void)hipSetDevice(c->device);
  const size_t M = (size_t)batch * chunk;
  // tables and per-step environment lists, rebuilt when the budgets change
  std::vector<int32_t> key;
  key.reserve(2 + M);
  key.push_back(batch);
  key.push_back(chunk);
  key.insert(key.end(), budgets, budgets + M);
  if (key != c->bud_key) {
    std::vector<float> t(kMaxTrSteps * M), dt(kMaxTrSteps * M);
    std::vector<uint8_t> mk(kMaxTrSteps * M);
    int32_t n = 0;
    std::string err;
    if (!build_schedule_host(budgets, batch, chunk, kMaxTrSteps, &n, t.data(), dt.data(), mk.data(), &err))
      return fail(c, UAD_E_INVALID, fn + ": " + err + " (budgets must lie in 1..64)");
    // environment b has an active token at step k while its largest budget exceeds k
    const int maxb = c->cfg.max_batch;
    std::vector<int32_t> map((size_t)n * maxb, 0);
    std::vector<uint16_t> act(n);
    for (int k = 0; k < n; ++k) {
      int cnt = 0;
      for (int b = 0; b < batch; ++b) {
        int nb = 0;
        for (int i = 0; i < chunk; ++i) nb = std::max(nb, budgets[(size_t)b * chunk + i]);
        if (nb > k || c->ada) map[(size_t)k * maxb + cnt++] = b;  // adaptive norm: every environment
      }
      act[k] = (uint16_t)cnt;
    }
    hipError_t e = hipStreamSynchronize(c->stream);  // queued work may read the previous tables
    if (e == hipSuccess) e = hipMemcpy(c->bud_t, t.data(), n * M * sizeof(float), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(c->bud_dt, dt.data(), n * M * sizeof(float), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(c->bud_mask, mk.data(), n * M, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(c->bud_map, map.data(), map.size() * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      c->bud_key.clear();
      return hip_fail(c, e, "uad_denoise_budgets: step tables");
    }
    c->bud_key = key;
    c->bud_active = act;
  }
  GraphKey k{};
  k.kind = 3;
  k.x = x; k.B = batch; k.H = chunk; k.n_steps = (int)c->bud_active.size();
  k.released = released; k.release_step = release_step; k.step_ticks = step_ticks;
  for (int i = 0; i < k.n_steps; ++i) k.active[i] = c->bud_active[i];
  return run_work(c, k);
}

uad_status uad_denoise_release(uad_ctx *c, float *x, int32_t batch, int32_t chunk, int32_t U, int32_t K,
                               int32_t Nstar, int32_t S, int32_t mode, float *urgent_out, float *executed_out,
                               const uint8_t *gac_mask, float *urgent_host, void *release_event,
                               uint64_t *step_ticks) {
  if (!c) return UAD_E_INVALID;
  const char *fn = "uad_denoise_release";
  if (!x || !urgent_out) return fail(c, UAD_E_INVALID, std::string(fn) + ": null x/urgent_out");
  if (batch < 1 || chunk < 1) return fail(c, UAD_E_INVALID, std::string(fn) + ": batch and chunk must be >= 1");
  if (batch > c->cfg.max_batch || chunk > c->cfg.max_chunk)
    return fail(c, UAD_E_SHAPE, std::string(fn) + ": batch/chunk beyond the context maxima");
  if (mode != UAD_RELEASE_UAER && mode != UAD_RELEASE_TR) return fail(c, UAD_E_INVALID, std::string(fn) + ": bad mode");
  if (!(1 <= K && K < Nstar && Nstar <= kMaxTrSteps))
    return fail(c, UAD_E_INVALID, std::string(fn) + ": need 1 <= K < N* <= 64");
  if (!(1 <= U && U < S && S <= chunk)) return fail(c, UAD_E_INVALID, std::string(fn) + ": need 1 <= U < S <= chunk");
  if (executed_out && mode != UAD_RELEASE_TR)
    return fail(c, UAD_E_INVALID, std::string(fn) + ": Ghost Action Correction needs Trajectory Reconciliation");
  if (!c->dbg) {
    if (!c->weights_loaded) return fail(c, UAD_E_STATE, std::string(fn) + ": weights not loaded");
    if (!c->prefix_set) return fail(c, UAD_E_STATE, std::string(fn) + ": prefix K/V not set");
    if (batch > c->prefix_batch) return fail(c, UAD_E_STATE, std::string(fn) + ": prefix set for fewer environments");
  }
  (void)hipSetDevice(c->device);
  const int reconcile = mode == UAD_RELEASE_TR ? 1 : 0;
  const size_t M = (size_t)batch * chunk;
  // step tables: steps < K from the budgets (K urgent, N* tail); later steps from
  // the uniform N* schedule with TR, else from the budgets (urgent frozen)
  const int key[6] = {batch, chunk, U, K, Nstar, reconcile};
  if (!std::equal(key, key + 6, c->tr_key)) {
    std::vector<int32_t> bud(M, Nstar), uni(M, Nstar);
    for (int b = 0; b < batch; ++b)
      for (int i = 0; i < U; ++i) bud[(size_t)b * chunk + i] = K;
    std::vector<float> t1(Nstar * M), d1(Nstar * M), t2(Nstar * M), d2(Nstar * M);
    std::vector<uint8_t> m1(Nstar * M), m2(Nstar * M);
    int32_t n1 = 0, n2 = 0;
    std::string err;
    if (!build_schedule_host(bud.data(), batch, chunk, Nstar, &n1, t1.data(), d1.data(), m1.data(), &err) ||
        !build_schedule_host(uni.data(), batch, chunk, Nstar, &n2, t2.data(), d2.data(), m2.data(), &err))
      return fail(c, UAD_E_INVALID, std::string(fn) + ": " + err);
    if (reconcile) {
      std::copy(t2.begin() + K * M, t2.end(), t1.begin() + K * M);
      std::copy(d2.begin() + K * M, d2.end(), d1.begin() + K * M);
      std::copy(m2.begin() + K * M, m2.end(), m1.begin() + K * M);
    }
    // the tables may be in use by queued work of the previous configuration
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e == hipSuccess) e = hipMemcpy(c->tr_t, t1.data(), Nstar * M * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(c->tr_dt, d1.data(), Nstar * M * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(c->tr_mask, m1.data(), Nstar * M, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(c, e, "uad_denoise_release: step tables");
    std::copy(key, key + 6, c->tr_key);
  }
  // Pinned urgent_host: the release kernel writes it through its device
  // address (a cross-stream copy after the release cost ~90 us of the time to
  // first release at batch 1); other host memory is copied on the release stream.
  // (looked up on every call: a freed pinned buffer's address may come back as pageable memory)
  float *host_dev = nullptr;
  if (urgent_host) {
    hipPointerAttribute_t pa{};
    if (hipPointerGetAttributes(&pa, urgent_host) == hipSuccess && pa.type == hipMemoryTypeHost && pa.devicePointer)
      host_dev = (float *)pa.devicePointer;
    (void)hipGetLastError();  // pageable memory: the query's error is expected
  }
  if (c->ada && !c->dbg && M <= 256) ensure_ada_rows(c, (size_t)Nstar * c->m_alloc);
  GraphKey k{};
  k.kind = 1;
  k.x = x; k.B = batch; k.H = chunk; k.n_steps = Nstar; k.step_ticks = step_ticks;
  k.U = U; k.Kr = K; k.Nstar = Nstar; k.S = S; k.reconcile = reconcile;
  k.urgent = urgent_out; k.executed = executed_out; k.gac_mask = gac_mask; k.urgent_host = host_dev;
  uad_status rs = run_work(c, k);
  if (rs != UAD_OK) return rs;
  // release: the urgent actions (and their pinned host copy) are final here;
  // a pageable host buffer gets its copy on the release stream while the
  // tail continues on the context stream
  hipError_t e = hipEventRecord(c->ev_rel, c->stream);
  if (e == hipSuccess && urgent_host && !host_dev) {
    e = hipStreamWaitEvent(c->rel_stream, c->ev_rel, 0);
    if (e == hipSuccess)
      e = hipMemcpyAsync(urgent_host, urgent_out, (size_t)batch * U * c->Da * sizeof(float), hipMemcpyDeviceToHost,
                         c->rel_stream);
    if (e == hipSuccess && release_event) e = hipEventRecord((hipEvent_t)release_event, c->rel_stream);
  } else if (e == hipSuccess && release_event) {
    e = hipEventRecord((hipEvent_t)release_event, c->stream);
  }
  if (e != hipSuccess) return hip_fail(c, e, "uad_denoise_release: release");
  k.kind = 2;
  k.urgent_host = nullptr;
  return run_work(c, k);
}

uad_status uad_synchronize(uad_ctx *c) {
  if (!c) return UAD_E_INVALID;
  (void)hipSetDevice(c->device);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  // the device status word of the work just finished (read, then cleared)
  unsigned w = 0;
  e = hipMemcpy(&w, c->status, sizeof(w), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(c, e, "uad_synchronize: status word");
  if (w == 0) return UAD_OK;
  e = hipMemset(c->status, 0, sizeof(w));
  if (e != hipSuccess) return hip_fail(c, e, "uad_synchronize: status word");
  if (w & kStatusTimeout)
    return fail(c, UAD_E_HIP, "uad_synchronize: an in-kernel wait gave up (results of that work are invalid)");
  return fail(c, UAD_E_RANGE,
              "uad_synchronize: an fp16 GEMM / attention operand was not finite (|value| > 65504 or NaN); "
              "results of that work are invalid");
}

uad_status uad_tick_rate_hz(uad_ctx *c, double *hz) {
  if (!c || !hz) return UAD_E_INVALID;
  *hz = c->tick_hz;
  return UAD_OK;
}

uad_status uad_debug_velocity_field(uad_ctx *c, int32_t enable, float alpha, float beta) {
  if (!c) return UAD_E_INVALID;
  c->dbg = enable != 0;
  c->dbg_alpha = alpha;
  c->dbg_beta = beta;
  return UAD_OK;
}

uad_status uad_profile_enable(uad_ctx *c, int32_t enable) {
  if (!c) return UAD_E_INVALID;
  (void)hipSetDevice(c->device);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  for (auto &r : c->prof_pending) {
    c->ev_pool.push_back(r.a);
    c->ev_pool.push_back(r.b);
  }
  c->prof_pending.clear();
  c->prof_ms.assign(K_NCLASS, 0.0);
  c->prof_n.assign(K_NCLASS, 0);
  c->prof_on = enable != 0;
  return UAD_OK;
}

uad_status uad_profile_read(uad_ctx *c, int32_t index, char *name, int32_t name_cap, double *total_ms,
                            int64_t *launches) {
  if (!c) return UAD_E_INVALID;
  if (index < 0 || index >= K_NCLASS) return fail(c, UAD_E_INVALID, "uad_profile_read: index out of range");
  (void)hipSetDevice(c->device);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  if (c->prof_ms.size() != K_NCLASS) {
    c->prof_ms.assign(K_NCLASS, 0.0);
    c->prof_n.assign(K_NCLASS, 0);
  }
  for (auto &r : c->prof_pending) {
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventElapsedTime");
    c->prof_ms[r.cls] += ms;
    c->prof_n[r.cls] += 1;
    c->ev_pool.push_back(r.a);
    c->ev_pool.push_back(r.b);
  }
  c->prof_pending.clear();
  if (name && name_cap > 0) {
    std::strncpy(name, kClassNames[index], name_cap - 1);
    name[name_cap - 1] = 0;
  }
  if (total_ms) *total_ms = c->prof_ms[index];
  if (launches) *launches = c->prof_n[index];
  return UAD_OK;
}

uad_status uad_build_schedule(const int32_t *budgets, int32_t batch, int32_t chunk, int32_t max_steps,
                              int32_t *n_steps, float *t, float *dt, uint8_t *mask) {
  std::string err;
  return build_schedule_host(budgets, batch, chunk, max_steps, n_steps, t, dt, mask, &err) ? UAD_OK
                                                                                           : UAD_E_INVALID;
}

}  // extern "C"
