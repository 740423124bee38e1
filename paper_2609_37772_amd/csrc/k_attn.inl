// Joint attention of the chunk's queries over [cached prefix ; chunk] keys.
//
// Every action token attends to all P prefix tokens and all H chunk tokens
// (no mask), query head j reading KV head floor(j*Hkv/Hq).  The grouped query
// heads of one KV head are packed into the row dimension (row r = head-in-group
// * H + token), so one K/V tile read serves all of them.
//
// Per workgroup: one (environment, KV head), 64 packed query rows (4 waves x
// 16), and a contiguous range of 32-key blocks (split-KV when the batch is
// small).  Keys are processed in chunks of NB blocks: a chunk's K and V^T
// tiles go straight from global memory into LDS (LDS-direct loads, shared by
// the 4 waves, double buffered), all issued at once, and the next chunk's
// loads are in flight while a chunk is used, so a split of at most NB blocks
// costs one memory round trip.
// Each wave computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16 so that a
// lane ends up holding 8 scores of ONE query, which are exactly the 8 k-values
// of its operand for the P V product: no transpose through LDS.  Softmax
// statistics are reduced across the 4 lanes that share a query with
// wavefront shuffles (online softmax, fp32, exp2 domain, accumulators
// rescaled only when the running max moves by more than 2^8).  With split-KV the
// unnormalised partial outputs and (max, sum) pairs are merged in fixed split
// order by attn_combine_kernel.
#include "uad_internal.h"

namespace uad {

// One 32-key block in LDS, filled by LDS-direct global loads (16 bytes per
// lane, lane-linear placement) and read as MFMA fragments.  Rows are stored
// unpadded with their 16-byte chunks XOR-swizzled so that the 8 lanes served
// per LDS cycle hit distinct banks:
//   K:   32 keys x HD,  chunk j of key row r stored at chunk j ^ (r & 7);
//   V^T: HD x 32 keys (permuted, see vt_index), chunk g of column row c
//        stored at chunk g ^ ((c >> 1) & 3).
template <int HD>
struct AttnBlock {
  __bf16 k[32 * HD];
  __bf16 vt[HD * 32];
};

// Softmax rescaling threshold (log2 domain): the running max of a query is
// only raised when a block's max exceeds it by more than this, so most blocks
// skip rescaling the accumulators; probabilities stay <= 2^8.
constexpr float kRescaleThreshold = 8.0f;

// Blocks per chunk (one memory round trip); two chunks are resident (double
// buffer), 2 * NB * 32 * HD * 4 bytes of LDS.
template <int HD>
constexpr int attn_chunk_blocks() {
  return HD == 256 ? 2 : 4;
}

// Blocks per stage of the tall batched workgroups (6-8 waves): the waves
// meet once per stage.  Same-machine A/B per launch: HD = 128 (2048 tokens x 1152
// keys) 33.2 -> 32.4 us with 2 blocks (4 blocks: 33.2); HD = 256 (3200 tokens x
// 866 keys) 45.3 -> 46.2 us with 2, so one there.
template <int HD>
constexpr int attn_tall_blocks() {
  return HD == 256 ? 1 : 2;
}

typedef __attribute__((address_space(3))) void lds_void;


// Workgroup wg of pf.wgs reads its 4 KiB-aligned share of the prefetch ranges
// (16 bytes per lane per load, 8 loads in flight per lane: measured best of
// 4 / 8 / 16 at batch 1, where fewer ran past the attention workgroups and
// more slowed their own loads); what it read is
// folded into one word that is stored only on an impossible match, which
// keeps the loads from being removed.
__device__ __forceinline__ void prefetch_share(const Prefetch &pf, int wg, unsigned *sink) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const uint32_t total = pf.bytes[0] + pf.bytes[1];
  const uint32_t per = ((total + pf.wgs - 1) / pf.wgs + 4095u) & ~4095u;
  const uint32_t beg = (uint32_t)wg * per, end = min(beg + per, total);
  const uint32_t stride = blockDim.x * 16;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (uint32_t off0 = beg + threadIdx.x * 16; off0 < end; off0 += 8 * stride) {
    u32x4 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t off = min(off0 + i * stride, end - 16);
      const char *src = off < pf.bytes[0] ? pf.p[0] + off : pf.p[1] + (off - pf.bytes[0]);
      v[i] = *(const u32x4 *)src;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) acc ^= v[i];
  }
  const unsigned w = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (w == 0x9e3779b9u && threadIdx.x == 0 && wg == 0) *sink = w;
}

// LOWREG: the K fragments of each 16-key half and the V fragments of each
// half of the output columns are read just before their MFMAs (fewer live
// registers: two waves per SIMD at HD = 256) instead of all up front.
// NW waves (16 query rows each) per workgroup; NW > 4 only without split-KV
// (a.qblocks counts blocks of 16 * NW rows).
template <int HD, int NB, bool LOWREG, int NW>
__global__ __launch_bounds__(64 * NW) void attn_kernel(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char attn_smem[];
  AttnBlock<HD> *bufs = (AttnBlock<HD> *)attn_smem;  // [2][NB]
  constexpr int KS = HD / 32;   // k-steps of the QK^T product
  constexpr int NTO = HD / 16;  // 16-column output tiles
  constexpr int CPR = HD / 8;   // 16-byte chunks per K row
  constexpr int TI = HD / 16;   // LDS-direct instructions (64 lanes x 16 B) per K or V^T tile
  constexpr int INS = (TI + NW - 1) / NW;  // per wave, the last ones guarded
  if ((int)blockIdx.x >= (int)gridDim.x - a.pre_attn.wgs) {  // prefetch workgroups follow the attention ones
    prefetch_share(a.pre_attn, blockIdx.x - (gridDim.x - a.pre_attn.wgs), a.pf_sink);
    return;
  }
  const int lane = threadIdx.x & 63;
  // the batched variants take the wave index through readfirstlane (scalar
  // per-wave addressing; 64 environments 39.7 -> 39.0 us)
  const int wave = LOWREG ? __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) : threadIdx.x >> 6;
  // XCD-aware placement: the query blocks of one (environment-head, split)
  // group read the same K/V tiles, so the group's workgroups get ids on one
  // XCD (workgroup i runs on XCD i % 8) and share its L2; groups are dealt
  // round-robin over the 8 XCDs.
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int rgrp = slot / a.qblocks, qblock = slot - rgrp * a.qblocks;
  const int grp = xcd + 8 * rgrp;
  if (grp >= a.n_eh * a.splits) return;  // padding of the last round (whole workgroup)
  const int eh = grp / a.splits;  // env * Hkv + kv head
  const int split = grp - eh * a.splits;
  const int b = eh / a.n_kv_heads;
  const int g = eh - b * a.n_kv_heads;
  // K/V store slot of this environment (compacted steps run a subset)
  const int ehkv = (a.env_map ? a.env_map[b] : b) * a.n_kv_heads + g;

  const __bf16 *kbase = a.kc + (size_t)ehkv * a.s_alloc * HD;
  const __bf16 *vbase = a.vtc + vt_index(ehkv, 0, 0, HD, a.s_alloc);

  const int n_blocks = (a.n_keys + 31) / 32;
  const int blk0 = split * a.blocks_per_split;
  int blk1 = blk0 + a.blocks_per_split;
  if (blk1 > n_blocks) blk1 = n_blocks;

  // This lane's query (as the B operand of S^T): packed row r0 + (lane & 15).
  const int r0 = qblock * (16 * NW) + wave * 16;
  const int my_r = r0 + (lane & 15);
  bf16x8 qf[KS];
  {
    const bool ok = my_r < a.rows;
    const int hg = ok ? my_r / a.chunk : 0;
    const int tok = ok ? my_r - hg * a.chunk : 0;
    const int head = g * a.group + hg;
    const __bf16 *qp = a.q + (size_t)(b * a.chunk + tok) * a.ldq + head * HD + (lane >> 4) * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = ok ? *(const bf16x8 *)(qp + ks * 32) : bf16x8{};
  }

  // LDS-direct loads of the chunk starting at block c0 into buffer set `which`
  // (blocks past the split's end re-read its last block; never used).
  auto issue = [&](int c0, int which) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int blk = min(c0 + j, blk1 - 1);
      AttnBlock<HD> &dst = bufs[which * NB + j];
      const __bf16 *kb = kbase + (size_t)blk * 32 * HD;
      const __bf16 *vb = vbase + (size_t)blk * 32 * HD;
      // wave w issues the contiguous instructions [w*TI/NW, (w+1)*TI/NW)
      const int ins0 = wave * TI / NW, ins1 = (wave + 1) * TI / NW;
#pragma unroll
      for (int i = 0; i < INS; ++i) {
        if (TI % NW != 0 && ins0 + i >= ins1) break;  // wave-uniform
        const int q0 = (ins0 + i) * 64;  // first LDS chunk of this instruction
        const int q = q0 + lane;
        const int kr = q / CPR, kp = q - kr * CPR;
        __builtin_amdgcn_global_load_lds((const void *)(kb + kr * HD + ((kp ^ (kr & 7)) * 8)),
                                         (lds_void *)(dst.k + q0 * 8), 16, 0, 0);
        const int vr = q >> 2, vp = q & 3;
        __builtin_amdgcn_global_load_lds((const void *)(vb + vr * 32 + ((vp ^ ((vr >> 1) & 3)) * 8)),
                                         (lds_void *)(dst.vt + q0 * 8), 16, 0, 0);
      }
    }
  };
  if (blk0 < blk1) issue(blk0, 0);

  f32x4 o[NTO];
#pragma unroll
  for (int nt = 0; nt < NTO; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // reference max (log2 domain) of query (lane & 15), within 2^8 of the true max
  float l_run = 0.f;        // this lane's partial sum of exp2

  int which = 0;
  for (int c0 = blk0; c0 < blk1; c0 += NB, which ^= 1) {
    const int nb = min(NB, blk1 - c0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this chunk's LDS-direct loads (and q) landed
    __syncthreads();  // ... for every wave; the other buffer set is free again
    if (c0 + NB < blk1) issue(c0 + NB, which ^ 1);

#pragma nounroll
    for (int j = 0; j < nb; ++j) {
      const AttnBlock<HD> &blk = bufs[which * NB + j];
      const int k0 = (c0 + j) * 32;
      // S^T for two 16-key halves: s[h][r] = score(query lane&15, key k0+16h+4(lane>>4)+r).
      // All K and V fragments of the block are read up front.
      f32x4 s[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
      bf16x8 vf[LOWREG ? 1 : NTO];
      if constexpr (LOWREG) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int row = 16 * h + (lane & 15);
          bf16x8 kf1[KS];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            kf1[ks] = *(const bf16x8 *)&blk.k[row * HD + (((ks * 4 + (lane >> 4)) ^ (row & 7)) * 8)];
          __builtin_amdgcn_sched_barrier(0);  // all reads of the half issued before its MFMAs
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf1[ks], qf[ks], s[h], 0, 0, 0);
        }
      } else {
        bf16x8 kf[2][KS];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int row = 16 * h + (lane & 15);
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            kf[h][ks] = *(const bf16x8 *)&blk.k[row * HD + (((ks * 4 + (lane >> 4)) ^ (row & 7)) * 8)];
        }
#pragma unroll
        for (int nt = 0; nt < NTO; ++nt) {
          const int c = nt * 16 + (lane & 15);
          vf[nt] = *(const bf16x8 *)&blk.vt[c * 32 + (((lane >> 4) ^ ((c >> 1) & 3)) * 8)];
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int h = 0; h < 2; ++h) s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[h][ks], qf[ks], s[h], 0, 0, 0);
      }
      // raw scores; keys past the end (last block only) masked to -inf; the
      // scale (> 0) is applied to the block max and folded into exp2's FMA
      if (k0 + 32 > a.n_keys) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (k0 + 16 * h + (lane >> 4) * 4 + r >= a.n_keys) s[h][r] = -INFINITY;
      }
      float mloc = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                         fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
      mloc = max_pair32(max_pair16(mloc)) * a.scale_log2;
      // lazy rescale: raise the running max only past the threshold (whole wave)
      if (__any(mloc > m_run + kRescaleThreshold)) {
        const float m_new = fmaxf(m_run, mloc);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // arguments <= 0
        m_run = m_new;
        l_run *= alpha;
        // output rows (row 4*(lane>>4)+r of the tile) take their query's alpha
        float al[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) al[r] = __shfl(alpha, (lane >> 4) * 4 + r);
#pragma unroll
        for (int nt = 0; nt < NTO; ++nt)
#pragma unroll
          for (int r = 0; r < 4; ++r) o[nt][r] *= al[r];
      }
      float psum = 0.f;
      bf16x8 pf;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[h][r], a.scale_log2, -m_run));
          psum += p;
          pf[h * 4 + r] = (__bf16)p;
        }
      l_run += psum;
      // O += P V : B operand lane l = V[keys of pf][col 16nt + (l&15)]
      if constexpr (LOWREG) {
        constexpr int HALF = NTO / 2;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          bf16x8 vf1[HALF];
#pragma unroll
          for (int q = 0; q < HALF; ++q) {
            const int c = (hh * HALF + q) * 16 + (lane & 15);
            vf1[q] = *(const bf16x8 *)&blk.vt[c * 32 + (((lane >> 4) ^ ((c >> 1) & 3)) * 8)];
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int q = 0; q < HALF; ++q)
            o[hh * HALF + q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf, vf1[q], o[hh * HALF + q], 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int nt = 0; nt < NTO; ++nt) o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf, vf[nt], o[nt], 0, 0, 0);
      }
    }
  }

  const float l_tot = sum_pair32(sum_pair16(l_run));

  // Output rows of this lane: r0 + 4*(lane>>4) + r, column 16*nt + (lane&15)
  float lr[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) lr[r] = __shfl(l_tot, (lane >> 4) * 4 + r);
  unsigned bad = 0;  // fp16 range flag of this lane's stores
  if (a.splits == 1) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = r0 + (lane >> 4) * 4 + r;
      if (row >= a.rows) continue;
      const int hg = row / a.chunk, tok = row - hg * a.chunk;
      const int head = g * a.group + hg;
      const int orow = b * a.chunk + tok;
      const float inv = 1.0f / lr[r];
#pragma unroll
      for (int nt = 0; nt < NTO; ++nt)
        store_op(a.o + afrag_index(orow, head * HD + nt * 16 + (lane & 15), a.ldo / kTileK), o[nt][r] * inv, bad);
    }
    flush_range(a.status, bad);
  } else {
    // Partials o_s / l_s in fp16 (bounded by max |V|), in the accumulator's
    // own layout: per 16-row tile, [nt][lane][4] (one 8-byte store per lane and
    // column tile), and (m, l) per row in fp32.
    const size_t tile = ((size_t)split * a.n_eh + eh) * (a.rows_pad / 16) + (r0 >> 4);
    op_t *op = a.opart + tile * (16 * HD) + lane * 4;
    float inv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) inv[r] = 1.0f / lr[r];
#pragma unroll
    for (int nt = 0; nt < NTO; ++nt) {
      const float p0 = o[nt][0] * inv[0], p1 = o[nt][1] * inv[1], p2 = o[nt][2] * inv[2], p3 = o[nt][3] * inv[3];
      *(f16x4 *)(op + nt * 256) = f16x4{(op_t)p0, (op_t)p1, (op_t)p2, (op_t)p3};
      check_op4(p0, p1, p2, p3, bad);
    }
    // lanes 0..15 hold the statistics of their own query row r0 + lane
    if (lane < 16) *(float2 *)(a.mlpart + (tile * 16 + lane) * 2) = float2{m_run, l_tot};
    flush_range(a.status, bad);
  }
}

// Merge split-KV partials: with o_s = O_s / l_s stored,
// o = sum_s 2^(m_s - M) l_s o_s / sum_s 2^(m_s - M) l_s, splits in fixed order.  One wave per (16-row tile, 16-column tile): lane l
// owns the float4 of the accumulator layout (rows 4*(l>>4)..+3, column l&15)
// and reads the (m, l) pairs of its 4 rows itself, so all loads are issued
// up front and the merge needs no LDS or barrier.  W waves per workgroup take
// W neighbouring column tiles.
template <int SMAX, int W>
__global__ __launch_bounds__(64 * W) void attn_combine_kernel(AttnArgs a, int hd) {
  const int rt = blockIdx.x;                                               // 16-row tile
  const int nt = blockIdx.y * W + (W > 1 ? (int)(threadIdx.x >> 6) : 0);  // 16-column tile
  const int eh = blockIdx.z;
  const int n_eh = a.n_eh;
  if (eh >= n_eh) {  // the extra slice prefetches
    prefetch_share(a.pre_comb, blockIdx.y * gridDim.x + blockIdx.x, a.pf_sink);
    return;
  }
  const int b = eh / a.n_kv_heads, g = eh - b * a.n_kv_heads;
  const int splits = a.splits;
  const int ntiles = a.rows_pad / 16;
  const int lane = threadIdx.x & 63;
  const int rbase = (lane >> 4) * 4;
  unsigned bad = 0;  // fp16 range flag of this lane's stores
  f16x4 os[SMAX];
  float2 ml[SMAX][4];
#pragma unroll
  for (int sp = 0; sp < SMAX; ++sp) {
    const size_t tile = ((size_t)min(sp, splits - 1) * n_eh + eh) * ntiles + rt;
    const f16x4 ov = *(const f16x4 *)(a.opart + tile * (16 * (size_t)hd) + nt * 256 + lane * 4);
    os[sp] = sp < splits ? ov : f16x4{};
    // the (m, l) pairs of this lane's 4 rows are 32 contiguous bytes: two 16-byte loads
    const f32x4 *mp = (const f32x4 *)(a.mlpart + (tile * 16 + rbase) * 2);
    const f32x4 v01 = mp[0], v23 = mp[1];
    const bool ok = sp < splits;
    ml[sp][0] = ok ? float2{v01[0], v01[1]} : float2{-INFINITY, 0.f};
    ml[sp][1] = ok ? float2{v01[2], v01[3]} : float2{-INFINITY, 0.f};
    ml[sp][2] = ok ? float2{v23[0], v23[1]} : float2{-INFINITY, 0.f};
    ml[sp][3] = ok ? float2{v23[2], v23[3]} : float2{-INFINITY, 0.f};
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float M = -INFINITY;
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) M = fmaxf(M, ml[sp][r].x);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) {
      const float w = sp < splits ? __builtin_amdgcn_exp2f(ml[sp][r].x - M) * ml[sp][r].y : 0.f;
      num += w * (float)os[sp][r];
      den += w;
    }
    const int row = rt * 16 + rbase + r;
    if (row >= a.rows) continue;
    const int hg = row / a.chunk, tok = row - hg * a.chunk;
    const int head = g * a.group + hg;
    store_op(a.o + afrag_index(b * a.chunk + tok, head * hd + nt * 16 + (lane & 15), a.ldo / kTileK), num / den,
             bad);
  }
  flush_range(a.status, bad);
}

static int g_attn_cus = 256;  // compute units of the device (set by attention_init)

template <int HD>
static hipError_t launch_hd(const AttnArgs &a, int batch, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  constexpr int NB = attn_chunk_blocks<HD>();
  if (a.qblocks != (a.rows + 63) / 64 || a.n_eh != batch * a.n_kv_heads) return hipErrorInvalidValue;
  const int groups = a.n_eh * a.splits;
  if (a.pre_attn.wgs < 0 || a.pre_comb.wgs < 0 || ((a.pre_attn.wgs || a.pre_comb.wgs) && !a.pf_sink))
    return hipErrorInvalidValue;
  dim3 grid(8 * ((groups + 7) / 8) * a.qblocks + a.pre_attn.wgs);
  hipEvent_t end_attn = a.splits == 1 ? ev1 : nullptr;
  // Long splits (batched steps, one split per query block): one 32-key block
  // per stage and K/V fragments streamed in halves, so that two workgroups
  // (8 waves) share a CU and hide each other's LDS reads and softmax; short
  // splits (batch 1): NB blocks per stage, one memory round trip per split.
  const bool streamed = a.blocks_per_split > 2 * NB;
  const uint32_t lds = (uint32_t)(2 * (streamed ? 1 : NB) * sizeof(AttnBlock<HD>));
  if (streamed && a.splits == 1 && a.pre_attn.wgs == 0) {
    // Without split-KV every workgroup of a group re-reads the group's whole
    // K/V, so fewer, taller query blocks cut that traffic; 4-wave workgroups
    // run two per CU, 6- and 8-wave ones one.  Take the row block that gives
    // the fewest 16-row tasks on the busiest CU, then the fewest workgroups.
    int best_nw = 4, best_load = 0, best_wgs = 0;
    for (int nw : {4, 6, 7, 8}) {
      const int wgs = groups * ((a.rows + 16 * nw - 1) / (16 * nw));
      const int per_cu = nw == 4 ? 2 : 1;
      const int load = (wgs + g_attn_cus * per_cu - 1) / (g_attn_cus * per_cu) * per_cu * nw;
      if (nw == 4 || load < best_load || (load == best_load && wgs < best_wgs)) {
        best_nw = nw;
        best_load = load;
        best_wgs = wgs;
      }
    }
    if (best_nw != 4) {
      AttnArgs at = a;
      at.qblocks = (a.rows + 16 * best_nw - 1) / (16 * best_nw);
      const dim3 g2(8 * ((groups + 7) / 8) * at.qblocks);
      constexpr int TB = attn_tall_blocks<HD>();
      const uint32_t lds_tall = (uint32_t)(2 * TB * sizeof(AttnBlock<HD>));
      if (best_nw == 6)
        UAD_LAUNCH((attn_kernel<HD, TB, true, 6>), g2, dim3(384), lds_tall, s, ev0, end_attn, at);
      else if (best_nw == 7)
        UAD_LAUNCH((attn_kernel<HD, TB, true, 7>), g2, dim3(448), lds_tall, s, ev0, end_attn, at);
      else
        UAD_LAUNCH((attn_kernel<HD, TB, true, 8>), g2, dim3(512), lds_tall, s, ev0, end_attn, at);
      return hipGetLastError();
    }
  }
  if (streamed)
    UAD_LAUNCH((attn_kernel<HD, 1, true, 4>), grid, dim3(256), lds, s, ev0, end_attn, a);
  else
    UAD_LAUNCH((attn_kernel<HD, NB, false, 4>), grid, dim3(256), lds, s, ev0, end_attn, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  hipEvent_t none = nullptr;
  AttnArgs ac = a;
  // Beyond 8 splits (one chunk each: batch 1) four waves per workgroup, a
  // quarter of the workgroups to dispatch (the merge and its read-ahead slice
  // are ~900 one-wave workgroups at batch 1): same-machine, three pairs,
  // 0.7066 -> 0.7037 ms per step; at 8 environments (4 splits) one wave per
  // workgroup stays ahead (1.663 vs 1.677 ms).
  const int W = a.splits > 8 ? 4 : 1;
  ac.pre_comb.wgs = a.pre_comb.wgs ? (a.rows_pad / 16) * (HD / (16 * W)) : 0;  // one extra z slice
  const dim3 cgrid(a.rows_pad / 16, HD / (16 * W), batch * a.n_kv_heads + (ac.pre_comb.wgs ? 1 : 0));
  if (a.splits <= 4)
    UAD_LAUNCH((attn_combine_kernel<4, 1>), cgrid, dim3(64), 0, s, none, ev1, ac, HD);
  else if (a.splits <= 8)
    UAD_LAUNCH((attn_combine_kernel<8, 1>), cgrid, dim3(64), 0, s, none, ev1, ac, HD);
  else if (a.splits <= 16)
    UAD_LAUNCH((attn_combine_kernel<16, 4>), cgrid, dim3(256), 0, s, none, ev1, ac, HD);
  else if (a.splits <= 32)
    UAD_LAUNCH((attn_combine_kernel<32, 4>), cgrid, dim3(256), 0, s, none, ev1, ac, HD);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int HD>
static hipError_t init_hd() {
  constexpr int NB = attn_chunk_blocks<HD>();
  constexpr int streamed_lds = (int)(2 * sizeof(AttnBlock<HD>));
  hipError_t e = hipFuncSetAttribute((const void *)attn_kernel<HD, NB, false, 4>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)(2 * NB * sizeof(AttnBlock<HD>)));
  if (e == hipSuccess)
    e = hipFuncSetAttribute((const void *)attn_kernel<HD, 1, true, 4>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            streamed_lds);
  constexpr int TB = attn_tall_blocks<HD>();
  constexpr int tall_lds = (int)(2 * TB * sizeof(AttnBlock<HD>));
  static_assert(tall_lds <= 160 * 1024, "stages exceed the LDS of a CU");
  if (e == hipSuccess)
    e = hipFuncSetAttribute((const void *)attn_kernel<HD, TB, true, 6>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            tall_lds);
  if (e == hipSuccess)
    e = hipFuncSetAttribute((const void *)attn_kernel<HD, TB, true, 7>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            tall_lds);
  if (e == hipSuccess)
    e = hipFuncSetAttribute((const void *)attn_kernel<HD, TB, true, 8>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            tall_lds);
  return e;
}

hipError_t attention_init() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&g_attn_cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess && g_attn_cus < 1) e = hipErrorInvalidDevice;
  if (e == hipSuccess) e = init_hd<64>();
  if (e == hipSuccess) e = init_hd<128>();
  if (e == hipSuccess) e = init_hd<256>();
  return e;
}

int attention_max_splits(int) { return 32; }

int attention_chunk_blocks(int head_dim) {
  switch (head_dim) {
    case 64: return attn_chunk_blocks<64>();
    case 128: return attn_chunk_blocks<128>();
    case 256: return attn_chunk_blocks<256>();
  }
  return 1;
}

hipError_t launch_attention(const AttnArgs &a, int batch, int head_dim, hipStream_t s, hipEvent_t ev0,
                            hipEvent_t ev1) {
  switch (head_dim) {
    case 64: return launch_hd<64>(a, batch, s, ev0, ev1);
    case 128: return launch_hd<128>(a, batch, s, ev0, ev1);
    case 256: return launch_hd<256>(a, batch, s, ev0, ev1);
  }
  return hipErrorInvalidValue;
}

}  // namespace uad
