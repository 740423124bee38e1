// Joint attention of the chunk's queries over [cached prefix ; chunk] keys.
//
// Every action token attends to all P prefix tokens and all H chunk tokens
// (no mask), query head j reading KV head floor(j*Hkv/Hq).  The grouped query
// heads of one KV head are packed into the row dimension (row r = head-in-group
// * H + token), so one K/V tile read serves all of them.
//
// Per workgroup: one (environment, KV head), 64 packed query rows (4 waves x
// 16), and a contiguous range of 32-key blocks (split-KV when the batch is
// small).  K and V^T blocks are staged in LDS and shared by the 4 waves; the
// next block's global loads are issued before the current block is used.
// Each wave computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16 so that a
// lane ends up holding 8 scores of ONE query, which are exactly the 8 k-values
// of its operand for the P V product: no transpose through LDS.  Softmax
// statistics are reduced across the 4 lanes that share a query with
// wavefront shuffles (online softmax, fp32, exp2 domain).  With split-KV the
// unnormalised partial outputs and (max, sum) pairs are merged in fixed split
// order by attn_combine_kernel.
#include "uad_internal.h"

namespace uad {

template <int HD>
struct AttnSmem {
  __bf16 k[32][HD + 8];   // 32 keys x HD (+16 B pad: conflict-free 16 B reads)
  __bf16 vt[HD][32 + 4];  // HD x 32 keys (+8 B pad: conflict-free 8 B reads)
};

template <int HD>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  __shared__ AttnSmem<HD> sm;
  constexpr int KS = HD / 32;  // k-steps of the QK^T product
  constexpr int NTO = HD / 16; // 16-column output tiles
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int qblock = blockIdx.x;
  const int split = blockIdx.y;
  const int eh = blockIdx.z;  // env * Hkv + kv head
  const int b = eh / a.n_kv_heads;
  const int g = eh - b * a.n_kv_heads;

  const __bf16 *kbase = a.kc + (size_t)eh * a.s_alloc * HD;
  const __bf16 *vbase = a.vtc + (size_t)eh * HD * a.s_alloc;

  // This lane's query (as the B operand of S^T) : packed row r0 + (lane & 15)
  const int r0 = qblock * 64 + wave * 16;
  const int my_r = r0 + (lane & 15);
  bf16x8 qf[KS];
  {
    const bool ok = my_r < a.rows;
    const int hg = ok ? my_r / a.chunk : 0;
    const int tok = ok ? my_r - hg * a.chunk : 0;
    const int head = g * a.group + hg;
    const __bf16 *qp = a.q + (size_t)(b * a.chunk + tok) * a.ldq + head * HD + (lane >> 4) * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ok)
        qf[ks] = *(const bf16x8 *)(qp + ks * 32);
      else
        qf[ks] = bf16x8{};
    }
  }

  f32x4 o[NTO];
#pragma unroll
  for (int nt = 0; nt < NTO; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // running max (log2 domain) of query (lane & 15)
  float l_run = 0.f;        // this lane's partial sum of exp2

  const int n_blocks = (a.n_keys + 31) / 32;
  const int blk0 = split * a.blocks_per_split;
  int blk1 = blk0 + a.blocks_per_split;
  if (blk1 > n_blocks) blk1 = n_blocks;

  // K/V blocks are prefetched into registers one block ahead, so the global
  // loads of block b+1 are in flight while block b is multiplied from LDS.
  constexpr int KCH = 32 * HD / 8 / 256;  // 16-byte K chunks per thread
  constexpr int VCH = HD * 4 / 256;       // 16-byte V^T chunks per thread
  bf16x8 kreg[KCH], vreg[VCH];
  auto fetch = [&](int blk) {
    const int k0 = blk * 32;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = threadIdx.x + 256 * i;
      const int row = c / (HD / 8), col = (c - row * (HD / 8)) * 8;
      kreg[i] = *(const bf16x8 *)(kbase + (size_t)(k0 + row) * HD + col);
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = threadIdx.x + 256 * i;
      const int row = c >> 2, col = (c & 3) * 8;
      vreg[i] = *(const bf16x8 *)(vbase + (size_t)row * a.s_alloc + k0 + col);
    }
  };
  if (blk0 < blk1) fetch(blk0);

  for (int blk = blk0; blk < blk1; ++blk) {
    const int k0 = blk * 32;
    __syncthreads();  // previous block fully consumed
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = threadIdx.x + 256 * i;
      const int row = c / (HD / 8), col = (c - row * (HD / 8)) * 8;
      *(bf16x8 *)&sm.k[row][col] = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int c = threadIdx.x + 256 * i;
      const int row = c >> 2, col = (c & 3) * 8;
      const bf16x8 v = vreg[i];
      *(bf16x4 *)&sm.vt[row][col] = bf16x4{v[0], v[1], v[2], v[3]};
      *(bf16x4 *)&sm.vt[row][col + 4] = bf16x4{v[4], v[5], v[6], v[7]};
    }
    __syncthreads();
    if (blk + 1 < blk1) fetch(blk + 1);

    // S^T for two 16-key halves: s[h][r] = score(query lane&15, key k0+16h+4(lane>>4)+r)
    f32x4 s[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      s[h] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 kf = *(const bf16x8 *)&sm.k[16 * h + (lane & 15)][ks * 32 + (lane >> 4) * 8];
        s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], s[h], 0, 0, 0);
      }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + 16 * h + (lane >> 4) * 4 + r;
        float v = s[h][r] * a.scale_log2;
        if (key >= a.n_keys) v = -INFINITY;
        s[h][r] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
    bf16x8 pf;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = exp2f(s[h][r] - m_new);
        psum += p;
        pf[h * 4 + r] = (__bf16)p;
      }
    l_run = l_run * alpha + psum;
    // rescale output rows (row 4*(lane>>4)+r of the tile) by their query's alpha
    float al[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) al[r] = __shfl(alpha, (lane >> 4) * 4 + r);
#pragma unroll
    for (int nt = 0; nt < NTO; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[nt][r] *= al[r];
    // O += P V : B operand lane l = V[keys of pf][col 16nt + (l&15)]
#pragma unroll
    for (int nt = 0; nt < NTO; ++nt) {
      const __bf16 *vr = &sm.vt[nt * 16 + (lane & 15)][0];
      const bf16x4 v0 = *(const bf16x4 *)(vr + (lane >> 4) * 4);
      const bf16x4 v1 = *(const bf16x4 *)(vr + 16 + (lane >> 4) * 4);
      const bf16x8 vf = bf16x8{v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
      o[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf, vf, o[nt], 0, 0, 0);
    }
  }

  float l_tot = l_run;
  l_tot += __shfl_xor(l_tot, 16);
  l_tot += __shfl_xor(l_tot, 32);

  // Output rows of this lane: r0 + 4*(lane>>4) + r, column 16*nt + (lane&15)
  float lr[4], mr[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    lr[r] = __shfl(l_tot, (lane >> 4) * 4 + r);
    mr[r] = __shfl(m_run, (lane >> 4) * 4 + r);
  }
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
        store_op(a.o + afrag_index(orow, head * HD + nt * 16 + (lane & 15), a.ldo / kTileK), o[nt][r] * inv);
    }
  } else {
    const size_t pbase = ((size_t)split * gridDim.z + eh) * a.rows_pad;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = r0 + (lane >> 4) * 4 + r;
      if (row >= a.rows) continue;
      float *op = a.opart + (pbase + row) * HD + (lane & 15);
#pragma unroll
      for (int nt = 0; nt < NTO; ++nt) op[nt * 16] = o[nt][r];
      if ((lane & 15) == 0) {
        a.mlpart[(pbase + row) * 2 + 0] = mr[r];
        a.mlpart[(pbase + row) * 2 + 1] = lr[r];
      }
    }
  }
}

// Merge split-KV partials: o = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s,
// splits in fixed order.  The (m_s, l_s) pairs of the row are staged in LDS
// by one vector load per thread; every partial load is issued up front.
constexpr int kMaxKvSplits = 32;
template <int HD>
__global__ __launch_bounds__(HD) void attn_combine_kernel(AttnArgs a) {
  __shared__ float2 mls[kMaxKvSplits];
  const int row = blockIdx.x;
  const int eh = blockIdx.y;
  const int b = eh / a.n_kv_heads, g = eh - b * a.n_kv_heads;
  const int c = threadIdx.x;
  const int n_eh = gridDim.y;
  const int splits = a.splits;
  const float *__restrict__ opart = a.opart;
  if (c < kMaxKvSplits)
    mls[c] = c < splits ? *(const float2 *)(a.mlpart + (((size_t)c * n_eh + eh) * a.rows_pad + row) * 2)
                        : float2{-INFINITY, 0.f};
  float os[kMaxKvSplits];
#pragma unroll
  for (int s = 0; s < kMaxKvSplits; ++s)
    os[s] = s < splits ? opart[(((size_t)s * n_eh + eh) * a.rows_pad + row) * HD + c] : 0.f;
  __syncthreads();
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < kMaxKvSplits; ++s) M = fmaxf(M, mls[s].x);
  float num = 0.f, den = 0.f;
#pragma unroll
  for (int s = 0; s < kMaxKvSplits; ++s) {
    if (s < splits) {
      const float w = exp2f(mls[s].x - M);
      num += w * os[s];
      den += w * mls[s].y;
    }
  }
  const int hg = row / a.chunk, tok = row - hg * a.chunk;
  const int head = g * a.group + hg;
  store_op(a.o + afrag_index(b * a.chunk + tok, head * HD + c, a.ldo / kTileK), num / den);
}

template <int HD>
static hipError_t launch_hd(const AttnArgs &a, int batch, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  dim3 grid((a.rows + 63) / 64, a.splits, batch * a.n_kv_heads);
  hipEvent_t end_attn = a.splits == 1 ? ev1 : nullptr;
  UAD_LAUNCH((attn_kernel<HD>), grid, dim3(256), 0, s, ev0, end_attn, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  hipEvent_t none = nullptr;
  UAD_LAUNCH((attn_combine_kernel<HD>), dim3(a.rows, batch * a.n_kv_heads), dim3(HD), 0, s, none, ev1, a);
  return hipGetLastError();
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
