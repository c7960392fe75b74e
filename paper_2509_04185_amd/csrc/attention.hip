// Block-hybrid grouped-query attention of the SBD block forward.
//
// For sequence b with cache length L and block rows j = 0..k-1 (stored at positions
// L + j), row j attends to key position kv iff kv < L + j + 1 when j is a causal row
// (j < n_causal) and to every key kv < L + k when j is in the prediction block: the
// inference mask of the paper (App. A, Fig. 3) restricted to the rows of the block.
//
// Work split: one workgroup per (split, KV head x row block, sequence).  The rows of a
// KV head are the group*k (query head, block row) pairs that read it; each wave takes 16
// of them (one MFMA tile) and walks the keys of its split in 32-key steps:
//   S^T = K Q^T   (v_mfma_f32_16x16x32_bf16: keys on M, query rows on N, d_h in 4 steps;
//                  Q as hi + lo bf16, two MFMAs per step)
//   online softmax per query row in base 2 (queries carry log2(e)/sqrt(d_h))
//   O^T += V^T P^T (P as hi + lo bf16 in the B-operand layout straight from the score
//                   tile; V^T comes from the transposed, permuted cache blocks)
// Each split leaves unnormalised (max, sum, O) per row; a merge kernel combines the
// splits with log-sum-exp weights in split order.

#include "sbd_device.h"

namespace sbd {

__device__ __forceinline__ int64_t attn_head_base(int layer, int slot, int g, int n_slots,
                                                  int n_kv, int64_t cap, int d_h) {
  return (((int64_t)layer * n_slots + slot) * n_kv + g) * cap * d_h;
}

template <int DH>
__global__ __launch_bounds__(256) void attn_split_kernel(AttnArgs a) {
  constexpr int NDT = DH / 16;  // 16-wide dimension tiles
  constexpr int NKS = DH / 32;  // 32-wide reduction steps for the scores
  const int split = blockIdx.x;
  const int g = blockIdx.y / a.n_rowblocks;
  const int rb = blockIdx.y % a.n_rowblocks;
  const int b = blockIdx.z;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 15, grp = lane >> 4;
  const SeqParam sp = a.seqs[b];
  const int L = sp.cache_len, nc = sp.n_causal, k = a.k;
  const int G = a.n_q / a.n_kv;
  const int R = G * k;

  const int rho = rb * 64 + w * 16 + r;
  const bool row_ok = rho < R;
  const int hh = row_ok ? rho / k : 0;
  const int j = row_ok ? rho % k : 0;
  const int hq = g * G + hh;
  const int kend = row_ok ? ((j >= nc) ? L + k : L + j + 1) : 0;

  // Key blocks this wave visits: its split's range, clipped to its rows' last key.
  int kend_w = kend;
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) kend_w = max(kend_w, __shfl_xor(kend_w, o));
  const int nblk_w = (kend_w + 31) / 32;
  const int blk0 = split * a.blocks_per_split;
  const int blk1 = min(blk0 + a.blocks_per_split, nblk_w);

  // Query fragments (B operand, hi and lo): row r, dims 32*s + 8*grp .. +8.
  i32x4 qf[NKS], ql[NKS];
  const int64_t qoff = ((int64_t)(b * k + j) * a.n_q + hq) * DH;
#pragma unroll
  for (int s = 0; s < NKS; ++s) {
    qf[s] = row_ok ? ld16(a.q + qoff + 32 * s + 8 * grp) : i32x4{0, 0, 0, 0};
    ql[s] = row_ok ? ld16(a.q_lo + qoff + 32 * s + 8 * grp) : i32x4{0, 0, 0, 0};
  }

  const int64_t hb = attn_head_base(a.layer, sp.slot, g, a.n_slots, a.n_kv, a.cap, DH);
  const bf16_t* kbase = a.kcache + hb;
  const bf16_t* vbase = a.vcache + hb;

  f32x4 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  for (int kb = blk0; kb < blk1; ++kb) {
    const int key0 = kb * 32;
    f32x4 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      const bf16_t* kp = kbase + (int64_t)(key0 + 16 * t + r) * DH + 8 * grp;
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        const i32x4 kf = ld16(kp + 32 * s);
        st[t] = mfma16x16x32(kf, qf[s], st[t]);
        st[t] = mfma16x16x32(kf, ql[s], st[t]);
      }
    }
    // st[t][i]: score of key key0 + 16t + 4grp + i for query row r.
    float mloc = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kv = key0 + 16 * t + 4 * grp + i;
        if (kv >= kend) st[t][i] = -INFINITY;
        mloc = fmaxf(mloc, st[t][i]);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    const float scale = (m_run == -INFINITY) ? 0.f : exp2f(m_run - m_new);
    float p[8];
    float lsum = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float v = (st[t][i] == -INFINITY) ? 0.f : exp2f(st[t][i] - m_new);
        p[4 * t + i] = v;
        lsum += v;
      }
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    l_run = l_run * scale + lsum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) o[dt] *= scale;
    // P as hi/lo bf16 (B operand): element e holds key 16*(e/4) + 4*grp + e%4.
    i32x4 pf, pl;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      bf16_t h0, l0, h1, l1;
      split_bf16(p[2 * e], h0, l0);
      split_bf16(p[2 * e + 1], h1, l1);
      pf[e] = (int)((uint32_t)h0 | ((uint32_t)h1 << 16));
      pl[e] = (int)((uint32_t)l0 | ((uint32_t)l1 << 16));
    }
    const bf16_t* vb = vbase + (int64_t)kb * DH * 32 + 8 * grp;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const i32x4 vf = ld16(vb + (int64_t)(16 * dt + r) * 32);
      o[dt] = mfma16x16x32(vf, pf, o[dt]);
      o[dt] = mfma16x16x32(vf, pl, o[dt]);
    }
  }

  if (!row_ok) return;
  const int64_t item = (int64_t)(b * k + j) * a.n_q + hq;
  const int64_t n_items = (int64_t)a.B * k * a.n_q;
  if (grp == 0) {
    float* ml = a.part_ml + ((int64_t)split * n_items + item) * 2;
    ml[0] = m_run;
    ml[1] = l_run;
  }
  float* po = a.part_o + ((int64_t)split * n_items + item) * DH;
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) *(f32x4*)(po + 16 * dt + 4 * grp) = o[dt];
}

// One wave per (row, query head): combine the splits, normalise, store hi/lo bf16.
// Lane s reads split s's (max, sum); the split weights 2^(m_s - M) are broadcast from
// their lanes while every lane accumulates its own dimensions over the splits.
template <int DH>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  const int64_t n_items = (int64_t)a.B * a.k * a.n_q;
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= n_items) return;
  const int lane = threadIdx.x & 63;
  const int ns = a.n_splits;  // <= 64
  float ms = -INFINITY, ls = 0.f;
  if (lane < ns) {
    const float2 v = *(const float2*)(a.part_ml + ((int64_t)lane * n_items + item) * 2);
    ms = v.x;
    ls = v.y;
  }
  const float mx = wave_max(ms);
  const float wgt = (ms == -INFINITY) ? 0.f : exp2f(ms - mx);
  const float lsum = wave_sum(wgt * ls);
  constexpr int PER = DH / 64;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  const float* po = a.part_o + item * DH + lane;
  const int64_t split_stride = n_items * DH;
  int s = 0;
  for (; s + 4 <= ns; s += 4) {
    float v[4][PER];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int e = 0; e < PER; ++e) v[u][e] = po[(int64_t)(s + u) * split_stride + 64 * e];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float wu = __shfl(wgt, s + u);
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] += wu * v[u][e];
    }
  }
  for (; s < ns; ++s) {
    const float wu = __shfl(wgt, s);
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += wu * po[(int64_t)s * split_stride + 64 * e];
  }
  const float inv = 1.0f / lsum;
  const int64_t orow = item / a.n_q;
  const int hq = (int)(item % a.n_q);
  const int64_t dst = orow * (int64_t)a.n_q * DH + (int64_t)hq * DH;
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    bf16_t hi, lo;
    split_bf16(acc[e] * inv, hi, lo);
    a.out[dst + lane + 64 * e] = hi;
    a.out_lo[dst + lane + 64 * e] = lo;
  }
}

hipError_t launch_attention_split(const AttnArgs& a, const Exec& ex) {
  dim3 grid(a.n_splits, a.n_kv * a.n_rowblocks, a.B);
  if (a.d_h == 128)
    SBD_KLAUNCH(attn_split_kernel<128>, grid, dim3(256), ex, a);
  else if (a.d_h == 64)
    SBD_KLAUNCH(attn_split_kernel<64>, grid, dim3(256), ex, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention_merge(const AttnArgs& a, const Exec& ex) {
  const int64_t n_items = (int64_t)a.B * a.k * a.n_q;
  dim3 grid((unsigned)((n_items + 3) / 4));
  if (a.d_h == 128)
    SBD_KLAUNCH(attn_merge_kernel<128>, grid, dim3(256), ex, a);
  else if (a.d_h == 64)
    SBD_KLAUNCH(attn_merge_kernel<64>, grid, dim3(256), ex, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sbd
