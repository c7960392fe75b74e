// QKV epilogue of the decode GEMM (gemv.hip): per-head q/k RMSNorm, rotate-half RoPE, q as
// scaled hi/lo bf16, K and V into the cache at cache_len + j.
#pragma once

#include "sbd_device.h"

namespace sbd {

// What the epilogue reads besides the accumulators, loaded before the weight stream so
// that none of it is on the kernel's tail: for the lane's rows 4g + i, the cache position
// and slot, and the rotary (cos, sin) of the dims 16 pr + r it rotates; the q/k norm gains
// of the dims it holds.
template <int DH>
struct QkvPre {
  static constexpr int tph = DH / 16, ptiles = tph / 2;
  int p_cache[4], slot[4];
  float cs[4][ptiles], sn[4][ptiles];
  float gq[tph], gk[tph];
};

template <int DH>
__device__ __forceinline__ void qkv_epi_prefetch(const QkvEpi& e, int M, QkvPre<DH>& pre) {
  constexpr int tph = DH / 16, ptiles = tph / 2, half = DH / 2;
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = min(4 * g + i, M - 1);
    const SeqParam sp = e.seqs[m / e.kblk];
    const int pos = e.rows[m].pos;
    pre.p_cache[i] = sp.cache_len + m % e.kblk;
    pre.slot[i] = sp.slot;
#pragma unroll
    for (int pr = 0; pr < ptiles; ++pr) {
      const float2 v = *(const float2*)(e.rope + ((int64_t)pos * half + pr * 16 + r) * 2);
      pre.cs[i][pr] = v.x;
      pre.sn[i][pr] = v.y;
    }
  }
  // one branch around all the gain loads, so that they are in flight together
  if (e.qk_norm) {
#pragma unroll
    for (int t = 0; t < tph; ++t) {
      pre.gq[t] = bf2f(e.q_norm[16 * t + r]);
      pre.gk[t] = bf2f(e.k_norm[16 * t + r]);
    }
  } else {
#pragma unroll
    for (int t = 0; t < tph; ++t) pre.gq[t] = pre.gk[t] = 1.f;
  }
}

// QKV epilogue of one packed group (8 tiles = 128 columns = 128 / DH whole heads), run by a
// wave holding all 8 accumulator tiles: of the lane's rows 4g + i, those with i == i_sel
// (every i when i_sel < 0), so that four waves can share the rows.
template <int DH>
__device__ __forceinline__ void qkv_epilogue(const QkvEpi& e, int M, int grp, const f32x4 (&acc)[8],
                                             const float (&rinv)[4], const QkvPre<DH>& pre, int i_sel = -1) {
  constexpr int tph = DH / 16, ptiles = tph / 2, half = DH / 2, heads = 8 / tph;
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (i_sel >= 0 && i != i_sel) continue;
    const int m = 4 * g + i;
    const bool row_ok = m < M;
    const float rv = row_ok ? rinv[i] : 0.f;
    float u[8];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) u[ct] = acc[ct][i] * rv;
#pragma unroll
    for (int hh = 0; hh < heads; ++hh) {
      const int h = grp * heads + hh;  // q heads, then k heads, then v heads
      if (e.qk_norm && h < e.n_q + e.n_kv) {
        float ss = 0.f;
#pragma unroll
        for (int t = 0; t < tph; ++t) ss += u[hh * tph + t] * u[hh * tph + t];
        ss += __shfl_xor(ss, 1);
        ss += __shfl_xor(ss, 2);
        ss += __shfl_xor(ss, 4);
        ss += __shfl_xor(ss, 8);
        const float rn = 1.0f / sqrtf(ss / (float)DH + e.eps);
#pragma unroll
        for (int t = 0; t < tph; ++t) u[hh * tph + t] *= rn * (h < e.n_q ? pre.gq[t] : pre.gk[t]);
      }
    }
    if (!row_ok) continue;
    const int p_cache = pre.p_cache[i];
#pragma unroll
    for (int hh = 0; hh < heads; ++hh) {
      const int h = grp * heads + hh;
      if (h >= e.n_q + e.n_kv) {  // V: transposed cache block, slot order of misc.hip vslot()
        const int gk = h - e.n_q - e.n_kv;
        const int64_t blk = (((int64_t)e.layer * e.n_slots + pre.slot[i]) * e.n_kv + gk) * e.cap * DH +
                            (int64_t)(p_cache / 32) * DH * 32;
        const int p = p_cache & 31;
        const int sl = ((p & 15) >> 2) * 8 + (p >> 4) * 4 + (p & 3);
#pragma unroll
        for (int t = 0; t < tph; ++t) kv_store(e.vcache, blk + (16 * t + r) * 32 + sl, u[hh * tph + t], e.kv_fp8, e.kv_inv);
        continue;
      }
#pragma unroll
      for (int pr = 0; pr < ptiles; ++pr) {
        const int dim = pr * 16 + r;
        const float cs = pre.cs[i][pr], sn = pre.sn[i][pr];
        const float u0 = u[hh * tph + pr], u1 = u[hh * tph + pr + ptiles];
        const float r0 = u0 * cs - u1 * sn;
        const float r1 = u1 * cs + u0 * sn;
        if (h < e.n_q) {
          const int64_t o = ((int64_t)m * e.n_q + h) * DH;
          bf16_t hi, lo;
          split_bf16(r0 * e.q_scale, hi, lo);
          e.q[o + dim] = hi;
          e.q_lo[o + dim] = lo;
          split_bf16(r1 * e.q_scale, hi, lo);
          e.q[o + dim + half] = hi;
          e.q_lo[o + dim + half] = lo;
        } else {
          const int gk = h - e.n_q;
          const int64_t dst = (((int64_t)e.layer * e.n_slots + pre.slot[i]) * e.n_kv + gk) * e.cap * DH +
                              (int64_t)p_cache * DH;
          kv_store(e.kcache, dst + dim, r0, e.kv_fp8, e.kv_inv);
          kv_store(e.kcache, dst + dim + half, r1, e.kv_fp8, e.kv_inv);
        }
      }
    }
  }
}

}  // namespace sbd
