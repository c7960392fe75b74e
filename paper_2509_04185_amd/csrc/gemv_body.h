// The weight stream of the decode-sized GEMM (M <= 16 rows), shared by gemv.hip and the
// per-XCD layer kernels (layer_xcd.hip).
//
// One wave accumulates acc[ct] += A W_t^T over its K steps for C tiles t of a packed matrix
// (v_mfma_f32_16x16x32_bf16; A as hi and lo bf16, two MFMAs per step).  Steps come in
// batches of U, double-buffered: the loads of batch b + 1 are issued before the MFMAs of
// batch b wait for theirs (scheduling barriers keep the compiler from interleaving them),
// so 2U steps of weights are in flight per wave.  The last batch clamps its step index (a
// repeated fragment, no extra HBM traffic) and zeroes the activation fragments of steps
// past the end, which then add nothing.
#pragma once

#include "sbd_device.h"

namespace sbd {

// Weight fragments: a lane's 8 weights of a tile's 16 x 32 step, as bf16 (i32x4, 16 bytes)
// or as OCP e4m3 bytes (i32x2, 8 bytes) widened to bf16 right before the MFMA.  The fp8
// packing is the bf16 one element for element (kPackStep and packed_frag count elements),
// one byte per element.  A matrix in fp8 carries a power-of-two scale per output row (the
// lane's row of the tile): the widening multiplies by it exactly (gfx950's scaled
// conversion), so the MFMA sees the exact bf16 values q * 2^e.
template <class WT> struct WFrag;
template <> struct WFrag<bf16_t> { using T = i32x4; };
template <> struct WFrag<fp8_t> { using T = i32x2; };

__device__ __forceinline__ i32x4 ld_w(const bf16_t* p) { return ld16_stream(p); }
__device__ __forceinline__ i32x2 ld_w(const fp8_t* p) { return __builtin_nontemporal_load((const i32x2*)p); }

__device__ __forceinline__ i32x4 w_operand(i32x4 w, float) { return w; }
__device__ __forceinline__ i32x4 w_operand(i32x2 w, float sc) { return e4m3x8_to_bf16(w, sc); }

// The lane's per-row weight scales of tiles t0 .. t0 + C - 1 (row 16 t + r); 1 for bf16.
template <class WT, int C>
__device__ __forceinline__ void load_wscale(const float* wscale, int t0, int r, float (&sc)[C]) {
#pragma unroll
  for (int ct = 0; ct < C; ++ct) sc[ct] = (sizeof(WT) == 1) ? wscale[(int64_t)(t0 + ct) * 16 + r] : 1.0f;
}

// Weight fragments of steps b0 .. b0 + U - 1 (clamped to ns - 1) of the C tiles.
template <int C, int U, class WT>
__device__ __forceinline__ void gemv_issue_w(const WT* const (&wt)[C], int b0, int ns,
                                             typename WFrag<WT>::T (&wv)[U][C]) {
#pragma unroll
  for (int uu = 0; uu < U; ++uu) {
    const int st = min(b0 + uu, ns - 1);
#pragma unroll
    for (int ct = 0; ct < C; ++ct) wv[uu][ct] = ld_w(wt[ct] + (int64_t)st * kPackStep);
  }
}

// Activation fragments (hi, lo) of the same steps; a_off is this lane's byte offset at step
// 0 (a step is 32 bf16 = 64 bytes further).  POL: cache policy of the loads.
template <int U, int POL>
__device__ __forceinline__ void gemv_issue_a(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t ral, uint32_t a_off,
                                             int b0, int ns, i32x4 (&xa)[U], i32x4 (&xl)[U]) {
#pragma unroll
  for (int uu = 0; uu < U; ++uu) {
    const uint32_t o = a_off + (uint32_t)min(b0 + uu, ns - 1) * 64u;
    xa[uu] = __builtin_amdgcn_raw_buffer_load_b128(ra, o, 0, POL);
    xl[uu] = __builtin_amdgcn_raw_buffer_load_b128(ral, o, 0, POL);
  }
}

template <int C, int U, class WR>
__device__ __forceinline__ void gemv_mfma(const WR (&wv)[U][C], const i32x4 (&xa)[U], const i32x4 (&xl)[U],
                                          int b0, int ns, const float (&sc)[C], f32x4 (&acc)[C]) {
#pragma unroll
  for (int uu = 0; uu < U; ++uu) {
    const bool ok = b0 + uu < ns;
    const i32x4 a_hi = ok ? xa[uu] : i32x4{0, 0, 0, 0};
    const i32x4 a_lo = ok ? xl[uu] : i32x4{0, 0, 0, 0};
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      const i32x4 w = w_operand(wv[uu][ct], sc[ct]);
      acc[ct] = mfma16x16x32(a_hi, w, acc[ct]);
      acc[ct] = mfma16x16x32(a_lo, w, acc[ct]);
    }
  }
}

// acc += the wave's steps [0, ns).  wt[ct]: this lane's piece of tile ct's fragment at step
// 0.  PRE: the caller already issued the weights of batch 0 into w0 (gemv_issue_w), e.g.
// before waiting for the activations; otherwise w0 is scratch.  sc: the lane's weight scales.
template <int C, int U, int POL, bool PRE, class WT>
__device__ __forceinline__ void gemv_stream(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t ral, uint32_t a_off,
                                            const WT* const (&wt)[C], int ns, typename WFrag<WT>::T (&w0)[U][C],
                                            const float (&sc)[C], f32x4 (&acc)[C]) {
  if (ns <= 0) return;
  const int nb = (ns + U - 1) / U;
  typename WFrag<WT>::T w1[U][C];
  i32x4 xa0[U], xl0[U], xa1[U], xl1[U];
  gemv_issue_a<U, POL>(ra, ral, a_off, 0, ns, xa0, xl0);
  if constexpr (!PRE) gemv_issue_w<C, U>(wt, 0, ns, w0);
  for (int b = 0; b < nb; b += 2) {
    if (b + 1 < nb) {
      gemv_issue_a<U, POL>(ra, ral, a_off, (b + 1) * U, ns, xa1, xl1);
      gemv_issue_w<C, U>(wt, (b + 1) * U, ns, w1);
    }
    __builtin_amdgcn_sched_barrier(0);
    gemv_mfma<C, U>(w0, xa0, xl0, b * U, ns, sc, acc);
    __builtin_amdgcn_sched_barrier(0);
    if (b + 1 < nb) {
      if (b + 2 < nb) {
        gemv_issue_a<U, POL>(ra, ral, a_off, (b + 2) * U, ns, xa0, xl0);
        gemv_issue_w<C, U>(wt, (b + 2) * U, ns, w0);
      }
      __builtin_amdgcn_sched_barrier(0);
      gemv_mfma<C, U>(w1, xa1, xl1, (b + 1) * U, ns, sc, acc);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

}  // namespace sbd

namespace sbd {

// ---- the same stream with the activations taken from the fixed-point residual
//
// The per-XCD layer kernels keep the residual stream x as int64 fixed point (value * 2^32):
// partial sums from several XCDs are then added with integer atomics, exactly and in any
// order.  A consumer forms its operand itself: x = hi32 + lo32 * 2^-32 in fp32, times the
// norm gain g[k], split into hi/lo bf16; it also accumulates x^2 of the elements it reads,
// the input of its RMSNorm scale.  A lane reads 8 consecutive k of its row per step: 64
// bytes of x plus 16 bytes of g.

constexpr float kFixScale = 4294967296.0f;  // 2^32
__device__ __forceinline__ float fix_to_f32(int lo, int hi) {
  return (float)hi + (float)(uint32_t)lo * (1.0f / kFixScale);
}

template <int U>
__device__ __forceinline__ void gemv_issue_x64(__amdgpu_buffer_rsrc_t rx, __amdgpu_buffer_rsrc_t rg, uint32_t x_off,
                                               uint32_t g_off, int b0, int ns, i32x4 (&xv)[U][4], i32x4 (&gv)[U]) {
#pragma unroll
  for (int uu = 0; uu < U; ++uu) {
    const uint32_t st = (uint32_t)min(b0 + uu, ns - 1);
#pragma unroll
    for (int q = 0; q < 4; ++q) xv[uu][q] = __builtin_amdgcn_raw_buffer_load_b128(rx, x_off + st * 256u + q * 16u, 0, 0);
    gv[uu] = __builtin_amdgcn_raw_buffer_load_b128(rg, g_off + st * 64u, 0, 0);
  }
}

// hi/lo bf16 operands of 8 elements; ss += their x^2 (steps past the end add nothing).
__device__ __forceinline__ void x64_operand(const i32x4 (&xv)[4], i32x4 gv, bool ok, i32x4& a_hi, i32x4& a_lo, float& ss) {
  float v[8];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    v[2 * q] = fix_to_f32(xv[q][0], xv[q][1]);
    v[2 * q + 1] = fix_to_f32(xv[q][2], xv[q][3]);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) ss += ok ? v[e] * v[e] : 0.f;
  float xg[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t gw = (uint32_t)gv[e];
    xg[2 * e] = v[2 * e] * __uint_as_float(gw << 16);
    xg[2 * e + 1] = v[2 * e + 1] * __uint_as_float(gw & 0xffff0000u);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t h = pack_bf2(xg[2 * e], xg[2 * e + 1]);
    a_hi[e] = ok ? (int)h : 0;
    a_lo[e] = ok ? (int)pack_bf2(xg[2 * e] - __uint_as_float(h << 16), xg[2 * e + 1] - __uint_as_float(h & 0xffff0000u)) : 0;
  }
}

template <int C, int U, class WR>
__device__ __forceinline__ void gemv_mfma_x64(const WR (&wv)[U][C], const i32x4 (&xv)[U][4], const i32x4 (&gv)[U],
                                              int b0, int ns, const float (&sc)[C], f32x4 (&acc)[C], float& ss) {
#pragma unroll
  for (int uu = 0; uu < U; ++uu) {
    i32x4 a_hi, a_lo;
    x64_operand(xv[uu], gv[uu], b0 + uu < ns, a_hi, a_lo, ss);
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      const i32x4 w = w_operand(wv[uu][ct], sc[ct]);
      acc[ct] = mfma16x16x32(a_hi, w, acc[ct]);
      acc[ct] = mfma16x16x32(a_lo, w, acc[ct]);
    }
  }
}

// gemv_stream with the operand formed from the fixed-point residual: x_off is this lane's
// byte offset into x at step 0 (8 bytes per element), g_off its byte offset into the gain.
template <int C, int U, class WT>
__device__ __forceinline__ void gemv_stream_x64(__amdgpu_buffer_rsrc_t rx, __amdgpu_buffer_rsrc_t rg, uint32_t x_off,
                                                uint32_t g_off, const WT* const (&wt)[C], int ns,
                                                const float (&sc)[C], f32x4 (&acc)[C], float& ss) {
  if (ns <= 0) return;
  const int nb = (ns + U - 1) / U;
  typename WFrag<WT>::T w0[U][C], w1[U][C];
  i32x4 x0[U][4], x1[U][4], g0[U], g1[U];
  gemv_issue_x64<U>(rx, rg, x_off, g_off, 0, ns, x0, g0);
  gemv_issue_w<C, U>(wt, 0, ns, w0);
  for (int b = 0; b < nb; b += 2) {
    if (b + 1 < nb) {
      gemv_issue_x64<U>(rx, rg, x_off, g_off, (b + 1) * U, ns, x1, g1);
      gemv_issue_w<C, U>(wt, (b + 1) * U, ns, w1);
    }
    __builtin_amdgcn_sched_barrier(0);
    gemv_mfma_x64<C, U>(w0, x0, g0, b * U, ns, sc, acc, ss);
    __builtin_amdgcn_sched_barrier(0);
    if (b + 1 < nb) {
      if (b + 2 < nb) {
        gemv_issue_x64<U>(rx, rg, x_off, g_off, (b + 2) * U, ns, x0, g0);
        gemv_issue_w<C, U>(wt, (b + 2) * U, ns, w0);
      }
      __builtin_amdgcn_sched_barrier(0);
      gemv_mfma_x64<C, U>(w1, x1, g1, (b + 1) * U, ns, sc, acc, ss);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// A value as fixed point (v * 2^32, rounded to nearest), and the atomic add of such values to
// the residual (exact; any order gives the same sum).
__device__ __forceinline__ long long fix_q(float v) { return __double2ll_rn((double)v * 4294967296.0); }
__device__ __forceinline__ void fix_add_q(int64_t* p, long long q) {
  atomicAdd(reinterpret_cast<unsigned long long*>(p), (unsigned long long)q);
}

}  // namespace sbd
