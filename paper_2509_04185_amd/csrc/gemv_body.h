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

// Weight fragments of steps b0 .. b0 + U - 1 (clamped to ns - 1) of the C tiles.
template <int C, int U>
__device__ __forceinline__ void gemv_issue_w(const bf16_t* const (&wt)[C], int b0, int ns, i32x4 (&wv)[U][C]) {
#pragma unroll
  for (int uu = 0; uu < U; ++uu) {
    const int st = min(b0 + uu, ns - 1);
#pragma unroll
    for (int ct = 0; ct < C; ++ct) wv[uu][ct] = ld16_stream(wt[ct] + (int64_t)st * kPackStep);
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

template <int C, int U>
__device__ __forceinline__ void gemv_mfma(const i32x4 (&wv)[U][C], const i32x4 (&xa)[U], const i32x4 (&xl)[U],
                                          int b0, int ns, f32x4 (&acc)[C]) {
#pragma unroll
  for (int uu = 0; uu < U; ++uu) {
    const bool ok = b0 + uu < ns;
    const i32x4 a_hi = ok ? xa[uu] : i32x4{0, 0, 0, 0};
    const i32x4 a_lo = ok ? xl[uu] : i32x4{0, 0, 0, 0};
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      acc[ct] = mfma16x16x32(a_hi, wv[uu][ct], acc[ct]);
      acc[ct] = mfma16x16x32(a_lo, wv[uu][ct], acc[ct]);
    }
  }
}

// acc += the wave's steps [0, ns).  wt[ct]: this lane's piece of tile ct's fragment at step
// 0.  PRE: the caller already issued the weights of batch 0 into w0 (gemv_issue_w), e.g.
// before waiting for the activations; otherwise w0 is scratch.
template <int C, int U, int POL, bool PRE>
__device__ __forceinline__ void gemv_stream(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t ral, uint32_t a_off,
                                            const bf16_t* const (&wt)[C], int ns, i32x4 (&w0)[U][C],
                                            f32x4 (&acc)[C]) {
  if (ns <= 0) return;
  const int nb = (ns + U - 1) / U;
  i32x4 w1[U][C], xa0[U], xl0[U], xa1[U], xl1[U];
  gemv_issue_a<U, POL>(ra, ral, a_off, 0, ns, xa0, xl0);
  if constexpr (!PRE) gemv_issue_w<C, U>(wt, 0, ns, w0);
  for (int b = 0; b < nb; b += 2) {
    if (b + 1 < nb) {
      gemv_issue_a<U, POL>(ra, ral, a_off, (b + 1) * U, ns, xa1, xl1);
      gemv_issue_w<C, U>(wt, (b + 1) * U, ns, w1);
    }
    __builtin_amdgcn_sched_barrier(0);
    gemv_mfma<C, U>(w0, xa0, xl0, b * U, ns, acc);
    __builtin_amdgcn_sched_barrier(0);
    if (b + 1 < nb) {
      if (b + 2 < nb) {
        gemv_issue_a<U, POL>(ra, ral, a_off, (b + 2) * U, ns, xa0, xl0);
        gemv_issue_w<C, U>(wt, (b + 2) * U, ns, w0);
      }
      __builtin_amdgcn_sched_barrier(0);
      gemv_mfma<C, U>(w1, xa1, xl1, (b + 1) * U, ns, acc);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

}  // namespace sbd
