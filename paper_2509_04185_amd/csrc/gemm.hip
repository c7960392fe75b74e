// Skinny weight-streaming GEMM for the block forward: y[m][n] = sum_k A[m][k] W[n][k].
//
// The block forward multiplies M = batch * k activation rows (16 at batch 1, k = 16) by
// every weight matrix of the decoder, so it is bound by streaming the weights from HBM.
// Each workgroup owns 16*C output columns (C 16-wide MFMA tiles) and a row block; its
// NW waves split the reduction dimension K and stream disjoint K ranges of the same
// weight rows with 16-byte non-temporal loads, double-buffered in registers.  The
// activations come as hi/lo bf16 pairs (two MFMAs per step, see GemmArgs).  Partial
// sums meet in LDS and are added in a fixed wave order (deterministic), and the
// epilogue applies the operation that follows the product in the decoder block:
//   EPI_SCALED_STORE  out = rinv[m] * y           (QKV projection, LM head)
//   EPI_RESID         x += y; xn = bf16(x * g_next); per-row sums of x^2 over each
//                     16 columns (O and down projections: residual add, the next
//                     RMSNorm's inputs)
//   EPI_SWIGLU        act = bf16(silu(rinv*gate) * rinv*up)  (gate/up projection)
// RMSNorm is split across two kernels: the producer writes x * g (gain applied, bf16)
// plus per-16-column partial sums of squares; the consumer adds the partials of a row
// and scales its fp32 result by 1/sqrt(mean(x^2) + eps), which equals normalising the
// input first because the scale is constant along a row.
//
// MFMA v_mfma_f32_16x16x32_bf16: lane l holds row (l % 16) of A and column (l % 16) of
// B^T for the 8 consecutive k of group l / 16; the result holds rows 4*(l/16)+i of
// column l % 16.

#include "sbd_device.h"

namespace sbd {

template <int MT, int C, int NW, int U, int EPI>
__global__ __launch_bounds__(NW * 64) void gemm_kernel(GemmArgs a) {
  constexpr int NC = 16 * C;  // output columns of the workgroup
  __shared__ float red[NW][MT * 16][NC + 1];
  __shared__ float rinv_s[MT * 16];

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int r = lane & 15;
  const int g = lane >> 4;
  // Row blocks vary fastest so the blocks re-reading one weight tile run together.
  const int tile = blockIdx.y;
  const int row0 = blockIdx.x * (MT * 16);
  const int K = a.K;

  // Weight row feeding column 16*ct + r of this workgroup.
  const bf16_t* wrow[C];
  if (EPI == EPI_SWIGLU) {
    // columns [0, 8C) are gate rows j0.., columns [8C, 16C) the matching up rows
    const int j0 = tile * 8 * C;
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      const int c = 16 * ct + r;
      wrow[ct] = (c < 8 * C) ? a.W0 + (int64_t)(j0 + c) * K : a.W1 + (int64_t)(j0 + c - 8 * C) * K;
    }
  } else {
    const int n = tile * NC;
    const bf16_t* base;
    int nloc;
    if (n < a.n0) {
      base = a.W0; nloc = n;
    } else if (n < a.n0 + a.n1) {
      base = a.W1; nloc = n - a.n0;
    } else {
      base = a.W2; nloc = n - a.n0 - a.n1;
    }
#pragma unroll
    for (int ct = 0; ct < C; ++ct) wrow[ct] = base + (int64_t)(nloc + 16 * ct + r) * K;
  }
  const bf16_t* arow[MT];
  const bf16_t* arow_lo[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int m = row0 + mt * 16 + r;
    if (m >= a.M) m = a.M - 1;
    arow[mt] = a.A + (int64_t)m * a.lda;
    arow_lo[mt] = a.A_lo + (int64_t)m * a.lda;
  }

  // This wave's share of the K/32 steps.
  const int S = K / 32;
  const int base_steps = S / NW, rem = S % NW;
  const int s0 = w * base_steps + (w < rem ? w : rem);
  const int ns = base_steps + (w < rem ? 1 : 0);
  const int kbase = s0 * 32 + g * 8;

  f32x4 acc[MT][C];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ct = 0; ct < C; ++ct) acc[mt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  i32x4 wb0[U][C], ab0[U][MT], al0[U][MT], wb1[U][C], ab1[U][MT], al1[U][MT];

#define SBD_LOAD(WB, AB, AL, STEP)                                                 \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                                 \
    const int kk = kbase + ((STEP) + u) * 32;                                     \
    _Pragma("unroll") for (int ct = 0; ct < C; ++ct) WB[u][ct] = ld16_stream(wrow[ct] + kk); \
    _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) {                           \
      AB[u][mt] = ld16(arow[mt] + kk);                                            \
      AL[u][mt] = ld16(arow_lo[mt] + kk);                                         \
    }                                                                              \
  }
#define SBD_COMPUTE(WB, AB, AL)                                                    \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                                 \
    _Pragma("unroll") for (int mt = 0; mt < MT; ++mt)                             \
      _Pragma("unroll") for (int ct = 0; ct < C; ++ct) {                          \
        acc[mt][ct] = mfma16x16x32(AB[u][mt], WB[u][ct], acc[mt][ct]);            \
        acc[mt][ct] = mfma16x16x32(AL[u][mt], WB[u][ct], acc[mt][ct]);            \
      }                                                                            \
  }

  const int nchunks = ns / U;
  if (nchunks > 0) { SBD_LOAD(wb0, ab0, al0, 0); }

  // Per-row 1/rms from the producer's partial sums of squares (overlaps the first loads).
  if (EPI != EPI_RESID) {
    const int half = threadIdx.x >> 5, hl = threadIdx.x & 31;
    for (int rr = half; rr < MT * 16; rr += NW * 2) {
      const int m = row0 + rr;
      float sq = 0.f;
      if (a.sumsq_in != nullptr && m < a.M)
        for (int p = hl; p < a.n_part; p += 32) sq += a.sumsq_in[(int64_t)m * a.n_part + p];
      sq = half_wave_sum(sq);
      if (hl == 0) rinv_s[rr] = (a.sumsq_in != nullptr) ? 1.0f / sqrtf(sq * a.inv_d + a.eps) : 1.0f;
    }
  }

  for (int c = 0; c < nchunks; c += 2) {
    if (c + 1 < nchunks) { SBD_LOAD(wb1, ab1, al1, (c + 1) * U); }
    SBD_COMPUTE(wb0, ab0, al0);
    if (c + 1 < nchunks) {
      if (c + 2 < nchunks) { SBD_LOAD(wb0, ab0, al0, (c + 2) * U); }
      SBD_COMPUTE(wb1, ab1, al1);
    }
  }
  for (int st = nchunks * U; st < ns; ++st) {
    const int kk = kbase + st * 32;
    i32x4 wv[C];
#pragma unroll
    for (int ct = 0; ct < C; ++ct) wv[ct] = ld16_stream(wrow[ct] + kk);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const i32x4 av = ld16(arow[mt] + kk);
      const i32x4 avl = ld16(arow_lo[mt] + kk);
#pragma unroll
      for (int ct = 0; ct < C; ++ct) {
        acc[mt][ct] = mfma16x16x32(av, wv[ct], acc[mt][ct]);
        acc[mt][ct] = mfma16x16x32(avl, wv[ct], acc[mt][ct]);
      }
    }
  }
#undef SBD_LOAD
#undef SBD_COMPUTE

#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ct = 0; ct < C; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[w][mt * 16 + 4 * g + i][16 * ct + r] = acc[mt][ct][i];
  __syncthreads();

  // Epilogue: thread idx -> (row idx / NC, column idx % NC); each 16-lane group holds
  // 16 consecutive columns of one row.
  constexpr int TOTAL = MT * 16 * NC;
  constexpr int STRIDE = NW * 64;
  for (int idx = threadIdx.x; idx < (TOTAL + STRIDE - 1) / STRIDE * STRIDE; idx += STRIDE) {
    const bool in = idx < TOTAL;
    const int rr = in ? idx / NC : 0, col = idx % NC;
    const int m = row0 + rr;
    const bool ok = in && m < a.M;
    float y = 0.f;
    if (in) {
#pragma unroll
      for (int w2 = 0; w2 < NW; ++w2) y += red[w2][rr][col];
    }
    if (EPI == EPI_SCALED_STORE) {
      if (ok) a.out_f32[(int64_t)m * a.ldo + tile * NC + col] = y * rinv_s[rr];
    } else if (EPI == EPI_RESID) {
      const int n = tile * NC + col;
      float xv = 0.f;
      if (ok) {
        float* xp = a.x + (int64_t)m * a.ldx + n;
        xv = *xp + y;
        *xp = xv;
        bf16_t hi, lo;
        split_bf16(xv * bf2f(a.g_next[n]), hi, lo);
        a.xn[(int64_t)m * a.ldx + n] = hi;
        a.xn_lo[(int64_t)m * a.ldx + n] = lo;
      }
      float s2 = xv * xv;
      s2 += __shfl_xor(s2, 8);
      s2 += __shfl_xor(s2, 4);
      s2 += __shfl_xor(s2, 2);
      s2 += __shfl_xor(s2, 1);
      if ((col & 15) == 0 && ok) a.sumsq_out[(int64_t)m * a.n_part + n / 16] = s2;
    } else {  // EPI_SWIGLU
      if (ok && col < 8 * C) {
        float yu = 0.f;
#pragma unroll
        for (int w2 = 0; w2 < NW; ++w2) yu += red[w2][rr][col + 8 * C];
        const float gt = y * rinv_s[rr];
        const float up = yu * rinv_s[rr];
        const float sg = gt / (1.0f + expf(-gt));
        bf16_t hi, lo;
        split_bf16(sg * up, hi, lo);
        a.act[(int64_t)m * a.ld_act + tile * 8 * C + col] = hi;
        a.act_lo[(int64_t)m * a.ld_act + tile * 8 * C + col] = lo;
      }
    }
  }
}

template <int MT, int C, int NW, int U, int EPI>
static void launch_cfg(const GemmArgs& a, hipStream_t s) {
  // n_tiles counts 32-column tiles; this configuration covers 16*C columns per workgroup.
  const int tiles = a.n_tiles * 32 / (16 * C);
  dim3 grid((a.M + 16 * MT - 1) / (16 * MT), tiles);
  hipLaunchKernelGGL((gemm_kernel<MT, C, NW, U, EPI>), grid, dim3(NW * 64), 0, s, a);
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 16)
    launch_cfg<1, 2, 8, 4, EPI>(a, s);
  else if (a.M <= 32)
    launch_cfg<2, 2, 8, 4, EPI>(a, s);
  else
    launch_cfg<4, 2, 4, 2, EPI>(a, s);
  return hipGetLastError();
}

hipError_t launch_gemm(GemmEpi epi, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_SCALED_STORE: return launch_epi<EPI_SCALED_STORE>(a, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, s);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace sbd
