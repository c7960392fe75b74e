// Skinny weight-streaming GEMM for the block forward: y[m][n] = sum_k A[m][k] W[n][k].
//
// The block forward multiplies M = batch * k activation rows (16 at batch 1, k = 16) by
// every weight matrix of the decoder, so it is bound by streaming the weights from HBM.
// Each workgroup owns 32 output columns (two 16-wide MFMA tiles) and the row block; its
// NW waves split the reduction dimension K and stream disjoint K ranges of the same 32
// weight rows with 16-byte non-temporal loads, double-buffered in registers.  Partial
// sums meet in LDS and are added in a fixed wave order (deterministic), and the
// epilogue applies the operation that follows the product in the decoder block:
//   EPI_SCALED_STORE  out = rinv[m] * y           (QKV projection, LM head)
//   EPI_RESID         x += y; xn = bf16(x * g_next); per-row sum of x^2 of the tile
//                     (O and down projections: residual add, next RMSNorm's inputs)
//   EPI_SWIGLU        act = bf16(silu(rinv*gate) * rinv*up)  (gate/up projection)
// RMSNorm is split across two kernels: the producer writes x * g (gain applied, bf16)
// plus per-32-column partial sums of squares; the consumer adds the partials of a row
// and scales its fp32 result by 1/sqrt(mean(x^2) + eps), which equals normalising the
// input first because the scale is constant along a row.
//
// MFMA v_mfma_f32_16x16x32_bf16: lane l holds row (l % 16) of A and column (l % 16) of
// B^T for the 8 consecutive k of group l / 16; the result holds rows 4*(l/16)+i of
// column l % 16.

#include "sbd_device.h"

namespace sbd {

template <int MT, int NW, int U, int EPI>
__global__ __launch_bounds__(NW * 64) void gemm_kernel(GemmArgs a) {
  __shared__ float red[NW][MT * 16][33];
  __shared__ float rinv_s[MT * 16];

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int r = lane & 15;
  const int g = lane >> 4;
  // Row blocks vary fastest so the blocks re-reading one weight tile run together.
  const int tile = blockIdx.y;
  const int row0 = blockIdx.x * (MT * 16);
  const int K = a.K;

  // Weight rows of the two 16-wide column tiles.
  const bf16_t* wrow0;
  const bf16_t* wrow1;
  if (EPI == EPI_SWIGLU) {
    const int j0 = tile * 16;
    wrow0 = a.W0 + (int64_t)(j0 + r) * K;
    wrow1 = a.W1 + (int64_t)(j0 + r) * K;
  } else {
    const int n = tile * 32;
    const bf16_t* base;
    int nloc;
    if (n < a.n0) {
      base = a.W0; nloc = n;
    } else if (n < a.n0 + a.n1) {
      base = a.W1; nloc = n - a.n0;
    } else {
      base = a.W2; nloc = n - a.n0 - a.n1;
    }
    wrow0 = base + (int64_t)(nloc + r) * K;
    wrow1 = base + (int64_t)(nloc + 16 + r) * K;
  }
  const bf16_t* arow[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int m = row0 + mt * 16 + r;
    if (m >= a.M) m = a.M - 1;
    arow[mt] = a.A + (int64_t)m * a.lda;
  }

  // This wave's share of the K/32 steps.
  const int S = K / 32;
  const int base_steps = S / NW, rem = S % NW;
  const int s0 = w * base_steps + (w < rem ? w : rem);
  const int ns = base_steps + (w < rem ? 1 : 0);
  const int kbase = s0 * 32 + g * 8;

  f32x4 acc[MT][2];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    acc[mt][0] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc[mt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  i32x4 wb0[U][2], ab0[U][MT], wb1[U][2], ab1[U][MT];

#define SBD_LOAD(WB, AB, STEP)                                              \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                          \
    const int kk = kbase + ((STEP) + u) * 32;                              \
    WB[u][0] = ld16_stream(wrow0 + kk);                                    \
    WB[u][1] = ld16_stream(wrow1 + kk);                                    \
    _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) AB[u][mt] = ld16(arow[mt] + kk); \
  }
#define SBD_COMPUTE(WB, AB)                                                 \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                          \
    _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) {                    \
      acc[mt][0] = mfma16x16x32(AB[u][mt], WB[u][0], acc[mt][0]);          \
      acc[mt][1] = mfma16x16x32(AB[u][mt], WB[u][1], acc[mt][1]);          \
    }                                                                       \
  }

  const int nchunks = ns / U;
  if (nchunks > 0) { SBD_LOAD(wb0, ab0, 0); }
  for (int c = 0; c < nchunks; c += 2) {
    if (c + 1 < nchunks) { SBD_LOAD(wb1, ab1, (c + 1) * U); }
    SBD_COMPUTE(wb0, ab0);
    if (c + 1 < nchunks) {
      if (c + 2 < nchunks) { SBD_LOAD(wb0, ab0, (c + 2) * U); }
      SBD_COMPUTE(wb1, ab1);
    }
  }
  for (int st = nchunks * U; st < ns; ++st) {
    const int kk = kbase + st * 32;
    const i32x4 w0 = ld16_stream(wrow0 + kk);
    const i32x4 w1 = ld16_stream(wrow1 + kk);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const i32x4 av = ld16(arow[mt] + kk);
      acc[mt][0] = mfma16x16x32(av, w0, acc[mt][0]);
      acc[mt][1] = mfma16x16x32(av, w1, acc[mt][1]);
    }
  }
#undef SBD_LOAD
#undef SBD_COMPUTE

  // Per-row 1/rms from the producer's partial sums of squares.
  if (EPI != EPI_RESID) {
    const int half = threadIdx.x >> 5, hl = threadIdx.x & 31;
    for (int rr = half; rr < MT * 16; rr += NW * 2) {
      const int m = row0 + rr;
      float s = 0.f;
      if (a.sumsq_in != nullptr && m < a.M)
        for (int p = hl; p < a.n_part; p += 32) s += a.sumsq_in[(int64_t)m * a.n_part + p];
      s = half_wave_sum(s);
      if (hl == 0) rinv_s[rr] = (a.sumsq_in != nullptr) ? 1.0f / sqrtf(s * a.inv_d + a.eps) : 1.0f;
    }
  }

#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      red[w][mt * 16 + 4 * g + i][r] = acc[mt][0][i];
      red[w][mt * 16 + 4 * g + i][16 + r] = acc[mt][1][i];
    }
  __syncthreads();

  for (int idx = threadIdx.x; idx < MT * 16 * 32; idx += NW * 64) {
    const int rr = idx >> 5, col = idx & 31;
    const int m = row0 + rr;
    float y = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < NW; ++w2) y += red[w2][rr][col];
    if (EPI == EPI_SCALED_STORE) {
      if (m < a.M) a.out_f32[(int64_t)m * a.ldo + tile * 32 + col] = y * rinv_s[rr];
    } else if (EPI == EPI_RESID) {
      const int n = tile * 32 + col;
      float xv = 0.f;
      if (m < a.M) {
        float* xp = a.x + (int64_t)m * a.ldx + n;
        xv = *xp + y;
        *xp = xv;
        a.xn[(int64_t)m * a.ldx + n] = f2bf(xv * bf2f(a.g_next[n]));
      }
      const float s2 = half_wave_sum(xv * xv);
      if (col == 0 && m < a.M) a.sumsq_out[(int64_t)m * a.n_part + tile] = s2;
    } else {  // EPI_SWIGLU
      if (col < 16 && m < a.M) {
        float yu = 0.f;
#pragma unroll
        for (int w2 = 0; w2 < NW; ++w2) yu += red[w2][rr][col + 16];
        const float gt = y * rinv_s[rr];
        const float up = yu * rinv_s[rr];
        const float sg = gt / (1.0f + expf(-gt));
        a.act[(int64_t)m * a.ld_act + tile * 16 + col] = f2bf(sg * up);
      }
    }
  }
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 16) {
    dim3 grid((a.M + 15) / 16, a.n_tiles);
    hipLaunchKernelGGL((gemm_kernel<1, 8, 8, EPI>), grid, dim3(8 * 64), 0, s, a);
  } else if (a.M <= 32) {
    dim3 grid((a.M + 31) / 32, a.n_tiles);
    hipLaunchKernelGGL((gemm_kernel<2, 8, 4, EPI>), grid, dim3(8 * 64), 0, s, a);
  } else {
    dim3 grid((a.M + 63) / 64, a.n_tiles);
    hipLaunchKernelGGL((gemm_kernel<4, 4, 2, EPI>), grid, dim3(4 * 64), 0, s, a);
  }
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
