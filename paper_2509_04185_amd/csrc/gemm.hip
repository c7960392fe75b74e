// Skinny weight-streaming GEMM for the block forward: y[m][n] = sum_k A[m][k] W[n][k].
//
// The block forward multiplies M = batch * k activation rows (16 at batch 1, k = 16) by
// every weight matrix of the decoder, so it is bound by streaming the weights from HBM.
//
// Weights are repacked once (pack_kernel) into MFMA fragment order.  A matrix with N rows
// and K columns is cut into 16-row tiles; the 16-byte piece of lane l in step s of tile t
// holds W[16t + l%16][32s + 8(l/16) .. +8], so one 16-byte load per lane reads a 1 KB
// fragment that lands directly in the B operand of v_mfma_f32_16x16x32_bf16.  Tiles are
// grouped by 8 (128 rows) and a group's 8 fragments of one step are stored together:
// [N/128 groups][K/32 steps][8 tiles][64 lanes][8] (packed_frag() in sbd_device.h), so a
// decode-sized GEMM reading several tiles of a group per step reads contiguous memory.
// The gate and up projections share one packed matrix whose tile t holds gate rows
// 8t..8t+7 followed by up rows 8t..8t+7, so SwiGLU pairs stay inside one tile.
//
// This kernel serves M > 16 (prefill chunks, large batches); decode-sized products go
// through gemv.hip.  Each workgroup owns C consecutive tiles (16*C output columns) and a
// row block; its NW waves split the K/32 steps and stream disjoint contiguous ranges with
// non-temporal loads, double-buffered in registers.  The activations come as hi/lo bf16
// pairs (two MFMAs per step, see GemmArgs).  Partial sums meet in LDS and are added in a
// fixed wave order (deterministic); the epilogue applies what follows the product in the
// block:
//   EPI_SCALED_STORE  out = rinv[m] * y           (QKV projection, LM head)
//   EPI_RESID         x += y; xn = x * g_next as hi/lo; per-row sums of x^2 over each 16
//                     columns (O and down projections: residual add, the next RMSNorm's
//                     inputs)
//   EPI_SWIGLU        act = silu(rinv*gate) * rinv*up as hi/lo (gate/up projection)
// RMSNorm is split across two kernels: the producer writes x * g (gain applied) plus
// per-16-column partial sums of squares; the consumer adds the partials of a row and
// scales its fp32 result by 1/sqrt(mean(x^2) + eps), which equals normalising the input
// first because the scale is constant along a row.
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

  // This wave's share of the K/32 steps.
  const int S_all = K / 32;
  const int base_steps = S_all / NW, rem = S_all % NW;
  const int s0 = w * base_steps + (w < rem ? w : rem);
  const int ns = base_steps + (w < rem ? 1 : 0);
  const int kbase = s0 * 32 + g * 8;

  const bf16_t* wbase[C];
#pragma unroll
  for (int ct = 0; ct < C; ++ct)
    wbase[ct] = a.Wp + packed_frag(tile * C + ct, s0, S_all) + lane * 8;
  const bf16_t* arow[MT];
  const bf16_t* arow_lo[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int m = row0 + mt * 16 + r;
    if (m >= a.M) m = a.M - 1;
    arow[mt] = a.A + (int64_t)m * a.lda + kbase;
    arow_lo[mt] = a.A_lo + (int64_t)m * a.lda + kbase;
  }

  f32x4 acc[MT][C];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ct = 0; ct < C; ++ct) acc[mt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  i32x4 wb0[U][C], ab0[U][MT], al0[U][MT], wb1[U][C], ab1[U][MT], al1[U][MT];

#define SBD_LOAD(WB, AB, AL, STEP)                                                 \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                                 \
    const int st_ = (STEP) + u;                                                   \
    _Pragma("unroll") for (int ct = 0; ct < C; ++ct)                              \
      WB[u][ct] = ld16_stream(wbase[ct] + (int64_t)st_ * kPackStep);              \
    _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) {                           \
      AB[u][mt] = ld16(arow[mt] + st_ * 32);                                      \
      AL[u][mt] = ld16(arow_lo[mt] + st_ * 32);                                   \
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
    i32x4 wv[C];
#pragma unroll
    for (int ct = 0; ct < C; ++ct) wv[ct] = ld16_stream(wbase[ct] + (int64_t)st * kPackStep);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const i32x4 av = ld16(arow[mt] + st * 32);
      const i32x4 avl = ld16(arow_lo[mt] + st * 32);
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

  // Sum the waves' partial tiles into red[0] (fixed wave order).
  constexpr int TOTAL = MT * 16 * NC;
  constexpr int STRIDE = NW * 64;
  for (int idx = threadIdx.x; idx < TOTAL; idx += STRIDE) {
    const int rr = idx / NC, col = idx % NC;
    float y = red[0][rr][col];
#pragma unroll
    for (int w2 = 1; w2 < NW; ++w2) y += red[w2][rr][col];
    red[0][rr][col] = y;
  }

  __syncthreads();

  // Epilogue: thread idx -> (row idx / NC, column idx % NC); each 16-lane group holds
  // the 16 columns of one tile of one row.
  for (int idx = threadIdx.x; idx < (TOTAL + STRIDE - 1) / STRIDE * STRIDE; idx += STRIDE) {
    const bool in = idx < TOTAL;
    const int rr = in ? idx / NC : 0, col = idx % NC;
    const int m = row0 + rr;
    const bool ok = in && m < a.M;
    const float y = in ? red[0][rr][col] : 0.f;
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
    } else {  // EPI_SWIGLU: column c < 8 of a tile is gate j, column c + 8 the matching up
      const int c = col & 15;
      if (ok && c < 8) {
        const float gt = y * rinv_s[rr];
        const float up = red[0][rr][col + 8] * rinv_s[rr];
        const float sg = gt / (1.0f + expf(-gt));
        const int j = (tile * C + (col >> 4)) * 8 + c;
        bf16_t hi, lo;
        split_bf16(sg * up, hi, lo);
        a.act[(int64_t)m * a.ld_act + j] = hi;
        a.act_lo[(int64_t)m * a.ld_act + j] = lo;
      }
    }
  }
}

template <int MT, int C, int NW, int U, int EPI>
static void launch_cfg(const GemmArgs& a, const Exec& ex) {
  dim3 grid((a.M + 16 * MT - 1) / (16 * MT), a.n_tiles / C);
  SBD_KLAUNCH((gemm_kernel<MT, C, NW, U, EPI>), grid, dim3(NW * 64), ex, a);
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, const Exec& ex) {
  if (a.M <= 16)
    launch_cfg<1, 2, 4, 4, EPI>(a, ex);
  else if (a.M <= 32)
    launch_cfg<2, 2, 8, 4, EPI>(a, ex);
  else
    launch_cfg<4, 2, 4, 2, EPI>(a, ex);
  return hipGetLastError();
}

hipError_t launch_gemm(GemmEpi epi, const GemmArgs& a, const Exec& ex) {
  if (a.M < 1 || a.K < 32 || a.K % 32 || a.n_tiles % 8) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_SCALED_STORE: return launch_epi<EPI_SCALED_STORE>(a, ex);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, ex);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(a, ex);
    default: return hipErrorInvalidValue;
  }
}

// One thread per 16-byte piece of the packed matrix (layout at the top of this file).
// Mode 0: packed row n is src0 row n.  Mode 1 (gate/up): packed tile t holds src0 rows
// 8t..8t+7 then src1 rows 8t..8t+7.
__global__ __launch_bounds__(256) void pack_kernel(const bf16_t* src0, const bf16_t* src1,
                                                   bf16_t* dst, int64_t n_pieces, int K, int mode) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_pieces) return;
  const int S = K / 32;
  const int lane = (int)(i % 64);
  const int64_t tt = (i / 64) % 8;            // tile inside the group
  const int64_t s = (i / 512) % S;            // K step
  const int64_t t = (i / (512 * (int64_t)S)) * 8 + tt;
  const int rr = lane & 15;
  const int64_t k0 = 32 * s + 8 * (lane >> 4);
  const bf16_t* row;
  if (mode == 0)
    row = src0 + (t * 16 + rr) * (int64_t)K;
  else
    row = (rr < 8) ? src0 + (t * 8 + rr) * (int64_t)K : src1 + (t * 8 + rr - 8) * (int64_t)K;
  *(i32x4*)(dst + i * 8) = *(const i32x4*)(row + k0);
}

hipError_t launch_pack(const bf16_t* src0, const bf16_t* src1, bf16_t* dst, int64_t rows, int K,
                       int mode, hipStream_t s) {
  if (rows % 128 || K % 32) return hipErrorInvalidValue;
  const int64_t n_pieces = rows * K / 8;
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)((n_pieces + 255) / 256)), dim3(256), 0, s, src0,
                     src1, dst, n_pieces, K, mode);
  return hipGetLastError();
}

}  // namespace sbd
