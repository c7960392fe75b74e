// Decode-sized GEMM (M <= 16 rows): y[m][n] = sum_k A[m][k] W[n][k].
//
// At M <= 16 every projection of the block forward is a stream of its weights from HBM.
// The kernel is shaped by three measured costs: bytes in flight per CU, the activation
// fragments re-read for every weight fragment, and the fixed latency at the start and end
// of a launch.
//   - A workgroup owns C consecutive tiles (C = 1..8; they may straddle packed groups) and
//     a K range; a K step then reads C KB of weights against 2 KB of activation fragments
//     (hi and lo).  C need not divide 8, so a projection can be cut into exactly as many
//     workgroups as the chip has CUs (gate/up at the 8B shape: 1792 tiles = 256 x 7).
//   - Its NW waves split the K range and stream it (gemv_body.h: batches of U steps,
//     double-buffered, 2U steps in flight per wave).  A short kernel is a few memory round
//     trips long; what it needs from memory besides the weights (norm partials, residual
//     rows, rotary rows, positions) is requested before the weight stream starts.
//   - The NW partial tiles are added in LDS in wave order.  When the K range is split over
//     KS workgroups, all of them run on one XCD: each parks its partial tiles in that XCD's
//     L2 and the last to arrive adds the KS slices in order and runs the epilogue.  Results
//     are deterministic; no workgroup waits for another.
//
// Epilogues (acc in the v_mfma_f32_16x16x32_bf16 D layout: lane l holds column l % 16 of
// a tile, rows 4*(l/16) + i):
//   EPI_SCALED_STORE  out = rinv[m] * y                      (LM head)
//   EPI_LOGITS_EB     the same (stores optional) plus, per row and 64-column chunk (4 of
//                     the C = 8 tiles), the EB softmax statistics (eb_stats.h)
//   EPI_RESID         x += y; xn = x * g_next as hi/lo bf16; one partial sum of x^2 per
//                     row and workgroup for the next RMSNorm (O, down projections)
//   EPI_SWIGLU        act = silu(rinv*gate) * rinv*up as hi/lo (gate/up: packed tile t
//                     holds gate rows 8t..8t+7 then up rows 8t..8t+7)
//   EPI_QKV           C = 8 (128 columns = whole heads): per-head q/k RMSNorm, rotate-half
//                     RoPE, q as scaled hi/lo, K and V into the cache at cache_len + j
// Activations are hi/lo bf16 pairs: two MFMAs per step, exact products in fp32.
// RMSNorm is split between kernels: the producer of x (EPI_RESID, or the embedding) writes
// x * g and partial sums of x^2; the consumer adds the partials of its rows, loaded before
// its weight stream starts, and scales its fp32 products by rinv[m] = 1/sqrt(mean(x^2) +
// eps), which equals normalising the input because the scale is constant along a row.

#include <algorithm>

#include "eb_stats.h"
#include "gemv_body.h"
#include "qkv_epilogue.h"

namespace sbd {

// Tile ct of a workgroup is summed and finished by wave ct % NW.
template <int NW>
__device__ __forceinline__ bool owns_tile(int ct, int wave) { return ct % NW == wave; }

template <int C, int NW, int U, int EPI, int DH, class WT>
__global__ __launch_bounds__(NW * 64) void gemv_kernel(GemvArgs a) {
  static_assert(C >= 1 && C <= 8, "a workgroup takes one to eight tiles");
  static_assert(EPI != EPI_QKV || C == 8, "the QKV epilogue works on whole groups");
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  // Workgroup x runs on XCD x % 8; the KS slices of unit `sub` (tiles sub*C .. sub*C + C-1)
  // all sit on XCD sub % 8, so their hand-off stays in that XCD's L2.  The unit count is
  // padded to a multiple of 8; padding workgroups leave at once.
  const int KS = a.splits;
  const int sub = (int)((blockIdx.x >> 3) / KS) * 8 + (int)(blockIdx.x & 7);
  const int kc = (int)((blockIdx.x >> 3) % KS);
  if (sub * C >= a.n_tiles) return;
  const int t0 = sub * C;
  const int S = a.K / 32;
  const int z0 = (int)((int64_t)S * kc / KS), z1 = (int)((int64_t)S * (kc + 1) / KS);
  const int s_b = z0 + (z1 - z0) * wave / NW, s_e = z0 + (z1 - z0) * (wave + 1) / NW;
  const int ns = s_e - s_b;

  // Consumers: the partial sums of squares of the input rows, loaded before the weight
  // stream; thread t adds partials q, q + tpr, ... of row t / tpr (tpr threads per row).
  constexpr int tpr = NW * 4;
  constexpr int kPre = 8;
  float sq_pre[kPre];
  const int sq_m = threadIdx.x / tpr, sq_q = threadIdx.x % tpr;
  const bool sq_on = EPI != EPI_RESID && a.sumsq_in != nullptr && sq_m < a.M;
#pragma unroll
  for (int j = 0; j < kPre; ++j) {
    const int p = sq_q + j * tpr;
    sq_pre[j] = (sq_on && p < a.n_part_in) ? a.sumsq_in[(int64_t)sq_m * a.n_part_in + p] : 0.f;
  }
  // EPI_RESID: the residual rows and the next norm's gain for the tiles this wave finishes
  float x_pre[(C + NW - 1) / NW][4], g_pre[(C + NW - 1) / NW];
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int k2 = 0; k2 < (C + NW - 1) / NW; ++k2) {
      const int ct = wave + k2 * NW;
      const int n = (t0 + (ct < C ? ct : 0)) * 16 + r;
      g_pre[k2] = bf2f(a.g_next[n]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 4 * g + i;
        x_pre[k2][i] = (ct < C && m < a.M) ? a.x[(int64_t)m * a.ldx + n] : 0.f;
      }
    }
  }

  QkvPre<DH> qpre;
  if constexpr (EPI == EPI_QKV) qkv_epi_prefetch<DH>(a.qkv, a.M, qpre);

  const int arow_m = r < a.M ? r : a.M - 1;
  const uint32_t a_off = (uint32_t)(((int64_t)arow_m * a.lda + g * 8 + s_b * 32) * 2);
  // tile t0 + ct at step s_b; consecutive steps of a tile are kPackStep apart
  const WT* wbase;
  if constexpr (sizeof(WT) == 1) wbase = a.Wp8; else wbase = a.Wp;
  const WT* wt[C];
#pragma unroll
  for (int ct = 0; ct < C; ++ct) wt[ct] = wbase + packed_frag(t0 + ct, s_b, S) + lane * 8;
  float wsc[C];
  load_wscale<WT, C>(a.wscale, t0, r, wsc);

  f32x4 acc[C];
#pragma unroll
  for (int ct = 0; ct < C; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  {
    typename WFrag<WT>::T w0[U][C];
    gemv_stream<C, U, 0, false>(buf_rsrc(a.A), buf_rsrc(a.A_lo), a_off, wt, ns, w0, wsc, acc);
  }

  // ---- 1/rms of this lane's accumulator rows 4g + i
  __shared__ float rinv_s[16];
  __shared__ float ssq_s[C][16];  // EPI_RESID: per-tile sums of x^2 of each row
  float rinv[4] = {1.f, 1.f, 1.f, 1.f};
  if constexpr (EPI != EPI_RESID) {
    if (a.sumsq_in != nullptr) {
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < kPre; ++j) s += sq_pre[j];
      for (int p = sq_q + kPre * tpr; sq_on && p < a.n_part_in; p += tpr)
        s += a.sumsq_in[(int64_t)sq_m * a.n_part_in + p];
#pragma unroll
      for (int o = tpr / 2; o >= 1; o /= 2) s += __shfl_xor(s, o);
      if (sq_q == 0 && sq_m < 16) rinv_s[sq_m] = 1.0f / sqrtf(s * a.inv_d + a.eps);
      __syncthreads();
#pragma unroll
      for (int i = 0; i < 4; ++i) rinv[i] = rinv_s[4 * g + i];
    }
  }

  // ---- the NW partial tiles, added in LDS in wave order
  if constexpr (NW > 1) {
    __shared__ f32x4 red[NW][C][64];
#pragma unroll
    for (int ct = 0; ct < C; ++ct) red[wave][ct][lane] = acc[ct];
    __syncthreads();
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      if (!owns_tile<NW>(ct, wave)) continue;
      f32x4 s = red[0][ct][lane];
      for (int w = 1; w < NW; ++w) s += red[w][ct][lane];
      acc[ct] = s;
    }
  }

  // ---- K split over workgroups: park the slice, the last to arrive adds all in order
  if (KS > 1) {
    const __amdgpu_buffer_rsrc_t rp = buf_rsrc(a.part);
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      if (!owns_tile<NW>(ct, wave)) continue;
      *(f32x4*)(a.part + (((int64_t)kc * a.n_tiles + t0 + ct) * 64 + lane) * 4) = acc[ct];
    }
    if (!last_arrival_xcd(a.counters + (int64_t)sub * kCtrStride, KS)) return;
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      if (!owns_tile<NW>(ct, wave)) continue;
      f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int z0 = 0; z0 < KS; z0 += 4) {  // four slices in flight, added in slice order
        i32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          v[u] = z0 + u < KS ? ld16_l2(rp, (uint32_t)((((int64_t)(z0 + u) * a.n_tiles + t0 + ct) * 64 + lane) * 16))
                             : i32x4{0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < 4; ++u) s += __builtin_bit_cast(f32x4, v[u]);
      }
      acc[ct] = s;
    }
  }

  // ---- epilogue
  if constexpr (EPI == EPI_QKV) {
    if constexpr (NW > 1) {  // gather the group's 8 tiles in wave 0
      __shared__ f32x4 fin[C][64];
#pragma unroll
      for (int ct = 0; ct < C; ++ct)
        if (owns_tile<NW>(ct, wave)) fin[ct][lane] = acc[ct];
      __syncthreads();
      if (wave != 0) return;
#pragma unroll
      for (int ct = 0; ct < C; ++ct) acc[ct] = fin[ct][lane];
    }
    qkv_epilogue<DH>(a.qkv, a.M, sub, acc, rinv, qpre);
    return;
  } else if constexpr (EPI == EPI_LOGITS_EB) {
    static_assert(C == 8 && NW == 1, "the logits statistics take whole groups in one wave");
    // the logits as EPI_SCALED_STORE; the fp32 products staged in LDS as [16 rows][128
    // columns]; then lane L reduces 32 columns of row L / 4 (quarter L % 4), two lanes per
    // 64-column chunk
    __shared__ __attribute__((aligned(16))) float st[16][8 * 16 + 4];
#pragma unroll
    for (int ct = 0; ct < C; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 4 * g + i;
        if (a.out_f32 != nullptr && m < a.M) a.out_f32[(int64_t)m * a.ldo + (t0 + ct) * 16 + r] = acc[ct][i] * rinv[i];
        st[m][ct * 16 + r] = acc[ct][i];
      }
    __builtin_amdgcn_wave_barrier();
    const int row = lane >> 2, seg = lane & 3;
    float mx;
    int arg;
    double z, sz;
    eb_seg_stats<32, 2>(&st[row][seg * 32], a.sumsq_in != nullptr ? rinv_s[row] : 1.f, t0 * 16 + seg * 32, a.eb_mask_id, mx, arg, z, sz);
    if ((seg & 1) == 0 && row < a.M) eb_chunk_store(a.eb_part, a.eb_arg, a.eb_chunks, row, t0 / 4 + seg / 2, mx, arg, z, sz);
    return;
  } else {
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      if (!owns_tile<NW>(ct, wave)) continue;
      const int tile = t0 + ct;
      if constexpr (EPI == EPI_SCALED_STORE) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = 4 * g + i;
          if (m < a.M) a.out_f32[(int64_t)m * a.ldo + tile * 16 + r] = acc[ct][i] * rinv[i];
        }
      } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = 4 * g + i;
          const float v = acc[ct][i] * (m < a.M ? rinv[i] : 0.f);
          const float up = __shfl_xor(v, 8);
          if (r < 8 && m < a.M) {
            const int jj = tile * 8 + r;
            bf16_t hi, lo;
            split_bf16(v / (1.0f + expf(-v)) * up, hi, lo);
            a.act[(int64_t)m * a.ld_act + jj] = hi;
            a.act_lo[(int64_t)m * a.ld_act + jj] = lo;
          }
        }
      } else {  // EPI_RESID
        const int k2 = ct / NW;
        const int n = tile * 16 + r;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = 4 * g + i;
          float xv = 0.f;
          if (m < a.M) {
            xv = x_pre[k2][i] + acc[ct][i];
            a.x[(int64_t)m * a.ldx + n] = xv;
            bf16_t hi, lo;
            split_bf16(xv * g_pre[k2], hi, lo);
            a.xn[(int64_t)m * a.ldx + n] = hi;
            a.xn_lo[(int64_t)m * a.ldx + n] = lo;
          }
          float s2 = xv * xv;
          s2 += __shfl_xor(s2, 1);
          s2 += __shfl_xor(s2, 2);
          s2 += __shfl_xor(s2, 4);
          s2 += __shfl_xor(s2, 8);
          if (r == 0) ssq_s[ct][m] = s2;
        }
      }
    }
  }

  if constexpr (EPI == EPI_RESID) {
    // one partial sum of x^2 per row for this workgroup's C tiles, added in tile order
    __syncthreads();
    if (threadIdx.x < a.M) {
      float s = 0.f;
#pragma unroll
      for (int ct = 0; ct < C; ++ct) s += ssq_s[ct][threadIdx.x];
      a.sumsq[(int64_t)threadIdx.x * a.n_part + sub] = s;
    }
  }
}

// An fp8 matrix keeps the bf16 shape's bytes in flight with twice the steps per batch.
template <int C, int NW, int U, int EPI, int DH = 128>
static void launch_gemv_cfg(const GemvArgs& a, int KS, const Exec& ex) {
  const int units = (a.n_tiles / C + 7) / 8 * 8;
  GemvArgs b = a;
  b.splits = KS;
  if (a.Wp8 != nullptr)
    SBD_KLAUNCH((gemv_kernel<C, NW, 2 * U, EPI, DH, fp8_t>), dim3((unsigned)(units * KS)), dim3(NW * 64), ex, b);
  else
    SBD_KLAUNCH((gemv_kernel<C, NW, U, EPI, DH, bf16_t>), dim3((unsigned)(units * KS)), dim3(NW * 64), ex, b);
}

// Launch shapes from sweeps over the 8B decode shapes (M = 16), timed as chains of launches
// over rotating weight copies.  Many tiles (LM head, gate/up): whole groups, few waves, no
// split.  Few tiles (QKV, O, down): the K range is split over workgroups until about one
// workgroup per CU streams (QKV 48 groups x 5, O and down 64 half groups x 4), keeping at
// least 8 K steps per workgroup.
GemvShape gemv_pick(GemmEpi epi, int n_tiles, int K) {
  const int groups = n_tiles / 8, S = K / 32;
  if (groups >= 512) return GemvShape{8, 1, 2, 1};
  if (groups >= 192) return GemvShape{8, 4, 1, 1};
  if (epi == EPI_QKV) {
    int KS = std::max(1, std::min(256 / groups, kGemvMaxSplit));
    while (KS > 1 && S / KS < 8) --KS;
    return GemvShape{8, 4, 1, KS};
  }
  const int units = n_tiles / 4;
  int KS = std::max(1, std::min(256 / std::max(units, 1), kGemvMaxSplit));
  while (KS > 1 && S / KS < 8) --KS;
  return GemvShape{4, 8, (S / KS) / 8 >= 8 ? 2 : 4, KS};
}

template <int EPI, int DH = 128>
static bool dispatch(const GemvArgs& a, GemvShape sh, const Exec& ex) {
  const int c = sh.C * 1000 + sh.NW * 10 + sh.U;
  if constexpr (EPI == EPI_LOGITS_EB) {  // one shape: whole groups, one wave, no split
    if (c != 8012 || sh.KS != 1) return false;
    launch_gemv_cfg<8, 1, 2, EPI>(a, 1, ex);
    return true;
  } else {
    switch (c) {
      case 8041: launch_gemv_cfg<8, 4, 1, EPI, DH>(a, sh.KS, ex); return true;
      case 8012: launch_gemv_cfg<8, 1, 2, EPI, DH>(a, sh.KS, ex); return true;
      default: break;
    }
    if constexpr (EPI != EPI_QKV) {
      switch (c) {
        case 4084: launch_gemv_cfg<4, 8, 4, EPI>(a, sh.KS, ex); return true;
        case 4082: launch_gemv_cfg<4, 8, 2, EPI>(a, sh.KS, ex); return true;
        default: break;
      }
    }
    return false;
  }
}

hipError_t launch_gemv(GemmEpi epi, const GemvArgs& a, GemvShape sh, const Exec& ex) {
  if (a.M < 1 || a.M > 16 || a.K < 32 || a.K % 32 || a.n_tiles < 8 || a.n_tiles % 8) return hipErrorInvalidValue;
  if (a.Wp8 != nullptr && a.wscale == nullptr) return hipErrorInvalidValue;
  if (sh.C == 0) sh = epi == EPI_LOGITS_EB ? GemvShape{8, 1, 2, 1} : gemv_pick(epi, a.n_tiles, a.K);
  if (a.no_split) sh.KS = 1;
  if (epi == EPI_LOGITS_EB && (a.eb_part == nullptr || a.eb_arg == nullptr || a.eb_chunks * kEbFChunk != a.n_tiles * 16))
    return hipErrorInvalidValue;
  if (sh.KS < 1 || sh.KS > kGemvMaxSplit || a.n_tiles % sh.C) return hipErrorInvalidValue;
  if (sh.KS > 1 && (int64_t)(a.n_tiles / sh.C + 7) / 8 * 8 * kCtrStride > kLayerCtr0) return hipErrorInvalidValue;
  if (sh.KS > 1 && a.counters == nullptr) return hipErrorInvalidValue;
  if (epi == EPI_RESID && (a.sumsq == nullptr || a.n_part != a.n_tiles / sh.C)) return hipErrorInvalidValue;
  if (sh.KS > 1 && (a.part == nullptr || (int64_t)sh.KS * a.n_tiles * 256 > a.part_cap))
    return hipErrorInvalidValue;
  bool ok = false;
  switch (epi) {
    case EPI_QKV:
      if (sh.C != 8) return hipErrorInvalidValue;
      if (a.qkv.d_h == 128)
        ok = dispatch<EPI_QKV, 128>(a, sh, ex);
      else if (a.qkv.d_h == 64)
        ok = dispatch<EPI_QKV, 64>(a, sh, ex);
      break;
    case EPI_RESID: ok = dispatch<EPI_RESID>(a, sh, ex); break;
    case EPI_SWIGLU: ok = dispatch<EPI_SWIGLU>(a, sh, ex); break;
    case EPI_SCALED_STORE: ok = dispatch<EPI_SCALED_STORE>(a, sh, ex); break;
    case EPI_LOGITS_EB: ok = dispatch<EPI_LOGITS_EB>(a, sh, ex); break;
  }
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sbd

namespace sbd {

// Packing of e4m3 matrices: one thread per 8-element piece, in the order of the bf16 packing
// (gemm.hip's pack_kernel; mode 1 interleaves gate and up rows per tile).  WIDEN: write the
// piece as bf16 values q * 2^e (the scaled conversion, exact) into the bf16 packing, else the
// bytes themselves into the fp8 packing.
template <bool WIDEN>
__global__ __launch_bounds__(256) void pack_fp8_kernel(const fp8_t* src0, const fp8_t* src1, float sc0, float sc1,
                                                       void* dst, int64_t n_pieces, int K, int mode) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_pieces) return;
  const int S = K / 32;
  const int lane = (int)(i % 64);
  const int64_t tt = (i / 64) % 8;
  const int64_t s = (i / 512) % S;
  const int64_t t = (i / (512 * (int64_t)S)) * 8 + tt;
  const int rr = lane & 15;
  const int64_t k0 = 32 * s + 8 * (lane >> 4);
  const bool second = mode == 1 && rr >= 8;
  const fp8_t* row = mode == 0 ? src0 + (t * 16 + rr) * (int64_t)K
                               : (second ? src1 + (t * 8 + rr - 8) * (int64_t)K : src0 + (t * 8 + rr) * (int64_t)K);
  const i32x2 q = *reinterpret_cast<const i32x2*>(row + k0);
  if constexpr (WIDEN)
    *reinterpret_cast<i32x4*>(static_cast<bf16_t*>(dst) + i * 8) = w_operand(q, second ? sc1 : sc0);
  else
    *reinterpret_cast<i32x2*>(static_cast<fp8_t*>(dst) + i * 8) = q;
}

static hipError_t pack_fp8(bool widen, const fp8_t* src0, const fp8_t* src1, float sc0, float sc1, void* dst,
                           int64_t rows, int K, int mode, hipStream_t s) {
  if (rows % 128 || K % 32) return hipErrorInvalidValue;
  const int64_t n_pieces = rows * K / 8;
  const dim3 grid((unsigned)((n_pieces + 255) / 256));
  if (widen)
    hipLaunchKernelGGL(pack_fp8_kernel<true>, grid, dim3(256), 0, s, src0, src1, sc0, sc1, dst, n_pieces, K, mode);
  else
    hipLaunchKernelGGL(pack_fp8_kernel<false>, grid, dim3(256), 0, s, src0, src1, sc0, sc1, dst, n_pieces, K, mode);
  return hipGetLastError();
}

hipError_t launch_pack_fp8(const fp8_t* src0, const fp8_t* src1, fp8_t* dst, int64_t rows, int K, int mode,
                           hipStream_t s) {
  return pack_fp8(false, src0, src1, 1.f, 1.f, dst, rows, K, mode, s);
}

hipError_t launch_pack_fp8_widen(const fp8_t* src0, const fp8_t* src1, int e0, int e1, bf16_t* dst, int64_t rows,
                                 int K, int mode, hipStream_t s) {
  return pack_fp8(true, src0, src1, ldexpf(1.f, e0), ldexpf(1.f, e1), dst, rows, K, mode, s);
}

}  // namespace sbd
