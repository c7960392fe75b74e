// Fused decode forward: every layer of a decode-sized block forward (M <= 16 rows) and the
// LM head in one launch of one persistent workgroup per CU.
//
// A forward of M <= 16 rows is a stream of the weights from HBM interrupted by short
// dependency chains (RMSNorm needs whole rows, attention needs the new K and V, ...).  As
// separate kernels, every boundary costs the launch, the first load latency of the next
// kernel and the tail of the previous one.  Here NWG workgroups (one per CU, all resident)
// walk through the phases of every layer in order:
//   QKV projection (+ q/k norm, RoPE, K/V into the cache) -> attention splits -> attention
//   merge -> O projection (+ residual) -> gate/up (+ SwiGLU) -> down (+ residual),
// and finally the LM head.  Phases are separated by counters, not kernel boundaries: a
// workgroup raises a counter once its stores for the next phase have completed, and waits
// for the counters its inputs depend on.  Before it waits, every wave requests the first
// U steps of its weights for the next phase (weights never depend on activations), so the
// weight stream overlaps the dependency chain: 4 waves x U x 8 KB per CU in flight.
//
// Weight streaming is balanced exactly: a GEMM phase's (group, K step) units (a group is
// 128 output columns, a unit 8 KB of packed weights) are divided into NWG equal contiguous
// ranges, one per workgroup, and each range into 4 per wave.  A range spans at most two
// groups; the waves' partial tiles meet in LDS, and a group shared by several workgroups
// is finished by the last of them to arrive, which adds the parked partials in workgroup
// order (deterministic) and runs the epilogue.
//
// Data that a workgroup writes for a workgroup of the same launch crosses XCDs, whose L2
// caches are not coherent with each other: such data is written and read with
// device-scope (sc1) accesses, and a producer raises a counter only after its stores have
// completed.  A wait polls with device-scope loads and gives up after a bounded number of
// polls, raising an error flag: a launch that cannot make progress ends, it never hangs.
//
// Two copies of the normalised activations and their partial sums of squares are kept:
// one written by the O projection (read by gate/up), one by the embedding or the down
// projection (read by the next QKV projection and the LM head).

#include "attention_body.h"
#include "qkv_epilogue.h"

namespace sbd {

constexpr int kFwdSmem = 98304;   // LDS per workgroup: more than half a CU's, so one per CU
constexpr int kSpinLimit = 1 << 20;  // polls before a wait is declared failed (~1 s)
constexpr int kFwdU = 4;          // K steps of weights requested per batch
constexpr int kC = 8;             // tiles (16 columns each) of a 128-column group
// LDS layout (bytes): [0, 64K) partial tiles [4 waves][2 groups][8 tiles][64 lanes] f32x4,
// or the attention's K/V chunks; then the QKV gather buffer, rinv and sums of squares.
constexpr int kSmemGather = 65536;
constexpr int kSmemRinv = kSmemGather + 8192;
constexpr int kSmemSsq = kSmemRinv + 64;

// Wait until *ctr >= target: thread 0 polls, then the workgroup proceeds.  Every later read
// of data produced in this launch is a device-scope load.
__device__ __forceinline__ void fwd_wait(const FwdArgs& f, int* ctr, int target, int what) {
  if (threadIdx.x == 0) {
    int it = 0;
    while (ld_i32_dev(ctr) < target) {
      __builtin_amdgcn_s_sleep(2);
      if ((++it & 1023) == 0 && ld_i32_dev(f.err) != 0) break;  // another wait already failed
      if (it > kSpinLimit) {
        atomicExch(f.err + 1, what);
        atomicOr(f.err, 1);
        break;
      }
    }
  }
  __syncthreads();
}

// Raise *ctr by n once every store of this workgroup has completed.
__device__ __forceinline__ void fwd_signal(int* ctr, int n) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) atomicAdd(ctr, n);
}

__device__ __forceinline__ int* layer_ctr(const FwdArgs& f, int layer, int which) {
  return f.ctl + f.plan.ctr0 + layer * f.plan.ctr_stride + which;
}

// One GEMM phase.
struct PGemm {
  const bf16_t* A;       // activations hi [M][lda] (device-scope loads)
  const bf16_t* A_lo;
  int lda, M, K;
  const bf16_t* W;       // packed weights
  int n_groups;
  const float* ssq_in;   // consumers: partial sums of x^2 of the A rows [M][n_part_in]
  int n_part_in;
  int* dep;              // wait until *dep >= dep_target before reading A
  int dep_target, dep_what;
  int* arr;              // arrival counters, one per group
  int phase;
};

// Units [u0, u1) of workgroup w out of nwg over T units.
__device__ __forceinline__ int64_t wg_unit(int64_t T, int w, int nwg) { return T * w / nwg; }
// The workgroup whose range holds unit u.
__device__ __forceinline__ int wg_of(int64_t u, int64_t T, int nwg) { return (int)(((u + 1) * nwg + T - 1) / T - 1); }

// Epilogue of group grp (C = 8 tiles) by one workgroup; wave v holds the final sums of tiles
// v and v + 4 in fin[0], fin[1].
template <int EPI, int DH>
__device__ __forceinline__ void group_epilogue(const FwdArgs& f, const PGemm& p, int layer, int grp,
                                               const f32x4 (&fin)[2], const float (&rinv)[4], char* smem) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  if constexpr (EPI == EPI_QKV) {
    f32x4* gat = reinterpret_cast<f32x4*>(smem + kSmemGather);
    gat[wave * 64 + lane] = fin[0];
    gat[(wave + 4) * 64 + lane] = fin[1];
    __syncthreads();
    if (wave == 0) {
      f32x4 acc[kC];
#pragma unroll
      for (int ct = 0; ct < kC; ++ct) acc[ct] = gat[ct * 64 + lane];
      QkvEpi e{};
      e.rows = f.rows; e.seqs = f.seqs; e.kblk = f.k; e.layer = layer;
      e.n_q = f.n_q; e.n_kv = f.n_kv; e.d_h = DH; e.qk_norm = f.qk_norm; e.eps = f.eps; e.q_scale = f.q_scale;
      e.rope = f.rope; e.q_norm = f.gains[layer].q_norm; e.k_norm = f.gains[layer].k_norm;
      e.q = f.q; e.q_lo = f.q_lo; e.kcache = f.kcache; e.vcache = f.vcache; e.cap = f.cap; e.n_slots = f.n_slots;
      qkv_epilogue<DH, true>(e, p.M, grp, acc, rinv);
    }
    // the heads of this group are complete: raise their KV groups' counters
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
      constexpr int heads = 128 / DH;
      const int G = f.n_q / f.n_kv;
      for (int hh = 0; hh < heads; ++hh) {
        const int h = grp * heads + hh;
        const int kvg = h < f.n_q ? h / G : (h < f.n_q + f.n_kv ? h - f.n_q : h - f.n_q - f.n_kv);
        atomicAdd(layer_ctr(f, layer, f.plan.c_attn_ready + kvg), 1);
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int tile = grp * kC + wave + 4 * q;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 4 * g + i;
        const float v = fin[q][i] * (m < p.M ? rinv[i] : 0.f);
        const float up = __shfl_xor(v, 8);
        if (r < 8 && m < p.M) {
          const int jj = tile * 8 + r;
          bf16_t hi, lo;
          split_bf16(v / (1.0f + expf(-v)) * up, hi, lo);
          st_bf16_dev(f.act + m * f.ffn + jj, hi);
          st_bf16_dev(f.act_lo + m * f.ffn + jj, lo);
        }
      }
    }
    fwd_signal(layer_ctr(f, layer, f.plan.c_gu_done), 1);
  } else {  // EPI_RESID (O: after attention; down: after the MLP)
    const bool is_o = p.phase == PH_O;
    const bf16_t* gn = is_o ? f.gains[layer].mlp_norm
                            : (layer + 1 < f.n_layers ? f.gains[layer + 1].attn_norm : f.final_norm);
    bf16_t* xo = is_o ? f.xn_o : f.xn_d;
    bf16_t* xo_lo = is_o ? f.xn_o_lo : f.xn_d_lo;
    float* ssq_out = is_o ? f.ssq_o : f.ssq_d;
    float* ssq_s = reinterpret_cast<float*>(smem + kSmemSsq);  // [8 tiles][16 rows]
    float xr[2][4];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int n = (grp * kC + wave + 4 * q) * 16 + r;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 4 * g + i;
        xr[q][i] = m < p.M ? ld_f32_dev(f.x + m * f.d + n) : 0.f;
      }
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int ct = wave + 4 * q;
      const int n = (grp * kC + ct) * 16 + r;
      const float gw = bf2f(gn[n]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 4 * g + i;
        float xv = 0.f;
        if (m < p.M) {
          xv = xr[q][i] + fin[q][i];
          st_f32_dev(f.x + m * f.d + n, xv);
          bf16_t hi, lo;
          split_bf16(xv * gw, hi, lo);
          st_bf16_dev(xo + m * f.d + n, hi);
          st_bf16_dev(xo_lo + m * f.d + n, lo);
        }
        float s2 = xv * xv;
        s2 += __shfl_xor(s2, 1);
        s2 += __shfl_xor(s2, 2);
        s2 += __shfl_xor(s2, 4);
        s2 += __shfl_xor(s2, 8);
        if (r == 0) ssq_s[ct * 16 + m] = s2;
      }
    }
    __syncthreads();
    if (threadIdx.x < p.M) {
      float s = 0.f;
#pragma unroll
      for (int ct = 0; ct < kC; ++ct) s += ssq_s[ct * 16 + threadIdx.x];
      st_f32_dev(ssq_out + threadIdx.x * p.n_groups + grp, s);
    }
    fwd_signal(layer_ctr(f, layer, is_o ? f.plan.c_o_done : f.plan.c_down_done), 1);
  }
}

// Stream the K steps [s0, s1) of group grp into this wave's accumulators.  w0 holds the
// weights of the first min(U, s1 - s0) steps, already requested.
__device__ __forceinline__ void stream_steps(const bf16_t* W, int S, int grp, int s0, int s1,
                                             __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t ral,
                                             uint32_t a_row_off, const i32x4 (&w0)[kFwdU][kC],
                                             f32x4 (&acc)[kC]) {
  constexpr int U = kFwdU, C = kC;
  const int lane = threadIdx.x & 63;
  const bf16_t* wb = W + packed_frag((int64_t)grp * C, s0, S) + lane * 8;
  const int ns = s1 - s0;
  {
    i32x4 xa[U], xl[U];
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      xa[uu] = (uu < ns) ? ld16_dev(ra, a_row_off + (s0 + uu) * 64) : i32x4{0, 0, 0, 0};
      xl[uu] = (uu < ns) ? ld16_dev(ral, a_row_off + (s0 + uu) * 64) : i32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      if (uu < ns) {
#pragma unroll
        for (int ct = 0; ct < C; ++ct) {
          acc[ct] = mfma16x16x32(xa[uu], w0[uu][ct], acc[ct]);
          acc[ct] = mfma16x16x32(xl[uu], w0[uu][ct], acc[ct]);
        }
      }
    }
  }
  int st = U;
#pragma unroll 1
  for (; st + U <= ns; st += U) {
    i32x4 wv[U][C], xa[U], xl[U];
#pragma unroll
    for (int uu = 0; uu < U; ++uu) {
      xa[uu] = ld16_dev(ra, a_row_off + (s0 + st + uu) * 64);
      xl[uu] = ld16_dev(ral, a_row_off + (s0 + st + uu) * 64);
    }
#pragma unroll
    for (int uu = 0; uu < U; ++uu)
#pragma unroll
      for (int ct = 0; ct < C; ++ct) wv[uu][ct] = ld16_stream(wb + (int64_t)(st + uu) * kPackStep + ct * 512);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int uu = 0; uu < U; ++uu)
#pragma unroll
      for (int ct = 0; ct < C; ++ct) {
        acc[ct] = mfma16x16x32(xa[uu], wv[uu][ct], acc[ct]);
        acc[ct] = mfma16x16x32(xl[uu], wv[uu][ct], acc[ct]);
      }
  }
#pragma unroll 1
  for (; st < ns; ++st) {
    const i32x4 xa = ld16_dev(ra, a_row_off + (s0 + st) * 64), xl = ld16_dev(ral, a_row_off + (s0 + st) * 64);
    i32x4 wv[C];
#pragma unroll
    for (int ct = 0; ct < C; ++ct) wv[ct] = ld16_stream(wb + (int64_t)st * kPackStep + ct * 512);
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      acc[ct] = mfma16x16x32(xa, wv[ct], acc[ct]);
      acc[ct] = mfma16x16x32(xl, wv[ct], acc[ct]);
    }
  }
}

// Request the weights of steps [s0, s0 + min(U, ns)) of group grp.
__device__ __forceinline__ void prefetch_steps(const bf16_t* W, int S, int grp, int s0, int ns,
                                               i32x4 (&w0)[kFwdU][kC]) {
  const bf16_t* wb = W + packed_frag((int64_t)grp * kC, s0, S) + (threadIdx.x & 63) * 8;
#pragma unroll
  for (int uu = 0; uu < kFwdU; ++uu)
#pragma unroll
    for (int ct = 0; ct < kC; ++ct)
      w0[uu][ct] = (uu < ns) ? ld16_stream(wb + (int64_t)uu * kPackStep + ct * 512) : i32x4{0, 0, 0, 0};
}

// 1/rms of this lane's rows 4g + i from the partial sums of squares (16 threads per row).
__device__ __forceinline__ void row_rinv(const FwdArgs& f, const float* ssq, int n_part, int M, char* smem,
                                         float (&rinv)[4]) {
  float* rinv_s = reinterpret_cast<float*>(smem + kSmemRinv);
  const int m = threadIdx.x / 16, q = threadIdx.x % 16;
  float s = 0.f;
  if (ssq != nullptr && m < M)
    for (int p = q; p < n_part; p += 16) s += ld_f32_dev(ssq + m * n_part + p);
#pragma unroll
  for (int o = 8; o >= 1; o /= 2) s += __shfl_xor(s, o);
  if (q == 0) rinv_s[m] = ssq != nullptr ? 1.0f / sqrtf(s / (float)f.d + f.eps) : 1.f;
  __syncthreads();
  const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) rinv[i] = rinv_s[4 * g + i];
}

// One GEMM phase for workgroup w of nwg: stream the workgroup's share of the units, combine
// the waves' partial tiles in LDS, finish the groups it alone covers, park the others and
// finish those for which it arrives last.
template <int EPI, int DH>
__device__ __forceinline__ void gemm_phase(const FwdArgs& f, const PGemm& p, int layer, int w, int nwg,
                                           char* smem) {
  constexpr int C = kC;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int S = p.K / 32;
  const int64_t T = (int64_t)p.n_groups * S;
  const int64_t wu0 = wg_unit(T, w, nwg), wu1 = wg_unit(T, w + 1, nwg);
  const int64_t u0 = wu0 + (wu1 - wu0) * wave / 4, u1 = wu0 + (wu1 - wu0) * (wave + 1) / 4;
  const int g0 = (int)(wu0 / S);  // first group of the workgroup

  // segments of this wave: [u0, m1) in group ga, [m1, u1) in group ga + 1
  const int ga = (int)(u0 / S);
  const int64_t m1 = u0 < u1 ? std::min<int64_t>(u1, (int64_t)(ga + 1) * S) : u0;
  i32x4 w0[kFwdU][C];
  if (u0 < u1) prefetch_steps(p.W, S, ga, (int)(u0 - (int64_t)ga * S), (int)(m1 - u0), w0);
  if (p.dep != nullptr) fwd_wait(f, p.dep, p.dep_target, p.dep_what);

  const __amdgpu_buffer_rsrc_t ra = buf_rsrc(p.A), ral = buf_rsrc(p.A_lo);
  const int arow_m = r < p.M ? r : p.M - 1;
  const uint32_t a_row_off = (uint32_t)(((int64_t)arow_m * p.lda + g * 8) * 2);
  f32x4* slot = reinterpret_cast<f32x4*>(smem);  // [wave][2][C][64]
  f32x4 acc[C];
#pragma unroll
  for (int ct = 0; ct < C; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (u0 < u1)
    stream_steps(p.W, S, ga, (int)(u0 - (int64_t)ga * S), (int)(m1 - (int64_t)ga * S), ra, ral, a_row_off, w0, acc);
  // partial of the first group (local index ga - g0), then of the second
  const int la = u0 < u1 ? ga - g0 : 0;
#pragma unroll
  for (int lg = 0; lg < 2; ++lg)
#pragma unroll
    for (int ct = 0; ct < C; ++ct)
      slot[((wave * 2 + lg) * C + ct) * 64 + lane] =
          (u0 < u1 && lg == la) ? acc[ct] : f32x4{0.f, 0.f, 0.f, 0.f};
  if (m1 < u1) {
#pragma unroll
    for (int ct = 0; ct < C; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    prefetch_steps(p.W, S, ga + 1, 0, (int)(u1 - m1), w0);
    stream_steps(p.W, S, ga + 1, 0, (int)(u1 - m1), ra, ral, a_row_off, w0, acc);
#pragma unroll
    for (int ct = 0; ct < C; ++ct) slot[((wave * 2 + la + 1) * C + ct) * 64 + lane] = acc[ct];
  }

  float rinv[4] = {1.f, 1.f, 1.f, 1.f};
  if constexpr (EPI != EPI_RESID) row_rinv(f, p.ssq_in, p.n_part_in, p.M, smem, rinv);
  __syncthreads();  // all partial tiles are in LDS
  if (wu0 >= wu1) return;
  const int g1 = (int)((wu1 - 1) / S);
  for (int grp = g0; grp <= g1; ++grp) {  // workgroup-uniform
    const int lg = grp - g0;
    // this wave's tiles ct = wave and wave + 4, summed over the 4 waves
    f32x4 fin[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int ct = wave + 4 * q;
      f32x4 s = slot[((0 * 2 + lg) * C + ct) * 64 + lane];
#pragma unroll
      for (int v = 1; v < 4; ++v) s += slot[((v * 2 + lg) * C + ct) * 64 + lane];
      fin[q] = s;
    }
    const int w_first = wg_of((int64_t)grp * S, T, nwg), w_last = wg_of((int64_t)grp * S + S - 1, T, nwg);
    if (w_last > w_first) {
      // park this workgroup's part; the last contributor adds all parts in workgroup order
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        float* pp = f.part + ((int64_t)(w * 2 + lg) * C + wave + 4 * q) * 256 + lane;
#pragma unroll
        for (int i = 0; i < 4; ++i) st_f32_dev(pp + i * 64, fin[q][i]);
      }
      // contributors: the workgroups in [w_first, w_last] with a non-empty range (with fewer
      // units than workgroups, empty ones lie in between)
      int n_contrib = 0;
      for (int w2 = w_first; w2 <= w_last; ++w2) n_contrib += wg_unit(T, w2, nwg) < wg_unit(T, w2 + 1, nwg);
      if (!last_arrival(p.arr + grp, n_contrib)) continue;
#pragma unroll
      for (int q = 0; q < 2; ++q) fin[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int w2 = w_first; w2 <= w_last; ++w2) {
        const int64_t b2 = wg_unit(T, w2, nwg);
        if (b2 >= wg_unit(T, w2 + 1, nwg)) continue;
        const int lg2 = grp - (int)(b2 / S);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const float* pp = f.part + ((int64_t)(w2 * 2 + lg2) * C + wave + 4 * q) * 256 + lane;
#pragma unroll
          for (int i = 0; i < 4; ++i) fin[q][i] += ld_f32_dev(pp + i * 64);
        }
      }
    }
    group_epilogue<EPI, DH>(f, p, layer, grp, fin, rinv, smem);
  }
}

// LM head: whole groups, one per wave, full K; logits for the next launch.
template <int DH>
__device__ __forceinline__ void lm_head_phase(const FwdArgs& f, int w, int nwg, char* smem) {
  constexpr int C = kC;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int n_groups = f.vocab / 128, S = f.d / 32, M = f.lm_rows;
  const FwdPlan& P = f.plan;
  const bf16_t* W = f.wpack + f.wp_lm;
  const bf16_t* A = f.xn_d + (int64_t)f.lm_row0 * f.d;
  const bf16_t* A_lo = f.xn_d_lo + (int64_t)f.lm_row0 * f.d;
  const int gw0 = w * 4 + wave;
  i32x4 w0[kFwdU][C];
  if (gw0 < n_groups) prefetch_steps(W, S, gw0, 0, S, w0);
  fwd_wait(f, layer_ctr(f, f.n_layers - 1, P.c_down_done), P.groups[PH_DOWN], 1000000);
  float rinv[4];
  const int np = P.groups[PH_DOWN];
  row_rinv(f, f.ssq_d + (int64_t)f.lm_row0 * np, np, M, smem, rinv);
  const __amdgpu_buffer_rsrc_t ra = buf_rsrc(A), ral = buf_rsrc(A_lo);
  const int arow_m = r < M ? r : M - 1;
  const uint32_t a_row_off = (uint32_t)(((int64_t)arow_m * f.d + g * 8) * 2);
  for (int grp = gw0; grp < n_groups; grp += nwg * 4) {
    f32x4 acc[C];
#pragma unroll
    for (int ct = 0; ct < C; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (grp != gw0) prefetch_steps(W, S, grp, 0, S, w0);
    stream_steps(W, S, grp, 0, S, ra, ral, a_row_off, w0, acc);
#pragma unroll
    for (int ct = 0; ct < C; ++ct) {
      const int tile = grp * C + ct;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 4 * g + i;
        if (m < M) f.logits[(int64_t)m * f.vocab + tile * 16 + r] = acc[ct][i] * rinv[i];
      }
    }
  }
}

// The launch arguments, read afresh from the kernel-argument segment.  The layer loop would
// otherwise keep every field it uses in scalar registers from the start of the kernel to
// the end, far more than there are; an empty asm hides the pointer from loop-invariant code
// motion, so each phase loads only what it uses, when it uses it (scalar loads, cached).
__device__ __forceinline__ const FwdArgs& fwd_args() {
  auto p = __builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(p));
  return *(const FwdArgs*)p;
}

template <int DH>
__global__ __launch_bounds__(256) void fused_forward_kernel(FwdArgs) {
  __shared__ __attribute__((aligned(16))) char smem[kFwdSmem];
  const int w = blockIdx.x, nwg = gridDim.x;
  const int n_layers = fwd_args().n_layers;
  for (int l = 0; l < n_layers; ++l) {
    const int wb = l * 16;
    {  // QKV projection
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      PGemm p{};
      p.A = f.xn_d; p.A_lo = f.xn_d_lo; p.lda = f.d; p.M = f.M; p.K = f.d;
      p.W = f.wpack + (int64_t)l * f.wp_layer; p.n_groups = P.groups[PH_QKV];
      p.ssq_in = f.ssq_d; p.n_part_in = l == 0 ? f.n_part_embed : P.groups[PH_DOWN];
      if (l > 0) {
        p.dep = layer_ctr(f, l - 1, P.c_down_done);
        p.dep_target = P.groups[PH_DOWN]; p.dep_what = wb + PH_QKV;
      }
      p.arr = layer_ctr(f, l, P.c_arr_q); p.phase = PH_QKV;
      gemm_phase<EPI_QKV, DH>(f, p, l, w, nwg, smem);
    }
    {  // attention splits
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      AttnArgs a{};
      a.seqs = f.seqs; a.B = f.B; a.k = f.k; a.layer = l; a.n_q = f.n_q; a.n_kv = f.n_kv; a.d_h = DH;
      a.q = f.q; a.q_lo = f.q_lo; a.kcache = f.kcache; a.vcache = f.vcache; a.cap = f.cap; a.n_slots = f.n_slots;
      a.n_rowblocks = f.n_rowblocks; a.n_splits = f.n_splits; a.blocks_per_split = f.blocks_per_split;
      a.part_ml = f.part_ml; a.part_o = f.part_o; a.out = f.attn; a.out_lo = f.attn_lo;
      const int n_attn = f.B * f.n_kv * f.n_rowblocks * f.n_splits;
      for (int t = w; t < n_attn; t += nwg) {
        const int split = t % f.n_splits;
        const int gy = (t / f.n_splits) % (f.n_kv * f.n_rowblocks);
        const int b = t / (f.n_splits * f.n_kv * f.n_rowblocks);
        fwd_wait(f, layer_ctr(f, l, P.c_attn_ready + gy / f.n_rowblocks), f.n_q / f.n_kv + 2, wb + PH_ATTN);
        attn_split_body<DH, true>(a, split, gy, b, smem);
        fwd_signal(layer_ctr(f, l, P.c_attn_done), 1);
      }
    }
    {  // merge: one item per wave
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      AttnArgs a{};
      a.B = f.B; a.k = f.k; a.n_q = f.n_q; a.n_kv = f.n_kv; a.d_h = DH;
      a.n_rowblocks = f.n_rowblocks; a.n_splits = f.n_splits;
      a.part_ml = f.part_ml; a.part_o = f.part_o; a.out = f.attn; a.out_lo = f.attn_lo;
      const int n_attn = f.B * f.n_kv * f.n_rowblocks * f.n_splits;
      const int n_items = f.M * f.n_q;
      const int n_merge = (n_items + 3) / 4;
      for (int t = w; t < n_merge; t += nwg) {
        fwd_wait(f, layer_ctr(f, l, P.c_attn_done), n_attn, wb + PH_MERGE);
        const int item = t * 4 + (threadIdx.x >> 6);
        if (item < n_items) attn_merge_body<DH, true>(a, item);
        fwd_signal(layer_ctr(f, l, P.c_merge_done), 1);
      }
    }
    {  // O projection + residual
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      PGemm p{};
      p.A = f.attn; p.A_lo = f.attn_lo; p.lda = f.n_q * DH; p.M = f.M; p.K = f.n_q * DH;
      p.W = f.wpack + (int64_t)l * f.wp_layer + f.wp_o; p.n_groups = P.groups[PH_O];
      p.dep = layer_ctr(f, l, P.c_merge_done); p.dep_target = (f.M * f.n_q + 3) / 4; p.dep_what = wb + PH_O;
      p.arr = layer_ctr(f, l, P.c_arr_o); p.phase = PH_O;
      gemm_phase<EPI_RESID, DH>(f, p, l, w, nwg, smem);
    }
    {  // gate/up + SwiGLU
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      PGemm p{};
      p.A = f.xn_o; p.A_lo = f.xn_o_lo; p.lda = f.d; p.M = f.M; p.K = f.d;
      p.W = f.wpack + (int64_t)l * f.wp_layer + f.wp_gu; p.n_groups = P.groups[PH_GU];
      p.ssq_in = f.ssq_o; p.n_part_in = P.groups[PH_O];
      p.dep = layer_ctr(f, l, P.c_o_done); p.dep_target = P.groups[PH_O]; p.dep_what = wb + PH_GU;
      p.arr = layer_ctr(f, l, P.c_arr_gu); p.phase = PH_GU;
      gemm_phase<EPI_SWIGLU, DH>(f, p, l, w, nwg, smem);
    }
    {  // down + residual
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      PGemm p{};
      p.A = f.act; p.A_lo = f.act_lo; p.lda = f.ffn; p.M = f.M; p.K = f.ffn;
      p.W = f.wpack + (int64_t)l * f.wp_layer + f.wp_down; p.n_groups = P.groups[PH_DOWN];
      p.dep = layer_ctr(f, l, P.c_gu_done); p.dep_target = P.groups[PH_GU]; p.dep_what = wb + PH_DOWN;
      p.arr = layer_ctr(f, l, P.c_arr_d); p.phase = PH_DOWN;
      gemm_phase<EPI_RESID, DH>(f, p, l, w, nwg, smem);
    }
  }
  const FwdArgs& f = fwd_args();
  if (f.logits != nullptr) lm_head_phase<DH>(f, w, nwg, smem);
}

// Group counts and counter layout for the shapes in f, for nwg persistent workgroups.
bool fused_plan(FwdArgs& f, int nwg, int64_t part_cap_floats) {
  FwdPlan& P = f.plan;
  P = FwdPlan{};
  if (f.M < 1 || f.M > 16 || f.d % 128 || f.ffn % 64 || f.vocab % 128 || (f.d_h != 64 && f.d_h != 128))
    return false;
  if (((f.n_q + 2 * f.n_kv) * f.d_h) % 128 || (f.n_q * f.d_h) % 32 || f.n_splits < 1 || f.n_splits > 64)
    return false;
  P.groups[PH_QKV] = (f.n_q + 2 * f.n_kv) * f.d_h / 128;
  P.groups[PH_O] = f.d / 128;
  P.groups[PH_GU] = 2 * f.ffn / 128;
  P.groups[PH_DOWN] = f.d / 128;
  // a workgroup's share of a GEMM phase must span at most two groups
  for (int p : {PH_QKV, PH_O, PH_GU, PH_DOWN})
    if (P.groups[p] > nwg) return false;
  if (nwg > kFwdMaxWorkgroups || (int64_t)nwg * kFwdPartFloats > part_cap_floats) return false;
  int c = 0;
  P.c_down_done = c++;
  P.c_attn_ready = c; c += f.n_kv;
  P.c_attn_done = c++;
  P.c_merge_done = c++;
  P.c_o_done = c++;
  P.c_gu_done = c++;
  P.c_arr_q = c; c += P.groups[PH_QKV];
  P.c_arr_o = c; c += P.groups[PH_O];
  P.c_arr_gu = c; c += P.groups[PH_GU];
  P.c_arr_d = c; c += P.groups[PH_DOWN];
  P.ctr0 = 0;
  P.ctr_stride = c;
  P.n_ctl = f.n_layers * c;
  return c == fused_counters_per_layer(f.n_kv, (int64_t)(f.n_q + 2 * f.n_kv) * f.d_h, f.d, f.ffn);
}

hipError_t launch_fused_forward(const FwdArgs& f, int nwg, const Exec& ex) {
  if (f.d_h == 128)
    SBD_KLAUNCH(fused_forward_kernel<128>, dim3((unsigned)nwg), dim3(256), ex, f);
  else
    SBD_KLAUNCH(fused_forward_kernel<64>, dim3((unsigned)nwg), dim3(256), ex, f);
  return hipGetLastError();
}

}  // namespace sbd
