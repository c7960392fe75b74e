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
// weight stream overlaps the dependency chain.
//
// GEMM phases.  The unit of work is a group (128 output columns, 8 MFMA tiles) over a slice
// of K.  With G groups and NWG workgroups, kw = NWG / G workgroups share each group, each
// taking 1/kw of K (kw = 1: a workgroup takes whole groups, G > NWG: several in turn).  The
// four waves of a workgroup split its K slice and meet in LDS.  A group shared by kw > 1
// workgroups is finished as a reduce-scatter: every contributor parks its partial tile in
// global memory and waits for the group's kw arrivals; then contributor i adds the rows
// M*i/kw .. M*(i+1)/kw - 1 of all kw partials (in contributor order: deterministic) and runs
// the epilogue for those rows.  No workgroup reads more than one group's worth of partials.
//
// Attention.  Split tasks (sequence, KV head, row block, key split) raise a per-(sequence,
// KV head, row block) counter; the same workgroups then merge the splits, each a slice of
// that row block's query rows, and raise a per-KV-head counter.  A workgroup of the O
// projection waits only for the KV heads its K slice reads.
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

namespace sbd {

constexpr int kFwdSmem = 98304;   // LDS per workgroup: more than half a CU's, so one per CU
constexpr int kSpinLimit = 1 << 20;  // polls before a wait is declared failed (~1 s)
constexpr int kFwdU = 4;          // K steps of weights requested per batch
constexpr int kC = 8;             // tiles (16 columns each) of a 128-column group
// LDS layout (bytes).  [0, 32K): the waves' partial tiles [4 waves][8 tiles][64 lanes]
// f32x4, or the attention's K/V chunks [0, kAttnSmem); then the row-major group tile
// [16 rows][kRmStride] f32, 1/rms per row, per-row positions and the rotary rows of the
// forward's rows (filled once at the start).
constexpr int kRmStride = 132;
constexpr int kSmemRm = 65536 + 256;
constexpr int kSmemRinv = kSmemRm + 16 * kRmStride * 4;
constexpr int kSmemRows = kSmemRinv + 16 * 4;
constexpr int kSmemRope = kSmemRows + 16 * 16;
constexpr int kSmemEnd = kSmemRope + 16 * 64 * 2 * 4;
static_assert(kSmemEnd <= kFwdSmem, "fused forward LDS layout");
static_assert(kAttnSmem <= kSmemRm, "attention chunks overlap the group tile");

struct RowInfo {
  int pos;      // RoPE position
  int p_cache;  // cache position of the row's K and V
  int slot;     // cache slot of its sequence
  int pad;
};

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
  int n_groups, kw;      // groups; workgroups per group
  const float* ssq_in;   // consumers: partial sums of x^2 of the A rows [M][n_part_in]
  int n_part_in;
  int* dep;              // wait until *dep >= dep_target before reading A (null: none)
  int dep_target;
  int* merge_dep;        // O projection: per-KV-head merge counters, each >= merge_target
  int merge_target;
  int what;              // task code reported by a failed wait
  int* arr;              // arrival counters, one per group
  int* done;             // raised once per finished unit (null for the QKV phase)
  int phase;
};

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

// 1/rms of the rows [0, M) from their partial sums of squares, 16 threads per row: this
// thread's share of the partials (requested early), then the row sums into LDS (kSmemRinv;
// 1 where ssq is null).
__device__ __forceinline__ float row_ssq_share(const float* ssq, int n_part, int M) {
  const int m = threadIdx.x / 16, q = threadIdx.x % 16;
  float s = 0.f;
  if (ssq != nullptr && m < M)
    for (int p = q; p < n_part; p += 16) s += ld_f32_dev(ssq + m * n_part + p);
  return s;
}
__device__ __forceinline__ void row_rinv_finish(const FwdArgs& f, bool have, float s, char* smem) {
  float* rinv_s = reinterpret_cast<float*>(smem + kSmemRinv);
#pragma unroll
  for (int o = 8; o >= 1; o /= 2) s += __shfl_xor(s, o);
  if (threadIdx.x % 16 == 0) rinv_s[threadIdx.x / 16] = have ? 1.0f / sqrtf(s / (float)f.d + f.eps) : 1.f;
}
__device__ __forceinline__ void row_rinv(const FwdArgs& f, const float* ssq, int n_part, int M, char* smem) {
  row_rinv_finish(f, ssq != nullptr, row_ssq_share(ssq, n_part, M), smem);
  __syncthreads();
}

// Epilogue inputs requested before a group's partials are complete.
struct EpiPre {
  f32x4 x[2];      // RESID: residual quads of this thread's two passes
  float gw[2][4];  // RESID: norm gains of the same columns
  float gq[2];     // QKV: q/k norm gains of dims p and p + DH/2
};

// Epilogue thread layouts over the rows [m0, m1) of group grp (128 columns):
//  RESID  pass ps, thread t: quad e = t + 256 ps -> row m0 + e / 32, columns 4 (e % 32) ..+3
//  SWIGLU thread t: row m0 + t / 16, activation quad t % 16 (gate and up columns of 4 outputs)
//  QKV    wave v: rows m0 + v, m0 + v + 4, ...; lane: a head of the group and a dim pair
template <int EPI, int DH>
__device__ __forceinline__ void epi_prefetch(const FwdArgs& f, const PGemm& p, int layer, int grp, int m0, int m1,
                                             EpiPre& pre) {
  if constexpr (EPI == EPI_RESID) {
    const bool is_o = p.phase == PH_O;
    const bf16_t* gn = is_o ? f.gains[layer].mlp_norm
                            : (layer + 1 < f.n_layers ? f.gains[layer + 1].attn_norm : f.final_norm);
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
      const int e = threadIdx.x + 256 * ps;
      const int m = m0 + (e >> 5), n = grp * 128 + (e & 31) * 4;
      pre.x[ps] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i) pre.gw[ps][i] = 0.f;
      if (m < m1) {
        pre.x[ps] = __builtin_bit_cast(f32x4, ld16_dev(buf_rsrc(f.x), (uint32_t)((m * f.d + n) * 4)));
        const i32x2 gv = *(const i32x2*)(gn + n);
        pre.gw[ps][0] = __uint_as_float((uint32_t)gv[0] << 16);
        pre.gw[ps][1] = __uint_as_float((uint32_t)gv[0] & 0xffff0000u);
        pre.gw[ps][2] = __uint_as_float((uint32_t)gv[1] << 16);
        pre.gw[ps][3] = __uint_as_float((uint32_t)gv[1] & 0xffff0000u);
      }
    }
  } else if constexpr (EPI == EPI_QKV) {
    constexpr int half = DH / 2, heads = 128 / DH;
    const int lane = threadIdx.x & 63;
    const int hh = lane / half, pp = lane % half;
    const int h = grp * heads + hh;
    pre.gq[0] = pre.gq[1] = 1.f;
    if (f.qk_norm && h < f.n_q + f.n_kv) {
      const bf16_t* gn = h < f.n_q ? f.gains[layer].q_norm : f.gains[layer].k_norm;
      pre.gq[0] = bf2f(gn[pp]);
      pre.gq[1] = bf2f(gn[pp + half]);
    }
  }
}

// Epilogue of rows [m0, m1) of group grp from the row-major tile in LDS.
template <int EPI, int DH>
__device__ __forceinline__ void epilogue_rows(const FwdArgs& f, const PGemm& p, int layer, int grp, int m0, int m1,
                                              const EpiPre& pre, char* smem) {
  const float* rm = reinterpret_cast<const float*>(smem + kSmemRm);
  const float* rinv_s = reinterpret_cast<const float*>(smem + kSmemRinv);
  if constexpr (EPI == EPI_RESID) {
    const bool is_o = p.phase == PH_O;
    bf16_t* xo = is_o ? f.xn_o : f.xn_d;
    bf16_t* xo_lo = is_o ? f.xn_o_lo : f.xn_d_lo;
    float* ssq_out = is_o ? f.ssq_o : f.ssq_d;
    const __amdgpu_buffer_rsrc_t rx = buf_rsrc(f.x), rh = buf_rsrc(xo), rl = buf_rsrc(xo_lo);
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
      const int e = threadIdx.x + 256 * ps;
      const int m = m0 + (e >> 5), c4 = e & 31;
      const int n = grp * 128 + c4 * 4;
      float s2 = 0.f;
      if (m < m1) {  // uniform over each half-wave
        const f32x4 v = *(const f32x4*)(rm + m * kRmStride + c4 * 4);
        const f32x4 xv = pre.x[ps] + v;
        st16_dev(rx, (uint32_t)((m * f.d + n) * 4), __builtin_bit_cast(i32x4, xv));
        const f32x4 xg = {xv[0] * pre.gw[ps][0], xv[1] * pre.gw[ps][1], xv[2] * pre.gw[ps][2], xv[3] * pre.gw[ps][3]};
        i32x2 hi, lo;
        split_bf16x4(xg, hi, lo);
        st8_dev(rh, (uint32_t)((m * f.d + n) * 2), hi);
        st8_dev(rl, (uint32_t)((m * f.d + n) * 2), lo);
        s2 = xv[0] * xv[0] + xv[1] * xv[1] + xv[2] * xv[2] + xv[3] * xv[3];
      }
      s2 = half_wave_sum(s2);
      if (m < m1 && c4 == 0) st_f32_dev(ssq_out + m * p.n_groups + grp, s2);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int m = m0 + (threadIdx.x >> 4), aq = threadIdx.x & 15;
    if (m < m1) {
      const float rv = rinv_s[m];
      const int c = (aq >> 1) * 16 + (aq & 1) * 4;  // gate columns; up columns at c + 8
      const f32x4 gt = *(const f32x4*)(rm + m * kRmStride + c) * rv;
      const f32x4 up = *(const f32x4*)(rm + m * kRmStride + c + 8) * rv;
      f32x4 a;
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = gt[i] / (1.0f + expf(-gt[i])) * up[i];
      i32x2 hi, lo;
      split_bf16x4(a, hi, lo);
      const int j = grp * 64 + aq * 4;
      st8_dev(buf_rsrc(f.act), (uint32_t)((m * f.ffn + j) * 2), hi);
      st8_dev(buf_rsrc(f.act_lo), (uint32_t)((m * f.ffn + j) * 2), lo);
    }
  } else {  // EPI_QKV
    constexpr int half = DH / 2, heads = 128 / DH;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int hh = lane / half, pp = lane % half;
    const int h = grp * heads + hh;  // q heads, then k heads, then v heads
    const RowInfo* ri = reinterpret_cast<const RowInfo*>(smem + kSmemRows);
    const float* rope_s = reinterpret_cast<const float*>(smem + kSmemRope);
    for (int m = m0 + wave; m < m1; m += 4) {  // wave-uniform
      const float rv = rinv_s[m];
      float u0 = rm[m * kRmStride + hh * DH + pp] * rv;
      float u1 = rm[m * kRmStride + hh * DH + pp + half] * rv;
      if (f.qk_norm && h < f.n_q + f.n_kv) {
        float ss = u0 * u0 + u1 * u1;
#pragma unroll
        for (int o = half / 2; o >= 1; o /= 2) ss += __shfl_xor(ss, o);
        const float rn = 1.0f / sqrtf(ss / (float)DH + f.eps);
        u0 *= rn * pre.gq[0];
        u1 *= rn * pre.gq[1];
      }
      const RowInfo rw = ri[m];
      if (h >= f.n_q + f.n_kv) {  // V: transposed cache block, positions in the slot order of its reads
        const int gk = h - f.n_q - f.n_kv;
        bf16_t* blk = f.vcache + (((int64_t)layer * f.n_slots + rw.slot) * f.n_kv + gk) * f.cap * DH +
                      (int64_t)(rw.p_cache / 32) * DH * 32;
        const int q = rw.p_cache & 31;
        const int sl = ((q & 15) >> 2) * 8 + (q >> 4) * 4 + (q & 3);
        st_bf16_dev(blk + pp * 32 + sl, f2bf(u0));
        st_bf16_dev(blk + (pp + half) * 32 + sl, f2bf(u1));
        continue;
      }
      const float cs = rope_s[(m * 64 + pp) * 2], sn = rope_s[(m * 64 + pp) * 2 + 1];
      const float r0 = u0 * cs - u1 * sn;
      const float r1 = u1 * cs + u0 * sn;
      if (h < f.n_q) {
        const int64_t o = ((int64_t)m * f.n_q + h) * DH;
        bf16_t hi, lo;
        split_bf16(r0 * f.q_scale, hi, lo);
        st_bf16_dev(f.q + o + pp, hi);
        st_bf16_dev(f.q_lo + o + pp, lo);
        split_bf16(r1 * f.q_scale, hi, lo);
        st_bf16_dev(f.q + o + pp + half, hi);
        st_bf16_dev(f.q_lo + o + pp + half, lo);
      } else {
        const int gk = h - f.n_q;
        bf16_t* dst = f.kcache + (((int64_t)layer * f.n_slots + rw.slot) * f.n_kv + gk) * f.cap * DH +
                      (int64_t)rw.p_cache * DH;
        st_bf16_dev(dst + pp, f2bf(r0));
        st_bf16_dev(dst + pp + half, f2bf(r1));
      }
    }
  }
}

// One unit: group grp over K steps [s0, s1); contributor sl of kw.  first: the unit that
// waits for the phase's inputs (its weights are requested before the wait).
template <int EPI, int DH>
__device__ __forceinline__ void gemm_unit(const FwdArgs& f, const PGemm& p, int layer, int grp, int sl, int s0,
                                          int s1, bool first, char* smem) {
  constexpr int C = kC;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int S = p.K / 32;
  const int kw = p.kw;
  // this wave's quarter of the K slice
  const int a0 = s0 + (s1 - s0) * wave / 4, a1 = s0 + (s1 - s0) * (wave + 1) / 4;
  i32x4 w0[kFwdU][C];
  if (a0 < a1) prefetch_steps(p.W, S, grp, a0, a1 - a0, w0);
  if (first) {
    if (p.dep != nullptr) fwd_wait(f, p.dep, p.dep_target, p.what);
    if (p.merge_dep != nullptr && s0 < s1) {  // the KV heads whose attention outputs this slice reads
      const int G = f.n_q / f.n_kv;
      const int g0 = (s0 * 32 / DH) / G, g1 = ((s1 * 32 - 1) / DH) / G;
      for (int kg = g0; kg <= g1; ++kg) fwd_wait(f, p.merge_dep + kg, p.merge_target, p.what);
    }
  }
  // requested now, used after the stream: the consumer's row norms and the epilogue's
  // inputs (all final once the phase's dependencies are met)
  const int m0 = kw > 1 ? p.M * sl / kw : 0, m1 = kw > 1 ? p.M * (sl + 1) / kw : p.M;
  const float ssq_share = EPI != EPI_RESID ? row_ssq_share(p.ssq_in, p.n_part_in, p.M) : 0.f;
  EpiPre pre;
  epi_prefetch<EPI, DH>(f, p, layer, grp, m0, m1, pre);
  const __amdgpu_buffer_rsrc_t ra = buf_rsrc(p.A), ral = buf_rsrc(p.A_lo);
  const int arow_m = r < p.M ? r : p.M - 1;
  const uint32_t a_row_off = (uint32_t)(((int64_t)arow_m * p.lda + g * 8) * 2);
  f32x4 acc[C];
#pragma unroll
  for (int ct = 0; ct < C; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (a0 < a1) stream_steps(p.W, S, grp, a0, a1, ra, ral, a_row_off, w0, acc);
  f32x4* slot = reinterpret_cast<f32x4*>(smem);  // [wave][C][64]
#pragma unroll
  for (int ct = 0; ct < C; ++ct) slot[(wave * C + ct) * 64 + lane] = acc[ct];
  if constexpr (EPI != EPI_RESID) row_rinv_finish(f, p.ssq_in != nullptr, ssq_share, smem);
  __syncthreads();  // all partial tiles (and the row norms) are in LDS
  // wave v adds tiles v and v + 4 over the waves into the row-major tile
  float* rm = reinterpret_cast<float*>(smem + kSmemRm);
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int ct = wave + 4 * q;
    f32x4 s = slot[(0 * C + ct) * 64 + lane];
#pragma unroll
    for (int v = 1; v < 4; ++v) s += slot[(v * C + ct) * 64 + lane];
#pragma unroll
    for (int i = 0; i < 4; ++i) rm[(4 * g + i) * kRmStride + ct * 16 + r] = s[i];
  }
  __syncthreads();
  if (kw > 1) {
    // reduce-scatter: park, wait for the group's kw parts, add this contributor's rows
    const __amdgpu_buffer_rsrc_t rp = buf_rsrc(f.part + (int64_t)grp * kw * kFwdPartFloats);
    for (int e = threadIdx.x; e < p.M * 32; e += 256) {
      const int m = e >> 5, c4 = e & 31;
      st16_dev(rp, (uint32_t)(((sl * 16 + m) * 128 + c4 * 4) * 4),
               __builtin_bit_cast(i32x4, *(const f32x4*)(rm + m * kRmStride + c4 * 4)));
    }
    fwd_signal(p.arr + grp, 1);
    fwd_wait(f, p.arr + grp, kw, p.what + 8);
    for (int e = threadIdx.x; e < (m1 - m0) * 32; e += 256) {
      const int m = m0 + (e >> 5), c4 = e & 31;
      f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int c0 = 0; c0 < kw; c0 += 8) {
        i32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          v[u] = (c0 + u < kw) ? ld16_dev(rp, (uint32_t)((((c0 + u) * 16 + m) * 128 + c4 * 4) * 4))
                               : i32x4{0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < 8; ++u) s += __builtin_bit_cast(f32x4, v[u]);
      }
      *(f32x4*)(rm + m * kRmStride + c4 * 4) = s;
    }
    __syncthreads();
  }
  epilogue_rows<EPI, DH>(f, p, layer, grp, m0, m1, pre, smem);
  if constexpr (EPI == EPI_QKV) {
    // this unit's rows of the group's heads are in place: raise their KV heads' counters
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
  } else {
    fwd_signal(p.done, 1);
  }
}

// One GEMM phase for workgroup w of nwg.
template <int EPI, int DH>
__device__ __forceinline__ void gemm_phase(const FwdArgs& f, const PGemm& p, int layer, int w, int nwg,
                                           char* smem) {
  const int S = p.K / 32;
  if (p.kw == 1) {
    for (int grp = w; grp < p.n_groups; grp += nwg)  // workgroup-uniform
      gemm_unit<EPI, DH>(f, p, layer, grp, 0, 0, S, grp == w, smem);
  } else if (w < p.n_groups * p.kw) {
    const int grp = w / p.kw, sl = w % p.kw;
    gemm_unit<EPI, DH>(f, p, layer, grp, sl, S * sl / p.kw, S * (sl + 1) / p.kw, true, smem);
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
  fwd_wait(f, layer_ctr(f, f.n_layers - 1, P.c_down_done), P.units[PH_DOWN], 1000000);
  const int np = P.groups[PH_DOWN];
  row_rinv(f, f.ssq_d + (int64_t)f.lm_row0 * np, np, M, smem);
  const float* rinv_s = reinterpret_cast<const float*>(smem + kSmemRinv);
  float rinv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) rinv[i] = rinv_s[4 * g + i];
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

__device__ __forceinline__ PGemm make_gemm(const FwdArgs& f, int ph, int layer) {
  const FwdPlan& P = f.plan;
  PGemm p{};
  p.M = f.M;
  p.n_groups = P.groups[ph];
  p.kw = P.kw[ph];
  p.phase = ph;
  p.what = layer * 16 + ph;
  return p;
}

template <int DH>
__global__ __launch_bounds__(256) void fused_forward_kernel(FwdArgs) {
  __shared__ __attribute__((aligned(16))) char smem[kFwdSmem];
  const int w = blockIdx.x, nwg = gridDim.x;
  {  // per-row positions and rotary rows, for every QKV epilogue of the launch
    const FwdArgs& f = fwd_args();
    RowInfo* ri = reinterpret_cast<RowInfo*>(smem + kSmemRows);
    float* rope_s = reinterpret_cast<float*>(smem + kSmemRope);
    if (threadIdx.x < f.M) {
      const int m = threadIdx.x;
      const SeqParam sp = f.seqs[m / f.k];
      ri[m] = RowInfo{f.rows[m].pos, sp.cache_len + m % f.k, sp.slot, 0};
    }
    constexpr int half = DH / 2;
    for (int e = threadIdx.x; e < f.M * half; e += 256) {
      const int m = e / half, pp = e % half;
      const float2 cs = *(const float2*)(f.rope + ((int64_t)f.rows[m].pos * half + pp) * 2);
      rope_s[(m * 64 + pp) * 2] = cs.x;
      rope_s[(m * 64 + pp) * 2 + 1] = cs.y;
    }
    __syncthreads();
  }
  const int n_layers = fwd_args().n_layers;
  for (int l = 0; l < n_layers; ++l) {
    {  // QKV projection
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      PGemm p = make_gemm(f, PH_QKV, l);
      p.A = f.xn_d; p.A_lo = f.xn_d_lo; p.lda = f.d; p.K = f.d;
      p.W = f.wpack + (int64_t)l * f.wp_layer;
      p.ssq_in = f.ssq_d; p.n_part_in = l == 0 ? f.n_part_embed : P.groups[PH_DOWN];
      if (l > 0) {
        p.dep = layer_ctr(f, l - 1, P.c_down_done);
        p.dep_target = P.units[PH_DOWN];
      }
      p.arr = layer_ctr(f, l, P.c_arr_q);
      gemm_phase<EPI_QKV, DH>(f, p, l, w, nwg, smem);
    }
    {  // attention: split tasks, then merges of the completed row blocks
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      AttnArgs a{};
      a.seqs = f.seqs; a.B = f.B; a.k = f.k; a.layer = l; a.n_q = f.n_q; a.n_kv = f.n_kv; a.d_h = DH;
      a.q = f.q; a.q_lo = f.q_lo; a.kcache = f.kcache; a.vcache = f.vcache; a.cap = f.cap; a.n_slots = f.n_slots;
      a.n_rowblocks = f.n_rowblocks; a.n_splits = f.n_splits; a.blocks_per_split = f.blocks_per_split;
      a.part_ml = f.part_ml; a.part_o = f.part_o; a.out = f.attn; a.out_lo = f.attn_lo;
      const int ns = f.n_splits, nrb = f.n_rowblocks;
      const int G = f.n_q / f.n_kv;
      const int n_attn = f.B * f.n_kv * nrb * ns;
      for (int t = w; t < n_attn; t += nwg) {
        const int split = t % ns;
        const int gy = (t / ns) % (f.n_kv * nrb);
        const int b = t / (ns * f.n_kv * nrb);
        fwd_wait(f, layer_ctr(f, l, P.c_attn_ready + gy / nrb), P.attn_ready_target, l * 16 + PH_ATTN);
        attn_split_body<DH, true>(a, split, gy, b, smem);
        fwd_signal(layer_ctr(f, l, P.c_arr_attn + b * f.n_kv * nrb + gy), 1);
      }
      for (int t = w; t < n_attn; t += nwg) {
        const int split = t % ns;
        const int gy = (t / ns) % (f.n_kv * nrb);
        const int b = t / (ns * f.n_kv * nrb);
        const int g = gy / nrb, rb = gy % nrb;
        fwd_wait(f, layer_ctr(f, l, P.c_arr_attn + b * f.n_kv * nrb + gy), ns, l * 16 + PH_MERGE);
        // this task's slice of the row block's query rows, one row per wave at a time
        const int r0 = rb * 64, n_rho = min(64, G * f.k - r0);
        const int q0 = n_rho * split / ns, q1 = n_rho * (split + 1) / ns;
        for (int q = q0 + (threadIdx.x >> 6); q < q1; q += 4) {  // wave-uniform
          const int rho = r0 + q;
          const int hh = rho / f.k, j = rho % f.k;
          attn_merge_body<DH, true>(a, (int64_t)(b * f.k + j) * f.n_q + g * G + hh);
        }
        fwd_signal(layer_ctr(f, l, P.c_merge_done + g), 1);
      }
    }
    {  // O projection + residual
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      PGemm p = make_gemm(f, PH_O, l);
      p.A = f.attn; p.A_lo = f.attn_lo; p.lda = f.n_q * DH; p.K = f.n_q * DH;
      p.W = f.wpack + (int64_t)l * f.wp_layer + f.wp_o;
      p.merge_dep = layer_ctr(f, l, P.c_merge_done); p.merge_target = P.merge_target;
      p.arr = layer_ctr(f, l, P.c_arr_o); p.done = layer_ctr(f, l, P.c_o_done);
      gemm_phase<EPI_RESID, DH>(f, p, l, w, nwg, smem);
    }
    {  // gate/up + SwiGLU
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      PGemm p = make_gemm(f, PH_GU, l);
      p.A = f.xn_o; p.A_lo = f.xn_o_lo; p.lda = f.d; p.K = f.d;
      p.W = f.wpack + (int64_t)l * f.wp_layer + f.wp_gu;
      p.ssq_in = f.ssq_o; p.n_part_in = P.groups[PH_O];
      p.dep = layer_ctr(f, l, P.c_o_done); p.dep_target = P.units[PH_O];
      p.arr = layer_ctr(f, l, P.c_arr_gu); p.done = layer_ctr(f, l, P.c_gu_done);
      gemm_phase<EPI_SWIGLU, DH>(f, p, l, w, nwg, smem);
    }
    {  // down + residual
      const FwdArgs& f = fwd_args();
      const FwdPlan& P = f.plan;
      PGemm p = make_gemm(f, PH_DOWN, l);
      p.A = f.act; p.A_lo = f.act_lo; p.lda = f.ffn; p.K = f.ffn;
      p.W = f.wpack + (int64_t)l * f.wp_layer + f.wp_down;
      p.dep = layer_ctr(f, l, P.c_gu_done); p.dep_target = P.units[PH_GU];
      p.arr = layer_ctr(f, l, P.c_arr_d); p.done = layer_ctr(f, l, P.c_down_done);
      gemm_phase<EPI_RESID, DH>(f, p, l, w, nwg, smem);
    }
  }
  const FwdArgs& f = fwd_args();
  if (f.logits != nullptr) lm_head_phase<DH>(f, w, nwg, smem);
}

// Group counts, workgroups per group and counter layout for the shapes in f, for nwg
// persistent workgroups.  False when the forward is outside what the launch implements.
bool fused_plan(FwdArgs& f, int nwg, int64_t part_cap_floats) {
  FwdPlan& P = f.plan;
  P = FwdPlan{};
  if (f.M < 1 || f.M > 16 || f.d % 128 || f.ffn % 64 || f.vocab % 128 || (f.d_h != 64 && f.d_h != 128))
    return false;
  if (((f.n_q + 2 * f.n_kv) * f.d_h) % 128 || (f.n_q * f.d_h) % 32 || f.n_q % f.n_kv)
    return false;
  if (f.n_splits < 1 || f.n_splits > kMaxSplits || nwg < 1 || nwg > kFwdMaxWorkgroups)
    return false;
  P.groups[PH_QKV] = (f.n_q + 2 * f.n_kv) * f.d_h / 128;
  P.groups[PH_O] = f.d / 128;
  P.groups[PH_GU] = 2 * f.ffn / 128;
  P.groups[PH_DOWN] = f.d / 128;
  const int ks[PH_N] = {f.d, 0, 0, f.n_q * f.d_h, f.d, f.ffn};
  for (int p : {PH_QKV, PH_O, PH_GU, PH_DOWN}) {
    const int S = ks[p] / 32;
    P.kw[p] = P.groups[p] >= nwg ? 1 : std::min(std::min(nwg / P.groups[p], S), kFwdMaxKw);
    P.units[p] = P.groups[p] * P.kw[p];
    // parked partials: 16 rows x 128 columns per unit of a shared group
    if (P.kw[p] > 1 && (int64_t)P.units[p] * kFwdPartFloats > part_cap_floats) return false;
  }
  const int G = f.n_q / f.n_kv;
  P.attn_ready_target = (G + 2) * P.kw[PH_QKV];
  P.merge_target = f.B * f.n_rowblocks * f.n_splits;
  int c = 0;
  P.c_down_done = c++;
  P.c_o_done = c++;
  P.c_gu_done = c++;
  P.c_attn_ready = c; c += f.n_kv;
  P.c_merge_done = c; c += f.n_kv;
  P.c_arr_attn = c; c += f.B * f.n_kv * f.n_rowblocks;
  P.c_arr_q = c; c += P.groups[PH_QKV];
  P.c_arr_o = c; c += P.groups[PH_O];
  P.c_arr_gu = c; c += P.groups[PH_GU];
  P.c_arr_d = c; c += P.groups[PH_DOWN];
  P.ctr0 = 0;
  P.ctr_stride = c;
  P.n_ctl = f.n_layers * c;
  return c <= fused_counters_per_layer(f.n_kv, (int64_t)(f.n_q + 2 * f.n_kv) * f.d_h, f.d, f.ffn,
                                       (int64_t)f.B * f.n_kv * f.n_rowblocks);
}

hipError_t launch_fused_forward(const FwdArgs& f, int nwg, const Exec& ex) {
  if (f.d_h == 128)
    SBD_KLAUNCH(fused_forward_kernel<128>, dim3((unsigned)nwg), dim3(256), ex, f);
  else
    SBD_KLAUNCH(fused_forward_kernel<64>, dim3((unsigned)nwg), dim3(256), ex, f);
  return hipGetLastError();
}

}  // namespace sbd
