// Weight-streaming GEMM for M > 16 rows: y[m][n] = sum_k A[m][k] W[n][k].
//
// Weights are repacked once (pack_kernel) into MFMA fragment order.  A matrix with N rows
// and K columns is cut into 16-row tiles; the 16-byte piece of lane l in step s of tile t
// holds W[16t + l%16][32s + 8(l/16) .. +8], so one 16-byte load per lane reads a 1 KB
// fragment in the B-operand order of v_mfma_f32_16x16x32_bf16.  Tiles are grouped by 8
// (128 rows) and a group's 8 fragments of one step are stored together:
// [N/128 groups][K/32 steps][8 tiles][64 lanes][8] (packed_frag() in sbd_device.h).  The
// gate and up projections share one packed matrix whose tile t holds gate rows 8t..8t+7
// followed by up rows 8t..8t+7, so SwiGLU pairs stay inside one tile.
//
// This kernel serves the block forwards of several sequences (M = batch * k up to a few
// hundred rows) and the prefill chunks; decode-sized products (M <= 16) go through
// gemv.hip.  At these M every projection still reads far more weight bytes than it does
// MFMA work per byte (M flop per weight byte, against a ridge of ~300), so the design
// streams every weight byte from HBM once:
//   - A workgroup owns a column block of NT tiles (128, 256, or for gate/up 192 columns) and a row block of
//     MT tiles (up to 128 rows; larger M is cut into row blocks that run on the same XCD
//     and meet the same weights in its L2), and a range of K steps.
//   - Weights and activations reach LDS by direct loads (global_load_lds, no registers)
//     in stages of one K step, a ring of NS stages, so NS - 1 steps are in flight while
//     the waves multiply the current one.  The four waves split the block into column
//     quarters (or halves x row halves); a wave reads its weight fragments and the A
//     fragments (hi and lo) of its rows from LDS and runs two MFMAs per pair.
//   - When there are too few column blocks to fill the chip, K is split over workgroups
//     of one XCD, all resident at once (plans of one round): each parks its partial tiles
//     in that XCD's L2 and waits for the others, then adds the slices of a share of the row
//     tiles in slice order (deterministic) and runs their epilogue, so the finishing work
//     of a unit is spread over its slices (e4m3 weights at M <= 32: the last slice to
//     arrive adds all slices and finishes the block, without waiting).
// Epilogues (acc in the MFMA D layout: lane l holds column l % 16 of a tile, rows
// 4*(l/16) + i):
//   EPI_SCALED_STORE  out = rinv[m] * y           (QKV projection, LM head)
//   EPI_LOGITS_EB     the same (stores optional) plus the EB softmax statistics of every
//                     row's 64-column chunks (LM head; eb_stats.h)
//   EPI_RESID         x += y; xn = x * g_next as hi/lo; the sum of x^2 over the block's
//                     columns per row (O and down projections: residual add, the next
//                     RMSNorm's inputs)
//   EPI_SWIGLU        act = silu(rinv*gate) * rinv*up as hi/lo (gate/up projection)
// RMSNorm is split across two kernels: the producer writes x * g (gain applied) plus
// partial sums of squares; the consumer adds the partials of a row and scales its fp32
// result by 1/sqrt(mean(x^2) + eps), which equals normalising the input first because the
// scale is constant along a row.

#include <algorithm>
#include <type_traits>
#include <utility>

#include "eb_stats.h"

namespace sbd {

template <int MT, int NT, bool W8>
struct MidCfg {
  // waves across the column block: 2 x 2 waves (each reads half the activation and half the
  // weight fragments of a stage from LDS: 16 KB per 16-tile stage, against 20 KB in a 4 x 1 split)
  static constexpr int WC = 2;
  static constexpr int WM = 4 / WC;            // waves across the row block
  static constexpr int CW = NT / WC;           // tiles per wave
  static constexpr int MTW = MT / WM;          // row tiles per wave
  // weight bytes of a K step: 1 KB per tile in bf16, 512 B in e4m3 (one 1 KB wave-load then
  // carries two tiles' fragments)
  static constexpr int WB = NT * (W8 ? 512 : 1024);
  static constexpr int NWL = WB / 1024;               // weight wave-loads per stage
  static constexpr int STAGE = WB + 2 * MT * 1024;    // one K step: weights + 2 MT A fragments
  static constexpr int NS = (144 * 1024) / STAGE > 8 ? 8 : (144 * 1024) / STAGE;  // ring stages
  static constexpr int FPW = (NWL + 2 * MT) / 4;      // wave-loads of each wave per stage
  static constexpr int NWU = NWL / 4;                 // of a wave's FPW loads, the first NWU are weights
  static_assert(MTW >= 1 && (NWL + 2 * MT) % 4 == 0 && NWL % 4 == 0, "unsupported tile shape");
  static_assert((NS - 1) * FPW <= 63, "vmcnt range");
};

// f(std::integral_constant<int, 0>{}), ..., f(std::integral_constant<int, N - 1>{})
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Wait until at most n stages of FPW loads each are still in flight (n in [0, NMAX]).
template <int FPW, int NMAX>
__device__ __forceinline__ void vm_wait_stages(int n) {
  if constexpr (NMAX > 0) {
    if (n >= NMAX) {
      vm_wait<NMAX * FPW>();
      return;
    }
    vm_wait_stages<FPW, NMAX - 1>(n);
  } else {
    vm_wait<0>();
  }
}
// Barrier between stages: LDS reads of this wave complete, then s_barrier.  The empty asm
// statements keep the compiler from moving LDS accesses across it.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Value of an XCD-local counter, read with an atomic (a load could be served by the CU's own
// L1); the zero comes from an instruction the compiler cannot see through, so the atomic
// stays one.
__device__ __forceinline__ int ctr_peek(int* ctr) {
  int zero;
  asm volatile("v_mov_b32 %0, 0" : "=v"(zero));
  return __hip_atomic_fetch_add(ctr, zero, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// The K slices of a unit (all on one XCD, all resident) wait until every one has parked its
// partials: word 0 of the unit's counter line counts arrivals, word 1 departures, and the
// last to depart resets both for the next launch.  The wait is bounded: one that gives up
// raises the sticky error and the workgroup goes on (its results are then wrong, and the
// next API call reports it).
__device__ __forceinline__ void slices_arrived(const GemmArgs& a, int* ctr, int ks, int what) {
  __builtin_amdgcn_s_waitcnt(0);  // this wave's stores have reached the L2
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    int it = 0;
    while (ctr_peek(ctr) < ks) {
      __builtin_amdgcn_s_sleep(1);
      if (++it > a.spin_limit) {
        atomicOr(a.err, 1);
        atomicExch(a.err + 1, what);
        if (a.err_host != nullptr) {
          __hip_atomic_store(a.err_host + 1, what, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          __hip_atomic_store(a.err_host, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
        break;
      }
    }
    if (__hip_atomic_fetch_add(ctr + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == ks - 1) {
      __hip_atomic_store(ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      __hip_atomic_store(ctr + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  }
  __syncthreads();
}

// STREAM: every weight byte is read by one workgroup (one row block): non-temporal loads.
// W8: the weights are e4m3 bytes (a.Wp8, per-row scales a.wscale) in the same packing, one
// byte per element; a fragment is widened to the bf16 MFMA operand (times its row's scale,
// exact) after its LDS read, so the products are those of the widened bf16 matrix.
template <int MT, int NT, int EPI, bool STREAM, bool W8>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs a) {
  using Cfg = MidCfg<MT, NT, W8>;
  constexpr int WC = Cfg::WC, CW = Cfg::CW, MTW = Cfg::MTW, NS = Cfg::NS, FPW = Cfg::FPW;
  constexpr int STAGE = Cfg::STAGE;
  constexpr int WB = Cfg::WB;    // weight bytes of a stage; A fragments follow
  constexpr int NWU = Cfg::NWU;
  typedef typename std::conditional<W8, i32x2, i32x4>::type WFr;  // a weight fragment in registers
  __shared__ __attribute__((aligned(16))) char smem[NS * STAGE];
  __shared__ float rinv_s[MT * 16];
  __shared__ float ssq_s[WC][MT * 16];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int wc = w % WC, wm = w / WC;

  // Workgroup i runs on XCD i % 8; the m_blocks x splits units of column block cb all sit
  // on XCD cb % 8.  The count is padded to a multiple of 8; padding workgroups leave.
  const int KS = a.splits, MB = a.m_blocks, P = KS * MB;
  const int jx = (int)(blockIdx.x >> 3);
  const int cb = (jx / P) * 8 + (int)(blockIdx.x & 7);
  // a last column block may be half full (n_tiles % NT == 8, LM head with bf16 weights and
  // two waves across the block: the second wave's tiles are past the end)
  const int n_cb = (a.n_tiles + NT - 1) / NT;
  if (cb >= n_cb) return;
  const int mb = (jx % P) / KS, kc = (jx % P) % KS;
  const int uid = cb * MB + mb;
  const int row0 = mb * MT * 16;
  const int S_all = a.K / 32;
  const int s_b = (int)((int64_t)S_all * kc / KS), s_e = (int)((int64_t)S_all * (kc + 1) / KS);
  const int nst = s_e - s_b;
  const int t0 = cb * NT;

  // Sources of this wave's loads: load u of a stage fills 1 KB f = w + 4u of it; f < NWL is
  // weight tile t0 + f (bf16) or the tiles t0 + 2f, t0 + 2f + 1 (e4m3: their fragments are
  // adjacent in the packing), else A fragment f - NWL = 2 * (row tile) + (0: hi, 1: lo).
  const char* src[FPW];
  int64_t stride[FPW];
#pragma unroll
  for (int u = 0; u < FPW; ++u) {
    const int f = w + 4 * u;
    if (u < NWU) {
      if constexpr (W8) {
        src[u] = (const char*)(a.Wp8 + packed_frag(t0 + 2 * f, s_b, S_all) + lane * 16);
        stride[u] = kPackStep;
      } else {
        // a half-full block's tiles past the end read the last tile (results discarded)
        constexpr bool kHalf = EPI == EPI_SCALED_STORE || EPI == EPI_LOGITS_EB;
        src[u] = (const char*)(a.Wp + packed_frag(kHalf ? min(t0 + f, a.n_tiles - 1) : t0 + f, s_b, S_all) + lane * 8);
        stride[u] = kPackStep * 2;
      }
    } else {
      const int ai = f - Cfg::NWL;
      int row = row0 + (ai >> 1) * 16 + r;
      if (row >= a.M) row = a.M - 1;  // rows past the end: valid data, results discarded
      const bf16_t* base = (ai & 1) ? a.A_lo : a.A;
      if (a.a_mtiles) {  // fragment order: one contiguous 1 KB per fragment
        src[u] = (const char*)(base + apack(a.a_row0 + row, (int64_t)s_b * 32 + g * 8, a.a_mtiles));
        stride[u] = (int64_t)a.a_mtiles * 1024;
      } else {
        src[u] = (const char*)(base + (int64_t)row * a.lda + (int64_t)s_b * 32 + g * 8);
        stride[u] = 64;
      }
    }
  }
  // stage st into ring slot st % NS
  auto issue = [&](int st) {
    char* dst = smem + (st % NS) * STAGE + w * 1024;
    constexpr int kPolW = STREAM ? 2 : 0;  // nt: read once
#pragma unroll
    for (int u = 0; u < NWU; ++u)
      __builtin_amdgcn_global_load_lds((const void*)(src[u] + st * stride[u]),
                                       (__attribute__((address_space(3))) void*)(dst + u * 4096), 16, 0, kPolW);
#pragma unroll
    for (int u = NWU; u < FPW; ++u)
      __builtin_amdgcn_global_load_lds((const void*)(src[u] + st * stride[u]),
                                       (__attribute__((address_space(3))) void*)(dst + u * 4096), 16, 0, 0);
  };

  f32x4 acc[MTW][CW];
#pragma unroll
  for (int mw = 0; mw < MTW; ++mw)
#pragma unroll
    for (int cw = 0; cw < CW; ++cw) acc[mw][cw] = f32x4{0.f, 0.f, 0.f, 0.f};

  // LDS reads of a stage with ds_read16 (sbd_device.h): the compiler would otherwise guard
  // every read of LDS with a wait for all direct loads in flight (it cannot tell the ring
  // slots apart), draining the ring at each step.  Ordering is explicit instead: the stage
  // barrier before the reads, lds_wait() after them, and the results pinned behind it.
  // The reads of stage c + 1 are issued before the MFMAs of stage c (two register sets), so
  // the LDS traffic of one step overlaps the matrix work of the previous one.
  constexpr int WFB = W8 ? 512 : 1024;  // bytes of one weight fragment in LDS
  const uint32_t lds_w = (uint32_t)(uintptr_t)smem + (uint32_t)(wc * CW * WFB + lane * (WFB / 64));
  const uint32_t lds_a = (uint32_t)(uintptr_t)smem + (uint32_t)(WB + wm * MTW * 2048 + lane * 16);
  // the lane's weight scales (row r of each of its tiles); 1 for bf16
  float wsc[CW];
#pragma unroll
  for (int cw = 0; cw < CW; ++cw) wsc[cw] = W8 ? a.wscale[(int64_t)(t0 + wc * CW + cw) * 16 + r] : 1.0f;
  auto read_frags = [&](int st, WFr (&wv)[CW], i32x4 (&av)[MTW][2]) {
    const uint32_t sb = (uint32_t)((st % NS) * STAGE);
    const uint32_t aw = lds_w + sb, aa = lds_a + sb;
    static_for<CW>([&](auto I) {
      if constexpr (W8) wv[decltype(I)::value] = ds_read8<decltype(I)::value * 512>(aw);
      else wv[decltype(I)::value] = ds_read16<decltype(I)::value * 1024>(aw);
    });
    static_for<MTW * 2>([&](auto I) {
      constexpr int i = decltype(I)::value;
      av[i / 2][i % 2] = ds_read16<i * 1024>(aa);
    });
  };
  auto pin_frags = [&](WFr (&wv)[CW], i32x4 (&av)[MTW][2]) {
#pragma unroll
    for (int cw = 0; cw < CW; ++cw) lds_pin(wv[cw]);
#pragma unroll
    for (int mw = 0; mw < MTW; ++mw)
#pragma unroll
      for (int h = 0; h < 2; ++h) lds_pin(av[mw][h]);
  };
  auto mfma_frags = [&](const WFr (&wv)[CW], const i32x4 (&av)[MTW][2]) {
    if constexpr (W8) {  // each fragment widened once; every accumulator still takes hi, then lo
#pragma unroll
      for (int cw = 0; cw < CW; ++cw) {
        const i32x4 wf = e4m3x8_to_bf16(wv[cw], wsc[cw]);
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int mw = 0; mw < MTW; ++mw) acc[mw][cw] = mfma16x16x32(av[mw][h], wf, acc[mw][cw]);
      }
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int mw = 0; mw < MTW; ++mw)
#pragma unroll
          for (int cw = 0; cw < CW; ++cw) acc[mw][cw] = mfma16x16x32(av[mw][h], wv[cw], acc[mw][cw]);
    }
  };

  // Consumers of a norm: the producer's partial sums of squares of this block's rows,
  // requested before the stream (thread t adds partials of row t / TPR, float4 at a time).
  constexpr int TPR = 256 / (MT * 16);
  constexpr int NPRE = 4;
  const int rr_t = threadIdx.x / TPR, q_t = threadIdx.x % TPR;
  const int m_t = row0 + rr_t;
  const bool norm_in = EPI != EPI_RESID && a.sumsq_in != nullptr;
  const bool vec4 = (a.n_part & 3) == 0;
  const int n4 = a.n_part >> 2;
  const f32x4* prow = reinterpret_cast<const f32x4*>(a.sumsq_in + (int64_t)min(m_t, a.M - 1) * a.n_part);
  f32x4 pre[NPRE];
#pragma unroll
  for (int j = 0; j < NPRE; ++j) {
    const int p4 = q_t + j * TPR;
    pre[j] = (norm_in && vec4 && m_t < a.M && p4 < n4) ? prow[p4] : f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // A kernel's code runs cold from the instruction cache in every workgroup: the ring is
  // driven by compact loops (slot = stage % NS at run time) rather than unrolled code.
  // NS stages in flight: stage c's slot is refilled once every wave holds its fragments.
#pragma unroll 1
  for (int st = 0; st < NS && st < nst; ++st) issue(st);
  WFr wv0[CW], wv1[CW];
  i32x4 av0[MTW][2], av1[MTW][2];
  vm_wait_stages<FPW, NS - 1>(min(NS - 1, nst - 1));  // stage 0 has landed (this wave's part)
  stage_barrier();                                    // ... and every wave's
  read_frags(0, wv0, av0);
  lds_wait();
  pin_frags(wv0, av0);
  // step c: the fragments of stage c are in registers; stage c + 1 is read meanwhile
  auto step = [&](int c, WFr (&wc_)[CW], i32x4 (&ac_)[MTW][2], WFr (&wn)[CW], i32x4 (&an)[MTW][2]) {
    if (c + 1 < nst) {
      vm_wait_stages<FPW, NS - 2>(min(NS - 2, nst - 2 - c));  // stage c + 1 has landed (this wave's part)
      stage_barrier();  // ... and every wave's; every wave holds stage c's fragments: its slot is free
      if (c + NS < nst) issue(c + NS);
      read_frags(c + 1, wn, an);
    }
    // the MFMAs stay between the reads and their wait (they do not touch memory, so the
    // compiler would otherwise move them past the wait)
    __builtin_amdgcn_sched_barrier(0);
    mfma_frags(wc_, ac_);
    __builtin_amdgcn_sched_barrier(0);
    lds_wait();
    pin_frags(wn, an);
  };
#pragma unroll 1
  for (int c = 0; c < nst; c += 2) {
    step(c, wv0, av0, wv1, av1);
    if (c + 1 < nst) step(c + 1, wv1, av1, wv0, av0);
  }

  // ---- K split over workgroups (a plan of one round: every slice of a unit is resident):
  // each slice parks its partial tiles and waits for the others; the epilogue then adds the
  // slices of the row tiles kc, kc + KS, ... of the block in slice order and finishes them
  // (every output is the same sum of the same slices, whichever slice finishes it).  The
  // accumulators are not written again after the K loop: the sums go straight to LDS.
  // e4m3 weights and two row tiles (M <= 32) keep the single finisher: the last slice to
  // arrive sums every slice into the accumulators and finishes the whole block (there the
  // shared sums made the compiler move accumulators between register files inside the K
  // loop, which cost more than the shared finishing saves)
  constexpr bool kSingle = W8 && MT == 2;
  auto own = [&](int rt) { return kSingle || rt % KS == kc; };
  const int64_t slot = ((int64_t)uid * 4 + w) * (MTW * CW);       // in 1 KB (64 x f32x4) pieces
  const int64_t zstride = (int64_t)n_cb * MB * 4 * MTW * CW;       // pieces per slice
  if (KS > 1) {
#pragma unroll
    for (int mw = 0; mw < MTW; ++mw)
#pragma unroll
      for (int cw = 0; cw < CW; ++cw)
        *(f32x4*)(a.part + ((kc * zstride + slot + mw * CW + cw) * 64 + lane) * 4) = acc[mw][cw];
    if constexpr (kSingle) {
      if (!last_arrival_xcd(a.counters + (int64_t)uid * kCtrStride, KS)) return;
      // ZB slices at a time, every piece of a slice in flight together; added in slice order
      constexpr int ZB = MTW * CW >= 32 ? 1 : (MTW * CW >= 16 ? 2 : 4);
      const __amdgpu_buffer_rsrc_t rp = buf_rsrc(a.part);
#pragma unroll
      for (int mw = 0; mw < MTW; ++mw)
#pragma unroll
        for (int cw = 0; cw < CW; ++cw) acc[mw][cw] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int z0 = 0; z0 < KS; z0 += ZB) {
        i32x4 v[ZB][MTW][CW];
#pragma unroll
        for (int zz = 0; zz < ZB; ++zz)
#pragma unroll
          for (int mw = 0; mw < MTW; ++mw)
#pragma unroll
            for (int cw = 0; cw < CW; ++cw)
              v[zz][mw][cw] = z0 + zz < KS ? ld16_l2(rp, (uint32_t)((((z0 + zz) * zstride + slot + mw * CW + cw) * 64 + lane) * 16))
                                           : i32x4{0, 0, 0, 0};
#pragma unroll
        for (int zz = 0; zz < ZB; ++zz)
#pragma unroll
          for (int mw = 0; mw < MTW; ++mw)
#pragma unroll
            for (int cw = 0; cw < CW; ++cw) acc[mw][cw] += __builtin_bit_cast(f32x4, v[zz][mw][cw]);
      }
    } else {
      slices_arrived(a, a.counters + (int64_t)uid * kCtrStride, KS, 65536 + EPI);
    }
  }

  // ---- 1/rms of the block's rows (partials beyond the prefetched ones read here)
  if constexpr (EPI != EPI_RESID) {
    float sq = 0.f;
    if (norm_in && m_t < a.M) {
      if (vec4) {
#pragma unroll
        for (int j = 0; j < NPRE; ++j) sq += (pre[j][0] + pre[j][1]) + (pre[j][2] + pre[j][3]);
        for (int p4 = q_t + NPRE * TPR; p4 < n4; p4 += TPR) {
          const f32x4 v = prow[p4];
          sq += (v[0] + v[1]) + (v[2] + v[3]);
        }
      } else {
        for (int p = q_t; p < a.n_part; p += TPR) sq += a.sumsq_in[(int64_t)m_t * a.n_part + p];
      }
    }
#pragma unroll
    for (int o = TPR / 2; o >= 1; o /= 2) sq += __shfl_xor(sq, o);
    if (q_t == 0) rinv_s[rr_t] = norm_in ? 1.0f / sqrtf(sq * a.inv_d + a.eps) : 1.0f;
  }
  __syncthreads();  // rinv_s written; every wave is past the ring, which now stages results

  // ---- epilogue.  Each wave passes its tiles through LDS one row tile at a time (16 rows x
  // 16 CW columns, rows padded by 4 floats), then lanes own 4 consecutive columns of a row:
  // a row's 16 CW columns are written by consecutive lanes as whole 16-byte pieces.
  constexpr int LDR = CW * 16 + 4;  // staged row length (floats)
  constexpr int CPR = CW * 4;       // float4 pieces per staged row
  float* stg = reinterpret_cast<float*>(smem) + w * 16 * LDR;
  const int n_w0 = (t0 + wc * CW) * 16;  // first output column of this wave
  // false only for the empty half of a half-full block (an LM head's last block)
  const bool cols_in = (EPI != EPI_SCALED_STORE && EPI != EPI_LOGITS_EB) || n_w0 < a.n_tiles * 16;
  // EPI_RESID: a lane's residual pieces of row tile mw + 1 are requested before the stores
  // of row tile mw (which the compiler may not move them past); the gain is the same for
  // every row of the lane.
  constexpr int NPASS = 16 * CPR / 64;  // read-back passes per row tile
  const int n_l = n_w0 + (lane % CPR) * 4;
  f32x4 xcur[NPASS], xnxt[NPASS];
  i32x2 gw{0, 0};
  auto load_x = [&](int mw, f32x4(&xv)[NPASS]) {
#pragma unroll
    for (int j = 0; j < NPASS; ++j) {
      const int m = row0 + (wm * MTW + mw) * 16 + (j * 64 + lane) / CPR;
      xv[j] = m < a.M ? *(const f32x4*)(a.x + (int64_t)m * a.ldx + n_l) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  if constexpr (EPI == EPI_RESID) {
    gw = *(const i32x2*)(a.g_next + n_l);
    if (own(wm * MTW)) load_x(0, xcur);
  }
#pragma unroll
  for (int mw = 0; mw < MTW; ++mw) {
    const int rl0 = (wm * MTW + mw) * 16;  // first local row of this row tile
    if constexpr (EPI == EPI_RESID) {
      if (mw + 1 < MTW && own(wm * MTW + mw + 1)) load_x(mw + 1, xnxt);
    }
    if (own(wm * MTW + mw) && cols_in) {
      if (!kSingle && KS > 1) {
        // the slices' sums of this wave's tiles of the row tile: ZR slices at a time, all
        // their pieces in flight
        constexpr int ZR = 4;
        const __amdgpu_buffer_rsrc_t rp = buf_rsrc(a.part);
        f32x4 sum[CW];
#pragma unroll
        for (int cw = 0; cw < CW; ++cw) sum[cw] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int z0 = 0; z0 < KS; z0 += ZR) {
          i32x4 v[ZR][CW];
#pragma unroll
          for (int zz = 0; zz < ZR; ++zz)
#pragma unroll
            for (int cw = 0; cw < CW; ++cw)
              v[zz][cw] = z0 + zz < KS ? ld16_l2(rp, (uint32_t)((((z0 + zz) * zstride + slot + mw * CW + cw) * 64 + lane) * 16))
                                       : i32x4{0, 0, 0, 0};
#pragma unroll
          for (int zz = 0; zz < ZR; ++zz)
#pragma unroll
            for (int cw = 0; cw < CW; ++cw) sum[cw] += __builtin_bit_cast(f32x4, v[zz][cw]);
        }
#pragma unroll
        for (int cw = 0; cw < CW; ++cw)
#pragma unroll
          for (int i = 0; i < 4; ++i) stg[(4 * g + i) * LDR + cw * 16 + r] = sum[cw][i];
      } else {
#pragma unroll
        for (int cw = 0; cw < CW; ++cw)
#pragma unroll
          for (int i = 0; i < 4; ++i) stg[(4 * g + i) * LDR + cw * 16 + r] = acc[mw][cw][i];
      }
      if constexpr (EPI == EPI_SWIGLU) {
        // task: (row, tile tt, half h) -> act columns 8 (tile) + 4 h .. + 3
        constexpr int NT2 = 16 * CW * 2;
#pragma unroll
        for (int j = 0; j < (NT2 + 63) / 64; ++j) {
          const int idx = j * 64 + lane;
          const int row = idx / (CW * 2), tt = (idx % (CW * 2)) >> 1, h = idx & 1;
          const int m = row0 + rl0 + row;
          if (idx < NT2 && m < a.M) {
            const f32x4 gt = *(const f32x4*)(stg + row * LDR + tt * 16 + h * 4);
            const f32x4 up = *(const f32x4*)(stg + row * LDR + tt * 16 + 8 + h * 4);
            const float rv = rinv_s[rl0 + row];
            f32x4 y;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float gv = gt[e] * rv;
              y[e] = gv / (1.0f + expf(-gv)) * (up[e] * rv);
            }
            i32x2 hi, lo;
            split_bf16x4(y, hi, lo);
            const int64_t o = aoff(m, (int64_t)(t0 + wc * CW + tt) * 8 + h * 4, a.ld_act, a.o_mtiles);
            *(i32x2*)(a.act + o) = hi;
            *(i32x2*)(a.act_lo + o) = lo;
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 16 * CPR / 64; ++j) {
          const int idx = j * 64 + lane;
          const int row = idx / CPR, pc = idx % CPR;
          const int m = row0 + rl0 + row;
          const int n = n_w0 + pc * 4;
          const f32x4 y = *(const f32x4*)(stg + row * LDR + pc * 4);
          if constexpr (EPI == EPI_SCALED_STORE) {
            if (m < a.M) *(f32x4*)(a.out_f32 + (int64_t)m * a.ldo + n) = y * rinv_s[rl0 + row];
          } else if constexpr (EPI == EPI_LOGITS_EB) {
            if (m < a.M && a.out_f32 != nullptr) *(f32x4*)(a.out_f32 + (int64_t)m * a.ldo + n) = y * rinv_s[rl0 + row];
          } else {  // EPI_RESID
            float s2 = 0.f;
            if (m < a.M) {
              const f32x4 xv = xcur[j] + y;
              *(f32x4*)(a.x + (int64_t)m * a.ldx + n) = xv;
              f32x4 xg;
              xg[0] = xv[0] * __uint_as_float((uint32_t)gw[0] << 16);
              xg[1] = xv[1] * __uint_as_float((uint32_t)gw[0] & 0xffff0000u);
              xg[2] = xv[2] * __uint_as_float((uint32_t)gw[1] << 16);
              xg[3] = xv[3] * __uint_as_float((uint32_t)gw[1] & 0xffff0000u);
              i32x2 hi, lo;
              split_bf16x4(xg, hi, lo);
              const int64_t on = aoff(m, n, a.ldx, a.o_mtiles);
              *(i32x2*)(a.xn + on) = hi;
              *(i32x2*)(a.xn_lo + on) = lo;
              s2 = (xv[0] * xv[0] + xv[1] * xv[1]) + (xv[2] * xv[2] + xv[3] * xv[3]);
            }
#pragma unroll
            for (int o = 1; o < CPR; o <<= 1) s2 += __shfl_xor(s2, o);  // the row's CPR lanes
            if (pc == 0) ssq_s[wc][rl0 + row] = s2;
          }
        }
      }
      if constexpr (EPI == EPI_LOGITS_EB) {
        // the staged row tile again: lane L reduces VPL = 4 CW consecutive columns of row L / 4,
        // 16 / CW lanes per 64-column chunk
        constexpr int VPL = 4 * CW, LPC = 16 / CW;
        static_assert(VPL * LPC == kEbFChunk, "a chunk is 64 columns");
        const int row = lane >> 2, seg = lane & 3;
        const int m = row0 + rl0 + row;
        const int col0 = n_w0 + seg * VPL;
        float mx;
        int arg;
        double z, sz;
        eb_seg_stats<VPL, LPC>(stg + row * LDR + seg * VPL, rinv_s[rl0 + row], col0, a.eb_mask_id, mx, arg, z, sz);
        if (seg % LPC == 0 && m < a.M) eb_chunk_store(a.eb_part, a.eb_arg, a.eb_chunks, m, col0 / kEbFChunk, mx, arg, z, sz);
      }
    }
    if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int j = 0; j < NPASS; ++j) xcur[j] = xnxt[j];
    }
  }
  if constexpr (EPI == EPI_RESID) {
    __syncthreads();
    if (threadIdx.x < MT * 16) {
      const int m = row0 + threadIdx.x;
      float s = ssq_s[0][threadIdx.x];
#pragma unroll
      for (int q = 1; q < WC; ++q) s += ssq_s[q][threadIdx.x];
      if (m < a.M && own((int)threadIdx.x / 16)) a.sumsq_out[(int64_t)m * a.n_part_out + cb] = s;
    }
  }
}

// ---- host side: plan and launch

GemmPlan gemm_plan(int M, int n_tiles, int K, int64_t part_cap, bool nt12, bool half_block) {
  GemmPlan best{};
  const int mt = M <= 32 ? 2 : (M <= 64 ? 4 : 8);
  const int mb = (M + mt * 16 - 1) / (mt * 16);
  const int S_all = K / 32;
  double best_cost = 1e300;
  // 12-tile blocks (gate/up only): Qwen 8B's 1536 gate/up tiles then fill all 32 CUs of an
  // XCD in one round (16 blocks x 2 K slices) where 16-tile blocks leave 8 idle
  for (int nt : {16, 12, 8}) {
    // half_block: 16-tile blocks also when n_tiles % 16 == 8, the last one half full (one K
    // slice: its empty half would otherwise park and sum nothing)
    const bool half = half_block && nt == 16 && n_tiles % 16 == 8;
    if ((n_tiles % nt && !half) || (nt == 12 && !nt12)) continue;
    const int n_cb = (n_tiles + nt - 1) / nt;
    for (int ks = 1; ks <= 8; ++ks) {
      if (ks > 1 && (S_all / ks < 4 || half)) break;
      if (ks > 1 && (int64_t)ks * n_cb * nt * 16 * mb * mt * 16 > part_cap) break;
      if (ks > 1 && (int64_t)n_cb * mb * kCtrStride > kLayerCtr0) break;  // one counter line per unit
      // one workgroup per CU, 32 CUs per XCD; units of a column block share its XCD.  The
      // slices of a unit wait for each other, so a split plan runs in one round.
      const int per_xcd = ((n_cb + 7) / 8) * mb * ks;
      if (ks > 1 && per_xcd > kXcdWgs) break;
      const int rounds = (per_xcd + 31) / 32;
      const double steps = (double)S_all / ks;
      const double w_time = steps * nt * 1024.0 / (8e12 / 256);                   // weights at a CU's share of HBM
      const double m_time = steps * nt * mt * 2.0 * 16.0 / 4.0 / 2.4e9;           // MFMA issue, 4 SIMDs
      const double part_bytes = ks > 1 ? 2.0 * ks * n_tiles * 16.0 * mb * mt * 16 * 4 : 0.0;
      const double a_bytes = (double)n_cb * mb * mt * 16 * K * 4;
      // the split's own cost (parked partials, the slices' wait, their sums): a price per slice
      // batch fitted to the single-finisher reduction this kernel used before; on the measured
      // shapes it still picks the faster plans (a model of the shared sums alone moved gate/up
      // to unsplit plans that ran 0.5 % slower per forward)
      const int nacc = (mt / 2) * (nt / 2);  // accumulator tiles per wave (2 x 2 waves)
      const int zb = nacc >= 32 ? 1 : (nacc >= 16 ? 2 : 4);
      const double reduce = ks > 1 ? 1e-6 + 0.6e-6 * ((ks + zb - 1) / zb) : 0.0;
      const double cost = rounds * std::max(w_time, m_time) + 0.5 * part_bytes / 8e12 + a_bytes / 32e12 + reduce;
      if (cost < best_cost) {
        best_cost = cost;
        best = GemmPlan{mt, nt, ks, mb, n_cb};
      }
    }
  }
  return best;
}

template <int MT, int NT, int EPI>
static void launch_cfg(const GemmArgs& a, const Exec& ex) {
  const int n_cb = (a.n_tiles + NT - 1) / NT;
  const unsigned grid = (unsigned)(((n_cb + 7) / 8) * 8 * a.splits * a.m_blocks);
  const bool w8 = a.Wp8 != nullptr;
  if constexpr (NT == 12) {  // bf16 weights only (gemm_plan)
    if (a.m_blocks == 1)
      SBD_KLAUNCH((gemm_kernel<MT, NT, EPI, true, false>), dim3(grid), dim3(256), ex, a);
    else
      SBD_KLAUNCH((gemm_kernel<MT, NT, EPI, false, false>), dim3(grid), dim3(256), ex, a);
  } else {
    if (a.m_blocks == 1 && w8)
      SBD_KLAUNCH((gemm_kernel<MT, NT, EPI, true, true>), dim3(grid), dim3(256), ex, a);
    else if (a.m_blocks == 1)
      SBD_KLAUNCH((gemm_kernel<MT, NT, EPI, true, false>), dim3(grid), dim3(256), ex, a);
    else if (w8)
      SBD_KLAUNCH((gemm_kernel<MT, NT, EPI, false, true>), dim3(grid), dim3(256), ex, a);
    else
      SBD_KLAUNCH((gemm_kernel<MT, NT, EPI, false, false>), dim3(grid), dim3(256), ex, a);
  }
}

template <int EPI>
static void launch_epi(const GemmArgs& a, int mt, int nt, const Exec& ex) {
  if constexpr (EPI == EPI_SWIGLU) {
    if (nt == 12) {
      if (mt == 2) launch_cfg<2, 12, EPI>(a, ex);
      else if (mt == 4) launch_cfg<4, 12, EPI>(a, ex);
      else launch_cfg<8, 12, EPI>(a, ex);
      return;
    }
  }
  if (nt == 16) {
    if (mt == 2) launch_cfg<2, 16, EPI>(a, ex);
    else if (mt == 4) launch_cfg<4, 16, EPI>(a, ex);
    else launch_cfg<8, 16, EPI>(a, ex);
  } else {
    if (mt == 2) launch_cfg<2, 8, EPI>(a, ex);
    else if (mt == 4) launch_cfg<4, 8, EPI>(a, ex);
    else launch_cfg<8, 8, EPI>(a, ex);
  }
}

hipError_t launch_gemm(GemmEpi epi, const GemmArgs& a0, const Exec& ex) {
  if (a0.M < 1 || a0.K < 32 || a0.K % 32 || a0.n_tiles < 8 || a0.n_tiles % 8) return hipErrorInvalidValue;
  if (a0.Wp8 != nullptr && a0.wscale == nullptr) return hipErrorInvalidValue;
  const bool nt12 = epi == EPI_SWIGLU && a0.Wp8 == nullptr;
  const bool half_block = (epi == EPI_SCALED_STORE || epi == EPI_LOGITS_EB) && a0.Wp8 == nullptr;
  const GemmPlan p = gemm_plan(a0.M, a0.n_tiles, a0.K, (a0.part && !a0.no_split) ? a0.part_cap : 0, nt12, half_block);
  if (p.nt == 0) return hipErrorInvalidValue;
  if (p.splits > 1 && (a0.counters == nullptr || (int64_t)p.n_cb * p.m_blocks * kCtrStride > kLayerCtr0))
    return hipErrorInvalidValue;
  if (epi == EPI_RESID && a0.n_part_out != p.n_cb) return hipErrorInvalidValue;
  // the epilogue writes 16-byte (fp32) and 8-byte (bf16) pieces of 4 columns
  if ((epi == EPI_SCALED_STORE && a0.ldo % 4) || (epi == EPI_RESID && a0.ldx % 4) ||
      (epi == EPI_SWIGLU && a0.ld_act % 4) || (epi == EPI_LOGITS_EB && a0.out_f32 && a0.ldo % 4))
    return hipErrorInvalidValue;
  if (epi == EPI_LOGITS_EB && (a0.eb_part == nullptr || a0.eb_arg == nullptr || a0.eb_chunks * kEbFChunk != a0.n_tiles * 16))
    return hipErrorInvalidValue;
  GemmArgs a = a0;
  a.splits = p.splits;
  a.m_blocks = p.m_blocks;
  // the slices of a unit wait for each other: only in a plan of one round (gemm_plan), on a
  // device that keeps every workgroup of an XCD resident at once
  if (p.splits > 1 && (!a0.wait_ok || a0.err == nullptr || ((p.n_cb + 7) / 8) * p.m_blocks * p.splits > kXcdWgs))
    return hipErrorInvalidValue;
  switch (epi) {
    case EPI_SCALED_STORE: launch_epi<EPI_SCALED_STORE>(a, p.mt, p.nt, ex); break;
    case EPI_RESID: launch_epi<EPI_RESID>(a, p.mt, p.nt, ex); break;
    case EPI_SWIGLU: launch_epi<EPI_SWIGLU>(a, p.mt, p.nt, ex); break;
    case EPI_LOGITS_EB: launch_epi<EPI_LOGITS_EB>(a, p.mt, p.nt, ex); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
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
