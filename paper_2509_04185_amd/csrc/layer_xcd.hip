// Per-XCD layer kernels: a decode-sized layer (M <= 16 block rows) of the SBD block forward
// as two launches, each of one workgroup per CU, with the work of every phase divided
// between the 8 XCDs so that every hand-off but the residual update stays inside one XCD.
//
// One kernel per projection (gemv.hip) pays, at every kernel boundary, the launch gap, the
// first-load latency of the next kernel and the tail of the previous one (wave reduction,
// split-K hand-off, epilogue).  At the 8B decode shapes that is 3-6 us per kernel against
// 6-35 us of weight streaming.  Here a layer is two launches:
//
//   layer_attn_kernel  XCD x owns KV head x.  Its 32 workgroups
//     1. project Q for the x-th group of G query heads, K and V of head x (G + 2 packed
//        groups, K split KS = 32 / (G + 2) ways; the last of a group's slices adds them and
//        runs the q/k-norm + RoPE epilogue, writing q and the new K/V cache rows);
//     2. run the attention of KV head x, one task per key range (32 / B per sequence);
//     3. merge the tasks, one wave per query row, into the attention output;
//     4. multiply that output - the K slice x of the O projection - by W_o, one packed group
//        (128 output columns) per workgroup, and add the product into the residual.
//   layer_mlp_kernel   XCD x owns columns [x F/8, (x+1) F/8) of the MLP.  Its 32 workgroups
//     1. project gate/up for those columns (F/2048 tiles each) with the SwiGLU epilogue;
//     2. multiply them - the K slice x of the down projection - by W_down, one packed group
//        per workgroup, and add the product into the residual.
//
// The residual is int64 fixed point (x * 2^32): the 8 XCDs' partial products of an output
// column are added with integer atomics, exact in any order, so no XCD waits for another
// and the result does not depend on timing.  The next consumer (QKV of the next layer,
// gate/up) forms x * g as hi/lo bf16 from it while it streams and adds up x^2 for its
// RMSNorm scale: the scale is constant along a row, so it is applied to the products.
//
// Phases 1-4 of a kernel depend on each other only within an XCD: a producer writes with
// plain stores (they reach the XCD's L2 before its vmcnt drops), raises an XCD counter with
// an atomic, and consumers poll it with atomics (a load could be served by the CU's own L1)
// and then read the data (lines their CU has not read before in the launch).  The weights
// of a phase never depend on activations, so each workgroup requests its first O / down
// weights before it waits for its inputs.
//
// Every wait is bounded: a wait that gives up raises a sticky error (device word and pinned
// host copy) that the next API call reports, and the launch runs to its end.  All 32
// workgroups of an XCD are resident at once (one per CU: the LDS request is more than half a
// CU's), so every wait is for work that is already running.

#include "attention_body.h"
#include "gemv_body.h"
#include "qkv_epilogue.h"

namespace sbd {

namespace {

constexpr int kLxSmem = 98304;       // LDS per workgroup: more than half a CU's, so one per CU
constexpr int kDH = 128;
constexpr int kLxMaxKs = 8;          // K slices of a QKV group at most (32 / (G + 2), G >= 2)
constexpr int kLxMergeBatch = kXcdWgs;  // attention tasks of one sequence at most
// counter lines of XCD x: [x * 64, x * 64 + 64); device-wide lines after all XCDs'
constexpr int kCtrQkv = 0;           // + group: last-arrival counters of the QKV slices
constexpr int kCtrQkvDone = 40;      // QKV groups finished (epilogue stored)
constexpr int kCtrAttnDone = 41;     // attention tasks finished
constexpr int kCtrMergeDone = 42;    // workgroups past the merge
constexpr int kCtrOStart = 43;       // workgroups past the O projection's wait
constexpr int kCtrGuDone = 44;       // workgroups past gate/up
constexpr int kCtrDownStart = 45;    // workgroups past the down projection's wait
constexpr int kCtrScratch = 63;      // a line nothing reads (target of l2_touch_keep)

__device__ __forceinline__ int* xcd_ctr(const LayerXArgs& a, int x, int line) {
  return a.ctr + (int64_t)(x * 64 + line) * kCtrStride;
}

// Add 1 to an XCD counter once every store of this workgroup has reached the L2.
__device__ __forceinline__ void xcd_signal(int* ctr) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Value of an XCD counter as the L2 holds it.  A load would do only once: a workgroup-scope
// load may be served by this CU's L1, which keeps the first value it fetched.  An atomic is
// always performed in the L2; adding a zero the compiler cannot see keeps it from turning
// the idempotent update back into a load.
template <int SCOPE = __HIP_MEMORY_SCOPE_WORKGROUP>
__device__ __forceinline__ int xcd_peek(int* ctr) {
  int zero;
  asm volatile("v_mov_b32 %0, 0" : "=v"(zero));
  return __hip_atomic_fetch_add(ctr, zero, __ATOMIC_RELAXED, SCOPE);
}

// Pull [p, p + bytes) into the L2 of this XCD: one 4-byte load per 128-byte line, spread
// over the workgroup.  Ordinary loads, so the compiler tracks their completion; their sum
// is returned for a use the compiler cannot remove (l2_touch_keep) and never matters.
__device__ __forceinline__ int l2_touch(const void* p, int64_t bytes) {
  const char* c = static_cast<const char*>(p);
  int sum = 0;
  for (int64_t o = (int64_t)threadIdx.x * 128; o < bytes; o += (int64_t)blockDim.x * 128)
    sum += *reinterpret_cast<const int*>(c + o);
  return sum;
}
// Consumes the sum of l2_touch: `never` is a value the sum cannot be told from at compile
// time; the store, into this workgroup's own scratch, is not reached in practice either
// way and changes nothing another phase reads.
__device__ __forceinline__ void l2_touch_keep(int sum, int never, int* scratch) {
  if (sum == never) scratch[threadIdx.x % kCtrStride] = sum;
}

// Wait until *ctr >= target (thread 0 polls, then the workgroup proceeds).  SCOPE: that of
// the counter's writers (device scope for a device-wide counter).
template <int SCOPE = __HIP_MEMORY_SCOPE_WORKGROUP>
__device__ __forceinline__ void xcd_wait(const LayerXArgs& a, int* ctr, int target, int what) {
  if (threadIdx.x == 0) {
    int it = 0;
    while (xcd_peek<SCOPE>(ctr) < target) {
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
  }
  __syncthreads();
}

// Counts workgroups past their last wait on this XCD's phase counters; the last of the 32
// resets those counters (and itself) for the next launch.
__device__ __forceinline__ void xcd_passed(const LayerXArgs& a, int x, int line, const int* resets, int n) {
  __syncthreads();
  if (threadIdx.x == 0) {
    int* c = xcd_ctr(a, x, line);
    if (__hip_atomic_fetch_add(c, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) == kXcdWgs - 1) {
      for (int i = 0; i < n; ++i)
        __hip_atomic_store(xcd_ctr(a, x, resets[i]), 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      __hip_atomic_store(c, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  }
}

// The 4 waves' partial tiles of a C-tile unit added in wave order; wave w ends with the sums
// of the tiles ct = w, w + 4, ... (the tiles it owns).  red: 4 * C KB of LDS.
template <int C>
__device__ __forceinline__ void reduce_waves(f32x4 (&acc)[C], char* red_mem) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  f32x4* red = reinterpret_cast<f32x4*>(red_mem);  // [4][C][64]
#pragma unroll
  for (int ct = 0; ct < C; ++ct) red[(wave * C + ct) * 64 + lane] = acc[ct];
  __syncthreads();
#pragma unroll
  for (int ct = 0; ct < C; ++ct) {
    if (ct % 4 != wave) continue;
    f32x4 s = red[(0 * C + ct) * 64 + lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) s += red[(w * C + ct) * 64 + lane];
    acc[ct] = s;
  }
  __syncthreads();  // red is free again
}

// Sum of x^2 of rows 0..15 over the lanes and waves of a workgroup: lane (r, g) of every
// wave holds a share of row r; the 4 waves' row sums are added in wave order.  Result in
// row_s[0..15] (LDS) after the call.
__device__ __forceinline__ void row_ss_reduce(float ss, float* tmp_s, float* row_s) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  ss += __shfl_xor(ss, 16);
  ss += __shfl_xor(ss, 32);
  if (lane < 16) tmp_s[wave * 16 + lane] = ss;
  __syncthreads();
  if (threadIdx.x < 16)
    row_s[threadIdx.x] = tmp_s[threadIdx.x] + tmp_s[16 + threadIdx.x] + tmp_s[32 + threadIdx.x] + tmp_s[48 + threadIdx.x];
  __syncthreads();
}

// The residual lives in three buffers used in turn: launch i reads x_src = R[i % 3], adds
// its products into x_dst = R[(i + 1) % 3] (zeroed by launch i - 1) and zeroes
// x_zero = R[(i + 2) % 3] (read by launch i - 1, so nobody uses it any more).  Nothing is
// read and updated in one launch, so no workgroup waits for the others' reads.  The old
// value of each output column is added exactly once: XCD x adds it for tile x of each
// packed group, together with its own partial product.

// Share `part` of `parts` of x_zero (rows [0, M)), 16 bytes per store.
__device__ __forceinline__ void residual_zero(const LayerXArgs& a, int part, int parts) {
  const int64_t n = (int64_t)a.M * a.d / 2;  // d is even
  longlong2* z = reinterpret_cast<longlong2*>(a.x_zero);
  for (int64_t e = (int64_t)part * 256 + threadIdx.x; e < n; e += (int64_t)parts * 256) z[e] = longlong2{0, 0};
}

// Old residual of the elements of tile x of group grp that this lane adds (rows 4 g4 + i,
// column r; wave x % 4 owns the tile); zero elsewhere.
__device__ __forceinline__ void residual_old(const LayerXArgs& a, int grp, int x, long long (&old)[4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) old[i] = 0;
  if (wave == (x & 3)) {
    const int n = (grp * 8 + x) * 16 + r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = 4 * g4 + i;
      if (m < a.M) old[i] = a.x_src[(int64_t)m * a.d + n];
    }
  }
}

// Add the summed tiles of packed group grp (wave w owns tiles w and w + 4) into x_dst, with
// the old values of tile x.
__device__ __forceinline__ void residual_add(const LayerXArgs& a, int grp, int x, const f32x4 (&acc)[8],
                                             const long long (&old)[4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2) {
    const int ct = wave + 4 * k2;
    const int n = (grp * 8 + ct) * 16 + r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = 4 * g4 + i;
      if (m < a.M) fix_add_q(a.x_dst + (int64_t)m * a.d + n, fix_q(acc[ct][i]) + (ct == x ? old[i] : 0));
    }
  }
}

}  // namespace

// WT: the weights' format (bf16_t, or fp8_t widened to bf16 in registers: twice the steps per
// batch keep the same bytes in flight).
template <class WT, bool KV8>
__global__ __launch_bounds__(256) void layer_attn_kernel(LayerXArgs a) {
  constexpr int UW = sizeof(WT) == 1 ? 2 : 1;  // batch scale of the weight streams
  __shared__ __attribute__((aligned(16))) char smem[kLxSmem];
  const int x = blockIdx.x & 7, lw = blockIdx.x >> 3;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g4 = lane >> 4;
  const int G = a.n_q / a.n_kv;
  const int ngrp = G + 2, KS = kXcdWgs / ngrp;
  float* xpart = a.xpart + (int64_t)x * kLxXcdFloats;
  // the workgroups without a QKV slice zero the next launch's residual buffer meanwhile
  const int n_idle = kXcdWgs - ngrp * KS;
  if (lw >= ngrp * KS) residual_zero(a, x * n_idle + (lw - ngrp * KS), kXcds * n_idle);

  bool finisher = false;  // this workgroup ran a QKV group's epilogue
  // ---- 1. QKV projection, unit (group gi of this XCD, K slice kc)
  if (lw < ngrp * KS) {
    const int gi = lw / KS, kc = lw % KS;
    const int grp = gi < G ? x * G + gi : (gi == G ? a.n_q + x : a.n_q + a.n_kv + x);
    const int S = a.d / 32;
    const int z0 = S * kc / KS, z1 = S * (kc + 1) / KS;
    const int s_b = z0 + (z1 - z0) * wave / 4, ns = z0 + (z1 - z0) * (wave + 1) / 4 - s_b;
    QkvEpi e{};
    e.rows = a.rows; e.seqs = a.seqs; e.kblk = a.k; e.layer = a.layer;
    e.n_q = a.n_q; e.n_kv = a.n_kv; e.d_h = kDH; e.qk_norm = a.qk_norm; e.eps = a.eps; e.q_scale = a.q_scale;
    e.rope = a.rope; e.q_norm = a.q_norm; e.k_norm = a.k_norm; e.q = a.q; e.q_lo = a.q_lo;
    e.kcache = a.kcache; e.vcache = a.vcache; e.cap = a.cap; e.n_slots = a.n_slots;
    e.kv_fp8 = KV8; e.kv_inv = a.kv_inv;
    QkvPre<kDH> qpre;
    qkv_epi_prefetch<kDH>(e, a.M, qpre);
    const int arow = r < a.M ? r : a.M - 1;
    const WT* wt[8];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) wt[ct] = static_cast<const WT*>(a.wqkv) + packed_frag(grp * 8 + ct, s_b, S) + lane * 8;
    float wsc[8];
    load_wscale<WT, 8>(a.sc_qkv, grp * 8, r, wsc);
    f32x4 acc[8];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    float ss = 0.f;  // x^2 of this lane's elements of row r: the slice's share of the RMSNorm sums
    gemv_stream_x64<8, UW>(buf_rsrc(a.x_src), buf_rsrc(a.g_attn), (uint32_t)(((int64_t)arow * a.d + g4 * 8 + s_b * 32) * 8),
                           (uint32_t)((g4 * 8 + s_b * 32) * 2), wt, ns, wsc, acc, ss);
    float* ss_s = reinterpret_cast<float*>(smem + 65536 + 1024);  // [64] wave shares, then [16] rows
    row_ss_reduce(r < a.M ? ss : 0.f, ss_s, ss_s + 64);
    reduce_waves<8>(acc, smem);
    // park this slice (tiles, then its 16 row sums of x^2) in the XCD's L2; the last of the
    // group's KS slices finishes the group
    float* qp = xpart + (int64_t)gi * KS * kLxQkvSlice;
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const int ct = wave + 4 * k2;
      *(f32x4*)(qp + (int64_t)kc * kLxQkvSlice + (ct * 64 + lane) * 4) = acc[ct];
    }
    if (threadIdx.x < 16) qp[(int64_t)kc * kLxQkvSlice + 2048 + threadIdx.x] = ss_s[64 + threadIdx.x];
    if (last_arrival_xcd(xcd_ctr(a, x, kCtrQkv + gi), KS)) {
      const __amdgpu_buffer_rsrc_t rq = buf_rsrc(qp);
      f32x4* fin = reinterpret_cast<f32x4*>(smem);  // [8][64]
      // Every reload of the group's slices (this wave's two tiles, and the row sums of x^2)
      // is requested before any is used: one round trip to the L2.  Slots past KS re-read
      // slice 0, which keeps the loads unconditional (a load behind a runtime condition
      // becomes a branch that waits for it), and are dropped from the sums.
      i32x4 v[2][kLxMaxKs];
      float t[kLxMaxKs];
      const int rs = threadIdx.x & 15;
#pragma unroll
      for (int z = 0; z < kLxMaxKs; ++z) {
        const int zz = z < KS ? z : 0;
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2)
          v[k2][z] = ld16_l2(rq, (uint32_t)(((int64_t)zz * kLxQkvSlice + ((wave + 4 * k2) * 64 + lane) * 4) * 4));
        t[z] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                             rq, (uint32_t)(((int64_t)zz * kLxQkvSlice + 2048 + rs) * 4), 0, kPolicyL2));
      }
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {  // added in slice order
        f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int z = 0; z < kLxMaxKs; ++z) sum += z < KS ? __builtin_bit_cast(f32x4, v[k2][z]) : f32x4{0.f, 0.f, 0.f, 0.f};
        fin[(wave + 4 * k2) * 64 + lane] = sum;
      }
      float* rinv_s = reinterpret_cast<float*>(smem + 65536 + 2048);  // [16]
      if (threadIdx.x < 16) {  // the KS slices' sums of x^2 of row threadIdx.x, in slice order
        float tt = 0.f;
#pragma unroll
        for (int z = 0; z < kLxMaxKs; ++z) tt += z < KS ? t[z] : 0.f;
        rinv_s[threadIdx.x] = 1.0f / sqrtf(tt / (float)a.d + a.eps);
      }
      __syncthreads();
#pragma unroll
      for (int ct = 0; ct < 8; ++ct) acc[ct] = fin[ct * 64 + lane];
      float rinv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) rinv[i] = rinv_s[4 * g4 + i];
      qkv_epilogue<kDH>(e, a.M, grp, acc, rinv, qpre, wave);  // wave w: rows 4g + w
      xcd_signal(xcd_ctr(a, x, kCtrQkvDone));
      finisher = true;
    }
  }

  // The first two steps of this wave's O weights (phase 4): requested now by the workgroups
  // that finished no QKV group (the memory system is idle until phase 4), by the others
  // before their wait in phase 4, so that nothing on the way to the attention waits for them.
  const int o_S = a.n_q * kDH / 32;
  const int o_z0 = x * G * kDH / 32, o_zn = G * kDH / 32;
  const int o_sb = o_z0 + o_zn * wave / 4, o_ns = o_z0 + o_zn * (wave + 1) / 4 - o_sb;
  const WT* o_wt[8];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) o_wt[ct] = static_cast<const WT*>(a.wo) + packed_frag(lw * 8 + ct, o_sb, o_S) + lane * 8;
  typename WFrag<WT>::T o_w01[2][8];
  if (!finisher && o_ns > 0) gemv_issue_w<8, 2>(o_wt, 0, o_ns, o_w01);

  // ---- 2. attention of KV head x: task t = (sequence, key range)
  const int n_tasks = a.B * a.n_tasks;
  float* att_ml = xpart + kLxQkvFloats;                         // [task][64 rows][2]
  float* att_o = att_ml + (int64_t)kLxAttnTasks * kLxRows * 2;  // [task][64 rows][128]
  if (lw < n_tasks) {
    const int b = lw / a.n_tasks, s = lw % a.n_tasks;
    const SeqParam sp = a.seqs[b];
    const int L = sp.cache_len;
    const int nblk = (L + a.k + 31) / 32;
    int touched = 0;
    {  // key blocks holding only positions cached before this forward: into the L2 now
      const int kb0 = nblk * s / a.n_tasks, kb1 = min(nblk * (s + 1) / a.n_tasks, L / 32);
      if (kb1 > kb0) {
        constexpr int es = KV8 ? 1 : 2;  // bytes per cached element
        const int64_t off = (attn_head_base(a.layer, sp.slot, x, a.n_slots, a.n_kv, a.cap, kDH) +
                             (int64_t)kb0 * 32 * kDH) * es;
        const int64_t bytes = (int64_t)(kb1 - kb0) * 32 * kDH * es;
        touched += l2_touch(static_cast<const char*>(a.kcache) + off, bytes);
        touched += l2_touch(static_cast<const char*>(a.vcache) + off, bytes);
      }
    }
    xcd_wait(a, xcd_ctr(a, x, kCtrQkvDone), ngrp, a.layer * 16 + 1);
    AttnArgs aa{};
    aa.seqs = a.seqs; aa.B = a.B; aa.k = a.k; aa.layer = a.layer; aa.n_q = a.n_q; aa.n_kv = a.n_kv; aa.d_h = kDH;
    aa.q = a.q; aa.q_lo = a.q_lo; aa.kcache = a.kcache; aa.vcache = a.vcache; aa.cap = a.cap; aa.n_slots = a.n_slots;
    aa.kv_fp8 = KV8; aa.kv_scale = a.kv_scale;
    aa.n_rowblocks = 1;
    AttnPart<kDH> pt;
    attn_core<kDH, kPolicyL2, KV8>(aa, x, 0, b, nblk * s / a.n_tasks, nblk * (s + 1) / a.n_tasks, smem, pt);
    if (pt.row_ok) {
      if (g4 == 0) *(float2*)(att_ml + ((int64_t)lw * kLxRows + pt.rho) * 2) = float2{pt.m, pt.l};
#pragma unroll
      for (int dt = 0; dt < kDH / 16; ++dt)
        *(f32x4*)(att_o + ((int64_t)lw * kLxRows + pt.rho) * kDH + 16 * dt + 4 * g4) = pt.o[dt];
    }
    xcd_signal(xcd_ctr(a, x, kCtrAttnDone));
    l2_touch_keep(touched, a.layer - (1 << 30), xcd_ctr(a, x, kCtrScratch));
  }

  // ---- 3. merge: one wave per query row (sequence b, row rho = head-in-group * k + j)
  {
    const int R = G * a.k, n_rows = a.B * R;
    const int row = lw * 4 + wave;
    if (lw * 4 < n_rows) {
      xcd_wait(a, xcd_ctr(a, x, kCtrAttnDone), n_tasks, a.layer * 16 + 2);
      if (row < n_rows) {
        const int b = row / R, rho = row % R;
        const int nt = a.n_tasks;
        const __amdgpu_buffer_rsrc_t rml = buf_rsrc(att_ml), ro = buf_rsrc(att_o);
        float2 ml = float2{-INFINITY, 0.f};
        if (lane < nt) {
          const i32x2 v = ld8_l2(rml, (uint32_t)((((int64_t)(b * nt + lane)) * kLxRows + rho) * 8));
          ml = float2{__int_as_float(v[0]), __int_as_float(v[1])};
        }
        const float mx = wave_max(ml.x);
        const float wgt = ml.x == -INFINITY ? 0.f : exp2f(ml.x - mx);
        const float lsum = wave_sum(wgt * ml.y);
        float acc0 = 0.f, acc1 = 0.f;
        // every task's partial requested at once (nt <= kLxMergeBatch: one round trip on the
        // layer's dependency chain), added in task order
        for (int t0 = 0; t0 < nt; t0 += kLxMergeBatch) {  // wave-uniform
          float v0[kLxMergeBatch], v1[kLxMergeBatch];
#pragma unroll
          for (int u = 0; u < kLxMergeBatch; ++u) {
            const int t = min(t0 + u, nt - 1);
            const uint32_t base = (uint32_t)((((int64_t)(b * nt + t)) * kLxRows + rho) * kDH * 4);
            v0[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ro, base + lane * 4, 0, kPolicyL2));
            v1[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(ro, base + (lane + 64) * 4, 0, kPolicyL2));
          }
#pragma unroll
          for (int u = 0; u < kLxMergeBatch; ++u) {
            const float wu = t0 + u < nt ? __shfl(wgt, t0 + u) : 0.f;
            acc0 += wu * v0[u];
            acc1 += wu * v1[u];
          }
        }
        const float inv = 1.0f / lsum;
        const int hh = rho / a.k, j = rho % a.k;
        const int64_t dst = ((int64_t)(b * a.k + j) * a.n_q + x * G + hh) * kDH;
        bf16_t hi, lo;
        split_bf16(acc0 * inv, hi, lo);
        a.attn[dst + lane] = hi;
        a.attn_lo[dst + lane] = lo;
        split_bf16(acc1 * inv, hi, lo);
        a.attn[dst + lane + 64] = hi;
        a.attn_lo[dst + lane + 64] = lo;
      }
    }
    xcd_signal(xcd_ctr(a, x, kCtrMergeDone));
  }

  // ---- 4. O projection: group lw, K slice x (the query heads of KV head x)
  {
    const int grp = lw;
    const int qd = a.n_q * kDH;
    const int ns = o_ns;
    // weights first: they wait for nothing.  Steps 0, 1 in o_w01, the rest in batches of 2.
    if (finisher && ns > 0) gemv_issue_w<8, 2>(o_wt, 0, ns, o_w01);
    const WT* wt2[8];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) wt2[ct] = o_wt[ct] + 2 * kPackStep;
    constexpr int U = 2 * UW;
    typename WFrag<WT>::T w0[U][8];
    if (ns > 2) gemv_issue_w<8, U>(wt2, 0, ns - 2, w0);
    float wsc[8];
    load_wscale<WT, 8>(a.sc_o, grp * 8, r, wsc);
    long long old[4];
    residual_old(a, grp, x, old);
    xcd_wait(a, xcd_ctr(a, x, kCtrMergeDone), kXcdWgs, a.layer * 16 + 3);
    {
      const int resets[3] = {kCtrQkvDone, kCtrAttnDone, kCtrMergeDone};
      xcd_passed(a, x, kCtrOStart, resets, 3);
    }
    f32x4 acc[8];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int arow = r < a.M ? r : a.M - 1;
    const __amdgpu_buffer_rsrc_t ra = buf_rsrc(a.attn), ral = buf_rsrc(a.attn_lo);
    const uint32_t a_off = (uint32_t)(((int64_t)arow * qd + g4 * 8 + o_sb * 32) * 2);
    if (ns > 0) {
      i32x4 xa[2], xl[2];
      gemv_issue_a<2, kPolicyL2>(ra, ral, a_off, 0, ns, xa, xl);
      gemv_mfma<8, 2>(o_w01, xa, xl, 0, ns, wsc, acc);
    }
    if (ns > 2) gemv_stream<8, U, kPolicyL2, true>(ra, ral, a_off + 2 * 64, wt2, ns - 2, w0, wsc, acc);
    reduce_waves<8>(acc, smem);
    residual_add(a, grp, x, acc, old);
  }
  if (n_idle == 0) residual_zero(a, blockIdx.x, gridDim.x);
}

template <int CG, class WT>
__global__ __launch_bounds__(256) void layer_mlp_kernel(LayerXArgs a) {
  constexpr int UW = sizeof(WT) == 1 ? 2 : 1;  // batch scale of the weight streams
  __shared__ __attribute__((aligned(16))) char smem[kLxSmem];
  const int x = blockIdx.x & 7, lw = blockIdx.x >> 3;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g4 = lane >> 4;
  float* ss_s = reinterpret_cast<float*>(smem + 65536 + 1024);  // [64] wave shares, then [16] rows

  // ---- 1. gate/up + SwiGLU: tiles t0 .. t0 + CG - 1 (activation columns 8 t .. 8 t + 7)
  {
    const int t0 = (x * kXcdWgs + lw) * CG;
    const int S = a.d / 32;
    const int s_b = S * wave / 4, ns = S * (wave + 1) / 4 - s_b;
    const int arow = r < a.M ? r : a.M - 1;
    const WT* wt[CG];
#pragma unroll
    for (int ct = 0; ct < CG; ++ct) wt[ct] = static_cast<const WT*>(a.wgu) + packed_frag(t0 + ct, s_b, S) + lane * 8;
    float wsc[CG];
    load_wscale<WT, CG>(a.sc_gu, t0, r, wsc);
    f32x4 acc[CG];
#pragma unroll
    for (int ct = 0; ct < CG; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    float ss = 0.f;  // the whole row passes through the 4 waves: its sum of x^2 for the RMSNorm
    gemv_stream_x64<CG, UW>(buf_rsrc(a.x_src), buf_rsrc(a.g_mlp), (uint32_t)(((int64_t)arow * a.d + g4 * 8 + s_b * 32) * 8),
                            (uint32_t)((g4 * 8 + s_b * 32) * 2), wt, ns, wsc, acc, ss);
    row_ss_reduce(r < a.M ? ss : 0.f, ss_s, ss_s + 64);
    float* rinv_s = ss_s + 64;
    if (threadIdx.x < 16) rinv_s[threadIdx.x] = 1.0f / sqrtf(rinv_s[threadIdx.x] / (float)a.d + a.eps);
    reduce_waves<CG>(acc, smem);
#pragma unroll
    for (int ct = 0; ct < CG; ++ct) {
      if (ct % 4 != wave) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 4 * g4 + i;
        const float v = acc[ct][i] * (m < a.M ? rinv_s[m] : 0.f);
        const float up = __shfl_xor(v, 8);
        if (r < 8 && m < a.M) {
          const int jj = (t0 + ct) * 8 + r;
          bf16_t hi, lo;
          split_bf16(v / (1.0f + expf(-v)) * up, hi, lo);
          a.act[(int64_t)m * a.ffn + jj] = hi;
          a.act_lo[(int64_t)m * a.ffn + jj] = lo;
        }
      }
    }
    xcd_signal(xcd_ctr(a, x, kCtrGuDone));
  }

  // ---- 2. down projection: group lw, K slice x (activation columns [x F/8, (x+1) F/8))
  {
    const int grp = lw;
    const int S = a.ffn / 32, zn = a.ffn / 8 / 32, z0 = x * zn;
    const int s_b = z0 + zn * wave / 4, ns = z0 + zn * (wave + 1) / 4 - s_b;
    const WT* wt[8];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) wt[ct] = static_cast<const WT*>(a.wdown) + packed_frag(grp * 8 + ct, s_b, S) + lane * 8;
    constexpr int U = 2 * UW;
    typename WFrag<WT>::T w0[U][8];
    if (ns > 0) gemv_issue_w<8, U>(wt, 0, ns, w0);  // weights first: they wait for nothing
    float wsc[8];
    load_wscale<WT, 8>(a.sc_down, grp * 8, r, wsc);
    long long old[4];
    residual_old(a, grp, x, old);
    xcd_wait(a, xcd_ctr(a, x, kCtrGuDone), kXcdWgs, a.layer * 16 + 5);
    {
      const int resets[1] = {kCtrGuDone};
      xcd_passed(a, x, kCtrDownStart, resets, 1);
    }
    f32x4 acc[8];
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int arow = r < a.M ? r : a.M - 1;
    gemv_stream<8, U, kPolicyL2, true>(buf_rsrc(a.act), buf_rsrc(a.act_lo),
                                       (uint32_t)(((int64_t)arow * a.ffn + g4 * 8 + s_b * 32) * 2), wt, ns, w0, wsc, acc);
    reduce_waves<8>(acc, smem);
    residual_add(a, grp, x, acc, old);
  }
  // the next launch's residual buffer, zeroed last: nothing here waits for these stores
  residual_zero(a, blockIdx.x, gridDim.x);
}

// After the last layer: the LM head's inputs from the fixed-point residual.  Row m =
// blockIdx.x, columns 1024 blockIdx.y + 4 t .. + 3 for thread t.
__global__ __launch_bounds__(256) void layer_finalize_kernel(FinalizeArgs a) {
  const int m = blockIdx.x;
  const int c = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (c >= a.d) return;  // d % 16 == 0: a 16-column group lies inside or outside as a whole
  const int64_t o = (int64_t)m * a.d + c;
  const longlong2 q0 = *reinterpret_cast<const longlong2*>(a.x64 + o);
  const longlong2 q1 = *reinterpret_cast<const longlong2*>(a.x64 + o + 2);
  const uint2 gv = *reinterpret_cast<const uint2*>(a.g + c);
  const long long q[4] = {q0.x, q0.y, q1.x, q1.y};
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = fix_to_f32((int)(uint32_t)(uint64_t)q[e], (int)(q[e] >> 32));
  *reinterpret_cast<float4*>(a.x + o) = float4{v[0], v[1], v[2], v[3]};
  const f32x4 xg = f32x4{v[0] * __uint_as_float(gv.x << 16), v[1] * __uint_as_float(gv.x & 0xffff0000u),
                         v[2] * __uint_as_float(gv.y << 16), v[3] * __uint_as_float(gv.y & 0xffff0000u)};
  i32x2 hi, lo;
  split_bf16x4(xg, hi, lo);
  *reinterpret_cast<i32x2*>(a.xn + o) = hi;
  *reinterpret_cast<i32x2*>(a.xn_lo + o) = lo;
  float s = v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  s += __shfl_xor(s, 1);
  s += __shfl_xor(s, 2);
  if ((threadIdx.x & 3) == 0) a.sumsq[(int64_t)m * (a.d / 16) + c / 16] = s;
}

bool layer_xcd_fits(const sbd_model_config& c, int n_cu, int B, int k) {
  if (n_cu != kXcds * kXcdWgs) return false;
  if (c.n_kv_heads != kXcds || c.head_dim != kDH || c.d_model != kXcdWgs * 128) return false;
  if (c.n_q_heads % c.n_kv_heads) return false;
  const int G = c.n_q_heads / c.n_kv_heads;
  if (G < 2 || G + 2 > kXcdWgs || (c.d_model / 32) / (kXcdWgs / (G + 2)) < 4) return false;
  if (c.ffn_dim % (kXcds * kXcdWgs * 8) != 0) return false;
  const int cg = c.ffn_dim / (kXcds * kXcdWgs * 8);
  if (cg < 6 || cg > 8) return false;
  if (B < 1 || k < 1 || B * k > kLxMaxRows || G * k > kLxRows || B > kLxAttnTasks) return false;
  if ((B * G * k + 3) / 4 > kXcdWgs) return false;  // one wave per merged row
  return true;
}

hipError_t launch_layer_attn(const LayerXArgs& a, bool fp8, const Exec& ex) {
  const dim3 grid(kXcds * kXcdWgs), block(256);
  if (fp8 && a.kv_fp8)
    SBD_KLAUNCH((layer_attn_kernel<fp8_t, true>), grid, block, ex, a);
  else if (fp8)
    SBD_KLAUNCH((layer_attn_kernel<fp8_t, false>), grid, block, ex, a);
  else if (a.kv_fp8)
    SBD_KLAUNCH((layer_attn_kernel<bf16_t, true>), grid, block, ex, a);
  else
    SBD_KLAUNCH((layer_attn_kernel<bf16_t, false>), grid, block, ex, a);
  return hipGetLastError();
}

hipError_t launch_layer_finalize(const FinalizeArgs& a, const Exec& ex) {
  if (a.d % 16 != 0) return hipErrorInvalidValue;
  SBD_KLAUNCH(layer_finalize_kernel, dim3(a.M, (a.d + 1023) / 1024), dim3(256), ex, a);
  return hipGetLastError();
}

template <class WT>
static hipError_t launch_layer_mlp_t(const LayerXArgs& a, const Exec& ex) {
  const int cg = a.ffn / (kXcds * kXcdWgs * 8);
  switch (cg) {
    case 6: SBD_KLAUNCH((layer_mlp_kernel<6, WT>), dim3(kXcds * kXcdWgs), dim3(256), ex, a); break;
    case 7: SBD_KLAUNCH((layer_mlp_kernel<7, WT>), dim3(kXcds * kXcdWgs), dim3(256), ex, a); break;
    case 8: SBD_KLAUNCH((layer_mlp_kernel<8, WT>), dim3(kXcds * kXcdWgs), dim3(256), ex, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_layer_mlp(const LayerXArgs& a, bool fp8, const Exec& ex) {
  return fp8 ? launch_layer_mlp_t<fp8_t>(a, ex) : launch_layer_mlp_t<bf16_t>(a, ex);
}

}  // namespace sbd
