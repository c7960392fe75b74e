// Block-hybrid grouped-query attention of the SBD block forward.
//
// For sequence b with cache length L and block rows j = 0..k-1 (stored at positions
// L + j), row j attends to key position kv iff kv < L + j + 1 when j is a causal row
// (j < n_causal) and to every key kv < L + k when j is in the prediction block: the
// inference mask of the paper (App. A, Fig. 3) restricted to the rows of the block.
//
// Work split: one workgroup per (split, KV head x row block, sequence).  The rows of a
// KV head are the group*k (query head, block row) pairs that read it; each wave takes 16
// of them (one MFMA tile) and walks the keys of its split in 32-key steps:
//   S^T = K Q^T   (v_mfma_f32_16x16x32_bf16: keys on M, query rows on N, d_h in 4 steps;
//                  Q as hi + lo bf16, two MFMAs per step)
//   online softmax per query row in base 2 (queries carry log2(e)/sqrt(d_h))
//   O^T += V^T P^T (P as hi + lo bf16 in the B-operand layout straight from the score
//                   tile; V^T comes from the transposed, permuted cache blocks)
// Each split leaves unnormalised (max, sum, O) per row; a merge kernel combines the
// splits with log-sum-exp weights in split order.  K and V blocks are staged in LDS by the
// whole workgroup (see the kernels: attention_body.h for the launches that share a
// workgroup with other phases, attn_split_kernel below for the standalone split kernel).

#include <type_traits>

#include "attention_body.h"

namespace sbd {

// The split kernel of the per-kernel path streams long key ranges, so it is shaped for
// bytes in flight: 8 waves, NRS row sets of 16 query rows times KP = 8 / NRS key parts (4 x 2,
// or 2 x 4 when a row block has at most 32 rows, so that no wave idles); the key positions
// of a ring stage (KP blocks of 32 keys of K and V from a bf16 cache, 2 KP from an fp8 cache;
// copied straight into LDS) are split between the KP waves holding the same 16 query rows,
// so each SIMD has two waves to overlap MFMA, softmax and LDS reads with the stream (an fp8
// wave takes two blocks per stage under one softmax update: the chain of a stage, not its
// bytes, sets its time); a ring of NBUF stages (128 KB) keeps NBUF - 1 stages in flight.  At
// the end the KP key parts of each row set are combined through LDS (log-sum-exp weights,
// in part order) into the split's partial.  LDS reads are ds_read16 (ds_read8 of an fp8
// cache), ordered by hand (see sbd_device.h).
template <int DH, bool KV8, int NRS>
__global__ __launch_bounds__(512) void attn_split_kernel(AttnArgs a) {
  using KB = KvBlk<DH, KV8>;    // a staged block's layout in LDS
  constexpr int NDT = DH / 16;  // 16-wide dimension tiles
  constexpr int NKS = DH / 32;  // 32-wide reduction steps for the scores
  constexpr int KP = 8 / NRS;                 // key parts
  constexpr int BLK = KB::BYTES;              // bytes of K (or of V) per 32-key block
  constexpr int BPW = KV8 ? 2 : 1;            // blocks per wave and stage
  constexpr int BPS = KP * BPW;               // blocks per stage
  constexpr int STAGE = BPS * 2 * BLK;        // K and V of the stage's blocks
  constexpr int NBUF = (128 * 1024) / STAGE > 8 ? 8 : (128 * 1024) / STAGE;
  constexpr int LPB = BLK / 1024;             // 1 KB wave-loads per part per block
  constexpr int PER_WAVE = STAGE / 1024 / 8;  // wave-loads of one wave per stage
  static_assert(NBUF >= 2 && (NBUF - 2) * PER_WAVE <= 63, "ring shape");
  static_assert(NRS * KP == 8 && (KP - 1) * NRS * 64 * (NDT * 16 + 16) <= NBUF * STAGE, "wave shape");
  __shared__ __attribute__((aligned(16))) char smem[NBUF * STAGE];
  __shared__ int s_kend[8];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rs = w % NRS, kh = w / NRS;  // row set (16 rows), key part of each stage
  const int r = lane & 15, grp = lane >> 4;
  const int split = blockIdx.x, g = blockIdx.y / a.n_rowblocks, rb = blockIdx.y % a.n_rowblocks, b = blockIdx.z;
  const SeqParam sp = a.seqs[b];
  const int L = sp.cache_len, nc = sp.n_causal, k = a.k;
  const int G = a.n_q / a.n_kv;
  const int R = G * k;
  const int rho = rb * 16 * NRS + rs * 16 + r;
  const bool row_ok = rho < R;
  const int hh = row_ok ? rho / k : 0;
  const int j = row_ok ? rho % k : 0;
  const int hq = g * G + hh;
  const int kend = row_ok ? ((j >= nc) ? L + k : L + j + 1) : 0;
  const int blk0 = split * a.blocks_per_split, blk_lim = blk0 + a.blocks_per_split;
  int kend_w = kend;
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) kend_w = max(kend_w, __shfl_xor(kend_w, o));
  const int blk1 = min(blk_lim, (kend_w + 31) / 32);  // this wave's blocks end here
  int kend_wg = kend_w;
  kend_wg = max(kend_wg, __shfl_xor(kend_wg, 16));
  kend_wg = max(kend_wg, __shfl_xor(kend_wg, 32));
  if (lane == 0) s_kend[w] = kend_wg;

  // queries (B operand, hi and lo): row r, dims 32 s + 8 grp .. + 8; complete before the ring
  i32x4 qf[NKS], ql[NKS];
  const int64_t qoff = ((int64_t)(b * k + j) * a.n_q + hq) * DH;
#pragma unroll
  for (int s2 = 0; s2 < NKS; ++s2) {
    qf[s2] = row_ok ? *(const i32x4*)(a.q + qoff + 32 * s2 + 8 * grp) : i32x4{0, 0, 0, 0};
    ql[s2] = row_ok ? *(const i32x4*)(a.q_lo + qoff + 32 * s2 + 8 * grp) : i32x4{0, 0, 0, 0};
  }
  vm_wait<0>();
  __syncthreads();
  for (int i = 0; i < 8; ++i) kend_wg = max(kend_wg, s_kend[i]);
  const int blk1_wg = min(blk_lim, (kend_wg + 31) / 32);
  const int n_st = blk1_wg > blk0 ? (blk1_wg - blk0 + BPS - 1) / BPS : 0;

  const int64_t hb = attn_head_base(a.layer, sp.slot, g, a.n_slots, a.n_kv, a.cap, DH);
  const char* kbase = static_cast<const char*>(a.kcache) + hb * KB::ES;
  const char* vbase = static_cast<const char*>(a.vcache) + hb * KB::ES;
  const float kv_sc = a.kv_scale;
  // Wave-load u of wave w in stage st: i = w + 8u -> block i / (2 LPB) of the stage, part
  // (i / LPB) % 2 (K, V), 1 KB slice i % LPB; pieces XOR-swizzled (KvBlk).
  auto issue = [&](int st) {
    char* buf = smem + (st % NBUF) * STAGE;
#pragma unroll
    for (int u = 0; u < PER_WAVE; ++u) {
      const int idx = w + 8 * u;
      const int bi = idx / (2 * LPB), part = (idx / LPB) % 2, sub = idx % LPB;
      int kb = blk0 + BPS * st + bi;
      if (kb >= blk1_wg) kb = blk1_wg - 1;  // past the end: a valid block, never used
      __builtin_amdgcn_global_load_lds((const void*)KB::src(kbase, vbase, kb, part, sub * 64 + lane),
                                       (__attribute__((address_space(3))) void*)(buf + (bi * 2 + part) * BLK + sub * 1024),
                                       16, 0, 2);  // nt: each cache byte is read once
    }
  };

  f32x4 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // this wave's block of stage st: scores, online softmax, O^T += V^T P^T
  auto compute = [&](int st) {
    const int kb0 = blk0 + BPS * st + kh * BPW;  // this wave's first block
    if (kb0 >= blk1) return;  // wave-uniform: nothing of its blocks is visible to its rows
    const char* blk = smem + (st % NBUF) * STAGE + (kh * BPW * 2) * BLK;  // block j: K at 2 j BLK, V after
    // fragments: KV8 reads 8 bytes and widens them once the reads are complete
    typedef typename std::conditional<KV8, i32x2, i32x4>::type Frag;
    auto rd = [](const char* p) -> Frag {
      if constexpr (KV8) return ds_read8(lds_addr(p));
      else return ds_read16(lds_addr(p));
    };
    auto widen = [&](Frag v) -> i32x4 {
      if constexpr (KV8) return e4m3x8_to_bf16(v, kv_sc);
      else return v;
    };
    Frag kr[BPW][2][NKS];
#pragma unroll
    for (int jb = 0; jb < BPW; ++jb)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int s2 = 0; s2 < NKS; ++s2) kr[jb][t][s2] = rd(blk + jb * 2 * BLK + KB::koff(16 * t + r, s2, grp));
    lds_wait();
#pragma unroll
    for (int jb = 0; jb < BPW; ++jb)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int s2 = 0; s2 < NKS; ++s2) lds_pin(kr[jb][t][s2]);
    f32x4 sc[BPW][2];
#pragma unroll
    for (int jb = 0; jb < BPW; ++jb)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        sc[jb][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s2 = 0; s2 < NKS; ++s2) {
          const i32x4 kf = widen(kr[jb][t][s2]);
          sc[jb][t] = mfma16x16x32(kf, qf[s2], sc[jb][t]);
          sc[jb][t] = mfma16x16x32(kf, ql[s2], sc[jb][t]);
        }
      }
    Frag vr[BPW][NDT];  // requested now: the softmax below hides their latency
#pragma unroll
    for (int jb = 0; jb < BPW; ++jb)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) vr[jb][dt] = rd(blk + (jb * 2 + 1) * BLK + KB::voff(16 * dt + r, grp));
    // sc[jb][t][i]: score of key 32 (kb0 + jb) + 16 t + 4 grp + i for query row r; a block
    // at or past blk1 (beyond this wave's last key, or in the next split) counts for nothing
    float mloc = -INFINITY;
#pragma unroll
    for (int jb = 0; jb < BPW; ++jb)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (kb0 + jb >= blk1 || 32 * (kb0 + jb) + 16 * t + 4 * grp + i >= kend) sc[jb][t][i] = -INFINITY;
          mloc = fmaxf(mloc, sc[jb][t][i]);
        }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    // exponents are <= 0 here: the hardware exp2 suffices (results below 2^-126 flush to 0)
    const float scale = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
    float p[BPW][8];
    float lsum = 0.f;
#pragma unroll
    for (int jb = 0; jb < BPW; ++jb)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float sv = sc[jb][t][i];
          const float v = (sv == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(sv - m_new);
          p[jb][4 * t + i] = v;
          lsum += v;
        }
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    l_run = l_run * scale + lsum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) o[dt] *= scale;
    lds_wait();
#pragma unroll
    for (int jb = 0; jb < BPW; ++jb)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) lds_pin(vr[jb][dt]);
#pragma unroll
    for (int jb = 0; jb < BPW; ++jb) {
      if (kb0 + jb >= blk1) continue;  // wave-uniform
      // P as hi/lo bf16 (B operand): element e holds key 16*(e/4) + 4*grp + e%4.
      i32x4 pf, pl;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = p[jb][2 * e], p1 = p[jb][2 * e + 1];
        const uint32_t hw = pack_bf2(p0, p1);
        pf[e] = (int)hw;
        pl[e] = (int)pack_bf2(p0 - __uint_as_float(hw << 16), p1 - __uint_as_float(hw & 0xffff0000u));
      }
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const i32x4 vf = widen(vr[jb][dt]);
        o[dt] = mfma16x16x32(vf, pf, o[dt]);
        o[dt] = mfma16x16x32(vf, pl, o[dt]);
      }
    }
  };

  // bare s_barrier between stages: the copies are complete once this wave's vmcnt dropped
  auto bar = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  for (int st = 0; st < NBUF - 1 && st < n_st; ++st) issue(st);
  for (int c = 0; c < n_st; ++c) {
    const int ahead = min(NBUF - 2, n_st - 1 - c);  // later stages still in flight
    if (ahead >= 6) vm_wait<6 * PER_WAVE>();
    else if (ahead == 5) vm_wait<5 * PER_WAVE>();
    else if (ahead == 4) vm_wait<4 * PER_WAVE>();
    else if (ahead == 3) vm_wait<3 * PER_WAVE>();
    else if (ahead == 2) vm_wait<2 * PER_WAVE>();
    else if (ahead == 1) vm_wait<PER_WAVE>();
    else vm_wait<0>();
    bar();  // every wave's part of stage c is in; every wave is done with stage c - 1
    if (c + NBUF - 1 < n_st) issue(c + NBUF - 1);
    compute(c);
  }
  __syncthreads();  // the ring is free: it holds the other key parts' states next

  // combine the key parts of each row set: parts 1 .. KP - 1 park (m, l, O), part 0 adds
  constexpr int SLOT = NDT * 16 + 16;  // bytes per lane (16-byte aligned pieces)
  auto park_of = [&](int part) { return smem + (((part - 1) * NRS + rs) * 64 + lane) * SLOT; };
  if (kh > 0) {
    char* park = park_of(kh);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) *(f32x4*)(park + dt * 16) = o[dt];
    *(float*)(park + NDT * 16) = m_run;
    *(float*)(park + NDT * 16 + 4) = l_run;
  }
  __syncthreads();
  if (kh > 0 || !row_ok) return;
  float mm = m_run;
#pragma unroll
  for (int part = 1; part < KP; ++part) mm = fmaxf(mm, *(const float*)(park_of(part) + NDT * 16));
  const float s0 = (m_run == -INFINITY) ? 0.f : exp2f(m_run - mm);
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) o[dt] *= s0;
  float ll = l_run * s0;
#pragma unroll
  for (int part = 1; part < KP; ++part) {
    const char* park = park_of(part);
    const float mp = *(const float*)(park + NDT * 16), lp = *(const float*)(park + NDT * 16 + 4);
    const float sp_ = (mp == -INFINITY) ? 0.f : exp2f(mp - mm);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) o[dt] += *(const f32x4*)(park + dt * 16) * sp_;
    ll += lp * sp_;
  }
  if (a.n_splits == 1) {  // the whole key range: normalise and store the output (no merge launch)
    const float inv = 1.0f / ll;
    const int64_t orow = (int64_t)b * k + j;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      i32x2 hi, lo;
      split_bf16x4(o[dt] * inv, hi, lo);
      const int64_t dst = aoff(orow, (int64_t)hq * DH + 16 * dt + 4 * grp, (int64_t)a.n_q * DH, a.out_mtiles);
      *(i32x2*)(a.out + dst) = hi;
      *(i32x2*)(a.out_lo + dst) = lo;
    }
    return;
  }

  // the split's unnormalised (max, sum, O) per row, as attn_split_body leaves them
  const int64_t item = (int64_t)(b * k + j) * a.n_q + hq;
  const int64_t n_items = (int64_t)a.B * k * a.n_q;
  if (grp == 0) {
    float* ml = a.part_ml + ((int64_t)split * n_items + item) * 2;
    ml[0] = mm;
    ml[1] = ll;
  }
  const int64_t po = ((int64_t)split * n_items + item) * DH;
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) *(f32x4*)(a.part_o + po + 16 * dt + 4 * grp) = o[dt];
}

template <int DH>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  const int64_t n_items = (int64_t)a.B * a.k * a.n_q;
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= n_items) return;
  attn_merge_body<DH, false>(a, item);
}

template <int DH, bool KV8>
static void launch_split_rs(const AttnArgs& a, dim3 grid, const Exec& ex) {
  // a row block of at most 32 rows (one block: n_rowblocks == 1) takes two row sets
  if ((a.n_q / a.n_kv) * a.k <= 32 && a.n_rowblocks == 1)
    SBD_KLAUNCH((attn_split_kernel<DH, KV8, 2>), grid, dim3(512), ex, a);
  else
    SBD_KLAUNCH((attn_split_kernel<DH, KV8, 4>), grid, dim3(512), ex, a);
}

hipError_t launch_attention_split(const AttnArgs& a, const Exec& ex) {
  dim3 grid(a.n_splits, a.n_kv * a.n_rowblocks, a.B);
  if (a.d_h == 128 && a.kv_fp8)
    launch_split_rs<128, true>(a, grid, ex);
  else if (a.d_h == 128)
    launch_split_rs<128, false>(a, grid, ex);
  else if (a.d_h == 64 && a.kv_fp8)
    launch_split_rs<64, true>(a, grid, ex);
  else if (a.d_h == 64)
    launch_split_rs<64, false>(a, grid, ex);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention_merge(const AttnArgs& a, const Exec& ex) {
  const int64_t n_items = (int64_t)a.B * a.k * a.n_q;
  dim3 grid((unsigned)((n_items + 3) / 4));
  if (a.d_h == 128)
    SBD_KLAUNCH(attn_merge_kernel<128>, grid, dim3(256), ex, a);
  else if (a.d_h == 64)
    SBD_KLAUNCH(attn_merge_kernel<64>, grid, dim3(256), ex, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sbd
