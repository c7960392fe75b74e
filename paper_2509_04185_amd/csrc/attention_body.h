// Device bodies of the block-hybrid attention (attention.hip has the description); shared
// by the standalone kernels and the fused decode forward.
#pragma once

#include "sbd_device.h"

namespace sbd {

constexpr int kAttnSmem = 65536 + 16;  // LDS of one attention workgroup (two K/V chunks)

__device__ __forceinline__ int64_t attn_head_base(int layer, int slot, int g, int n_slots,
                                                  int n_kv, int64_t cap, int d_h) {
  return (((int64_t)layer * n_slots + slot) * n_kv + g) * cap * d_h;
}

// A 32-key block of K (or of V) staged in LDS: 16-byte pieces, XOR-swizzled so that the
// fragment reads below are free of bank conflicts, and copied straight from the cache into
// LDS (global_load_lds: wave-load lane l fills LDS piece l of its 1 KB and reads the matching
// global piece).  The cache holds bf16 or (KV8) e4m3 codes; an fp8 block takes half the LDS
// and is widened to bf16 (times the cache's scale, exact) at the fragment reads.
//   K: row `key` (DH elements) holds its piece c at c ^ ksw(key);
//   V^T: row d (the block's 32 keys in slot order) holds its piece c at c ^ vsw(d).
template <int DH, bool KV8>
struct KvBlk {
  static constexpr int ES = KV8 ? 1 : 2;          // bytes per cached element
  static constexpr int BYTES = 32 * DH * ES;      // of K, or of V, per block
  static constexpr int KPR = DH * ES / 16;        // pieces per K row
  static constexpr int VPR = 32 * ES / 16;        // pieces per V^T row
  __device__ static int ksw(int key) { return KV8 ? (key / (256 / DH)) % KPR : key % KPR; }
  __device__ static int vsw(int d) { return KV8 ? (d >> 3) & 1 : (d >> 2) & 3; }
  // Global source of LDS piece q (< BYTES / 16) of block kb; part 0 K, 1 V.
  __device__ static const char* src(const char* kbase, const char* vbase, int kb, int part, int q) {
    if (part == 0) {
      const int key = q / KPR;
      return kbase + ((int64_t)(kb * 32 + key) * DH) * ES + ((q % KPR) ^ ksw(key)) * 16;
    }
    const int d = q / VPR;
    return vbase + ((int64_t)kb * DH * 32 + d * 32) * ES + ((q % VPR) ^ vsw(d)) * 16;
  }
  // LDS byte offset of this lane's K fragment (A operand: key `key`, dims 32 s + 8 grp .. +8)
  __device__ static int koff(int key, int s, int grp) {
    if (KV8) return key * DH + (((2 * s + (grp >> 1)) ^ ksw(key)) * 16) + (grp & 1) * 8;
    return key * DH * 2 + (((4 * s + grp) ^ ksw(key)) * 16);
  }
  // LDS byte offset of this lane's V^T fragment (A operand: dim d, slots 8 grp .. +8)
  __device__ static int voff(int d, int grp) {
    if (KV8) return d * 32 + (((grp >> 1) ^ vsw(d)) * 16) + (grp & 1) * 8;
    return d * 64 + ((grp ^ vsw(d)) * 16);
  }
  // The fragment at LDS byte address p as bf16 (sc: the cache's scale)
  __device__ static i32x4 frag(const char* p, float sc) {
    if constexpr (KV8)
      return e4m3x8_to_bf16(*(const i32x2*)p, sc);
    else
      return *(const i32x4*)p;
  }
};

// What one wave holds after its key range: unnormalised O^T tiles of its 16 query rows
// (lane: row r = lane % 16, dims 16 dt + 4 (lane / 16) + i), the running max and sum.
template <int DH>
struct AttnPart {
  f32x4 o[DH / 16];
  float m, l;
  bool row_ok;  // this lane's row exists
  int rho;      // its row within the KV head's rows (query head within the group, block row)
};

// One workgroup (4 waves) of the attention over key blocks [blk0, blk_lim) of KV head g,
// row block rb, sequence b.  smem: kAttnSmem bytes of LDS.  POL: cache policy of the loads
// of the queries and of the keys and values (they may have been written earlier in the same
// launch: kPolicyL2 when by the same XCD, kPolicyDevice when by any).
template <int DH, int POL, bool KV8 = false>
__device__ __forceinline__ void attn_core(const AttnArgs& a, int g, int rb, int b, int blk0, int blk_lim,
                                          char* smem, AttnPart<DH>& out) {
  constexpr int NDT = DH / 16;  // 16-wide dimension tiles
  constexpr int NKS = DH / 32;  // 32-wide reduction steps for the scores
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 15, grp = lane >> 4;
  const SeqParam sp = a.seqs[b];
  const int L = sp.cache_len, nc = sp.n_causal, k = a.k;
  const int G = a.n_q / a.n_kv;
  const int R = G * k;

  const int rho = rb * 64 + w * 16 + r;
  const bool row_ok = rho < R;
  const int hh = row_ok ? rho / k : 0;
  const int j = row_ok ? rho % k : 0;
  const int hq = g * G + hh;
  const int kend = row_ok ? ((j >= nc) ? L + k : L + j + 1) : 0;

  // Key blocks this wave visits: its split's range, clipped to its rows' last key.
  int kend_w = kend;
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) kend_w = max(kend_w, __shfl_xor(kend_w, o));
  const int nblk_w = (kend_w + 31) / 32;
  const int blk1 = min(blk_lim, nblk_w);

  // Query fragments (B operand, hi and lo): row r, dims 32*s + 8*grp .. +8.
  i32x4 qf[NKS], ql[NKS];
  const int64_t qoff = ((int64_t)(b * k + j) * a.n_q + hq) * DH;
  const __amdgpu_buffer_rsrc_t rq = buf_rsrc(a.q), rql = buf_rsrc(a.q_lo);
#pragma unroll
  for (int s = 0; s < NKS; ++s) {
    const uint32_t e = (uint32_t)((qoff + 32 * s + 8 * grp) * 2);
    qf[s] = row_ok ? __builtin_amdgcn_raw_buffer_load_b128(rq, e, 0, POL) : i32x4{0, 0, 0, 0};
    ql[s] = row_ok ? __builtin_amdgcn_raw_buffer_load_b128(rql, e, 0, POL) : i32x4{0, 0, 0, 0};
  }

  const int64_t hb = attn_head_base(a.layer, sp.slot, g, a.n_slots, a.n_kv, a.cap, DH);
  using KB = KvBlk<DH, KV8>;
  const char* kbase = static_cast<const char*>(a.kcache) + hb * KB::ES;
  const char* vbase = static_cast<const char*>(a.vcache) + hb * KB::ES;
  const float kv_sc = a.kv_scale;

  f32x4 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // The workgroup's key blocks are copied from the cache straight into LDS (global_load_lds,
  // no registers) in chunks of CH blocks, alternating between two buffers, so a chunk's
  // loads are all in flight at once and the next chunk streams in while the current one is
  // used (block layout in LDS: KvBlk).
  constexpr int BLK = KB::BYTES;            // bytes of K (or of V) per 32-key block
  constexpr int CH = 65536 / (4 * 32 * DH * 2);  // blocks per chunk (bf16: two buffers of K and V, 64 KB)
  constexpr int LPB = BLK / 1024;           // 1 KB wave-loads per part (K or V) per block
  constexpr int PER_WAVE = CH * 2 * LPB / 4;
  typedef char Chunk[CH][2][BLK];
  Chunk& lds_a = *reinterpret_cast<Chunk*>(smem);
  Chunk& lds_b = *reinterpret_cast<Chunk*>(smem + sizeof(Chunk));
  int* s_kend = reinterpret_cast<int*>(smem + 2 * sizeof(Chunk));
  int kend_wg = kend;
#pragma unroll
  for (int o2 = 1; o2 < 64; o2 <<= 1) kend_wg = max(kend_wg, __shfl_xor(kend_wg, o2));
  if (lane == 0) s_kend[w] = kend_wg;
  __syncthreads();
  kend_wg = max(max(s_kend[0], s_kend[1]), max(s_kend[2], s_kend[3]));
  const int blk1_wg = min(blk_lim, (kend_wg + 31) / 32);
  const int n_chunks = blk1_wg > blk0 ? (blk1_wg - blk0 + CH - 1) / CH : 0;

  // Wave-load u of wave w in chunk c: index i = w + 4u -> block i / (2 LPB), part
  // (i / LPB) % 2, 1 KB slice i % LPB.
  auto issue_chunk = [&](int c, char (&buf)[CH][2][BLK]) {
#pragma unroll
    for (int u = 0; u < PER_WAVE; ++u) {
      const int idx = w + 4 * u;
      const int bi = idx / (2 * LPB), part = (idx / LPB) % 2, sub = idx % LPB;
      int kb = blk0 + c * CH + bi;
      if (kb >= blk1_wg) kb = blk1_wg - 1;  // past the end: a valid block, never used
      __builtin_amdgcn_global_load_lds((const void*)KB::src(kbase, vbase, kb, part, sub * 64 + lane),
                                       (__attribute__((address_space(3))) void*)&buf[bi][part][sub * 1024],
                                       16, 0, POL);
    }
  };
  // s_waitcnt immediates: vmcnt(n) with the other counters left free
  constexpr int kWaitOne = ((PER_WAVE & 15) | ((PER_WAVE >> 4) << 14)) | (7 << 4) | (15 << 8);
  constexpr int kWaitAll = (7 << 4) | (15 << 8);

  // One chunk: the scores of all its blocks (independent MFMA chains), one online-softmax
  // update over the chunk's keys, then O^T += V^T P^T block by block.
  auto compute_chunk = [&](int c, const char (&buf)[CH][2][BLK]) {
    const int kb0 = blk0 + c * CH;
    const int nb = min(CH, blk1 - kb0);  // blocks of this chunk before this wave's last key
    if (nb <= 0) return;                 // wave-uniform
    f32x4 st[CH][2];
#pragma unroll
    for (int bi = 0; bi < CH; ++bi) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        st[bi][t] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (bi >= nb) continue;
        const int row = 16 * t + r;
#pragma unroll
        for (int s2 = 0; s2 < NKS; ++s2) {
          const i32x4 kf = KB::frag(buf[bi][0] + KB::koff(row, s2, grp), kv_sc);
          st[bi][t] = mfma16x16x32(kf, qf[s2], st[bi][t]);
          st[bi][t] = mfma16x16x32(kf, ql[s2], st[bi][t]);
        }
      }
    }
    // st[bi][t][i]: score of key 32 (kb0 + bi) + 16t + 4grp + i for query row r.
    float mloc = -INFINITY;
#pragma unroll
    for (int bi = 0; bi < CH; ++bi)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kv = 32 * (kb0 + bi) + 16 * t + 4 * grp + i;
          if (bi >= nb || kv >= kend) st[bi][t][i] = -INFINITY;
          mloc = fmaxf(mloc, st[bi][t][i]);
        }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    // exponents are <= 0 here: the hardware exp2 suffices (results below 2^-126 flush to 0)
    const float scale = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
    float p[CH][8];
    float lsum = 0.f;
#pragma unroll
    for (int bi = 0; bi < CH; ++bi)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float sv = st[bi][t][i];
          const float v = (sv == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(sv - m_new);
          p[bi][4 * t + i] = v;
          lsum += v;
        }
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    l_run = l_run * scale + lsum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) o[dt] *= scale;
#pragma unroll
    for (int bi = 0; bi < CH; ++bi) {
      if (bi >= nb) continue;
      // P as hi/lo bf16 (B operand): element e holds key 16*(e/4) + 4*grp + e%4.
      i32x4 pf, pl;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = p[bi][2 * e], p1 = p[bi][2 * e + 1];
        const uint32_t hw = pack_bf2(p0, p1);
        pf[e] = (int)hw;
        pl[e] = (int)pack_bf2(p0 - __uint_as_float(hw << 16), p1 - __uint_as_float(hw & 0xffff0000u));
      }
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const i32x4 vf = KB::frag(buf[bi][1] + KB::voff(16 * dt + r, grp), kv_sc);
        o[dt] = mfma16x16x32(vf, pf, o[dt]);
        o[dt] = mfma16x16x32(vf, pl, o[dt]);
      }
    }
  };

  // Chunks alternate between lds_a (even) and lds_b (odd).  The barriers are bare s_barrier
  // instructions: the copies into LDS are complete once this wave's vmcnt has dropped (the
  // explicit waits below), and a fenced barrier would also wait for the next chunk's copies
  // that are meant to stay in flight.  The empty asm statements keep the compiler from
  // moving LDS accesses across a barrier.
  auto bar = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  auto wait_chunk = [&](bool next_in_flight) {
    if (next_in_flight)
      __builtin_amdgcn_s_waitcnt(kWaitOne);
    else
      __builtin_amdgcn_s_waitcnt(kWaitAll);
  };
  if (n_chunks > 0) {
    issue_chunk(0, lds_a);
    if (n_chunks > 1) issue_chunk(1, lds_b);
    wait_chunk(n_chunks > 1);
    bar();
    compute_chunk(0, lds_a);
    bar();  // lds_a is free again
    if (n_chunks > 2) issue_chunk(2, lds_a);
  }
  for (int c = 1; c < n_chunks; c += 2) {
    wait_chunk(c + 1 < n_chunks);
    bar();
    compute_chunk(c, lds_b);
    bar();  // lds_b is free again
    if (c + 2 < n_chunks) issue_chunk(c + 2, lds_b);
    if (c + 1 < n_chunks) {
      wait_chunk(c + 2 < n_chunks);
      bar();
      compute_chunk(c + 1, lds_a);
      bar();  // lds_a is free again
      if (c + 3 < n_chunks) issue_chunk(c + 3, lds_a);
    }
  }

#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) out.o[dt] = o[dt];
  out.m = m_run;
  out.l = l_run;
  out.row_ok = row_ok;
  out.rho = rho;
}

// One workgroup of the split-KV attention: split `split` of the key blocks, KV head x row
// block gy, sequence b.  Leaves the split's unnormalised (max, sum, O) per row for the merge.
// DEV: the queries, keys and values were written earlier in the same launch (device-scope
// loads), and the partial results are read by another workgroup of it (device-scope stores).
template <int DH, bool DEV, bool KV8 = false>
__device__ __forceinline__ void attn_split_body(const AttnArgs& a, int split, int gy, int b, char* smem) {
  constexpr int NDT = DH / 16;
  const int g = gy / a.n_rowblocks, rb = gy % a.n_rowblocks;
  const int blk0 = split * a.blocks_per_split;
  AttnPart<DH> pt;
  attn_core<DH, DEV ? kPolicyDevice : 0, KV8>(a, g, rb, b, blk0, blk0 + a.blocks_per_split, smem, pt);
  if (!pt.row_ok) return;
  const int lane = threadIdx.x & 63, grp = lane >> 4;
  const int k = a.k, G = a.n_q / a.n_kv;
  const int hh = pt.rho / k, j = pt.rho % k, hq = g * G + hh;
  const int64_t item = (int64_t)(b * k + j) * a.n_q + hq;
  const int64_t n_items = (int64_t)a.B * k * a.n_q;
  if (grp == 0) {
    float* ml = a.part_ml + ((int64_t)split * n_items + item) * 2;
    if constexpr (DEV) {
      st_f32_dev(ml, pt.m);
      st_f32_dev(ml + 1, pt.l);
    } else {
      ml[0] = pt.m;
      ml[1] = pt.l;
    }
  }
  const int64_t po = ((int64_t)split * n_items + item) * DH;
  const __amdgpu_buffer_rsrc_t ro = buf_rsrc(a.part_o);
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
    if constexpr (DEV)
      st16_dev(ro, (uint32_t)((po + 16 * dt + 4 * grp) * 4), __builtin_bit_cast(i32x4, pt.o[dt]));
    else
      *(f32x4*)(a.part_o + po + 16 * dt + 4 * grp) = pt.o[dt];
  }
}

// One wave per (row, query head) item: combine the splits, normalise, store hi/lo bf16.
// Lane s reads split s's (max, sum); the split weights 2^(m_s - M) are broadcast from
// their lanes while every lane accumulates its own dimensions over the splits.  DEV as for
// attn_split_body.
template <int DH, bool DEV>
__device__ __forceinline__ void attn_merge_body(const AttnArgs& a, int64_t item) {
  const int64_t n_items = (int64_t)a.B * a.k * a.n_q;
  const int lane = threadIdx.x & 63;
  const __amdgpu_buffer_rsrc_t rml = buf_rsrc(a.part_ml), ro = buf_rsrc(a.part_o);
  const int ns = a.n_splits;  // <= 64
  constexpr int PER = DH / 64;
  const int64_t po = item * DH + lane;
  const int64_t split_stride = n_items * DH;
  auto ld_part = [&](int64_t e) -> float {
    if constexpr (DEV) return ld32_dev(ro, (uint32_t)(e * 4));
    else return a.part_o[e];
  };
  // Every load is requested before any is used: the (max, sum) pairs and the partial
  // outputs of the first kBatch splits, then the partial outputs kBatch splits at a time.
  constexpr int kBatch = 32;
  float v[kBatch][PER];
#pragma unroll
  for (int u = 0; u < kBatch; ++u)
#pragma unroll
    for (int e = 0; e < PER; ++e) v[u][e] = (u < ns) ? ld_part(po + (int64_t)u * split_stride + 64 * e) : 0.f;
  float ms = -INFINITY, ls = 0.f;
  if (lane < ns) {
    const int64_t e = ((int64_t)lane * n_items + item) * 2;
    if constexpr (DEV) {
      ms = ld32_dev(rml, (uint32_t)(e * 4));
      ls = ld32_dev(rml, (uint32_t)(e * 4 + 4));
    } else {
      const float2 mv = *(const float2*)(a.part_ml + e);
      ms = mv.x;
      ls = mv.y;
    }
  }
  const float mx = wave_max(ms);
  const float wgt = (ms == -INFINITY) ? 0.f : exp2f(ms - mx);
  const float lsum = wave_sum(wgt * ls);
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  for (int s0 = 0; s0 < ns; s0 += kBatch) {  // wave-uniform
    if (s0 > 0) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
#pragma unroll
        for (int e = 0; e < PER; ++e)
          v[u][e] = (s0 + u < ns) ? ld_part(po + (int64_t)(s0 + u) * split_stride + 64 * e) : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (s0 + u >= ns) break;  // wave-uniform
      const float wu = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wgt), s0 + u));
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] += wu * v[u][e];
    }
  }
  const float inv = 1.0f / lsum;
  const int64_t orow = item / a.n_q;
  const int hq = (int)(item % a.n_q);
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    bf16_t hi, lo;
    split_bf16(acc[e] * inv, hi, lo);
    const int64_t dst = aoff(orow, (int64_t)hq * DH + lane + 64 * e, (int64_t)a.n_q * DH, a.out_mtiles);
    if constexpr (DEV) {
      st_bf16_dev(a.out + dst, hi);
      st_bf16_dev(a.out_lo + dst, lo);
    } else {
      a.out[dst] = hi;
      a.out_lo[dst] = lo;
    }
  }
}

}  // namespace sbd
