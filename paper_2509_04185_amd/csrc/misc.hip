// Small per-row kernels of the block forward: embedding gather, RoPE + q/k-norm +
// KV staging, the RoPE angle table, and KV-cache import/export.
//
// KV-cache layout, per (layer, slot, KV head), capacity `cap` positions:
//   K: [cap][d_h] bf16, post-RoPE keys, one row per position.
//   V: [cap/32][d_h][32] bf16, each 32-position block stored transposed (dimension-major)
//      with its positions permuted by vslot() so that one 16-byte load gives the eight
//      values the attention kernel's P.V MFMA needs for one dimension.

#include "sbd_device.h"

namespace sbd {

// Storage slot inside a 32-position V block of position p (0..31): positions
// {16t + 4q + i : t in {0,1}, i < 4} (the keys lane group q holds after the score MFMA)
// become the contiguous slots 8q .. 8q + 7.
__device__ __forceinline__ int vslot(int p) { return ((p & 15) >> 2) * 8 + (p >> 4) * 4 + (p & 3); }

__device__ __forceinline__ int64_t kv_head_base(int layer, int slot, int g, int n_slots, int n_kv,
                                                int64_t cap, int d_h) {
  return (((int64_t)layer * n_slots + slot) * n_kv + g) * cap * d_h;
}

// Row m = blockIdx.x, columns 1024 blockIdx.y + 4 t .. + 3 for thread t (every load of a
// thread is issued at once): x[m] = E[tok[m]] (fp32), xn[m] = x * g as hi/lo bf16,
// sumsq[m][c/16] = sum over each 16 columns of x^2 (the consumer forms 1/rms).
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  const int m = blockIdx.x;
  const int c = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (c >= a.d) return;  // d % 16 == 0: a 16-column group lies inside or outside as a whole
  const int tok = a.rows[m].tok;
  const uint2 ev = *reinterpret_cast<const uint2*>(a.embed + (int64_t)tok * a.d + c);
  const uint2 gv = *reinterpret_cast<const uint2*>(a.g + c);
  const float v[4] = {__uint_as_float(ev.x << 16), __uint_as_float(ev.x & 0xffff0000u),
                      __uint_as_float(ev.y << 16), __uint_as_float(ev.y & 0xffff0000u)};
  const float g[4] = {__uint_as_float(gv.x << 16), __uint_as_float(gv.x & 0xffff0000u),
                      __uint_as_float(gv.y << 16), __uint_as_float(gv.y & 0xffff0000u)};
  const int64_t o = (int64_t)m * a.d + c;
  *reinterpret_cast<float4*>(a.x + o) = float4{v[0], v[1], v[2], v[3]};
  if (a.x64 != nullptr) {
    long long q[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) q[e] = __double2ll_rn((double)v[e] * 4294967296.0);
    *reinterpret_cast<longlong2*>(a.x64 + o) = longlong2{q[0], q[1]};
    *reinterpret_cast<longlong2*>(a.x64 + o + 2) = longlong2{q[2], q[3]};
    *reinterpret_cast<longlong2*>(a.x64_zero + o) = longlong2{0, 0};
    *reinterpret_cast<longlong2*>(a.x64_zero + o + 2) = longlong2{0, 0};
  }
  const f32x4 xg = f32x4{v[0] * g[0], v[1] * g[1], v[2] * g[2], v[3] * g[3]};
  i32x2 hi, lo;
  split_bf16x4(xg, hi, lo);
  const int64_t on = aoff(m, c, a.d, a.mtiles);  // 4 consecutive columns stay contiguous
  *reinterpret_cast<i32x2*>(a.xn + on) = hi;
  *reinterpret_cast<i32x2*>(a.xn_lo + on) = lo;
  float s = v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  s += __shfl_xor(s, 1);
  s += __shfl_xor(s, 2);
  if ((threadIdx.x & 3) == 0) a.sumsq[(int64_t)m * (a.d / 16) + c / 16] = s;
}

hipError_t launch_embed(const EmbedArgs& a, const Exec& ex) {
  if (a.d % 16 != 0) return hipErrorInvalidValue;
  SBD_KLAUNCH(embed_kernel, dim3(a.M, (a.d + 1023) / 1024), dim3(256), ex, a);
  return hipGetLastError();
}

// One wave per (row, head).  Lane i < d_h/2 owns the RoPE pair (i, i + d_h/2).
// Query heads: optional per-head RMSNorm, rotation, scaling, hi/lo bf16 store.
// Key heads: optional per-head RMSNorm, rotation, store into the cache at position
// cache_len + j.  Value heads: store into the transposed V block.
__global__ __launch_bounds__(64) void rope_stage_kernel(RopeStageArgs a) {
  const int h = blockIdx.x;
  const int m = blockIdx.y;
  const int lane = threadIdx.x;
  const int half = a.d_h / 2;
  const bool act = lane < half;
  const int b = m / a.k, j = m % a.k;
  const SeqParam sp = a.seqs[b];
  const int p_cache = sp.cache_len + j;
  const int pos = a.rows[m].pos;
  const float* src = a.qkv + (int64_t)m * (a.n_q + 2 * a.n_kv) * a.d_h + (int64_t)h * a.d_h;
  float u0 = act ? src[lane] : 0.f;
  float u1 = act ? src[lane + half] : 0.f;

  if (h < a.n_q + a.n_kv) {
    const bool is_q = h < a.n_q;
    if (a.qk_norm) {
      const float ss = wave_sum(u0 * u0 + u1 * u1);
      const float rinv = 1.0f / sqrtf(ss / (float)a.d_h + a.eps);
      const bf16_t* gn = is_q ? a.q_norm : a.k_norm;
      if (act) {
        u0 = u0 * rinv * bf2f(gn[lane]);
        u1 = u1 * rinv * bf2f(gn[lane + half]);
      }
    }
    if (!act) return;
    const float c = a.rope[((int64_t)pos * half + lane) * 2 + 0];
    const float sn = a.rope[((int64_t)pos * half + lane) * 2 + 1];
    const float r0 = u0 * c - u1 * sn;
    const float r1 = u1 * c + u0 * sn;
    if (is_q) {
      const int64_t o = ((int64_t)m * a.n_q + h) * a.d_h;
      bf16_t hi, lo;
      split_bf16(r0 * a.q_scale, hi, lo);
      a.q[o + lane] = hi;
      a.q_lo[o + lane] = lo;
      split_bf16(r1 * a.q_scale, hi, lo);
      a.q[o + lane + half] = hi;
      a.q_lo[o + lane + half] = lo;
    } else {
      const int g = h - a.n_q;
      const int64_t dst = kv_head_base(a.layer, sp.slot, g, a.n_slots, a.n_kv, a.cap, a.d_h) +
                          (int64_t)p_cache * a.d_h;
      kv_store(a.kcache, dst + lane, r0, a.kv_fp8, a.kv_inv);
      kv_store(a.kcache, dst + lane + half, r1, a.kv_fp8, a.kv_inv);
    }
  } else {
    if (!act) return;
    const int g = h - a.n_q - a.n_kv;
    const int64_t blk = kv_head_base(a.layer, sp.slot, g, a.n_slots, a.n_kv, a.cap, a.d_h) +
                        (int64_t)(p_cache / 32) * a.d_h * 32;
    const int sl = vslot(p_cache & 31);
    kv_store(a.vcache, blk + (int64_t)lane * 32 + sl, u0, a.kv_fp8, a.kv_inv);
    kv_store(a.vcache, blk + (int64_t)(lane + half) * 32 + sl, u1, a.kv_fp8, a.kv_inv);
  }
}

hipError_t launch_rope_stage(const RopeStageArgs& a, const Exec& ex) {
  SBD_KLAUNCH(rope_stage_kernel, dim3(a.n_q + 2 * a.n_kv, a.M), dim3(64), ex, a);
  return hipGetLastError();
}

// rope[p][i] = (cos, sin)(p * theta^(-2i/d_h)), angles in float64.
__global__ void rope_table_kernel(float* rope, int64_t cap, int d_h, double theta) {
  const int half = d_h / 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= cap * half) return;
  const int64_t p = idx / half;
  const int i = (int)(idx % half);
  const double inv_freq = pow(theta, -2.0 * (double)i / (double)d_h);
  const double phi = (double)p * inv_freq;
  rope[idx * 2 + 0] = (float)cos(phi);
  rope[idx * 2 + 1] = (float)sin(phi);
}

hipError_t launch_rope_table(float* rope, int64_t cap, int d_h, double theta, hipStream_t s) {
  const int64_t n = cap * (d_h / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, rope,
                     cap, d_h, theta);
  return hipGetLastError();
}

// grid (n, n_kv, n_layers); lanes walk the head dimension.
template <bool IMPORT>
__global__ __launch_bounds__(64) void kv_copy_kernel(KvCopyArgs a) {
  const int t = blockIdx.x, g = blockIdx.y, layer = blockIdx.z;
  const int p = a.pos0 + t;
  const int64_t hb = kv_head_base(layer, a.slot, g, a.n_slots, a.n_kv, a.cap, a.d_h);
  const int64_t io = (((int64_t)layer * a.n + t) * a.n_kv + g) * a.d_h;
  const int64_t kc = hb + (int64_t)p * a.d_h;
  const int64_t vb = hb + (int64_t)(p / 32) * a.d_h * 32;
  const int sl = vslot(p & 31);
  for (int i = threadIdx.x; i < a.d_h; i += 64) {
    const int64_t ki = kc + i, vi = vb + (int64_t)i * 32 + sl;
    if (IMPORT) {  // an fp8 cache gets the e4m3 code of the value (kv_store)
      kv_store(a.kcache, ki, bf2f(a.k_in[io + i]), a.kv_fp8, a.kv_inv);
      kv_store(a.vcache, vi, bf2f(a.v_in[io + i]), a.kv_fp8, a.kv_inv);
    } else if (a.kv_fp8) {  // widened: at most 4 significant bits, exact in bf16
      a.k_out[io + i] = f2bf(e4m3_to_f32(static_cast<const uint8_t*>(a.kcache)[ki], a.kv_scale));
      a.v_out[io + i] = f2bf(e4m3_to_f32(static_cast<const uint8_t*>(a.vcache)[vi], a.kv_scale));
    } else {
      a.k_out[io + i] = static_cast<const bf16_t*>(a.kcache)[ki];
      a.v_out[io + i] = static_cast<const bf16_t*>(a.vcache)[vi];
    }
  }
}

hipError_t launch_kv_import(const KvCopyArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(kv_copy_kernel<true>, dim3(a.n, a.n_kv, a.n_layers), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_kv_export(const KvCopyArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(kv_copy_kernel<false>, dim3(a.n, a.n_kv, a.n_layers), dim3(64), 0, s, a);
  return hipGetLastError();
}

// The XCD (accelerator complex die) each workgroup of a launch runs on, from the XCC_ID
// hardware register (bits 3:0): the per-XCD layer kernels and the split-K hand-offs rely on
// workgroup i running on XCD i % 8 and check it with this probe when a context is created.
__global__ __launch_bounds__(64) void xcd_probe_kernel(int* out) {
  const int id = (int)(__builtin_amdgcn_s_getreg((20) | (0 << 6) | ((4 - 1) << 11)) & 15);
  if (threadIdx.x == 0) out[blockIdx.x] = id;
}

hipError_t launch_xcd_probe(int* out, int n, hipStream_t s) {
  if (out == nullptr || n < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(xcd_probe_kernel, dim3(n), dim3(64), 0, s, out);
  return hipGetLastError();
}

}  // namespace sbd
