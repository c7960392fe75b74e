// Device-side helpers for the gfx950 kernels: vector types, bf16 conversion, wave
// reductions.  Included only by *.hip files.
#pragma once

#include <hip/hip_ext.h>

#include "sbd_internal.h"

// Launch on ex.s; the runtime records ex.start / ex.stop (when set) at the kernel's
// start and end.
#define SBD_KLAUNCH(kernel, grid, block, ex, ...) \
  hipExtLaunchKernelGGL(kernel, grid, block, 0, (ex).s, (ex).start, (ex).stop, 0, __VA_ARGS__)

namespace sbd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// float -> bf16, round to nearest even (the gfx950 conversion instruction); NaN stays NaN.
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// OCP e4m3 ("fn") code of v: round to nearest, ties to even, saturating at +-448 (the
// largest finite code; infinities saturate too), NaN -> 0x7f.  Below 2^-6 the codes are the
// subnormals m * 2^-9 (a rounding up to 8 * 2^-9 gives the smallest normal, code 8).
__device__ __forceinline__ uint32_t f32_to_e4m3(float v) {
  const uint32_t sign = (__float_as_uint(v) >> 24) & 0x80u;
  const float a = fabsf(v);
  if (!(a == a)) return 0x7fu;
  if (a >= 448.f) return sign | 0x7eu;
  if (a < 0.015625f) return sign | (uint32_t)rintf(a * 512.f);
  int e;
  const float r = frexpf(a, &e);                      // a = r 2^e, r in [0.5, 1)
  uint32_t m = (uint32_t)rintf((2.f * r - 1.f) * 8.f);  // a = (1 + m/8) 2^(e-1)
  int ex = e - 1;
  if (m == 8) {
    m = 0;
    ++ex;
  }
  return sign | min((uint32_t)((ex + 7) << 3) | m, 0x7eu);
}
// Value of an e4m3 code times s (exact for s a power of two in range).
__device__ __forceinline__ float e4m3_to_f32(uint32_t c, float s) {
  const uint32_t e = (c >> 3) & 15u, m = c & 7u;
  float a = e == 0 ? (float)m * 0.001953125f : ldexpf(1.f + (float)m * 0.125f, (int)e - 7);
  if (e == 15 && m == 7) a = __builtin_nanf("");
  return ((c & 0x80u) ? -a : a) * s;
}
// Eight e4m3 codes (byte i = element i) -> eight bf16 values times s, as an MFMA operand
// (the gfx950 scaled conversion; exact when s is a power of two and the products are in
// the normal range of bf16, which holds for every e4m3 value and the scales used here).
__device__ __forceinline__ i32x4 e4m3x8_to_bf16(i32x2 w, float s) {
  i32x4 o;
  o[0] = __builtin_bit_cast(int, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], s, false));
  o[1] = __builtin_bit_cast(int, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[0], s, true));
  o[2] = __builtin_bit_cast(int, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], s, false));
  o[3] = __builtin_bit_cast(int, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w[1], s, true));
  return o;
}
// One value into the KV cache at element idx: bf16, or the e4m3 code of v * inv (inv = 2^-e,
// the inverse of the cache's scale).
__device__ __forceinline__ void kv_store(void* base, int64_t idx, float v, int fp8, float inv) {
  if (fp8)
    static_cast<uint8_t*>(base)[idx] = (uint8_t)f32_to_e4m3(v * inv);
  else
    static_cast<bf16_t*>(base)[idx] = f2bf(v);
}

// Split v into hi = bf16(v) and lo = bf16(v - hi).
__device__ __forceinline__ void split_bf16(float v, bf16_t& hi, bf16_t& lo) {
  hi = f2bf(v);
  lo = f2bf(v - bf2f(hi));
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
// (bf16(a), bf16(b)) packed low to high in one 32-bit word.
__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{a, b}), bf16x2));
}

// Four floats as hi = bf16(v) and lo = bf16(v - hi), each packed into two 32-bit words.
__device__ __forceinline__ void split_bf16x4(f32x4 v, i32x2& hi, i32x2& lo) {
  const uint32_t h0 = pack_bf2(v[0], v[1]), h1 = pack_bf2(v[2], v[3]);
  hi = i32x2{(int)h0, (int)h1};
  lo = i32x2{(int)pack_bf2(v[0] - __uint_as_float(h0 << 16), v[1] - __uint_as_float(h0 & 0xffff0000u)),
             (int)pack_bf2(v[2] - __uint_as_float(h1 << 16), v[3] - __uint_as_float(h1 & 0xffff0000u))};
}

// 16-byte loads; the streaming variant marks the line non-temporal (read once).
__device__ __forceinline__ i32x4 ld16(const void* p) { return *(const i32x4*)p; }
__device__ __forceinline__ i32x4 ld16_stream(const void* p) {
  return __builtin_nontemporal_load((const i32x4*)p);
}

// Packed weights: 16-row tiles in groups of 8, [N/128][K/32 steps][8 tiles][64 lanes][8]
// bf16 (see gemm.hip).  Element offset of tile t's 1 KB fragment at K step s (S steps);
// consecutive steps of one tile are kPackStep elements apart.
constexpr int64_t kPackStep = 8 * 512;
__device__ __forceinline__ int64_t packed_frag(int64_t t, int64_t s, int64_t S) {
  return (((t >> 3) * S + s) * 8 + (t & 7)) * 512;
}

__device__ __forceinline__ f32x4 mfma16x16x32(i32x4 a, i32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Sum over the 32 lanes of each half-wave (fixed butterfly order: deterministic).
__device__ __forceinline__ float half_wave_sum(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 8);
  v += __shfl_xor(v, 4);
  v += __shfl_xor(v, 2);
  v += __shfl_xor(v, 1);
  return v;
}

// Device-scope (sc1) accesses for data that one workgroup writes and a workgroup on another
// XCD reads later in the same launch: the stores write through to the coherence point and
// the loads bypass possibly stale L2 lines.  Buffer forms take a wave-uniform base (a
// buffer resource) and a per-lane byte offset.
constexpr int kPolicyDevice = 16;  // cache-policy bits of a device-scope access (sc1)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ i32x4 ld16_dev(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, kPolicyDevice);
}
__device__ __forceinline__ float ld32_dev(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, kPolicyDevice));
}
__device__ __forceinline__ void st16_dev(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, i32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, byte_off, 0, kPolicyDevice);
}
__device__ __forceinline__ void st8_dev(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, i32x2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, byte_off, 0, kPolicyDevice);
}
__device__ __forceinline__ void st_bf16_dev(bf16_t* p, bf16_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_f32_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_f32_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_i32_dev(const int* p) {
  return __hip_atomic_load(const_cast<int*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// XCD-local hand-off.  A launch places workgroup i on XCD i % 8 (the round-robin dispatch
// of the 8 XCDs), and the 32 CUs of an XCD share one L2.  Workgroups that exchange data only
// with workgroups of their own XCD therefore need no device-scope traffic: partials are
// written with plain stores (the L1 is write-through: they are in the shared L2 once the
// writer's vmcnt drops), and the arrival counter is a workgroup-scope atomic, performed in
// that L2 (measured: such atomics are not seen across XCDs, and are not meant to be).  The
// reader's loads are workgroup-scope (sc0): they may be served by its own L1, so a line is
// read this way only if the reading CU has not read it earlier in the launch (the L1 is
// invalidated at every launch); a value that changes while being watched is polled with an
// atomic instead.  Every counter used this way sits on a 128-byte line of its own.
constexpr int kPolicyL2 = 1;    // cache-policy bits of a workgroup-scope access (sc0)
__device__ __forceinline__ i32x4 ld16_l2(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, kPolicyL2);
}
__device__ __forceinline__ i32x2 ld8_l2(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, kPolicyL2);
}

// Cross-workgroup reduction handshake for workgroups that all run on one XCD: every
// workgroup stores its partial results, then calls last_arrival_xcd(); it returns true in
// exactly one of the `expected` workgroups arriving at `counter` (the last), which then
// reads the others' partials with ld16_l2 / ld8_l2.  The counter is reset to 0 for the next
// launch.  No workgroup ever waits for another.
__device__ __forceinline__ bool last_arrival_xcd(int* counter, int expected) {
  __shared__ int s_last;
  __builtin_amdgcn_s_waitcnt(0);  // this wave's stores have reached the L2
  __syncthreads();
  if (threadIdx.x == 0) {
    const int prev = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    s_last = (prev == expected - 1) ? 1 : 0;
    if (s_last) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  __syncthreads();
  return s_last != 0;
}

// s_waitcnt vmcnt(N) (other counters left free)
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(((N & 15) | ((N >> 4) << 14)) | (7 << 4) | (15 << 8));
}

// Activation matrices of forwards of more than 16 rows (the GEMM's A operands: normalised
// residual, attention output, SwiGLU output) are stored in MFMA fragment order: the 1 KB
// fragment of 16-row tile t and 32-column step s sits at (s * mtiles + t) KB and holds, for
// lane (r, g) = (l % 16, l / 16), the 8 values of row 16 t + r, columns 32 s + 8 g .. + 8.
// The GEMM then reads a fragment with one contiguous 1 KB load instead of 16 pieces of 64
// bytes from 16 rows.  Element offset of (m, c) in such a matrix of `mtiles` row tiles:
__device__ __forceinline__ int64_t apack(int64_t m, int64_t c, int mtiles) {
  return ((((c >> 5) * mtiles + (m >> 4)) * 64 + ((c >> 3) & 3) * 16 + (m & 15)) << 3) + (c & 7);
}
// (m, c) in a row-major matrix of row stride ld (mtiles == 0) or in fragment order
__device__ __forceinline__ int64_t aoff(int64_t m, int64_t c, int64_t ld, int mtiles) {
  return mtiles ? apack(m, c, mtiles) : m * ld + c;
}

// LDS reads that the compiler does not see as such.  A kernel that fills LDS by direct
// loads (global_load_lds) while reading another part of it would otherwise get a wait for
// every direct load in flight before each LDS read (the compiler cannot tell the regions
// apart), which drains its prefetch.  The caller orders these reads itself: a barrier after
// the data has landed before them, lds_wait() after them, and lds_pin() on each result
// before its first use.
template <int OFF = 0>
__device__ __forceinline__ i32x4 ds_read16(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  i32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void lds_pin(i32x4& v) { asm volatile("" : "+v"(v)); }
template <int OFF = 0>
__device__ __forceinline__ i32x2 ds_read8(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  i32x2 v;
  asm volatile("ds_read_b64 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}
__device__ __forceinline__ void lds_pin(i32x2& v) { asm volatile("" : "+v"(v)); }
// LDS byte address of a __shared__ object
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }

__device__ __forceinline__ float wave_sum(float v) {
  v += __shfl_xor(v, 32);
  return half_wave_sum(v);
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, __shfl_xor(v, 32));
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 8));
  v = fmaxf(v, __shfl_xor(v, 4));
  v = fmaxf(v, __shfl_xor(v, 2));
  v = fmaxf(v, __shfl_xor(v, 1));
  return v;
}

}  // namespace sbd
