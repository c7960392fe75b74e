// EB-Sampler step (Sec. 2.2, eq. (eb_sampler)) on the block's fp32 logits.
//
// eb_partial: one workgroup per (vocabulary chunk of 4096, masked row).  It finds the
// chunk maximum m_c (and the smallest id reaching it, the mask column excluded), then
// with t = l - m_c in float64 accumulates Z_c = sum e^t and S_c = sum e^t t.  Sums are
// per-thread in a fixed order followed by a fixed tree, so results are reproducible.
//
// eb_select: one workgroup of 16 waves per sequence, one wave per row (rows w, w + 16, ...).
// Each masked row merges its chunks (one lane per chunk, fixed butterfly sums) with
// M = max m_c, delta_c = m_c - M:
//   Z = sum_c e^delta_c Z_c,  S = sum_c e^delta_c (S_c + delta_c Z_c),  H = log Z - S / Z
// (the entropy of softmax over the row; argmax = first chunk reaching M).  Then the
// masked rows are ranked by (H, row), lane 0 forms the running float64 sums c_r in
// that order, s = max{r >= 1 : c_{r-1} <= gamma}, and the first s rows are written out
// in ascending row order.  A row without a finite logit (outside the mask column) has
// entropy and confidence NaN and token -1; a NaN or infinite logit makes them NaN too.
// Such rows rank after every other row and are never accepted (with no other masked row,
// s = 0).

#include <mutex>

#include "eb_stats.h"

namespace sbd {

constexpr int kEbThreads = 256;
constexpr int kEbPer = kEbChunk / kEbThreads;  // 16 entries per thread

__global__ __launch_bounds__(kEbThreads) void eb_partial_kernel(EbArgs a) {
  __shared__ float smax[kEbThreads / 64];
  __shared__ int sarg[kEbThreads / 64];
  __shared__ double sz[kEbThreads / 64], ss[kEbThreads / 64];
  const int row = blockIdx.y;
  const int c = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // masks passed by value: an unmasked row's workgroups leave at once (a kernel-argument
  // read, so nothing waits on memory); an uploaded mask is read after the loads are issued
  if (a.is_mask == nullptr && !eb_row_masked(a, row)) return;
  const float* lr = a.logits + (int64_t)row * a.vocab;
  const int v0 = c * kEbChunk;

  // every load is unconditional (the index clamped into the row), so that all of them are
  // in flight at once; entries past the row end and the mask column are dropped afterwards
  float val[kEbPer];
#pragma unroll
  for (int e = 0; e < kEbPer; ++e) val[e] = lr[min(v0 + tid + e * kEbThreads, a.vocab - 1)];
  float mx = -INFINITY;
  int arg = INT32_MAX;
#pragma unroll
  for (int e = 0; e < kEbPer; ++e) {
    const int v = v0 + tid + e * kEbThreads;
    const bool ok = v < a.vocab && v != a.mask_id;
    if (!ok) val[e] = -INFINITY;
    if (ok && (val[e] > mx || (val[e] == mx && v < arg))) {
      mx = val[e];
      arg = v;
    }
  }
  // read after the chunk's loads are issued: the workgroup of an unmasked row stores nothing
  const bool masked = a.is_mask == nullptr || eb_row_masked(a, row);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float om = __shfl_xor(mx, o);
    const int oa = __shfl_xor(arg, o);
    if (om > mx || (om == mx && oa < arg)) {
      mx = om;
      arg = oa;
    }
  }
  if (lane == 0) {
    smax[w] = mx;
    sarg[w] = arg;
  }
  __syncthreads();
  mx = smax[0];
  arg = sarg[0];
  for (int i = 1; i < kEbThreads / 64; ++i)
    if (smax[i] > mx || (smax[i] == mx && sarg[i] < arg)) {
      mx = smax[i];
      arg = sarg[i];
    }

  double z = 0.0, s = 0.0;
  if (mx != -INFINITY) {
    const double md = (double)mx;
#pragma unroll
    for (int e = 0; e < kEbPer; ++e) {
      if (val[e] != -INFINITY) {
        const double t = (double)val[e] - md;
        const double ex = exp(t);
        z += ex;
        s += ex * t;
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    z += shfl_xor_d(z, o);
    s += shfl_xor_d(s, o);
  }
  if (lane == 0) {
    sz[w] = z;
    ss[w] = s;
  }
  __syncthreads();
  if (tid == 0 && masked) {
    double zt = 0.0, st = 0.0;
    for (int i = 0; i < kEbThreads / 64; ++i) {
      zt += sz[i];
      st += ss[i];
    }
    double* p = a.part + ((int64_t)row * a.n_chunks + c) * 3;
    p[0] = (double)mx;
    p[1] = zt;
    p[2] = st;
    a.part_arg[(int64_t)row * a.n_chunks + c] = (mx == -INFINITY) ? -1 : arg;
  }
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += shfl_xor_d(v, o);
  return v;
}

__device__ __forceinline__ double wave_max_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmax(v, shfl_xor_d(v, o));
  return v;
}

constexpr int kEbSelWaves = 16;

// One workgroup (16 waves) per sequence.  Wave w merges the chunk statistics of rows
// w, w + 16, ... with one lane per chunk; wave 0 then ranks and selects.
// MODE: kFromChunks (the partial kernel's chunk statistics, merged here), kFromEntropies
// (given entropies, no tokens), kFromRows (per-row entropy, confidence and token from
// eb_merge_kernel).
enum { kFromChunks = 0, kFromEntropies = 1, kFromRows = 2 };

template <int MODE>
__global__ __launch_bounds__(64 * kEbSelWaves) void eb_select_kernel(EbArgs a) {
  __shared__ double sh[64];
  __shared__ double sconf[64];
  __shared__ double skey[64];  // ranking key, ascending: H or -confidence
  __shared__ int smask[64];
  __shared__ int sbad[64];     // 1: the row's statistics are NaN (undefined softmax)
  __shared__ int stok[64];
  __shared__ int order[64];
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int k = a.k;
  const bool by_conf = a.rule != SBD_SELECT_EB_ENTROPY;

  for (int j = w; j < k; j += kEbSelWaves) {
    const int64_t row = (int64_t)b * k + j;
    const bool masked = eb_row_masked(a, row);
    double H = 0.0, conf = 0.0;
    int tok = -1;
    if (masked) {
      if (MODE == kFromEntropies) {
        H = a.entropy_in[row];
      } else if (MODE == kFromRows) {
        H = a.row_stats[row * 2];
        conf = a.row_stats[row * 2 + 1];
        tok = a.row_tok[row];
      } else {
        const double* p = a.part + row * a.n_chunks * 3;
        const int* pa = a.part_arg + row * a.n_chunks;
        // the lane's first chunk is read once, with its argmax; chunks past the 64th
        // (vocabularies above 256K entries) are read again in the second pass
        double m0 = -INFINITY, z0 = 0.0, s0 = 0.0;
        int g0 = -1;
        if (lane < a.n_chunks) {
          m0 = p[lane * 3];
          z0 = p[lane * 3 + 1];
          s0 = p[lane * 3 + 2];
          g0 = pa[lane];
        }
        double mloc = m0;
        for (int c = lane + 64; c < a.n_chunks; c += 64) mloc = fmax(mloc, p[c * 3]);
        const double M = wave_max_d(mloc);
        double z = 0.0, sacc = 0.0;
        int cfirst = INT32_MAX, carg = -1;  // the lane's first chunk reaching M, and its argmax
        if (m0 != -INFINITY) {
          const double d = m0 - M;
          const double f = exp(d);
          z += f * z0;
          sacc += f * (s0 + d * z0);
          if (m0 == M) {
            cfirst = lane;
            carg = g0;
          }
        }
        for (int c = lane + 64; c < a.n_chunks; c += 64) {
          const double mc = p[c * 3];
          if (mc == -INFINITY) continue;
          const double d = mc - M;
          const double f = exp(d);
          z += f * p[c * 3 + 1];
          sacc += f * (p[c * 3 + 2] + d * p[c * 3 + 1]);
          if (mc == M && c < cfirst) {
            cfirst = c;
            carg = pa[c];
          }
        }
        const double Z = wave_sum_d(z);
        const double S = wave_sum_d(sacc);
        int cmin = cfirst;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) cmin = min(cmin, __shfl_xor(cmin, o));
        const int from = cmin == INT32_MAX ? 0 : (cmin & 63);  // the lane holding chunk cmin
        const int t = __shfl(carg, from);
        if (cmin == INT32_MAX) {  // no finite logit in the row
          tok = -1;
          H = __builtin_nan("");
          conf = __builtin_nan("");
        } else {
          tok = t;
          H = log(Z) - S / Z;
          conf = 1.0 / Z;  // the largest probability: e^0 / Z
        }
      }
    }
    if (lane == 0) {
      sh[j] = H;
      sconf[j] = conf;
      const bool nan_stats = H != H || conf != conf;
      skey[j] = nan_stats ? 0.0 : (by_conf ? -conf : H);  // rows with NaN statistics: by row
      sbad[j] = nan_stats ? 1 : 0;
      smask[j] = masked ? 1 : 0;
      stok[j] = tok;
    }
  }
  __syncthreads();
  // Wave 0 ranks and selects; every value it needs from another lane is broadcast with
  // readlane (a uniform loop over the rows or ranks), not read back from LDS one by one.
  if (w != 0) return;
  const int j = lane;
  const bool in = j < k;
  const bool masked = in && smask[j] != 0;
  const double H = in ? sh[j] : 0.0;
  const double C = in ? sconf[j] : 0.0;
  const double key = in ? skey[j] : 0.0;
  const int bad = in ? sbad[j] : 0;
  // rank by (NaN statistics, key, row) ascending: a permutation of the masked rows whose
  // first n places hold the rows with usable statistics; only those can be accepted
  int rank = 0, n = 0;
  for (int i = 0; i < k; ++i) {  // uniform
    if (!__builtin_amdgcn_readlane((int)masked, i)) continue;
    const int bi = __builtin_amdgcn_readlane(bad, i);
    const double ki = readlane_d(key, i);
    n += bi ? 0 : 1;
    if (bi < bad || (bi == bad && (ki < key || (ki == key && i < j)))) ++rank;
  }
  if (masked) order[rank] = j;
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the wave's order[] stores are done
  // lane r holds the statistics of the row ranked r; the prefix sums run over the ranks in
  // order, one float64 addition after another, as the selection rule is written
  const int ro = lane < n ? order[lane] : 0;
  const double hr = lane < n ? sh[ro] : 0.0;
  const double cr = lane < n ? sconf[ro] : 0.0;
  int s = 0;
  if (a.rule == SBD_SELECT_EB_ENTROPY) {  // eq. (eb_sampler): c_{r-1} <= gamma
    double c = 0.0;
    for (int r = 0; r < n; ++r) {
      if (c <= a.gamma) s = r + 1;
      c += readlane_d(hr, r);
    }
  } else if (a.rule == SBD_SELECT_EB_CONFIDENCE) {  // App. B: sum - max of the prefix <= gamma
    double c = 0.0, top = -INFINITY;
    s = n > 0 ? 1 : 0;
    for (int r = 0; r < n; ++r) {
      const double h = readlane_d(hr, r);
      c += h;
      top = fmax(top, h);
      if (c - top <= a.gamma) s = r + 1;
    }
  } else {  // Factor: (r + 1)(1 - c_r) < f
    s = n > 0 ? 1 : 0;
    for (int r = 0; r < n; ++r)
      if ((double)(r + 2) * (1.0 - readlane_d(cr, r)) < a.gamma) s = r + 1;
  }
  if (lane == 0) a.n_accepted[b] = s;
  const bool acc = masked && rank < s;
  // output slot = number of accepted rows before j; accepted slots (< s) and the slots
  // cleared below (>= s) are disjoint
  const unsigned long long before = __ballot(acc) & ((1ull << j) - 1ull);
  const int idx = __popcll(before);
  const int64_t row = (int64_t)b * k + j;
  if (in) {
    if (j >= s) {
      a.accepted_pos[row] = -1;
      if (a.accepted_tok) a.accepted_tok[row] = -1;
    }
    if (a.entropy_out) a.entropy_out[row] = masked ? H : __builtin_nan("");
    if (a.conf_out) a.conf_out[row] = masked ? C : __builtin_nan("");
  }
  if (acc) {
    a.accepted_pos[(int64_t)b * k + idx] = j;
    if (a.accepted_tok) a.accepted_tok[(int64_t)b * k + idx] = stok[j];
  }
}

// Scratch of sbd_eb_select_noalloc, the entry point for callers that cannot allocate: the
// chunk statistics (max, Z, S) and the chunk argmaxes of up to kNoAllocRows rows of up to
// kNoAllocChunks vocabulary chunks each, 1.75 MiB per device for the life of the process.
// Every statistic a select reads is written by the partial kernel of the same call first, so
// nothing needs clearing between calls.
__device__ __align__(256) double scratch[(int64_t)kNoAllocRows * kNoAllocChunks * 3 +
                                         (int64_t)kNoAllocRows * kNoAllocChunks / 2];

hipError_t eb_noalloc_scratch(double** part, int32_t** part_arg) {
  static std::mutex mu;
  static void* addr[kNoAllocMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kNoAllocMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    // the array's name is a host-side stand-in: its device address comes from the runtime,
    // once per device, with that device current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *part = static_cast<double*>(addr[dev]);
  *part_arg = reinterpret_cast<int32_t*>(*part + (int64_t)kNoAllocRows * kNoAllocChunks * 3);
  return hipSuccess;
}

hipError_t launch_eb_partial(const EbArgs& a, const Exec& ex) {
  SBD_KLAUNCH(eb_partial_kernel, dim3(a.n_chunks, a.B * a.k), dim3(kEbThreads), ex, a);
  return hipGetLastError();
}

hipError_t launch_eb_select(const EbArgs& a, bool select_only, const Exec& ex) {
  if (select_only)
    SBD_KLAUNCH(eb_select_kernel<kFromEntropies>, dim3(a.B), dim3(64 * kEbSelWaves), ex, a);
  else if (a.row_stats != nullptr)
    SBD_KLAUNCH(eb_select_kernel<kFromRows>, dim3(a.B), dim3(64 * kEbSelWaves), ex, a);
  else
    SBD_KLAUNCH(eb_select_kernel<kFromChunks>, dim3(a.B), dim3(64 * kEbSelWaves), ex, a);
  return hipGetLastError();
}

// ---- rows of many chunks: the statistics of the LM head's 64-column chunks
//
// One workgroup of 512 threads per masked row.  Thread t takes chunks t, t + 512, ... (at
// most kMergePer: vocabularies up to 512 * 8 * 64 = 262144 entries), all loaded up front.
// M = max m_c (fixed reduction), the first chunk reaching M gives the token; then with
// delta_c = m_c - M, Z = sum_c e^delta_c Z_c and S = sum_c e^delta_c (S_c + delta_c Z_c),
// summed per thread in chunk order and then over lanes and waves in a fixed order; H =
// log Z - S / Z and the confidence 1 / Z, as the chunk merge of eb_select_kernel.
constexpr int kMergeThreads = 512;
constexpr int kMergePer = 8;

__global__ __launch_bounds__(kMergeThreads) void eb_merge_kernel(EbArgs a) {
  const int64_t row = blockIdx.x;
  if (a.is_mask == nullptr && !eb_row_masked(a, row)) return;
  __shared__ double red_d[2][kMergeThreads / 64];
  __shared__ int red_i[kMergeThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const double* p = a.part + row * a.n_chunks * 3;
  const int32_t* pa = a.part_arg + row * a.n_chunks;
  double mc[kMergePer], zc[kMergePer], sc[kMergePer];
  int ac[kMergePer];
#pragma unroll
  for (int i = 0; i < kMergePer; ++i) {  // clamped indices: every load is in flight at once
    const int c = min(tid + i * kMergeThreads, a.n_chunks - 1);
    mc[i] = p[c * 3];
    zc[i] = p[c * 3 + 1];
    sc[i] = p[c * 3 + 2];
    ac[i] = pa[c];
  }
  const bool masked = a.is_mask == nullptr || eb_row_masked(a, row);
#pragma unroll
  for (int i = 0; i < kMergePer; ++i)
    if (tid + i * kMergeThreads >= a.n_chunks) mc[i] = -INFINITY;
  double mloc = -INFINITY;
#pragma unroll
  for (int i = 0; i < kMergePer; ++i) mloc = fmax(mloc, mc[i]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) mloc = fmax(mloc, shfl_xor_d(mloc, o));
  if (lane == 0) red_d[0][w] = mloc;
  __syncthreads();
  double M = red_d[0][0];
#pragma unroll
  for (int i = 1; i < kMergeThreads / 64; ++i) M = fmax(M, red_d[0][i]);
  // the first chunk reaching M (none when every chunk is -inf)
  int cfirst = INT32_MAX;
#pragma unroll
  for (int i = kMergePer - 1; i >= 0; --i)
    if (mc[i] != -INFINITY && mc[i] == M) cfirst = tid + i * kMergeThreads;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) cfirst = min(cfirst, __shfl_xor(cfirst, o));
  double z = 0.0, s = 0.0;
#pragma unroll
  for (int i = 0; i < kMergePer; ++i) {
    if (mc[i] != -INFINITY) {
      const double d = mc[i] - M;
      const double f = exp(d);
      z += f * zc[i];
      s += f * (sc[i] + d * zc[i]);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    z += shfl_xor_d(z, o);
    s += shfl_xor_d(s, o);
  }
  __syncthreads();  // every thread has read red_d[0]
  if (lane == 0) {
    red_d[0][w] = z;
    red_d[1][w] = s;
    red_i[w] = cfirst;
  }
  __syncthreads();
  if (tid == 0 && masked) {
    double Z = 0.0, S = 0.0;
    int cmin = INT32_MAX;
    for (int i = 0; i < kMergeThreads / 64; ++i) {
      Z += red_d[0][i];
      S += red_d[1][i];
      cmin = min(cmin, red_i[i]);
    }
    double H, conf;
    int tok;
    if (cmin == INT32_MAX) {  // no finite logit in the row
      H = conf = __builtin_nan("");
      tok = -1;
    } else {
      H = log(Z) - S / Z;
      conf = 1.0 / Z;
      tok = pa[cmin];
    }
    a.row_stats[row * 2] = H;
    a.row_stats[row * 2 + 1] = conf;
    a.row_tok[row] = tok;
  }
}

hipError_t launch_eb_merge(const EbArgs& a, const Exec& ex) {
  if (a.n_chunks < 1 || a.n_chunks > kMergeThreads * kMergePer || a.row_stats == nullptr || a.row_tok == nullptr)
    return hipErrorInvalidValue;
  SBD_KLAUNCH(eb_merge_kernel, dim3(a.B * a.k), dim3(kMergeThreads), ex, a);
  return hipGetLastError();
}

}  // namespace sbd
