// Softmax statistics of 64-column chunks of logits rows, for the EB-Sampler's entropy
// (Sec. 2.2, eq. (eb_sampler)) straight from the LM head's epilogue (gemv.hip, gemm.hip):
// the logits then need not be stored and read back.  eb.hip merges the chunks of a row.
#pragma once

#include "sbd_device.h"

namespace sbd {

__device__ __forceinline__ double shfl_xor_d(double v, int m) {
  const int2 iv = *reinterpret_cast<int2*>(&v);
  int2 o;
  o.x = __shfl_xor(iv.x, m);
  o.y = __shfl_xor(iv.y, m);
  return *reinterpret_cast<double*>(&o);
}

// v of lane i (i uniform across the wave), in every lane
__device__ __forceinline__ double readlane_d(double v, int i) {
  const int2 iv = *reinterpret_cast<int2*>(&v);
  int2 o;
  o.x = __builtin_amdgcn_readlane(iv.x, i);
  o.y = __builtin_amdgcn_readlane(iv.y, i);
  return *reinterpret_cast<double*>(&o);
}

// One 64-column chunk of one row held by LPC adjacent lanes (xor distances below LPC), each
// with VPL consecutive columns col0 .. col0 + VPL - 1 staged in LDS at p (fp32 products,
// times `scale` = the row's norm scale gives the logit exactly as stored).  The mask column
// is left out.  Results, the same on the LPC lanes: the chunk maximum mx and the smallest
// column reaching it (INT32_MAX when no value is above -inf), then with t = l - mx in
// float64, Z = sum e^t and S = sum e^t t over the values above -inf (each lane in column
// order, then a fixed butterfly).  A NaN logit is never the maximum but makes Z and S NaN,
// an infinite maximum makes them NaN too (both as the EB partial kernel on stored logits).
template <int VPL, int LPC>
__device__ __forceinline__ void eb_seg_stats(const float* p, float scale, int col0, int mask_id, float& mx, int& arg,
                                             double& z, double& s) {
  float v[VPL];
#pragma unroll
  for (int e = 0; e < VPL; e += 4) {
    const f32x4 q = *reinterpret_cast<const f32x4*>(p + e);
#pragma unroll
    for (int u = 0; u < 4; ++u) v[e + u] = q[u] * scale;
  }
  mx = -INFINITY;
  arg = INT32_MAX;
#pragma unroll
  for (int e = 0; e < VPL; ++e) {
    if (col0 + e == mask_id) v[e] = -INFINITY;
    if (v[e] > mx) {  // columns ascend: the first of equal values is kept
      mx = v[e];
      arg = col0 + e;
    }
  }
#pragma unroll
  for (int o = 1; o < LPC; o <<= 1) {
    const float om = __shfl_xor(mx, o);
    const int oa = __shfl_xor(arg, o);
    if (om > mx || (om == mx && oa < arg)) {
      mx = om;
      arg = oa;
    }
  }
  z = 0.0;
  s = 0.0;
  if (mx != -INFINITY) {
    const double md = (double)mx;
#pragma unroll
    for (int e = 0; e < VPL; ++e) {
      if (v[e] != -INFINITY) {
        const double t = (double)v[e] - md;
        const double ex = exp(t);
        z += ex;
        s += ex * t;
      }
    }
  }
#pragma unroll
  for (int o = 1; o < LPC; o <<= 1) {  // a + b = b + a: the LPC lanes end with the same bits
    z += shfl_xor_d(z, o);
    s += shfl_xor_d(s, o);
  }
}

// Store the statistics of chunk `chunk` of row m: part [rows][n_chunks][3] = (max, Z, S),
// part_arg [rows][n_chunks] = the argmax column or -1.
__device__ __forceinline__ void eb_chunk_store(double* part, int32_t* part_arg, int n_chunks, int64_t m, int chunk,
                                               float mx, int arg, double z, double s) {
  double* p = part + (m * n_chunks + chunk) * 3;
  p[0] = (double)mx;
  p[1] = z;
  p[2] = s;
  part_arg[m * n_chunks + chunk] = mx == -INFINITY ? -1 : arg;
}

}  // namespace sbd
