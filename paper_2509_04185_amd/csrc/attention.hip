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
// whole workgroup (see the kernel).

#include "attention_body.h"

namespace sbd {

template <int DH>
__global__ __launch_bounds__(256) void attn_split_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[kAttnSmem];
  attn_split_body<DH, false>(a, blockIdx.x, blockIdx.y, blockIdx.z, smem);
}

template <int DH>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  const int64_t n_items = (int64_t)a.B * a.k * a.n_q;
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= n_items) return;
  attn_merge_body<DH, false>(a, item);
}

hipError_t launch_attention_split(const AttnArgs& a, const Exec& ex) {
  dim3 grid(a.n_splits, a.n_kv * a.n_rowblocks, a.B);
  if (a.d_h == 128)
    SBD_KLAUNCH(attn_split_kernel<128>, grid, dim3(256), ex, a);
  else if (a.d_h == 64)
    SBD_KLAUNCH(attn_split_kernel<64>, grid, dim3(256), ex, a);
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
