// combine.hip -- moe_unpermute_combine: y[t] = sum_j w[t][j] * o[inv[t][j]]
// + sum_s o[inv[t][k+s]], where each o row is the sum of its n_split slices.
// The weighted sum over a token's k experts is the output of the MoE layer
// (Sec. II-A); shared experts are added with weight 1.  Fixed order, fp32.
#include "common.hpp"

namespace moe {
namespace {

// One thread per 4 columns of a token.  The token's rows are taken in
// batches of NB (2, 4 or 8, the smallest that holds the k + S rows, else 8):
// the row indices, then the rows of the batch are loaded before the first add,
// so the loads overlap instead of waiting on each other; the adds keep the
// fixed order (slices ascending per row, then rows ascending into the fused
// multiply-add chain).
template <int NB>
__global__ void __launch_bounds__(256)
combine_kernel(const float* __restrict__ o, int n_split, int64_t ss, const int32_t* __restrict__ inv,
               const float* __restrict__ w, int T, int k, int S, int d, float* __restrict__ y) {
  const int per = d / 4;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= static_cast<int64_t>(T) * per) return;
  const int t = static_cast<int>(id / per);
  const int c4 = static_cast<int>(id % per);
  const int n = k + S;
  const int32_t* iv = inv + static_cast<int64_t>(t) * n;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int j0 = 0; j0 < n; j0 += NB) {
    int64_t p[NB];
    float wj[NB];
    f32x4 v[NB];
#pragma unroll
    for (int i = 0; i < NB; i++) {
      const int j = j0 + i;
      p[i] = j < n ? static_cast<int64_t>(iv[j]) : 0;
      wj[i] = j < k ? w[static_cast<int64_t>(t) * k + j] : 1.0f;
    }
#pragma unroll
    for (int i = 0; i < NB; i++)
      if (j0 + i < n) v[i] = reinterpret_cast<const f32x4*>(o + p[i] * d)[c4];
    for (int sp = 1; sp < n_split; sp++) {
      f32x4 u[NB];
#pragma unroll
      for (int i = 0; i < NB; i++)
        if (j0 + i < n) u[i] = reinterpret_cast<const f32x4*>(o + sp * ss + p[i] * d)[c4];
#pragma unroll
      for (int i = 0; i < NB; i++)
        if (j0 + i < n) v[i] = f32x4{v[i][0] + u[i][0], v[i][1] + u[i][1], v[i][2] + u[i][2], v[i][3] + u[i][3]};
    }
#pragma unroll
    for (int i = 0; i < NB; i++)
      if (j0 + i < n) {
#pragma unroll
        for (int c = 0; c < 4; c++) acc[c] = __fmaf_rn(wj[i], v[i][c], acc[c]);
      }
  }
  reinterpret_cast<f32x4*>(y + static_cast<int64_t>(t) * d)[c4] = acc;
}

}  // namespace
}  // namespace moe

extern "C" int moe_unpermute_combine(const float* o, int32_t n_split, int64_t split_stride,
                                     const int32_t* inv_perm, const float* topk_w, int32_t T,
                                     int32_t k, int32_t S, int32_t d, float* y, void* stream) {
  using namespace moe;
  if (T < 0 || k < 1 || k > MOE_MAX_TOPK || S < 0 || d <= 0 || d % 4 || n_split < 1)
    return MOE_ERR_ARG;
  if (T == 0) return MOE_OK;
  if (!o || !inv_perm || !topk_w || !y) return MOE_ERR_ARG;
  if (n_split > 1 && split_stride < static_cast<int64_t>(T) * (k + S) * d) return MOE_ERR_ARG;
  if (!aligned16(o) || !aligned16(y) || (n_split > 1 && split_stride % 4)) return MOE_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t n = static_cast<int64_t>(T) * (d / 4);
  const dim3 grid(static_cast<unsigned>(cdiv(n, 256)));
  if (k + S <= 2)
    hipLaunchKernelGGL(combine_kernel<2>, grid, dim3(256), 0, s, o, n_split, split_stride, inv_perm, topk_w,
                       T, k, S, d, y);
  else if (k + S <= 4)
    hipLaunchKernelGGL(combine_kernel<4>, grid, dim3(256), 0, s, o, n_split, split_stride, inv_perm, topk_w,
                       T, k, S, d, y);
  else
    hipLaunchKernelGGL(combine_kernel<8>, grid, dim3(256), 0, s, o, n_split, split_stride, inv_perm, topk_w,
                       T, k, S, d, y);
  return launch_status(s);
}
