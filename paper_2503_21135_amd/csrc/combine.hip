// combine.hip -- moe_unpermute_combine: y[t] = sum_j w[t][j] * o[inv[t][j]]
// + sum_s o[inv[t][k+s]], where each o row is the sum of its n_split slices.
// The weighted sum over a token's k experts is the output of the MoE layer
// (Sec. II-A); shared experts are added with weight 1.  Fixed order, fp32.
#include "common.hpp"

namespace moe {
namespace {

__global__ void __launch_bounds__(256)
combine_kernel(const float* __restrict__ o, int n_split, int64_t ss, const int32_t* __restrict__ inv,
               const float* __restrict__ w, int T, int k, int S, int d, float* __restrict__ y) {
  const int per = d / 4;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= static_cast<int64_t>(T) * per) return;
  const int t = static_cast<int>(id / per);
  const int c4 = static_cast<int>(id % per);
  const int32_t* iv = inv + static_cast<int64_t>(t) * (k + S);
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < k + S; j++) {
    const int64_t p = iv[j];
    f32x4 v = reinterpret_cast<const f32x4*>(o + p * d)[c4];
    for (int sp = 1; sp < n_split; sp++) {
      const f32x4 u = reinterpret_cast<const f32x4*>(o + sp * ss + p * d)[c4];
      v = f32x4{v[0] + u[0], v[1] + u[1], v[2] + u[2], v[3] + u[3]};
    }
    const float wj = j < k ? w[static_cast<int64_t>(t) * k + j] : 1.0f;
#pragma unroll
    for (int c = 0; c < 4; c++) acc[c] = __fmaf_rn(wj, v[c], acc[c]);
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
  hipLaunchKernelGGL(combine_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0, s, o,
                     n_split, split_stride, inv_perm, topk_w, T, k, S, d, y);
  return launch_status(s);
}
