// ffn_prep.hip -- activation preparation of moe_expert_ffn_mixed: fp32 group
// sums of the activation rows the streaming kernel reads, and the fp16 copy of
// the token rows the tile kernel reads.
#include "ffn_common.hpp"

namespace moe {
namespace ffn {

// ------------------------------------------------------------------ group sums
// out[j * rows + p] = sum over group j of the bf16 row of permuted row p, in
// fp32: each of g/8 lanes adds its 8 values in order, then an xor tree over
// those lanes.  The row of p starts at perm[p] * ld (gathered activations)
// or, with perm == NULL, at h_row(p) (hidden activations).  Rows p < p_split
// have K columns, the others K2 (routed and shared hidden rows in one
// launch); groups past a row's width are skipped.  Consecutive lane groups
// take consecutive p so the stores coalesce.
template <int NM>
__global__ void __launch_bounds__(256)
group_sum_kernel(FfnArgs a, const uint16_t* __restrict__ in, const int32_t* __restrict__ perm,
                 int64_t ld, int p0, int p1, int K, int p_split, int K2, float* __restrict__ out) {
  constexpr int g = NM * 32;
  constexpr int lanes = g / 8;
  const int G = max(K, K2) / g;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t n = static_cast<int64_t>(p1 - p0) * G * lanes;
  bool live = id < n;
  const int64_t item = id / lanes;
  const int q = static_cast<int>(id % lanes);
  const int np = p1 - p0;
  float s = 0.f;
  int p = 0, j = 0;
  if (live) {
    j = static_cast<int>(item / np);
    p = p0 + static_cast<int>(item % np);
    live = j < (p < p_split ? K : K2) / g;   // the same for every lane of the item
  }
  if (live) {
    const int64_t row = perm ? static_cast<int64_t>(perm[p]) * ld : h_row(a, p);
    const u32x4 v = *reinterpret_cast<const u32x4*>(in + row + static_cast<int64_t>(j) * g + q * 8);
#pragma unroll
    for (int c = 0; c < 4; c++) {
      s = s + bf16_lo(v[c]);
      s = s + bf16_hi(v[c]);
    }
  }
#pragma unroll
  for (int off = lanes / 2; off >= 1; off >>= 1) s = s + __shfl_xor(s, off, kWave);
  if (live && q == 0) out[static_cast<int64_t>(j) * a.rows + p] = s;
}

// x16[t][c] = fp16(x[t][c]) for the T tokens, the activation operand of the
// tile kernel, which reaches the row of permuted row p through perm[p] (one
// copy per token instead of one per routed and shared row; exact for
// |x| < 65504, the bf16 values being a subset of fp16's in that range); 8
// values per thread.
__global__ void __launch_bounds__(256) gather_f16_kernel(FfnArgs a, int T) {
  const int per_row = a.d / 8;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= static_cast<int64_t>(T) * per_row) return;
  const int p = static_cast<int>(id / per_row);
  const int c = static_cast<int>(id % per_row) * 8;
  const u32x4 v = *reinterpret_cast<const u32x4*>(a.x + static_cast<int64_t>(p) * a.d + c);
  u32x4 o;
  bool bad = false;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const float fl = bf16_lo(v[i]), fh = bf16_hi(v[i]);
    bad = bad || !fp16_finite(fl) || !fp16_finite(fh);
    const uint32_t lo = __builtin_bit_cast(uint16_t, static_cast<_Float16>(fl));
    const uint32_t hi = __builtin_bit_cast(uint16_t, static_cast<_Float16>(fh));
    o[i] = lo | (hi << 16);
  }
  *reinterpret_cast<u32x4*>(const_cast<uint16_t*>(a.x16) + static_cast<int64_t>(p) * a.d + c) = o;
  if (bad && a.status) *a.status = MOE_ERR_RANGE;
}

template __global__ void group_sum_kernel<2>(FfnArgs, const uint16_t*, const int32_t*, int64_t, int, int, int,
                                             int, int, float*);
template __global__ void group_sum_kernel<4>(FfnArgs, const uint16_t*, const int32_t*, int64_t, int, int, int,
                                             int, int, float*);

}  // namespace ffn
}  // namespace moe
