// route.hip -- moe_route_permute: router logits, top-k selection, combine
// weights and the permutation of token rows into per-expert segments.
//
// Sec. II-A: a fixed number k of experts is selected per token.  The token ->
// several experts mapping (Sec. I, Sec. II-A "Data-Weight Mappings") becomes
// a histogram of expert choices, an exclusive scan into segment offsets and a
// stable scatter of token indices.  Everything is bitwise reproducible: the
// logit reduction order is fixed (moe_quant.h), the exponential is the
// library's own, and the permutation's only atomics are bitwise ORs, whose
// result does not depend on their order.
#include "common.hpp"

#pragma clang fp contract(off)

namespace moe {
namespace {

constexpr int kChunk = 64;  // tokens per histogram chunk (one wave)

// Exponential for x <= 0 as the header defines it: Cody-Waite reduction by
// ln2 split into 2839/4096 (12 significant bits) and its fp32 remainder,
// Taylor polynomial of degree 7 in Horner form, scaling by 2^n.
__device__ float lib_exp_nonpos(float x) {
  if (x < -80.0f) return 0.0f;
  constexpr float kLog2e = static_cast<float>(1.4426950408889634);
  constexpr float kLn2Hi = 2839.0f / 4096.0f;
  constexpr float kLn2Lo = static_cast<float>(0.69314718055994531 - 2839.0 / 4096.0);
  constexpr float kC[8] = {static_cast<float>(1.0),
                           static_cast<float>(1.0),
                           static_cast<float>(1.0 / 2.0),
                           static_cast<float>(1.0 / 6.0),
                           static_cast<float>(1.0 / 24.0),
                           static_cast<float>(1.0 / 120.0),
                           static_cast<float>(1.0 / 720.0),
                           static_cast<float>(1.0 / 5040.0)};
  const float n = rintf(x * kLog2e);
  float r = __fmaf_rn(-n, kLn2Hi, x);
  r = __fmaf_rn(-n, kLn2Lo, r);
  float p = kC[7];
#pragma unroll
  for (int i = 6; i >= 0; i--) p = __fmaf_rn(p, r, kC[i]);
  return ldexpf(p, static_cast<int>(n));
}

// Wave-wide reduction of the 64 lane partials; lane 0 ends with the value of
// the header's halving tree (partial[l] += partial[l ^ off] pairs exactly the
// tree's operands at lane 0).
__device__ __forceinline__ float tree_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = v + __shfl_xor(v, off, kWave);
  return __shfl(v, 0, kWave);
}

constexpr int kMaxD = 8192;     // d_model limit of the router
constexpr int kRouteWaves = 8;  // waves per router workgroup

// Partial dot products of NE router rows (experts e0, e0 + es, ...) with the
// token row: lane l accumulates columns l, l + 64, l + 128, ... in ascending
// order with one fused multiply-add each, the header's per-lane order.  The
// activations are read straight from global memory (bf16 -> fp32 is exact),
// and each batch issues RB columns of every row before the first FMA so the
// whole batch is in flight at once.
template <int NE, int RB>
__device__ __forceinline__ void router_partials(const uint16_t* __restrict__ xr,
                                                const float* __restrict__ wr, int d, int e0,
                                                int es, int lane, float (&acc)[NE]) {
#pragma unroll
  for (int j = 0; j < NE; j++) acc[j] = 0.0f;
  int c0 = 0;
  for (; c0 + kWave * RB <= d; c0 += kWave * RB) {
    uint32_t xb[RB];
    float w[NE][RB];
#pragma unroll
    for (int i = 0; i < RB; i++) {
      const int c = c0 + kWave * i + lane;
      xb[i] = xr[c];
#pragma unroll
      for (int j = 0; j < NE; j++) w[j][i] = wr[static_cast<int64_t>(e0 + j * es) * d + c];
    }
#pragma unroll
    for (int i = 0; i < RB; i++) {
      const float xv = __uint_as_float(xb[i] << 16);
#pragma unroll
      for (int j = 0; j < NE; j++) acc[j] = __fmaf_rn(xv, w[j][i], acc[j]);
    }
  }
  for (int c = c0 + lane; c < d; c += kWave) {  // tail: fewer than RB columns per lane
    const float xv = __uint_as_float(static_cast<uint32_t>(xr[c]) << 16);
#pragma unroll
    for (int j = 0; j < NE; j++)
      acc[j] = __fmaf_rn(xv, wr[static_cast<int64_t>(e0 + j * es) * d + c], acc[j]);
  }
}

// Top k of one token's E logits src[0 .. E) by (logit desc, index asc; a
// NaN as -inf) and the softmax over the selected logits; one wave, every lane
// ends with the same picks, lane 0 writes the token's row of topk_ids /
// topk_w.
__device__ __forceinline__ void select_topk(const float* src, int E, int k, int t, int lane,
                                            int32_t* __restrict__ topk_ids,
                                            float* __restrict__ topk_w) {
  constexpr int kMaxPer = MOE_MAX_EXPERTS / kWave;
  float lg[kMaxPer];
#pragma unroll
  for (int m = 0; m < kMaxPer; m++) {
    const int e = m * kWave + lane;
    const float u = e < E ? src[e] : -INFINITY;
    lg[m] = u != u ? -INFINITY : u;   // a NaN ranks as -inf
  }
  // top-k by (logit desc, index asc); every lane ends with the same picks
  bool taken[kMaxPer];
  int ids[MOE_MAX_TOPK];
  float sel[MOE_MAX_TOPK];
#pragma unroll
  for (int m = 0; m < kMaxPer; m++) taken[m] = false;
  for (int j = 0; j < k; j++) {
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int m = 0; m < kMaxPer; m++) {
      const int e = m * kWave + lane;
      if (e < E && !taken[m] && (lg[m] > bv || (lg[m] == bv && e < bi))) {
        bv = lg[m];
        bi = e;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ov = __shfl_xor(bv, off, kWave);
      const int oi = __shfl_xor(bi, off, kWave);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
    ids[j] = bi;
    sel[j] = bv;
#pragma unroll
    for (int m = 0; m < kMaxPer; m++)
      if (bi == m * kWave + lane) taken[m] = true;
  }
  if (lane == 0) {
    float ex[MOE_MAX_TOPK];
    const float mref = sel[0];
    float S = 0.0f;
    for (int j = 0; j < k; j++) {
      ex[j] = lib_exp_nonpos(sel[j] - mref);
      S = S + ex[j];
    }
    for (int j = 0; j < k; j++) {
      topk_ids[static_cast<int64_t>(t) * k + j] = ids[j];
      topk_w[static_cast<int64_t>(t) * k + j] = ex[j] / S;
    }
  }
}

// One workgroup (8 waves) per token.  Wave w owns experts w, w + 8, ... and
// computes their logits four, two or one at a time; wave 0 then selects the
// top k and forms the weights.
__global__ void __launch_bounds__(kRouteWaves * kWave)
route_topk_kernel(const uint16_t* __restrict__ x, int T, int d, const float* __restrict__ wr,
                  const float* __restrict__ bias, int E, int k,
                  int32_t* __restrict__ topk_ids, float* __restrict__ topk_w) {
  __shared__ float lgs[MOE_MAX_EXPERTS];
  const int t = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const uint16_t* xr = x + static_cast<int64_t>(t) * d;
  const int mine = wv < E ? (E - 1 - wv) / kRouteWaves + 1 : 0;  // experts of this wave
  auto finish = [&](int e, float acc) {
    float v = tree_sum(acc);
    if (bias) v = v + bias[e];
    if (lane == 0) lgs[e] = v;
  };
  int m = 0;
  for (; m + 4 <= mine; m += 4) {
    float acc[4];
    router_partials<4, 32>(xr, wr, d, wv + m * kRouteWaves, kRouteWaves, lane, acc);
#pragma unroll
    for (int j = 0; j < 4; j++) finish(wv + (m + j) * kRouteWaves, acc[j]);
  }
  if (m + 2 <= mine) {
    float acc[2];
    router_partials<2, 32>(xr, wr, d, wv + m * kRouteWaves, kRouteWaves, lane, acc);
#pragma unroll
    for (int j = 0; j < 2; j++) finish(wv + (m + j) * kRouteWaves, acc[j]);
    m += 2;
  }
  if (m < mine) {
    float acc[1];
    router_partials<1, 64>(xr, wr, d, wv + m * kRouteWaves, kRouteWaves, lane, acc);
    finish(wv + m * kRouteWaves, acc[0]);
  }
  __syncthreads();
  if (wv != 0) return;
  select_topk(lgs, E, k, t, lane, topk_ids, topk_w);
}

constexpr int kLogitWaves = 4;      // waves of a logits workgroup
constexpr int kLogitExperts = 8;    // experts of a logits workgroup, two per wave
constexpr int kLogitTokens = 8;     // tokens of a logits workgroup
constexpr int kSplitRouterMinT = 256;   // batches from this size: logits, then top k
constexpr int kSplitRouterMinE = 16;    // smaller batches with this many experts too

// Router logits of large batches whose rows are not 16-byte aligned, with the
// experts spread over workgroups: workgroup (token block, expert block)
// computes 8 tokens x 8 experts, wave w
// experts 2w, 2w + 1 of the block, so a CU reads a slice of the router
// matrix once for 8 tokens instead of the whole matrix per token.  Each
// logit is the header's sum: lane l adds columns l, l + 64, ... in ascending
// order with one FMA each, then the halving tree over the lanes, then the
// bias.
template <int TB, int RB>
__global__ void __launch_bounds__(kLogitWaves * kWave)
route_logits_kernel(const uint16_t* __restrict__ x, int T, int d, const float* __restrict__ wr,
                    const float* __restrict__ bias, int E, float* __restrict__ logits) {
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int t0 = blockIdx.x * TB;
  const int e0 = blockIdx.y * kLogitExperts + 2 * wv;
  if (e0 >= E) return;   // wave-uniform; no barrier follows
  int er[2], tr[TB];
#pragma unroll
  for (int j = 0; j < 2; j++) er[j] = min(e0 + j, E - 1);   // clamped rows are computed, not stored
#pragma unroll
  for (int tb = 0; tb < TB; tb++) tr[tb] = min(t0 + tb, T - 1);
  float acc[TB][2];
#pragma unroll
  for (int tb = 0; tb < TB; tb++)
#pragma unroll
    for (int j = 0; j < 2; j++) acc[tb][j] = 0.0f;
  for (int c0 = 0; c0 < d; c0 += kWave * RB) {
    float w[2][RB];
    uint32_t xb[TB][RB];
#pragma unroll
    for (int i = 0; i < RB; i++) {
      if (c0 + kWave * i < d) {   // uniform: d is a multiple of 64
        const int c = c0 + kWave * i + lane;
#pragma unroll
        for (int j = 0; j < 2; j++) w[j][i] = wr[static_cast<int64_t>(er[j]) * d + c];
#pragma unroll
        for (int tb = 0; tb < TB; tb++) xb[tb][i] = x[static_cast<int64_t>(tr[tb]) * d + c];
      }
    }
#pragma unroll
    for (int i = 0; i < RB; i++) {
      if (c0 + kWave * i < d) {
#pragma unroll
        for (int tb = 0; tb < TB; tb++) {
          const float xv = __uint_as_float(xb[tb][i] << 16);
#pragma unroll
          for (int j = 0; j < 2; j++) acc[tb][j] = __fmaf_rn(xv, w[j][i], acc[tb][j]);
        }
      }
    }
  }
#pragma unroll
  for (int tb = 0; tb < TB; tb++)
#pragma unroll
    for (int j = 0; j < 2; j++) {
      float v = tree_sum(acc[tb][j]);
      if (bias) v = v + bias[er[j]];
      if (lane == 0 && t0 + tb < T && e0 + j < E) logits[static_cast<int64_t>(t0 + tb) * E + e0 + j] = v;
    }
}

// Reduce-scatter of the NV per-lane partial logits of a wave (NV a power of
// two, at most 64): at each offset of the header's halving tree (32, 16, ...,
// 1) a lane keeps one half of its values, hands the other half to the lane
// `off` away and adds what it receives, so a pair of lanes adds exactly the
// tree's operands (partial[l] + partial[l + off]; the two lanes add them in
// either order, which gives the same bits).  Once a lane holds a single value
// the remaining offsets are plain butterflies.  Value v ends in the lanes l
// with l / (64 / NV) == v.
template <int N, int OFF, int NV>
__device__ __forceinline__ void tree_scatter(float (&a)[NV], int lane) {
  if constexpr (OFF >= 1) {
    if constexpr (N > 1) {
      constexpr int H = N / 2;
      const bool hi = (lane & OFF) != 0;
#pragma unroll
      for (int i = 0; i < H; i++) {
        const float send = hi ? a[i] : a[i + H];
        const float keep = hi ? a[i + H] : a[i];
        a[i] = keep + __shfl_xor(send, OFF, kWave);
      }
      tree_scatter<H, OFF / 2, NV>(a, lane);
    } else {
      a[0] = a[0] + __shfl_xor(a[0], OFF, kWave);
      tree_scatter<1, OFF / 2, NV>(a, lane);
    }
  }
}

// Router logits staged through LDS: workgroup (token block of 4*WT tokens,
// expert block of WE experts) copies SC-column chunks of its token rows
// (bf16) and router rows (fp32) into LDS with 16-byte loads, the next
// chunk's loads in flight while the current one is used.  Wave w holds the
// logits of tokens WT*w .. WT*w + WT - 1 of the block against the WE experts,
// lane l adding columns l, l + 64, ... in ascending order with one FMA each
// (the header's per-lane order), then the halving tree over the lanes
// (tree_scatter) and the bias.  x and wr must be 16-byte aligned; tokens and
// experts past the ends are clamped (computed, not stored).
template <int WT, int WE, int SC>
__global__ void __launch_bounds__(4 * kWave)
route_logits_lds_kernel(const uint16_t* __restrict__ x, int T, int d, const float* __restrict__ wr,
                        const float* __restrict__ bias, int E, float* __restrict__ logits) {
  constexpr int TT = 4 * WT;                       // tokens of the block
  constexpr int NV = WT * WE;                      // partial logits per lane
  constexpr int XPT = TT * SC / 8 / 256;   // 16-byte x pieces per thread
  constexpr int WPT = WE * SC / 4 / 256;   // 16-byte router pieces per thread
  static_assert(NV <= kWave && (NV & (NV - 1)) == 0 && XPT >= 1 && WPT >= 1, "tile shape");
  __shared__ __attribute__((aligned(16))) uint16_t xs[TT][SC];
  __shared__ __attribute__((aligned(16))) float wsh[WE][SC];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n_eb = (E + WE - 1) / WE;   // expert blocks vary fastest: a token block's
  const int e0 = static_cast<int>(blockIdx.x % n_eb) * WE;   // workgroups run together
  const int t0 = static_cast<int>(blockIdx.x / n_eb) * TT;
  u32x4 xr[XPT] = {}, wrg[WPT] = {};
  auto load = [&](int c0) {
#pragma unroll
    for (int j = 0; j < XPT; j++) {
      const int i = tid + 256 * j, r = i / (SC / 8), c = c0 + (i % (SC / 8)) * 8;
      if (c < d)
        xr[j] = *reinterpret_cast<const u32x4*>(x + static_cast<int64_t>(min(t0 + r, T - 1)) * d + c);
    }
#pragma unroll
    for (int j = 0; j < WPT; j++) {
      const int i = tid + 256 * j, r = i / (SC / 4), c = c0 + (i % (SC / 4)) * 4;
      if (c < d)
        wrg[j] = *reinterpret_cast<const u32x4*>(wr + static_cast<int64_t>(min(e0 + r, E - 1)) * d + c);
    }
  };
  float acc[WT][WE];
#pragma unroll
  for (int tb = 0; tb < WT; tb++)
#pragma unroll
    for (int e = 0; e < WE; e++) acc[tb][e] = 0.0f;
  load(0);
  for (int c0 = 0; c0 < d; c0 += SC) {
    __syncthreads();   // every wave is done with the previous chunk
#pragma unroll
    for (int j = 0; j < XPT; j++) {
      const int i = tid + 256 * j;
      *reinterpret_cast<u32x4*>(&xs[i / (SC / 8)][(i % (SC / 8)) * 8]) = xr[j];
    }
#pragma unroll
    for (int j = 0; j < WPT; j++) {
      const int i = tid + 256 * j;
      *reinterpret_cast<u32x4*>(&wsh[i / (SC / 4)][(i % (SC / 4)) * 4]) = wrg[j];
    }
    __syncthreads();
    if (c0 + SC < d) load(c0 + SC);
#pragma unroll
    for (int i = 0; i < SC / kWave; i++) {
      if (c0 + kWave * i < d) {   // uniform: d is a multiple of 64
        const int c = kWave * i + lane;
        float xv[WT], wv_[WE];
#pragma unroll
        for (int tb = 0; tb < WT; tb++) xv[tb] = __uint_as_float(static_cast<uint32_t>(xs[wv * WT + tb][c]) << 16);
#pragma unroll
        for (int e = 0; e < WE; e++) wv_[e] = wsh[e][c];
#pragma unroll
        for (int tb = 0; tb < WT; tb++)
#pragma unroll
          for (int e = 0; e < WE; e++) acc[tb][e] = __fmaf_rn(xv[tb], wv_[e], acc[tb][e]);
      }
    }
  }
  float a[NV];
#pragma unroll
  for (int tb = 0; tb < WT; tb++)
#pragma unroll
    for (int e = 0; e < WE; e++) a[tb * WE + e] = acc[tb][e];
  tree_scatter<NV, kWave / 2, NV>(a, lane);
  constexpr int per = kWave / NV;   // lanes holding each value
  const int v = lane / per;
  const int t = t0 + wv * WT + v / WE, e = e0 + v % WE;
  if (lane % per == 0 && t < T && e < E) {
    float r = a[0];
    if (bias) r = r + bias[e];
    logits[static_cast<int64_t>(t) * E + e] = r;
  }
}

// Top k and weights of the logits rows, one wave per token, by rank: lane l
// holds logits l, l + 64, ... of the token and counts, for each, the logits
// that precede it in the order (logit descending, index ascending; a NaN is
// taken as -inf, so every rank is distinct); a logit of rank j < k is the
// pick of slot j.  The weights follow select_topk's arithmetic: e_j =
// cexp(l_j - l_0), S summed over the slots in order, w_j = e_j / S.
__global__ void __launch_bounds__(4 * kWave)
route_select_kernel(const float* __restrict__ logits, int T, int E, int k,
                    int32_t* __restrict__ topk_ids, float* __restrict__ topk_w) {
  constexpr int kMaxPer = MOE_MAX_EXPERTS / kWave;
  __shared__ __attribute__((aligned(16))) float lgs[4][MOE_MAX_EXPERTS];
  __shared__ float selv[4][MOE_MAX_TOPK], exs[4][MOE_MAX_TOPK];
  __shared__ int32_t seli[4][MOE_MAX_TOPK];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wv;
  const float* src = logits + static_cast<int64_t>(min(t, T - 1)) * E;
  const int E4 = (E + 3) & ~3;   // padded with -inf, which no logit follows
  float v[kMaxPer];
#pragma unroll
  for (int m = 0; m < kMaxPer; m++) {
    const int e = m * kWave + lane;
    float u = e < E ? src[e] : -INFINITY;
    if (u != u) u = -INFINITY;
    v[m] = u;
    if (e < E4) lgs[wv][e] = u;
  }
  __syncthreads();
  int rank[kMaxPer];
#pragma unroll
  for (int m = 0; m < kMaxPer; m++) rank[m] = 0;
  for (int e2 = 0; e2 < E4; e2 += 4) {
    const f32x4 u = *reinterpret_cast<const f32x4*>(&lgs[wv][e2]);
#pragma unroll
    for (int m = 0; m < kMaxPer; m++) {
      if (m * kWave < E) {   // uniform
        const int e = m * kWave + lane;
#pragma unroll
        for (int q = 0; q < 4; q++) rank[m] += (u[q] > v[m] || (u[q] == v[m] && e2 + q < e)) ? 1 : 0;
      }
    }
  }
#pragma unroll
  for (int m = 0; m < kMaxPer; m++) {
    const int e = m * kWave + lane;
    if (e < E && rank[m] < k) {
      selv[wv][rank[m]] = v[m];
      seli[wv][rank[m]] = e;
    }
  }
  __syncthreads();
  if (lane < k) exs[wv][lane] = lib_exp_nonpos(selv[wv][lane] - selv[wv][0]);
  __syncthreads();
  if (t >= T || lane >= k) return;
  float S = 0.0f;
  for (int j = 0; j < k; j++) S = S + exs[wv][j];
  topk_ids[static_cast<int64_t>(t) * k + lane] = seli[wv][lane];
  topk_w[static_cast<int64_t>(t) * k + lane] = exs[wv][lane] / S;
}
// One chunk's expert lane masks in LDS: bit l of mask[e] is set when token
// l of the chunk chose expert e (one LDS atomic OR per choice; OR does not
// depend on the order of the atomics).  The token's choices stay in
// registers, j < k a predicate of the compile-time loop.
__device__ __forceinline__ void chunk_masks(const int32_t* __restrict__ topk_ids, int T, int E, int k,
                                            int c, int lane, uint64_t* mask, int (&mine)[MOE_MAX_TOPK]) {
  const int t = c * kChunk + lane;
  const bool live = t < T;
#pragma unroll
  for (int j = 0; j < MOE_MAX_TOPK; j++)
    mine[j] = (live && j < k) ? topk_ids[static_cast<int64_t>(t) * k + j] : -1;
  for (int e = lane; e < E; e += kWave) mask[e] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < MOE_MAX_TOPK; j++)
    if (mine[j] >= 0) atomicOr(&mask[mine[j]], 1ull << lane);
  __syncthreads();
}

// hist[c][e] = number of tokens of chunk c that selected e.
__global__ void __launch_bounds__(64)
route_hist_kernel(const int32_t* __restrict__ topk_ids, int T, int E, int k,
                  int32_t* __restrict__ hist) {
  __shared__ uint64_t mask[MOE_MAX_EXPERTS];
  const int c = blockIdx.x;
  const int lane = threadIdx.x;
  int mine[MOE_MAX_TOPK];
  chunk_masks(topk_ids, T, E, k, c, lane, mask, mine);
  for (int e = lane; e < E; e += kWave) hist[static_cast<int64_t>(c) * E + e] = __popcll(mask[e]);
}

// offsets[] and per-chunk segment bases (single workgroup; one thread per
// expert column, chunks in order, their counts loaded 16 at a time).
__global__ void __launch_bounds__(256)
route_scan_kernel(const int32_t* __restrict__ hist, int n_chunks, int T, int E, int k, int S,
                  int32_t* __restrict__ base, int32_t* __restrict__ offsets) {
  __shared__ int32_t tot[MOE_MAX_EXPERTS];
  constexpr int kBatch = 16;
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    int s = 0;
    for (int c0 = 0; c0 < n_chunks; c0 += kBatch) {
      int v[kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; i++)
        v[i] = c0 + i < n_chunks ? hist[static_cast<int64_t>(c0 + i) * E + e] : 0;
#pragma unroll
      for (int i = 0; i < kBatch; i++) {
        if (c0 + i < n_chunks) base[static_cast<int64_t>(c0 + i) * E + e] = s;
        s += v[i];
      }
    }
    tot[e] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int e = 0; e < E; e++) {
      offsets[e] = acc;
      acc += tot[e];
    }
    for (int s2 = 0; s2 <= S; s2++) offsets[E + s2] = acc + s2 * T;
  }
}

// Stable scatter: rank of a token inside its chunk's share of segment e is
// the number of earlier lanes of the chunk that selected e, the popcount of
// the chunk's mask of e below the lane.
__global__ void __launch_bounds__(64)
route_scatter_kernel(const int32_t* __restrict__ topk_ids, int T, int E, int k, int S,
                     const int32_t* __restrict__ base, const int32_t* __restrict__ offsets,
                     int32_t* __restrict__ perm_token, int32_t* __restrict__ inv_perm) {
  __shared__ uint64_t mask[MOE_MAX_EXPERTS];
  const int c = blockIdx.x;
  const int lane = threadIdx.x;
  const int t = c * kChunk + lane;
  int mine[MOE_MAX_TOPK];
  chunk_masks(topk_ids, T, E, k, c, lane, mask, mine);
  if (t >= T) return;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int64_t row = static_cast<int64_t>(t) * (k + S);
#pragma unroll
  for (int j = 0; j < MOE_MAX_TOPK; j++) {
    if (j < k) {
      const int e = mine[j];
      const int p = offsets[e] + base[static_cast<int64_t>(c) * E + e] + __popcll(mask[e] & below);
      perm_token[p] = t;
      inv_perm[row + j] = p;
    }
  }
  for (int s = 0; s < S; s++) {
    const int p = offsets[E + s] + t;
    perm_token[p] = t;
    inv_perm[row + k + s] = p;
  }
}

constexpr int kPermWaves = 16;   // waves of the fused permutation workgroup
constexpr int kFusedChunks = 16; // token chunks the fused path holds in LDS

// Histogram, scans and stable scatter of up to kFusedChunks chunks in one
// workgroup (batches of up to 1024 tokens).  The segment order is the same as
// the three-kernel path's: experts ascending, then tokens ascending, shared
// experts last.  Each chunk keeps one 64-bit lane mask per expert (bit l set
// when token l of the chunk chose the expert), so a count is a popcount and a
// token's rank among the chunk's rows of an expert is the popcount of the mask
// below its lane: no thread loops over the experts.
__global__ void __launch_bounds__(kPermWaves * kWave)
route_permute_fused_kernel(const int32_t* __restrict__ topk_ids, int T, int E, int k, int S,
                           int32_t* __restrict__ offsets, int32_t* __restrict__ perm_token,
                           int32_t* __restrict__ inv_perm) {
  __shared__ uint64_t mask[kFusedChunks * MOE_MAX_EXPERTS];  // per chunk and expert
  __shared__ int32_t cb[kFusedChunks * MOE_MAX_EXPERTS];     // chunk bases per expert
  __shared__ int32_t seg[MOE_MAX_EXPERTS + 1];               // segment offsets, then the total
  const int lane = threadIdx.x & 63;
  const int n_chunks = (T + kChunk - 1) / kChunk;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  // wave c holds chunk c (n_chunks <= kPermWaves) and keeps its choices
  const int c = threadIdx.x >> 6;
  const int t = c * kChunk + lane;
  const bool live = t < T;
  // the token's choices in registers: loops over j run to the compile-time
  // bound with j < k as a predicate, so every load is issued at once and no
  // array is indexed at run time
  int mine[MOE_MAX_TOPK];
#pragma unroll
  for (int j = 0; j < MOE_MAX_TOPK; j++)
    mine[j] = (live && j < k) ? topk_ids[static_cast<int64_t>(t) * k + j] : -1;
  for (int i = threadIdx.x; i < n_chunks * E; i += blockDim.x) mask[i] = 0;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < MOE_MAX_TOPK; j++)
    if (mine[j] >= 0) atomicOr(&mask[c * E + mine[j]], 1ull << lane);
  __syncthreads();
  // per expert: exclusive scan of the chunk counts
  if (threadIdx.x < E) {
    const int e = threadIdx.x;
    int run = 0;
    for (int cc = 0; cc < n_chunks; cc++) {
      cb[cc * E + e] = run;
      run += __popcll(mask[cc * E + e]);
    }
    seg[e] = run;
  }
  __syncthreads();
  // exclusive scan of the segment sizes over experts: four per lane of wave 0
  if (c == 0) {
    int v[4];
    int sum = 0;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int e = 4 * lane + i;
      v[i] = e < E ? seg[e] : 0;
      sum += v[i];
    }
    int incl = sum;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int o = __shfl_up(incl, off, kWave);
      if (lane >= off) incl += o;
    }
    int run = incl - sum;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int e = 4 * lane + i;
      if (e < E) seg[e] = run;
      run += v[i];
    }
    if (lane == kWave - 1) seg[MOE_MAX_EXPERTS] = incl;
  }
  __syncthreads();
  const int routed = seg[MOE_MAX_EXPERTS];
  for (int e = threadIdx.x; e < E; e += blockDim.x) offsets[e] = seg[e];
  for (int s2 = threadIdx.x; s2 <= S; s2 += blockDim.x) offsets[E + s2] = routed + s2 * T;
  if (!live) return;
  const int64_t row = static_cast<int64_t>(t) * (k + S);
#pragma unroll
  for (int j = 0; j < MOE_MAX_TOPK; j++) {
    if (j < k) {
      const int i = c * E + mine[j];
      const int p = seg[mine[j]] + cb[i] + __popcll(mask[i] & below);
      perm_token[p] = t;
      inv_perm[row + j] = p;
    }
  }
  for (int s2 = 0; s2 < S; s2++) {
    const int p = routed + s2 * T + t;
    perm_token[p] = t;
    inv_perm[row + k + s2] = p;
  }
}

// x_perm[p] = x[perm_token[p]] (16-byte copies; d % 8 == 0).
__global__ void __launch_bounds__(256)
gather_rows_kernel(const uint16_t* __restrict__ x, int d, const int32_t* __restrict__ perm_token,
                   int rows, uint16_t* __restrict__ x_perm) {
  const int per_row = d / 8;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= static_cast<int64_t>(rows) * per_row) return;
  const int64_t p = id / per_row;
  const int q = static_cast<int>(id % per_row);
  const u32x4* src = reinterpret_cast<const u32x4*>(x + static_cast<int64_t>(perm_token[p]) * d) + q;
  reinterpret_cast<u32x4*>(x_perm + p * d)[q] = *src;
}

size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

}  // namespace
}  // namespace moe

extern "C" size_t moe_route_workspace_bytes(int32_t T, int32_t E, int32_t k, int32_t S) {
  (void)k;
  (void)S;
  if (T < 0 || E <= 0) return 0;
  const size_t n_chunks = static_cast<size_t>((T + moe::kChunk - 1) / moe::kChunk);
  // chunk histogram, chunk bases, then the logits [T][E] of large batches
  const bool split = T >= moe::kSplitRouterMinT || E >= moe::kSplitRouterMinE;
  const size_t logits = split ? sizeof(float) * static_cast<size_t>(T) * E : 0;
  return 2 * moe::align256(sizeof(int32_t) * (n_chunks > 0 ? n_chunks : 1) * E) + moe::align256(logits);
}

extern "C" int moe_route_permute(const uint16_t* x, int32_t T, int32_t d, const float* w_router,
                                 const float* bias, int32_t E, int32_t k, int32_t S,
                                 int32_t* topk_ids, float* topk_w, int32_t* offsets,
                                 int32_t* perm_token, int32_t* inv_perm, uint16_t* x_perm,
                                 void* ws, size_t ws_bytes, void* stream) {
  using namespace moe;
  if (T < 0 || d <= 0 || d % 64 || d > kMaxD || E <= 0 || S < 0 || E + S > MOE_MAX_EXPERTS)
    return MOE_ERR_ARG;
  if (k < 1 || k > E || k > MOE_MAX_TOPK) return MOE_ERR_ARG;
  if (!offsets || (T > 0 && (!x || !w_router || !topk_ids || !topk_w || !perm_token || !inv_perm)))
    return MOE_ERR_ARG;
  if (x_perm && (!aligned16(x_perm) || !aligned16(x))) return MOE_ERR_ALIGN;
  const size_t need = moe_route_workspace_bytes(T, E, k, S);
  if (!ws || ws_bytes < need) return MOE_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n_chunks = static_cast<int>(cdiv(T, kChunk));
  const size_t half = align256(sizeof(int32_t) * static_cast<size_t>(n_chunks > 0 ? n_chunks : 1) * E);
  int32_t* hist = static_cast<int32_t*>(ws);
  int32_t* base = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + half);
  const bool staged = aligned16(x) && aligned16(w_router);   // 16-byte row loads
  float* logits = reinterpret_cast<float*>(static_cast<char*>(ws) + 2 * half);
  const dim3 blk(4 * kWave);
  auto n_wg = [&](int tt, int te) { return static_cast<unsigned>(cdiv(T, tt) * cdiv(E, te)); };
  if (T > 0 && staged && (T >= kSplitRouterMinT || E >= kSplitRouterMinE)) {
    // logits over (token block, expert block) workgroups staged through LDS,
    // then the top k per token; on small batches of few experts the second
    // launch would cost more than it saves (one workgroup per token below)
    if (E <= 8)                          // 8 tokens x 8 experts
      hipLaunchKernelGGL((route_logits_lds_kernel<2, 8, 256>), dim3(n_wg(8, 8)), blk, 0, s, x, T, d, w_router,
                         bias, E, logits);
    else if (n_wg(16, 16) >= 256)        // 16 tokens x 16 experts
      hipLaunchKernelGGL((route_logits_lds_kernel<4, 16, 256>), dim3(n_wg(16, 16)), blk, 0, s, x, T, d,
                         w_router, bias, E, logits);
    else                                 // small batches: 4 tokens x 8 experts, 1024-column chunks
      hipLaunchKernelGGL((route_logits_lds_kernel<1, 8, 1024>), dim3(n_wg(4, 8)), blk, 0, s, x, T, d, w_router,
                         bias, E, logits);
    hipLaunchKernelGGL(route_select_kernel, dim3(static_cast<unsigned>(cdiv(T, 4))), blk, 0, s, logits, T, E, k,
                       topk_ids, topk_w);
  } else if (T >= kSplitRouterMinT) {    // rows off 16-byte alignment: a column per lane
    hipLaunchKernelGGL((route_logits_kernel<kLogitTokens, 16>),
                       dim3(static_cast<unsigned>(cdiv(T, kLogitTokens)), static_cast<unsigned>(cdiv(E, kLogitExperts))),
                       dim3(kLogitWaves * kWave), 0, s, x, T, d, w_router, bias, E, logits);
    hipLaunchKernelGGL(route_select_kernel, dim3(static_cast<unsigned>(cdiv(T, 4))), blk, 0, s, logits, T, E, k,
                       topk_ids, topk_w);
  } else if (T > 0) {
    hipLaunchKernelGGL(route_topk_kernel, dim3(static_cast<unsigned>(T)), dim3(kRouteWaves * kWave),
                       0, s, x, T, d, w_router, bias, E, k, topk_ids, topk_w);
  }
  if (n_chunks <= kFusedChunks) {
    hipLaunchKernelGGL(route_permute_fused_kernel, dim3(1), dim3(kPermWaves * kWave), 0, s,
                       topk_ids, T, E, k, S, offsets, perm_token, inv_perm);
  } else {
    hipLaunchKernelGGL(route_hist_kernel, dim3(n_chunks), dim3(64), 0, s, topk_ids, T, E, k, hist);
    hipLaunchKernelGGL(route_scan_kernel, dim3(1), dim3(256), 0, s, hist, n_chunks, T, E, k, S,
                       base, offsets);
    hipLaunchKernelGGL(route_scatter_kernel, dim3(n_chunks), dim3(64), 0, s, topk_ids, T, E, k, S,
                       base, offsets, perm_token, inv_perm);
  }
  if (T > 0) {
    if (x_perm) {
      const int64_t rows = static_cast<int64_t>(T) * (k + S);
      const int64_t n = rows * (d / 8);
      hipLaunchKernelGGL(gather_rows_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256),
                         0, s, x, d, perm_token, static_cast<int>(rows), x_perm);
    }
  }
  return launch_status(s);
}
