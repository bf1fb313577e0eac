// ffn.hip -- moe_expert_ffn_mixed: the routed and shared expert FFNs of one
// MoE layer over per-expert mixed-precision packed weights (2/3/4/8-bit
// codes, fp16 scale and zero per group of `group` inputs), with the channel
// switch applied row by row.
//
// Sec. IV-A: every expert has its own precision.  Sec. IV-B / V-A: a switched
// row reads its cached 8-bit copy instead of its base codes.  Sec. V-B: the
// packed codes are loaded in wide words, unpacked on chip, dequantized and fed
// to the matrix cores in one fused kernel.
//
// Dequantization, MI355X style.  The codes are turned into bf16 integers
// without any multiply: for b <= 4 a code q is OR-ed into the mantissa of the
// bf16 constant 128.0, giving exactly 128 + q; 8-bit codes go through the
// byte-to-float converter and give q.  The matrix cores then contract these
// exact integers with the bf16 activations in fp32, one quantization group
// at a time, and the group's scale and zero point are applied to the fp32
// partial sum:  sum_c s (q_c - z) x_c = s * (P - (off + z) * X),
// P = sum_c (off + q_c) x_c from the MFMA, X = sum_c x_c over the group.
// The weight operand is therefore exact; the only rounding besides fp32
// accumulation is the bf16 hidden activation h.
//
// Work decomposition (one wave = 64 lanes):
//   - a wave owns 16*ROWT rows (neurons for gate/up, output channels for
//     down) of one expert and streams its packed rows through all groups of
//     K (down: one of n_split slices of K);
//   - lane (r16 = lane % 16, kq = lane / 16) loads the group codes
//     [kq*g/4, (kq+1)*g/4) of row r16 -- one 16-byte load at 4 bits -- and
//     the matching activations of token r16 of the current 16-token tile;
//   - v_mfma_f32_16x16x32_bf16 with A = activations (tokens) and
//     B = weights (rows) leaves each lane the results of its own row r16 for
//     tokens 4*kq .. 4*kq+3, so the lane applies its own row's scale/zero.
#include <algorithm>

#include "common.hpp"

namespace moe {
namespace {

constexpr int kRowT = 2;                 // 16-row tiles per wave
constexpr int kRowsPerWave = 16 * kRowT;
constexpr uint32_t kMagic = 0x43004300u;  // two bf16 128.0

struct KindDev {
  const uint32_t* codes;
  const uint32_t* sz;
  const int64_t* code_off;
  const int64_t* sz_off;
  const uint32_t* copy_codes;
  const uint32_t* copy_sz;
  const int32_t* row_slot;
};

struct FfnArgs {
  KindDev kd[3];
  const int32_t* bits;
  const int32_t* order_gu;
  const int32_t* order_dn;
  const uint16_t* x;
  const float* xsum;
  const int32_t* offsets;
  const int32_t* perm;
  uint16_t* h;
  float* hsum;
  float* o;
  int64_t split_stride;
  int E, S, d, f, fs, group;
  int Tk;  // routed rows T*k
};

// Row-offset of permuted row p in the h buffer (routed rows have d_ff
// columns, shared rows d_ff_shared).
__device__ __forceinline__ int64_t h_row(const FfnArgs& a, int p) {
  return p < a.Tk ? static_cast<int64_t>(p) * a.f
                  : static_cast<int64_t>(a.Tk) * a.f + static_cast<int64_t>(p - a.Tk) * a.fs;
}
__device__ __forceinline__ int64_t hs_row(const FfnArgs& a, int p) {
  return p < a.Tk ? static_cast<int64_t>(p) * (a.f / a.group)
                  : static_cast<int64_t>(a.Tk) * (a.f / a.group) +
                        static_cast<int64_t>(p - a.Tk) * (a.fs / a.group);
}

// Where one row's codes and {scale, zero} words live.
struct RowSrc {
  const uint32_t* row;  // first code word of the row
  const uint32_t* sz;   // {s16, z} word of group 0
  int sz_stride;        // words between consecutive groups
  int bits;
};

__device__ __forceinline__ RowSrc row_source(const KindDev& k, int e, bool routed, int R, int K,
                                             int bits_e, int row, int group) {
  RowSrc r;
  const int slot = routed ? k.row_slot[static_cast<int64_t>(e) * R + row] : -1;
  if (slot < 0) {
    r.row = k.codes + k.code_off[e] + static_cast<int64_t>(row) * (K * bits_e / 32);
    r.sz = k.sz + k.sz_off[e] + row;
    r.sz_stride = R;
    r.bits = bits_e;
  } else {
    r.row = k.copy_codes + static_cast<int64_t>(slot) * (K / 4);
    r.sz = k.copy_sz + static_cast<int64_t>(slot) * (K / group);
    r.sz_stride = 1;
    r.bits = 8;
  }
  return r;
}

// Load `nw` code words (nw in {1,2,3,4,8}) of this lane's share of a group.
__device__ __forceinline__ void load_chunk(uint32_t (&cw)[8], const uint32_t* p, int nw) {
  if (nw == 8) {
    const u32x4 a = reinterpret_cast<const u32x4*>(p)[0];
    const u32x4 b = reinterpret_cast<const u32x4*>(p)[1];
    cw[0] = a[0]; cw[1] = a[1]; cw[2] = a[2]; cw[3] = a[3];
    cw[4] = b[0]; cw[5] = b[1]; cw[6] = b[2]; cw[7] = b[3];
  } else if (nw == 4) {
    const u32x4 a = reinterpret_cast<const u32x4*>(p)[0];
    cw[0] = a[0]; cw[1] = a[1]; cw[2] = a[2]; cw[3] = a[3];
  } else if (nw == 3) {
    cw[0] = p[0]; cw[1] = p[1]; cw[2] = p[2];
  } else if (nw == 2) {
    const u32x2 a = reinterpret_cast<const u32x2*>(p)[0];
    cw[0] = a[0]; cw[1] = a[1];
  } else {
    cw[0] = p[0];
  }
}

__device__ __forceinline__ uint32_t pair8(uint32_t w, int hi) {
  // bytes (c0, c2, c1, c3) -> bf16 pair (c0, c1) or (c2, c3), exact integers
  const float a = hi ? static_cast<float>((w >> 8) & 0xFFu) : static_cast<float>(w & 0xFFu);
  const float b = hi ? static_cast<float>(w >> 24) : static_cast<float>((w >> 16) & 0xFFu);
  return (__float_as_uint(a) >> 16) | (__float_as_uint(b) & 0xFFFF0000u);
}

// Codes of one lane's group share -> NM MFMA operands of 8 bf16 integers
// each (128 + q for b <= 4, q for b = 8), in natural K order.
template <int NM>
__device__ __forceinline__ void dequant(const uint32_t (&cw)[8], int bits, u32x4 (&wf)[NM]) {
  if (bits == 4) {
#pragma unroll
    for (int m = 0; m < NM; m++) {
      const uint32_t w = cw[m];
      wf[m] = u32x4{(w & 0x000F000Fu) | kMagic, ((w >> 4) & 0x000F000Fu) | kMagic,
                    ((w >> 8) & 0x000F000Fu) | kMagic, ((w >> 12) & 0x000F000Fu) | kMagic};
    }
  } else if (bits == 2) {
#pragma unroll
    for (int m = 0; m < NM; m++) {
      const uint32_t w = cw[m >> 1] >> ((m & 1) * 8);
      wf[m] = u32x4{(w & 0x00030003u) | kMagic, ((w >> 2) & 0x00030003u) | kMagic,
                    ((w >> 4) & 0x00030003u) | kMagic, ((w >> 6) & 0x00030003u) | kMagic};
    }
  } else if (bits == 8) {
#pragma unroll
    for (int m = 0; m < NM; m++)
      wf[m] = u32x4{pair8(cw[2 * m], 0), pair8(cw[2 * m], 1), pair8(cw[2 * m + 1], 0),
                    pair8(cw[2 * m + 1], 1)};
  } else {  // 3-bit planes, NM == 4
#pragma unroll
    for (int m = 0; m < NM; m++) {
      uint32_t v[4];
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const int p = 4 * m + j;
        const uint32_t lo = (cw[p >> 3] >> (2 * (p & 7))) & 0x00030003u;
        const uint32_t hi = ((cw[2] >> p) & 0x00010001u) << 2;
        v[j] = lo | hi | kMagic;
      }
      wf[m] = u32x4{v[0], v[1], v[2], v[3]};
    }
  }
}

__device__ __forceinline__ float silu_mul(float g, float u) {
  return g / (1.0f + __expf(-g)) * u;
}

// ------------------------------------------------------------------ gate/up
template <int NM, int NT>
__global__ void __launch_bounds__(256)
ffn_gateup_kernel(FfnArgs a, int e_begin, int n_exp, int R) {
  constexpr int g = NM * 32;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int bpe = R / kRowsPerWave;
  if (wave >= n_exp * bpe) return;
  const int e = e_begin + wave / bpe;
  const int rb = wave % bpe;
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15;
  const int kq = lane >> 4;
  const int seg0 = a.offsets[e];
  const int seg1 = a.offsets[e + 1];
  if (seg1 <= seg0) return;
  const bool routed = e < a.E;
  const int K = a.d;
  const int G = K / g;
  const int be = a.bits[e];

  int nrn[kRowT];
  RowSrc src[kRowT][2];
#pragma unroll
  for (int rt = 0; rt < kRowT; rt++) {
    const int i = rb * kRowsPerWave + rt * 16 + r16;
    nrn[rt] = routed ? a.order_gu[static_cast<int64_t>(e) * R + i] : i;
#pragma unroll
    for (int kk = 0; kk < 2; kk++)
      src[rt][kk] = row_source(a.kd[kk], e, routed, R, K, be, nrn[rt], g);
  }

  for (int t0 = seg0; t0 < seg1; t0 += NT * 16) {
    int xrow[NT];
    int stok[NT][4];
#pragma unroll
    for (int nt = 0; nt < NT; nt++) {
      const int p = t0 + nt * 16 + r16;
      xrow[nt] = p < seg1 ? a.perm[p] : -1;
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int pi = t0 + nt * 16 + 4 * kq + i;
        stok[nt][i] = pi < seg1 ? a.perm[pi] : -1;
      }
    }
    f32x4 acc[kRowT][2][NT];
#pragma unroll
    for (int rt = 0; rt < kRowT; rt++)
#pragma unroll
      for (int kk = 0; kk < 2; kk++)
#pragma unroll
        for (int nt = 0; nt < NT; nt++) acc[rt][kk][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int gi = 0; gi < G; gi++) {
      u32x4 xf[NT][NM];
      float X[NT][4];
#pragma unroll
      for (int nt = 0; nt < NT; nt++) {
        if (xrow[nt] >= 0) {
          const u32x4* px = reinterpret_cast<const u32x4*>(
              a.x + static_cast<int64_t>(xrow[nt]) * K + gi * g + kq * (g / 4));
#pragma unroll
          for (int m = 0; m < NM; m++) xf[nt][m] = px[m];
        } else {
#pragma unroll
          for (int m = 0; m < NM; m++) xf[nt][m] = u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int i = 0; i < 4; i++)
          X[nt][i] = stok[nt][i] >= 0 ? a.xsum[static_cast<int64_t>(stok[nt][i]) * G + gi] : 0.f;
      }
#pragma unroll
      for (int rt = 0; rt < kRowT; rt++) {
#pragma unroll
        for (int kk = 0; kk < 2; kk++) {
          const RowSrc& s = src[rt][kk];
          const int nw = g * s.bits / 128;
          uint32_t cw[8];
          load_chunk(cw, s.row + gi * (g * s.bits / 32) + kq * nw, nw);
          const uint32_t szw = s.sz[static_cast<int64_t>(gi) * s.sz_stride];
          const float sc = fp16_bits_to_f32(szw & 0xFFFFu);
          const float zz = fp16_bits_to_f32(szw >> 16) + (s.bits == 8 ? 0.f : 128.f);
          u32x4 wf[NM];
          dequant<NM>(cw, s.bits, wf);
#pragma unroll
          for (int nt = 0; nt < NT; nt++) {
            f32x4 tmp = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int m = 0; m < NM; m++) tmp = mfma16(xf[nt][m], wf[m], tmp);
#pragma unroll
            for (int i = 0; i < 4; i++)
              acc[rt][kk][nt][i] =
                  __fmaf_rn(sc, __fmaf_rn(-zz, X[nt][i], tmp[i]), acc[rt][kk][nt][i]);
          }
        }
      }
    }
    // SiLU-GLU epilogue: h = bf16(silu(g) * u)
#pragma unroll
    for (int rt = 0; rt < kRowT; rt++)
#pragma unroll
      for (int nt = 0; nt < NT; nt++)
#pragma unroll
        for (int i = 0; i < 4; i++) {
          const int p = t0 + nt * 16 + 4 * kq + i;
          if (p < seg1) {
            const float hv = silu_mul(acc[rt][0][nt][i], acc[rt][1][nt][i]);
            a.h[h_row(a, p) + nrn[rt]] = static_cast<uint16_t>(bf16_rne(hv));
          }
        }
  }
}

// ------------------------------------------------------------------ down
template <int NM, int NT>
__global__ void __launch_bounds__(256)
ffn_down_kernel(FfnArgs a, int e_begin, int n_exp, int n_split) {
  constexpr int g = NM * 32;
  const int R = a.d;
  const int bpe = R / kRowsPerWave;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wave >= n_exp * bpe * n_split) return;
  const int sp = wave % n_split;
  const int rb = (wave / n_split) % bpe;
  const int e = e_begin + wave / (n_split * bpe);
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15;
  const int kq = lane >> 4;
  const int seg0 = a.offsets[e];
  const int seg1 = a.offsets[e + 1];
  if (seg1 <= seg0) return;
  const bool routed = e < a.E;
  const int K = routed ? a.f : a.fs;
  const int G = K / g;
  const int g0 = sp * G / n_split;
  const int g1 = (sp + 1) * G / n_split;
  const int be = a.bits[e];

  int ch[kRowT];
  RowSrc src[kRowT];
#pragma unroll
  for (int rt = 0; rt < kRowT; rt++) {
    const int i = rb * kRowsPerWave + rt * 16 + r16;
    ch[rt] = routed ? a.order_dn[static_cast<int64_t>(e) * R + i] : i;
    src[rt] = row_source(a.kd[2], e, routed, R, K, be, ch[rt], g);
  }
  float* out = a.o + static_cast<int64_t>(sp) * a.split_stride;

  for (int t0 = seg0; t0 < seg1; t0 += NT * 16) {
    int hrow[NT];
    int hsr[NT][4];
#pragma unroll
    for (int nt = 0; nt < NT; nt++) {
      const int p = t0 + nt * 16 + r16;
      hrow[nt] = p < seg1 ? p : -1;
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int pi = t0 + nt * 16 + 4 * kq + i;
        hsr[nt][i] = pi < seg1 ? pi : -1;
      }
    }
    f32x4 acc[kRowT][NT];
#pragma unroll
    for (int rt = 0; rt < kRowT; rt++)
#pragma unroll
      for (int nt = 0; nt < NT; nt++) acc[rt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int gi = g0; gi < g1; gi++) {
      u32x4 hf[NT][NM];
      float X[NT][4];
#pragma unroll
      for (int nt = 0; nt < NT; nt++) {
        if (hrow[nt] >= 0) {
          const u32x4* ph =
              reinterpret_cast<const u32x4*>(a.h + h_row(a, hrow[nt]) + gi * g + kq * (g / 4));
#pragma unroll
          for (int m = 0; m < NM; m++) hf[nt][m] = ph[m];
        } else {
#pragma unroll
          for (int m = 0; m < NM; m++) hf[nt][m] = u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int i = 0; i < 4; i++)
          X[nt][i] = hsr[nt][i] >= 0 ? a.hsum[hs_row(a, hsr[nt][i]) + gi] : 0.f;
      }
#pragma unroll
      for (int rt = 0; rt < kRowT; rt++) {
        const RowSrc& s = src[rt];
        const int nw = g * s.bits / 128;
        uint32_t cw[8];
        load_chunk(cw, s.row + gi * (g * s.bits / 32) + kq * nw, nw);
        const uint32_t szw = s.sz[static_cast<int64_t>(gi) * s.sz_stride];
        const float sc = fp16_bits_to_f32(szw & 0xFFFFu);
        const float zz = fp16_bits_to_f32(szw >> 16) + (s.bits == 8 ? 0.f : 128.f);
        u32x4 wf[NM];
        dequant<NM>(cw, s.bits, wf);
#pragma unroll
        for (int nt = 0; nt < NT; nt++) {
          f32x4 tmp = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int m = 0; m < NM; m++) tmp = mfma16(hf[nt][m], wf[m], tmp);
#pragma unroll
          for (int i = 0; i < 4; i++)
            acc[rt][nt][i] = __fmaf_rn(sc, __fmaf_rn(-zz, X[nt][i], tmp[i]), acc[rt][nt][i]);
        }
      }
    }
#pragma unroll
    for (int rt = 0; rt < kRowT; rt++)
#pragma unroll
      for (int nt = 0; nt < NT; nt++)
#pragma unroll
        for (int i = 0; i < 4; i++) {
          const int p = t0 + nt * 16 + 4 * kq + i;
          if (p < seg1) out[static_cast<int64_t>(p) * R + ch[rt]] = acc[rt][nt][i];
        }
  }
}

// ------------------------------------------------------------------ group sums
// out[r * G + j] = sum of the bf16 values in[r*ld + j*g .. +g) in fp32: each
// of g/8 lanes adds its 8 values in order, then an xor tree over those lanes.
template <int NM>
__global__ void __launch_bounds__(256)
group_sum_kernel(const uint16_t* __restrict__ in, int64_t ld, int rows, int K,
                 float* __restrict__ out) {
  constexpr int g = NM * 32;
  constexpr int lanes = g / 8;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int G = K / g;
  const int64_t n = static_cast<int64_t>(rows) * G * lanes;
  const bool live = id < n;
  const int64_t gid = id / lanes;
  const int q = static_cast<int>(id % lanes);
  float s = 0.f;
  if (live) {
    const int64_t r = gid / G;
    const int j = static_cast<int>(gid % G);
    const u32x4 v = *reinterpret_cast<const u32x4*>(in + r * ld + static_cast<int64_t>(j) * g + q * 8);
#pragma unroll
    for (int c = 0; c < 4; c++) {
      s = s + bf16_lo(v[c]);
      s = s + bf16_hi(v[c]);
    }
  }
#pragma unroll
  for (int off = lanes / 2; off >= 1; off >>= 1) s = s + __shfl_xor(s, off, kWave);
  if (live && q == 0) out[gid] = s;
}

size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

struct Plan {
  int n_split;
  int nt_routed, nt_shared;
  size_t xsum_bytes, h_bytes, hsum_bytes, total;
};

int pick_nt(double tokens) {
  if (tokens <= 12.0) return 1;
  if (tokens <= 28.0) return 2;
  return 4;
}

Plan make_plan(const moe_layer_t* L, int T, int k) {
  Plan p{};
  const int E = L->n_experts, S = L->n_shared, g = L->group;
  const int64_t Tk = static_cast<int64_t>(T) * k;
  const int64_t base_waves = static_cast<int64_t>(E + S) * (L->d_model / kRowsPerWave);
  const int fmin = S > 0 ? std::min(L->d_ff, L->d_ff_shared) : L->d_ff;
  const int gmin = fmin / g;
  int ns = static_cast<int>(cdiv(4096, std::max<int64_t>(base_waves, 1)));
  ns = std::min(ns, 8);
  ns = std::min(ns, std::max(1, gmin / 8));
  p.n_split = std::max(ns, 1);
  p.nt_routed = pick_nt(static_cast<double>(Tk) / E);
  p.nt_shared = pick_nt(static_cast<double>(T));
  const int64_t hcols = Tk * L->d_ff + static_cast<int64_t>(S) * T * L->d_ff_shared;
  p.xsum_bytes = align256(sizeof(float) * static_cast<size_t>(T) * (L->d_model / g));
  p.h_bytes = align256(sizeof(uint16_t) * static_cast<size_t>(hcols));
  p.hsum_bytes = align256(sizeof(float) * static_cast<size_t>(hcols / g));
  p.total = p.xsum_bytes + p.h_bytes + p.hsum_bytes + 256;
  return p;
}

int validate_layer(const moe_layer_t* L) {
  if (!L) return MOE_ERR_ARG;
  const int E = L->n_experts, S = L->n_shared;
  if (E <= 0 || S < 0 || E + S > MOE_MAX_EXPERTS) return MOE_ERR_ARG;
  if (!(L->group == 64 || L->group == 128)) return MOE_ERR_ARG;
  if (L->d_model <= 0 || L->d_model % 64 || L->d_model % L->group) return MOE_ERR_ARG;
  if (L->d_ff <= 0 || L->d_ff % L->group || L->d_ff % kRowsPerWave) return MOE_ERR_ARG;
  if (S > 0 && (L->d_ff_shared <= 0 || L->d_ff_shared % L->group ||
                L->d_ff_shared % kRowsPerWave))
    return MOE_ERR_ARG;
  if (!L->bits || !L->bits_host || !L->order_gu || !L->order_dn) return MOE_ERR_ARG;
  for (int e = 0; e < E + S; e++) {
    if (!valid_bits(L->bits_host[e])) return MOE_ERR_BITS;
    if (L->bits_host[e] == 3 && L->group != 128) return MOE_ERR_ARG;
  }
  for (int kd = 0; kd < 3; kd++) {
    const moe_kind_desc_t& k = L->kind[kd];
    if (!k.codes || !k.sz || !k.code_off || !k.sz_off || !k.row_slot) return MOE_ERR_ARG;
    if (!aligned16(k.codes)) return MOE_ERR_ALIGN;
    if (k.n_slots < 0) return MOE_ERR_ARG;
    if (k.n_slots > 0) {
      if (!k.copy_codes || !k.copy_sz || !k.copy_hdr) return MOE_ERR_ARG;
      if (!aligned16(k.copy_codes)) return MOE_ERR_ALIGN;
    }
    if (k.code_off_host)
      for (int e = 0; e < E + S; e++)
        if (k.code_off_host[e] % 4) return MOE_ERR_ALIGN;
  }
  return MOE_OK;
}

template <int NM>
void launch_all(const FfnArgs& a, const Plan& p, int T, hipStream_t s) {
  const int E = a.E, S = a.S;
  // x group sums
  {
    const int64_t n = static_cast<int64_t>(T) * (a.d / (NM * 32)) * (NM * 4);
    hipLaunchKernelGGL(group_sum_kernel<NM>, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0,
                       s, a.x, static_cast<int64_t>(a.d), T, a.d, const_cast<float*>(a.xsum));
  }
  auto gateup = [&](int e0, int ne, int R, int nt) {
    const int64_t waves = static_cast<int64_t>(ne) * (R / kRowsPerWave);
    const dim3 grid(static_cast<unsigned>(cdiv(waves, 4)));
    if (nt == 1) hipLaunchKernelGGL((ffn_gateup_kernel<NM, 1>), grid, dim3(256), 0, s, a, e0, ne, R);
    else if (nt == 2) hipLaunchKernelGGL((ffn_gateup_kernel<NM, 2>), grid, dim3(256), 0, s, a, e0, ne, R);
    else hipLaunchKernelGGL((ffn_gateup_kernel<NM, 4>), grid, dim3(256), 0, s, a, e0, ne, R);
  };
  auto down = [&](int e0, int ne, int nt) {
    const int64_t waves = static_cast<int64_t>(ne) * (a.d / kRowsPerWave) * p.n_split;
    const dim3 grid(static_cast<unsigned>(cdiv(waves, 4)));
    if (nt == 1) hipLaunchKernelGGL((ffn_down_kernel<NM, 1>), grid, dim3(256), 0, s, a, e0, ne, p.n_split);
    else if (nt == 2) hipLaunchKernelGGL((ffn_down_kernel<NM, 2>), grid, dim3(256), 0, s, a, e0, ne, p.n_split);
    else hipLaunchKernelGGL((ffn_down_kernel<NM, 4>), grid, dim3(256), 0, s, a, e0, ne, p.n_split);
  };
  gateup(0, E, a.f, p.nt_routed);
  if (S > 0) gateup(E, S, a.fs, p.nt_shared);
  // h group sums
  {
    const int64_t n = static_cast<int64_t>(a.Tk) * (a.f / (NM * 32)) * (NM * 4);
    if (n > 0)
      hipLaunchKernelGGL(group_sum_kernel<NM>, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256),
                         0, s, a.h, static_cast<int64_t>(a.f), a.Tk, a.f, a.hsum);
    if (S > 0) {
      const int rows = S * T;
      const int64_t n2 = static_cast<int64_t>(rows) * (a.fs / (NM * 32)) * (NM * 4);
      hipLaunchKernelGGL(group_sum_kernel<NM>, dim3(static_cast<unsigned>(cdiv(n2, 256))), dim3(256),
                         0, s, a.h + static_cast<int64_t>(a.Tk) * a.f, static_cast<int64_t>(a.fs),
                         rows, a.fs, a.hsum + static_cast<int64_t>(a.Tk) * (a.f / (NM * 32)));
    }
  }
  down(0, E, p.nt_routed);
  if (S > 0) down(E, S, p.nt_shared);
}

}  // namespace
}  // namespace moe

extern "C" int moe_ffn_plan(const moe_layer_t* L, int32_t T, int32_t k, int32_t* n_split,
                            size_t* ws_bytes) {
  using namespace moe;
  const int st = validate_layer(L);
  if (st != MOE_OK) return st;
  if (T < 0 || k < 1 || k > L->n_experts) return MOE_ERR_ARG;
  const Plan p = make_plan(L, T, k);
  if (n_split) *n_split = p.n_split;
  if (ws_bytes) *ws_bytes = p.total;
  return MOE_OK;
}

extern "C" int moe_expert_ffn_mixed(const moe_layer_t* L, const uint16_t* x, int32_t T, int32_t k,
                                    const int32_t* offsets, const int32_t* perm_token, float* o,
                                    void* ws, size_t ws_bytes, void* stream) {
  using namespace moe;
  int st = validate_layer(L);
  if (st != MOE_OK) return st;
  if (T < 0 || k < 1 || k > L->n_experts || k > MOE_MAX_TOPK) return MOE_ERR_ARG;
  if (T == 0) return MOE_OK;
  if (!x || !offsets || !perm_token || !o) return MOE_ERR_ARG;
  if (!aligned16(x) || !aligned16(o)) return MOE_ERR_ALIGN;
  const Plan p = make_plan(L, T, k);
  if (!ws || ws_bytes < p.total) return MOE_ERR_WORKSPACE;
  FfnArgs a{};
  for (int kd = 0; kd < 3; kd++) {
    const moe_kind_desc_t& kk = L->kind[kd];
    a.kd[kd] = KindDev{kk.codes, kk.sz, kk.code_off, kk.sz_off, kk.copy_codes, kk.copy_sz, kk.row_slot};
  }
  a.bits = L->bits;
  a.order_gu = L->order_gu;
  a.order_dn = L->order_dn;
  a.x = x;
  a.offsets = offsets;
  a.perm = perm_token;
  a.E = L->n_experts;
  a.S = L->n_shared;
  a.d = L->d_model;
  a.f = L->d_ff;
  a.fs = L->n_shared > 0 ? L->d_ff_shared : L->group * 2;
  a.group = L->group;
  a.Tk = T * k;
  char* w = static_cast<char*>(ws);
  w = reinterpret_cast<char*>((reinterpret_cast<uintptr_t>(w) + 255) & ~static_cast<uintptr_t>(255));
  a.xsum = reinterpret_cast<float*>(w);
  a.h = reinterpret_cast<uint16_t*>(w + p.xsum_bytes);
  a.hsum = reinterpret_cast<float*>(w + p.xsum_bytes + p.h_bytes);
  a.o = o;
  a.split_stride = static_cast<int64_t>(T) * (k + L->n_shared) * L->d_model;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (L->group == 128)
    launch_all<4>(a, p, T, s);
  else
    launch_all<2>(a, p, T, s);
  return launch_status(s);
}
