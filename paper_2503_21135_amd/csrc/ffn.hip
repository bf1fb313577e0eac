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
#include <type_traits>

#include "common.hpp"

namespace moe {
namespace {

constexpr int kRowsPerWG = 128;          // rows of one kind per workgroup (64 at NT = 4)
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
  const int32_t* n_base;
  const uint16_t* x;
  const float* xsum;   // [d/g][rows] group sums of the gathered x rows
  const int32_t* offsets;
  const int32_t* perm;
  uint16_t* h;
  float* hsum;         // [max(f,fs)/g][rows] group sums of h rows
  float* o;
  int64_t split_stride;
  int E, S, d, f, fs, group;
  int Tk;    // routed rows T*k
  int rows;  // all permuted rows T*(k+S)
};

// Experts in the order their waves are launched (most bytes first).
struct Sched {
  int16_t e[MOE_MAX_EXPERTS];
};

// Row-offset of permuted row p in the h buffer (routed rows have d_ff
// columns, shared rows d_ff_shared).
__device__ __forceinline__ int64_t h_row(const FfnArgs& a, int p) {
  return p < a.Tk ? static_cast<int64_t>(p) * a.f
                  : static_cast<int64_t>(a.Tk) * a.f + static_cast<int64_t>(p - a.Tk) * a.fs;
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
template <int NW>
__device__ __forceinline__ void load_words(uint32_t (&cw)[NW], const uint32_t* p) {
  if constexpr (NW == 8) {
    const u32x4 a = reinterpret_cast<const u32x4*>(p)[0];
    const u32x4 b = reinterpret_cast<const u32x4*>(p)[1];
    cw[0] = a[0]; cw[1] = a[1]; cw[2] = a[2]; cw[3] = a[3];
    cw[4] = b[0]; cw[5] = b[1]; cw[6] = b[2]; cw[7] = b[3];
  } else if constexpr (NW == 4) {
    const u32x4 a = reinterpret_cast<const u32x4*>(p)[0];
    cw[0] = a[0]; cw[1] = a[1]; cw[2] = a[2]; cw[3] = a[3];
  } else if constexpr (NW == 2) {
    const u32x2 a = reinterpret_cast<const u32x2*>(p)[0];
    cw[0] = a[0]; cw[1] = a[1];
  } else {
#pragma unroll
    for (int i = 0; i < NW; i++) cw[i] = p[i];
  }
}

__device__ __forceinline__ void load_chunk(uint32_t (&cw)[8], const uint32_t* p, int nw) {
  if (nw == 8) {
    uint32_t t[8];
    load_words<8>(t, p);
#pragma unroll
    for (int i = 0; i < 8; i++) cw[i] = t[i];
  } else if (nw == 4) {
    uint32_t t[4];
    load_words<4>(t, p);
#pragma unroll
    for (int i = 0; i < 4; i++) cw[i] = t[i];
  } else if (nw == 3) {
    cw[0] = p[0]; cw[1] = p[1]; cw[2] = p[2];
  } else if (nw == 2) {
    uint32_t t[2];
    load_words<2>(t, p);
    cw[0] = t[0]; cw[1] = t[1];
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
template <int B, int NM, int NW>
__device__ __forceinline__ void dequant_b(const uint32_t (&cw)[NW], u32x4 (&wf)[NM]) {
  if constexpr (B == 4) {
#pragma unroll
    for (int m = 0; m < NM; m++) {
      const uint32_t w = cw[m];
      wf[m] = u32x4{(w & 0x000F000Fu) | kMagic, ((w >> 4) & 0x000F000Fu) | kMagic,
                    ((w >> 8) & 0x000F000Fu) | kMagic, ((w >> 12) & 0x000F000Fu) | kMagic};
    }
  } else if constexpr (B == 2) {
#pragma unroll
    for (int m = 0; m < NM; m++) {
      const uint32_t w = cw[m >> 1] >> ((m & 1) * 8);
      wf[m] = u32x4{(w & 0x00030003u) | kMagic, ((w >> 2) & 0x00030003u) | kMagic,
                    ((w >> 4) & 0x00030003u) | kMagic, ((w >> 6) & 0x00030003u) | kMagic};
    }
  } else if constexpr (B == 8) {
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

template <int NM>
__device__ __forceinline__ void dequant_rt(const uint32_t (&cw)[8], int bits, u32x4 (&wf)[NM]) {
  if (bits == 4) {
    uint32_t t[NM];
#pragma unroll
    for (int i = 0; i < NM; i++) t[i] = cw[i];
    dequant_b<4, NM, NM>(t, wf);
  } else if (bits == 2) {
    uint32_t t[NM / 2];
#pragma unroll
    for (int i = 0; i < NM / 2; i++) t[i] = cw[i];
    dequant_b<2, NM, NM / 2>(t, wf);
  } else if (bits == 8) {
    uint32_t t[2 * NM];
#pragma unroll
    for (int i = 0; i < 2 * NM; i++) t[i] = cw[i];
    dequant_b<8, NM, 2 * NM>(t, wf);
  } else {
    if constexpr (NM == 4) {
      uint32_t t[3] = {cw[0], cw[1], cw[2]};
      dequant_b<3, NM, 3>(t, wf);
    }
  }
}

__device__ __forceinline__ float silu_mul(float g, float u) {
  return g / (1.0f + __expf(-g)) * u;
}

// ------------------------------------------------------------------ streaming kernel
// One workgroup = 4 waves on one expert.  Each wave owns 16*RT consecutive
// positions of the expert's row order for each of NK weight kinds (NK = 2:
// the gate and up rows of the same neurons; NK = 1: down rows = output
// channels) and streams their packed codes through registers; the
// activations of the workgroup's token tile (NT*16 rows) are staged in LDS
// two groups at a time (double-buffered, one barrier per chunk), so every
// wave reads them from LDS rather than L2.  The codes of the next group are
// in flight while the current group is dequantized and contracted.
//
// Two passes cover an expert's rows: the base pass takes the leading rows of
// the order whose sources are all base codes (bit-width B of the expert, code
// registers sized for B); the switched pass takes the rest, each lane reading
// its own source (base codes or an 8-bit copy) at its own width.

constexpr int kWaves = 4;

// Workgroups [first[i], first[i+1]) of a launch serve expert e[i].
// Entry i is expert e[i] in the switched pass when sw[i] != 0, in the base
// pass otherwise.
struct WgMap {
  int n;
  int32_t first[2 * MOE_MAX_EXPERTS + 1];
  int16_t e[2 * MOE_MAX_EXPERTS];
  int8_t sw[2 * MOE_MAX_EXPERTS];
};

__device__ __forceinline__ int map_find(const WgMap& m, int wg) {
  int lo = 0, hi = m.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (m.first[mid] <= wg) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// B > 0: all rows read B-bit codes.  B == 0: per-lane width (<= 8 words).
template <int NM, int B>
struct CodeWords {
  static constexpr int value = B == 0 ? 8 : NM * B / 4;
};

template <int NM, int RT, int NK, int B>
struct CodeStage {
  uint32_t cw[RT][NK][CodeWords<NM, B>::value];
  uint32_t szw[RT][NK];
};

// Where the rows of one kind live for a wave.  B > 0: every row reads its
// expert's base codes, so the bases are wave-uniform and each lane keeps
// 32-bit offsets; B == 0: each lane keeps its own full source.
template <int RT, int NK, int B>
struct Rows {
  const uint32_t* cbase[NK];   // B > 0: codes of the expert
  const uint32_t* sbase[NK];   // B > 0: {scale, zero} words of the expert
  uint32_t coff[RT][NK];       // B > 0: word offset of the lane's row
  uint32_t soff[RT][NK];       // B > 0: offset of the lane's row, group 0
  int sstride;                 // B > 0: rows of the expert (group stride)
  RowSrc src[B == 0 ? RT : 1][B == 0 ? NK : 1];  // B == 0
};

template <int NM, int RT, int NK, int B>
__device__ __forceinline__ void load_stage(CodeStage<NM, RT, NK, B>& st, const Rows<RT, NK, B>& rw,
                                           const bool (&live)[RT], int gi, int kq) {
  constexpr int g = NM * 32;
  constexpr int NW = CodeWords<NM, B>::value;
#pragma unroll
  for (int rt = 0; rt < RT; rt++)
#pragma unroll
    for (int kk = 0; kk < NK; kk++) {
      if (!live[rt]) {
#pragma unroll
        for (int w = 0; w < NW; w++) st.cw[rt][kk][w] = 0u;
        st.szw[rt][kk] = 0u;
        continue;
      }
      if constexpr (B == 0) {
        const RowSrc& s = rw.src[rt][kk];
        const int nw = g * s.bits / 128;
        load_chunk(st.cw[rt][kk], s.row + gi * (g * s.bits / 32) + kq * nw, nw);
        st.szw[rt][kk] = s.sz[static_cast<int64_t>(gi) * s.sz_stride];
      } else {
        load_words<NW>(st.cw[rt][kk], rw.cbase[kk] + rw.coff[rt][kk] + gi * (g * B / 32) + kq * NW);
        st.szw[rt][kk] = rw.sbase[kk][rw.soff[rt][kk] + static_cast<uint32_t>(gi) * rw.sstride];
      }
    }
}

// Contract one group: A fragments (activations) come from LDS.
//
// All MFMA chains of the group are issued first and their results are read
// only after an explicit wait: a matrix-core result must not be read by a
// VALU instruction before the MFMA has finished writing it, and the code
// around this loop has short control-flow paths on which the compiler's own
// wait-state insertion was observed to fall short (the last accumulator
// element was read stale).  The 3 x s_nop 7 (24 wait states) cover the
// longest 16x16x32 bf16 MFMA latency on gfx950.
template <int NM, int NT, int RT, int NK, int B>
__device__ __forceinline__ void compute_group(const CodeStage<NM, RT, NK, B>& st,
                                              const Rows<RT, NK, B>& rw,
                                              const u32x4 (&af)[NT][NM], const f32x4 (&X)[NT],
                                              f32x4 (&acc)[RT][NK][NT]) {
  f32x4 tmp[RT][NK][NT];
  float sc[RT][NK], zz[RT][NK];
#pragma unroll
  for (int rt = 0; rt < RT; rt++)
#pragma unroll
    for (int kk = 0; kk < NK; kk++) {
      u32x4 wf[NM];
      float off;
      if constexpr (B == 0) {
        const int bits = rw.src[rt][kk].bits;
        dequant_rt<NM>(st.cw[rt][kk], bits, wf);
        off = bits == 8 ? 0.f : 128.f;
      } else {
        dequant_b<B, NM, CodeWords<NM, B>::value>(st.cw[rt][kk], wf);
        off = B == 8 ? 0.f : 128.f;
      }
      sc[rt][kk] = fp16_bits_to_f32(st.szw[rt][kk] & 0xFFFFu);
      zz[rt][kk] = fp16_bits_to_f32(st.szw[rt][kk] >> 16) + off;
#pragma unroll
      for (int nt = 0; nt < NT; nt++) {
        f32x4 t = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < NM; m++) t = mfma16(af[nt][m], wf[m], t);
        tmp[rt][kk][nt] = t;
      }
    }
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int rt = 0; rt < RT; rt++)
#pragma unroll
    for (int kk = 0; kk < NK; kk++)
#pragma unroll
      for (int nt = 0; nt < NT; nt++)
#pragma unroll
        for (int i = 0; i < 4; i++)
          acc[rt][kk][nt][i] = __fmaf_rn(sc[rt][kk], __fmaf_rn(-zz[rt][kk], X[nt][i], tmp[rt][kk][nt][i]),
                                         acc[rt][kk][nt][i]);
}

template <int NM, int NT>
struct XTile {
  static constexpr int g = NM * 32;
  static constexpr int KC = 2 * g;   // K columns per LDS chunk (2 groups)
  static constexpr int TOK = NT * 16;
  static constexpr int LDW = KC + 8;  // row stride in bf16 (16-byte pad)
  uint16_t x[2][TOK][LDW];
  float xs[2][2][TOK];
};

// The expert's rows at order positions [pos0, pos1) (lanes past pos1 idle),
// token tile passes over the expert's segment, K groups [g0, g1) of split sp.
template <int NM, int NT, int RT, int NK, int B>
__device__ void stream_body(const FfnArgs& a, XTile<NM, NT>& tl, int e, int pos0, int pos1,
                            int R, int sp, int n_split) {
  constexpr int g = NM * 32;
  constexpr int KC = XTile<NM, NT>::KC;
  constexpr int TOK = XTile<NM, NT>::TOK;
  constexpr int PIECES = TOK * KC / 8;   // 16-byte pieces per chunk
  constexpr int PPT = PIECES / 256;
  static_assert(PIECES % 256 == 0, "chunk must split evenly over the workgroup");
  const int tid = threadIdx.x;
  const int wv = tid >> 6;
  const int lane = tid & 63;
  const int r16 = lane & 15;
  const int kq = lane >> 4;
  const int seg0 = a.offsets[e];
  const int seg1 = a.offsets[e + 1];
  const bool routed = e < a.E;
  const bool down = NK == 1;
  const int K = down ? (routed ? a.f : a.fs) : a.d;
  const int G = K / g;
  const int g0 = sp * G / n_split;
  const int g1 = (sp + 1) * G / n_split;
  const int be = a.bits[e];
  const KindDev* kinds = down ? &a.kd[2] : &a.kd[0];
  const int32_t* order = down ? a.order_dn : a.order_gu;
  const float* xsum = down ? a.hsum : a.xsum;

  int row_id[RT];
  bool live[RT];
  Rows<RT, NK, B> rw;
  rw.sstride = R;
#pragma unroll
  for (int kk = 0; kk < NK; kk++) {
    rw.cbase[kk] = kinds[kk].codes + kinds[kk].code_off[e];
    rw.sbase[kk] = kinds[kk].sz + kinds[kk].sz_off[e];
  }
#pragma unroll
  for (int rt = 0; rt < RT; rt++) {
    const int pos = pos0 + wv * 16 * RT + rt * 16 + r16;
    live[rt] = pos < pos1;
    row_id[rt] = live[rt] ? (routed ? order[static_cast<int64_t>(e) * R + pos] : pos) : 0;
#pragma unroll
    for (int kk = 0; kk < NK; kk++) {
      if constexpr (B == 0) {
        rw.src[rt][kk] = row_source(kinds[kk], e, routed, R, K, be, row_id[rt], g);
      } else {
        rw.coff[rt][kk] = static_cast<uint32_t>(row_id[rt]) * static_cast<uint32_t>(K * B / 32);
        rw.soff[rt][kk] = static_cast<uint32_t>(row_id[rt]);
      }
    }
  }

  for (int t0 = seg0; t0 < seg1; t0 += TOK) {
    // piece q = tid + 256*i of a chunk: token row q / (KC/8), column (q % (KC/8))*8
    uint32_t arow[PPT];   // element offset of the row, 0xFFFFFFFF when absent
#pragma unroll
    for (int i = 0; i < PPT; i++) {
      const int p = t0 + (tid + 256 * i) / (KC / 8);
      arow[i] = p < seg1 ? static_cast<uint32_t>(down ? h_row(a, p)
                                                      : static_cast<int64_t>(a.perm[p]) * K)
                         : 0xFFFFFFFFu;
    }
    const uint16_t* abase = down ? a.h : a.x;
    const int acol = (tid % (KC / 8)) * 8;   // same column for every piece of a thread
    auto stage_x = [&](u32x4 (&v)[PPT], float& xsv, int gc) {
      const bool in_k = gc + acol / g < g1;   // the chunk's second group may not exist
#pragma unroll
      for (int i = 0; i < PPT; i++)
        v[i] = (arow[i] != 0xFFFFFFFFu && in_k)
                   ? *reinterpret_cast<const u32x4*>(abase + arow[i] + gc * g + acol)
                   : u32x4{0u, 0u, 0u, 0u};
      xsv = 0.f;
      if (tid < 2 * TOK) {
        const int gg = tid / TOK, j = tid % TOK;
        if (gc + gg < g1 && t0 + j < seg1)
          xsv = xsum[static_cast<int64_t>(gc + gg) * a.rows + t0 + j];
      }
    };
    auto write_x = [&](const u32x4 (&v)[PPT], float xsv, int buf) {
#pragma unroll
      for (int i = 0; i < PPT; i++)
        *reinterpret_cast<u32x4*>(&tl.x[buf][(tid + 256 * i) / (KC / 8)][acol]) = v[i];
      if (tid < 2 * TOK) tl.xs[buf][tid / TOK][tid % TOK] = xsv;
    };

    f32x4 acc[RT][NK][NT];
#pragma unroll
    for (int rt = 0; rt < RT; rt++)
#pragma unroll
      for (int kk = 0; kk < NK; kk++)
#pragma unroll
        for (int nt = 0; nt < NT; nt++) acc[rt][kk][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    CodeStage<NM, RT, NK, B> s0, s1;
    load_stage(s0, rw, live, g0, kq);
    if (g0 + 1 < g1) load_stage(s1, rw, live, g0 + 1, kq);
    {
      u32x4 v[PPT];
      float xsv;
      stage_x(v, xsv, g0);
      write_x(v, xsv, 0);
    }
    __syncthreads();
    int buf = 0;
    for (int gc = g0; gc < g1; gc += 2) {
      const bool more = gc + 2 < g1;
      u32x4 vn[PPT];
      float xsn = 0.f;
      if (more) stage_x(vn, xsn, gc + 2);
#pragma unroll
      for (int gg = 0; gg < 2; gg++) {
        if (gc + gg >= g1) break;
        u32x4 af[NT][NM];
        f32x4 X[NT];
#pragma unroll
        for (int nt = 0; nt < NT; nt++) {
#pragma unroll
          for (int m = 0; m < NM; m++)
            af[nt][m] = *reinterpret_cast<const u32x4*>(
                &tl.x[buf][nt * 16 + r16][gg * g + kq * (g / 4) + 8 * m]);
          X[nt] = *reinterpret_cast<const f32x4*>(&tl.xs[buf][gg][nt * 16 + 4 * kq]);
        }
        if (gg == 0) {
          compute_group<NM, NT, RT, NK, B>(s0, rw, af, X, acc);
          if (gc + 2 < g1) load_stage(s0, rw, live, gc + 2, kq);
        } else {
          compute_group<NM, NT, RT, NK, B>(s1, rw, af, X, acc);
          if (gc + 3 < g1) load_stage(s1, rw, live, gc + 3, kq);
        }
      }
      if (more) write_x(vn, xsn, buf ^ 1);
      __syncthreads();
      buf ^= 1;
    }

    if constexpr (NK == 2) {
      // SiLU-GLU epilogue: h = bf16(silu(g) * u)
#pragma unroll
      for (int rt = 0; rt < RT; rt++)
#pragma unroll
        for (int nt = 0; nt < NT; nt++)
#pragma unroll
          for (int i = 0; i < 4; i++) {
            const int p = t0 + nt * 16 + 4 * kq + i;
            if (live[rt] && p < seg1) {
              const float hv = silu_mul(acc[rt][0][nt][i], acc[rt][1][nt][i]);
              a.h[h_row(a, p) + row_id[rt]] = static_cast<uint16_t>(bf16_rne(hv));
            }
          }
    } else {
      float* out = a.o + static_cast<int64_t>(sp) * a.split_stride;
#pragma unroll
      for (int rt = 0; rt < RT; rt++)
#pragma unroll
        for (int nt = 0; nt < NT; nt++)
#pragma unroll
          for (int i = 0; i < 4; i++) {
            const int p = t0 + nt * 16 + 4 * kq + i;
            if (live[rt] && p < seg1) out[static_cast<int64_t>(p) * R + row_id[rt]] = acc[rt][0][nt][i];
          }
    }
  }
}

// Rows per workgroup of the base pass for an expert of bit-width B.
__host__ __device__ constexpr int base_rt(int B, int NT) { return (B == 8 || NT == 4) ? 1 : 2; }

// One launch serves both passes of a set of experts: the switched-pass
// workgroups come first in the grid (few, long, latency-bound), the base-pass
// workgroups fill the machine behind them.
template <int NM, int NT, int NK>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
ffn_stream_kernel(FfnArgs a, WgMap map, int n_split) {
  __shared__ __attribute__((aligned(16))) XTile<NM, NT> tl;
  const int wgi = blockIdx.x / n_split;
  const int sp = blockIdx.x % n_split;
  const int i = map_find(map, wgi);
  const int e = map.e[i];
  const int blk = wgi - map.first[i];
  if (a.offsets[e + 1] <= a.offsets[e]) return;
  const bool routed = e < a.E;
  const int R = NK == 1 ? a.d : (routed ? a.f : a.fs);
  const int nb = routed ? a.n_base[(NK == 1 ? a.E : 0) + e] : R;
  if (map.sw[i]) {
    // rows past n_base: per-lane sources, 64 positions per workgroup
    const int pos0 = nb + blk * kWaves * 16;
    if (pos0 >= R) return;
    const int pos1 = min(pos0 + kWaves * 16, R);
    stream_body<NM, NT, 1, NK, 0>(a, tl, e, pos0, pos1, R, sp, n_split);
    return;
  }
  const int B = a.bits[e];
  const int rows = kWaves * 16 * base_rt(B, NT);
  const int pos0 = blk * rows;
  if (pos0 >= nb) return;
  const int pos1 = min(pos0 + rows, nb);
  if (B == 8) {
    stream_body<NM, NT, base_rt(8, NT), NK, 8>(a, tl, e, pos0, pos1, R, sp, n_split);
  } else if (B == 4) {
    stream_body<NM, NT, base_rt(4, NT), NK, 4>(a, tl, e, pos0, pos1, R, sp, n_split);
  } else if (B == 2) {
    stream_body<NM, NT, base_rt(2, NT), NK, 2>(a, tl, e, pos0, pos1, R, sp, n_split);
  } else {
    if constexpr (NM == 4) stream_body<NM, NT, base_rt(3, NT), NK, 3>(a, tl, e, pos0, pos1, R, sp, n_split);
  }
}

// ------------------------------------------------------------------ group sums
// out[j * rows + p] = sum over group j of the bf16 row of permuted row p, in
// fp32: each of g/8 lanes adds its 8 values in order, then an xor tree over
// those lanes.  The row of p starts at perm[p] * ld (gathered activations)
// or, with perm == NULL, at h_row(p) (hidden activations, K = that row's
// width).  Consecutive lane groups take consecutive p so the stores coalesce.
template <int NM>
__global__ void __launch_bounds__(256)
group_sum_kernel(FfnArgs a, const uint16_t* __restrict__ in, const int32_t* __restrict__ perm,
                 int64_t ld, int p0, int p1, int K, float* __restrict__ out) {
  constexpr int g = NM * 32;
  constexpr int lanes = g / 8;
  const int G = K / g;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t n = static_cast<int64_t>(p1 - p0) * G * lanes;
  const bool live = id < n;
  const int64_t item = id / lanes;
  const int q = static_cast<int>(id % lanes);
  const int np = p1 - p0;
  float s = 0.f;
  int p = 0, j = 0;
  if (live) {
    j = static_cast<int>(item / np);
    p = p0 + static_cast<int>(item % np);
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
  const int64_t rows = static_cast<int64_t>(T) * (k + S);
  const int64_t base_waves = static_cast<int64_t>(E + S) * (L->d_model / 32);
  const int fmin = S > 0 ? std::min(L->d_ff, L->d_ff_shared) : L->d_ff;
  const int fmax = S > 0 ? std::max(L->d_ff, L->d_ff_shared) : L->d_ff;
  const int gmin = fmin / g;
  int ns = static_cast<int>(cdiv(4096, std::max<int64_t>(base_waves, 1)));
  ns = std::min(ns, 8);
  ns = std::min(ns, std::max(1, gmin / 8));
  p.n_split = std::max(ns, 1);
  p.nt_routed = pick_nt(static_cast<double>(Tk) / E);
  p.nt_shared = pick_nt(static_cast<double>(T));
  const int64_t hcols = Tk * L->d_ff + static_cast<int64_t>(S) * T * L->d_ff_shared;
  p.xsum_bytes = align256(sizeof(float) * static_cast<size_t>(rows) * (L->d_model / g));
  p.h_bytes = align256(sizeof(uint16_t) * static_cast<size_t>(hcols));
  p.hsum_bytes = align256(sizeof(float) * static_cast<size_t>(rows) * (fmax / g));
  p.total = p.xsum_bytes + p.h_bytes + p.hsum_bytes + 256;
  return p;
}

int validate_layer(const moe_layer_t* L) {
  if (!L) return MOE_ERR_ARG;
  const int E = L->n_experts, S = L->n_shared;
  if (E <= 0 || S < 0 || E + S > MOE_MAX_EXPERTS) return MOE_ERR_ARG;
  if (!(L->group == 64 || L->group == 128)) return MOE_ERR_ARG;
  if (L->d_model <= 0 || L->d_model % kRowsPerWG || L->d_model % L->group) return MOE_ERR_ARG;
  if (L->d_ff <= 0 || L->d_ff % L->group || L->d_ff % kRowsPerWG) return MOE_ERR_ARG;
  if (S > 0 && (L->d_ff_shared <= 0 || L->d_ff_shared % L->group ||
                L->d_ff_shared % kRowsPerWG))
    return MOE_ERR_ARG;
  if (!L->bits || !L->bits_host || !L->order_gu || !L->order_dn || !L->n_base) return MOE_ERR_ARG;
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

// Work map of one launch.  Switched pass (routed experts only): enough
// 64-row workgroups for the copies an expert can have.  Base pass: routed
// experts widest bit-width first (their workgroups stream the most bytes),
// R / rows-per-workgroup workgroups each; or the shared experts.
WgMap stream_map(const moe_layer_t* L, bool shared, bool down, int nt) {
  WgMap m{};
  int n = 0, wg = 0;
  auto add = [&](int e, int n_wg, int sw) {
    if (n_wg <= 0) return;
    m.e[n] = static_cast<int16_t>(e);
    m.sw[n] = static_cast<int8_t>(sw);
    m.first[n] = wg;
    wg += n_wg;
    n++;
  };
  const int E = L->n_experts;
  if (shared) {
    for (int i = 0; i < L->n_shared; i++) {
      const int e = E + i;
      const int R = down ? L->d_model : L->d_ff_shared;
      add(e, R / (kWaves * 16 * base_rt(L->bits_host[e], nt)), 0);
    }
  } else {
    const int R = down ? L->d_model : L->d_ff;
    int bound[MOE_MAX_EXPERTS] = {0};
    for (int kd = down ? 2 : 0; kd <= (down ? 2 : 1); kd++) {
      const moe_kind_desc_t& k = L->kind[kd];
      for (int s = 0; s < k.n_slots; s++) {
        const int e = k.copy_hdr_host ? k.copy_hdr_host[2 * s] : -1;
        if (e >= 0 && e < E) bound[e]++;
        else for (int x = 0; x < E; x++) bound[x] = R;   // headers unknown: any row
      }
    }
    for (int e = 0; e < E; e++)
      add(e, static_cast<int>(cdiv(std::min(R, bound[e]), kWaves * 16)), 1);
    for (int b : {8, 4, 3, 2})
      for (int e = 0; e < E; e++)
        if (L->bits_host[e] == b) add(e, R / (kWaves * 16 * base_rt(b, nt)), 0);
  }
  m.n = n;
  m.first[n] = wg;
  return m;
}

inline void mark(hipEvent_t* ev, int n_ev, int i, hipStream_t s) {
  if (ev && i < n_ev && ev[i]) (void)hipEventRecord(ev[i], s);
}

template <int NM>
void launch_all(const FfnArgs& a, const Plan& p, const moe_layer_t* L, int T, hipStream_t s,
                hipEvent_t* ev, int n_ev) {
  constexpr int g = NM * 32;
  const int S = a.S;
  mark(ev, n_ev, 0, s);
  {  // group sums of the gathered activations, [d/g][rows]
    const int64_t n = static_cast<int64_t>(a.rows) * (a.d / g) * (g / 8);
    hipLaunchKernelGGL(group_sum_kernel<NM>, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0,
                       s, a, a.x, a.perm, static_cast<int64_t>(a.d), 0, a.rows, a.d,
                       const_cast<float*>(a.xsum));
  }
  mark(ev, n_ev, 1, s);
  auto stream = [&](auto nk, const WgMap& m, int nt, int nsplit) {
    constexpr int NK = decltype(nk)::value;
    if (m.n == 0 || m.first[m.n] == 0) return;
    const dim3 grid(static_cast<unsigned>(m.first[m.n] * nsplit));
    if (nt == 1) hipLaunchKernelGGL((ffn_stream_kernel<NM, 1, NK>), grid, dim3(256), 0, s, a, m, nsplit);
    else if (nt == 2) hipLaunchKernelGGL((ffn_stream_kernel<NM, 2, NK>), grid, dim3(256), 0, s, a, m, nsplit);
    else hipLaunchKernelGGL((ffn_stream_kernel<NM, 4, NK>), grid, dim3(256), 0, s, a, m, nsplit);
  };
  using two = std::integral_constant<int, 2>;
  using one = std::integral_constant<int, 1>;
  stream(two{}, stream_map(L, false, false, p.nt_routed), p.nt_routed, 1);
  if (S > 0) stream(two{}, stream_map(L, true, false, p.nt_shared), p.nt_shared, 1);
  mark(ev, n_ev, 2, s);
  {  // group sums of h, [max(f,fs)/g][rows]
    const int64_t n = static_cast<int64_t>(a.Tk) * (a.f / g) * (g / 8);
    if (n > 0)
      hipLaunchKernelGGL(group_sum_kernel<NM>, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256),
                         0, s, a, a.h, static_cast<const int32_t*>(nullptr), int64_t{0}, 0, a.Tk,
                         a.f, a.hsum);
    if (S > 0) {
      const int64_t n2 = static_cast<int64_t>(a.rows - a.Tk) * (a.fs / g) * (g / 8);
      hipLaunchKernelGGL(group_sum_kernel<NM>, dim3(static_cast<unsigned>(cdiv(n2, 256))), dim3(256),
                         0, s, a, a.h, static_cast<const int32_t*>(nullptr), int64_t{0}, a.Tk, a.rows,
                         a.fs, a.hsum);
    }
  }
  mark(ev, n_ev, 3, s);
  stream(one{}, stream_map(L, false, true, p.nt_routed), p.nt_routed, p.n_split);
  if (S > 0) stream(one{}, stream_map(L, true, true, p.nt_shared), p.nt_shared, p.n_split);
  mark(ev, n_ev, 4, s);
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

namespace moe {
namespace {
int ffn_entry(const moe_layer_t* L, const uint16_t* x, int32_t T, int32_t k,
              const int32_t* offsets, const int32_t* perm_token, float* o, void* ws,
              size_t ws_bytes, void* stream, void* const* events, int32_t n_events) {
  int st = validate_layer(L);
  if (st != MOE_OK) return st;
  if (T < 0 || k < 1 || k > L->n_experts || k > MOE_MAX_TOPK) return MOE_ERR_ARG;
  if (T == 0) return MOE_OK;
  if (!x || !offsets || !perm_token || !o) return MOE_ERR_ARG;
  if (!aligned16(x) || !aligned16(o)) return MOE_ERR_ALIGN;
  const Plan p = make_plan(L, T, k);
  if (!ws || ws_bytes < p.total) return MOE_ERR_WORKSPACE;
  {  // activation offsets are 32-bit inside the kernels
    const int64_t rows = static_cast<int64_t>(T) * (k + L->n_shared);
    const int64_t fmax = std::max<int64_t>(L->d_ff, L->n_shared > 0 ? L->d_ff_shared : 0);
    if (rows * fmax >= (int64_t{1} << 32) || static_cast<int64_t>(T) * L->d_model >= (int64_t{1} << 32))
      return MOE_ERR_ARG;
  }
  FfnArgs a{};
  for (int kd = 0; kd < 3; kd++) {
    const moe_kind_desc_t& kk = L->kind[kd];
    a.kd[kd] = KindDev{kk.codes, kk.sz, kk.code_off, kk.sz_off, kk.copy_codes, kk.copy_sz, kk.row_slot};
  }
  a.bits = L->bits;
  a.order_gu = L->order_gu;
  a.order_dn = L->order_dn;
  a.n_base = L->n_base;
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
  a.rows = T * (k + L->n_shared);
  char* w = static_cast<char*>(ws);
  w = reinterpret_cast<char*>((reinterpret_cast<uintptr_t>(w) + 255) & ~static_cast<uintptr_t>(255));
  a.xsum = reinterpret_cast<float*>(w);
  a.h = reinterpret_cast<uint16_t*>(w + p.xsum_bytes);
  a.hsum = reinterpret_cast<float*>(w + p.xsum_bytes + p.h_bytes);
  a.o = o;
  a.split_stride = static_cast<int64_t>(T) * (k + L->n_shared) * L->d_model;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipEvent_t* ev = reinterpret_cast<hipEvent_t*>(const_cast<void**>(events));
  if (L->group == 128)
    launch_all<4>(a, p, L, T, s, ev, n_events);
  else
    launch_all<2>(a, p, L, T, s, ev, n_events);
  return launch_status(s);
}
}  // namespace
}  // namespace moe

extern "C" int moe_expert_ffn_mixed(const moe_layer_t* L, const uint16_t* x, int32_t T, int32_t k,
                                    const int32_t* offsets, const int32_t* perm_token, float* o,
                                    void* ws, size_t ws_bytes, void* stream) {
  return moe::ffn_entry(L, x, T, k, offsets, perm_token, o, ws, ws_bytes, stream, nullptr, 0);
}

extern "C" int moe_expert_ffn_mixed_ev(const moe_layer_t* L, const uint16_t* x, int32_t T,
                                       int32_t k, const int32_t* offsets,
                                       const int32_t* perm_token, float* o, void* ws,
                                       size_t ws_bytes, void* stream, void* const* events,
                                       int32_t n_events) {
  if (n_events < 0 || (n_events > 0 && !events)) return MOE_ERR_ARG;
  return moe::ffn_entry(L, x, T, k, offsets, perm_token, o, ws, ws_bytes, stream, events,
                        n_events);
}
