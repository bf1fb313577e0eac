// ffn.hip -- moe_expert_ffn_mixed: the routed and shared expert FFNs of one
// MoE layer over per-expert mixed-precision packed weights (2/3/4/6/8-bit
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
#include <functional>
#include <type_traits>
#include <vector>

#include <hip/hip_ext.h>

#include "common.hpp"

namespace moe {
namespace {

constexpr int kRowsPerWG = 128;          // row counts must be multiples of this
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
  const int32_t* class_cnt;
  const uint16_t* x;
  const float* xsum;   // [d/g][rows] group sums of the gathered x rows
  const int32_t* offsets;
  const int32_t* perm;
  uint16_t* h;
  float* hsum;         // [max(f,fs)/g][rows] group sums of h rows
  float* o;
  int64_t split_stride;
  int n_split_out;     // slices of o the combine adds (tile launches zero the others)
  int32_t* tile_prefix;   // workspace: 4 x (MOE_MAX_EXPERTS + 1) item prefixes
  const uint16_t* x16;  // [T][d] fp16 copy of x (tile kernel; row of permuted row p: perm[p])
  uint32_t x_bytes, h_bytes, xsum_bytes, hsum_bytes, x16_bytes;   // resource sizes (< 2^31)
  uint32_t copy_bytes[3], copy_sz_bytes[3];
  int E, S, d, f, fs, group;
  int Tk;    // routed rows T*k
  int rows;  // all permuted rows T*(k+S)
};

// Row-offset of permuted row p in the h buffer (routed rows have d_ff
// columns, shared rows d_ff_shared).
__device__ __forceinline__ int64_t h_row(const FfnArgs& a, int p) {
  return p < a.Tk ? static_cast<int64_t>(p) * a.f
                  : static_cast<int64_t>(a.Tk) * a.f + static_cast<int64_t>(p - a.Tk) * a.fs;
}

// Dequantization into exact bf16 integers.  b <= 4: a code q OR-ed into the
// mantissa of bf16 128.0 gives 128 + q; one v_and_or_b32 per output register
// (two codes) after a shift.  The OR operand must sit in a vector register:
// an instruction with three operands cannot take two literal constants here,
// and with the constant as a literal the compiler splits the operation in
// two.  `vm` holds 0x43004300 (two bf16 128.0) in a vector register.
// 8-bit codes go through the byte-to-float converter (q exactly), and one
// byte permute takes the upper halves (the bf16 patterns) of two floats.
// 3-bit codes use two contractions: the 2-bit plane as 128 + lo and the
// 1-bit plane as 512 + 4*hi (vh = 0x44004400, bf16 512.0, whose mantissa
// step is 4), so the sum carries lo + 4*hi + 640.  6-bit codes likewise:
// the 4-bit plane as 128 + lo and the 2-bit plane as 2048 + 16*hi
// (vh = 0x45004500, bf16 2048.0, mantissa step 16), offset 2176.
template <int B>
constexpr int kPlanes = (B == 3 || B == 6) ? 2 : 1;

template <int B>
constexpr float kOffset = B == 8 ? 0.f : (B == 3 ? 640.f : (B == 6 ? 2176.f : 128.f));

// bf16 constant of the high plane of a two-plane width
template <int BG, int BU>
constexpr uint32_t kHighMagic = (BG == 6 || BU == 6) ? 0x45004500u : 0x44004400u;

__device__ __forceinline__ uint32_t andor(uint32_t x, uint32_t mask, uint32_t vm) {
  return (x & mask) | vm;
}

// byte i of w as an fp32 bit pattern (selected as v_cvt_f32_ubyte<i>)
__device__ __forceinline__ uint32_t ubyte_f32(uint32_t w, int i) {
  return __float_as_uint(static_cast<float>((w >> (8 * i)) & 0xFFu));
}

__device__ __forceinline__ uint32_t pair8(uint32_t lo_f32, uint32_t hi_f32) {
  // bf16 halves: low 16 bits <- upper half of lo_f32, high 16 <- upper half of hi_f32
  return __builtin_amdgcn_perm(hi_f32, lo_f32, 0x07060302u);
}

// Codes of one lane's group share -> NM MFMA operands of 8 bf16 integers
// each per plane, in natural K order.
template <int B, int NM, int NW>
__device__ __forceinline__ void dequant_b(const uint32_t (&cw)[NW], u32x4 (&wf)[kPlanes<B>][NM],
                                          uint32_t vm, uint32_t vh) {
  if constexpr (B == 4) {
#pragma unroll
    for (int m = 0; m < NM; m++) {
      const uint32_t w = cw[m];
      wf[0][m] = u32x4{andor(w, 0x000F000Fu, vm), andor(w >> 4, 0x000F000Fu, vm),
                       andor(w >> 8, 0x000F000Fu, vm), andor(w >> 12, 0x000F000Fu, vm)};
    }
  } else if constexpr (B == 2) {
#pragma unroll
    for (int m = 0; m < NM; m++) {
      const uint32_t w = cw[m >> 1];
      const int sh = (m & 1) * 8;
      wf[0][m] = u32x4{andor(w >> sh, 0x00030003u, vm), andor(w >> (sh + 2), 0x00030003u, vm),
                       andor(w >> (sh + 4), 0x00030003u, vm), andor(w >> (sh + 6), 0x00030003u, vm)};
    }
  } else if constexpr (B == 8) {
#pragma unroll
    for (int m = 0; m < NM; m++) {
      // bytes (c0, c2, c1, c3) of each word -> pairs (c0, c1), (c2, c3)
      const uint32_t w0 = cw[2 * m], w1 = cw[2 * m + 1];
      wf[0][m] = u32x4{pair8(ubyte_f32(w0, 0), ubyte_f32(w0, 2)), pair8(ubyte_f32(w0, 1), ubyte_f32(w0, 3)),
                       pair8(ubyte_f32(w1, 0), ubyte_f32(w1, 2)), pair8(ubyte_f32(w1, 1), ubyte_f32(w1, 3))};
    }
  } else if constexpr (B == 6) {  // per 32-code block: words 0-3 bits 0..3, words 4-5 bits 4..5
    static_assert(NM % 4 == 0, "6-bit shares are whole 32-code blocks");
#pragma unroll
    for (int m = 0; m < NM; m++) {
      const int blk = 6 * (m / 4);
      const uint32_t w = cw[blk + m % 4];
      const uint32_t h = cw[blk + 4 + (m % 4) / 2];
      const int sh = (m & 1) * 8;
      wf[0][m] = u32x4{andor(w, 0x000F000Fu, vm), andor(w >> 4, 0x000F000Fu, vm),
                       andor(w >> 8, 0x000F000Fu, vm), andor(w >> 12, 0x000F000Fu, vm)};
      wf[1][m] = u32x4{andor(h >> sh, 0x00030003u, vh), andor(h >> (sh + 2), 0x00030003u, vh),
                       andor(h >> (sh + 4), 0x00030003u, vh), andor(h >> (sh + 6), 0x00030003u, vh)};
    }
  } else {  // 3-bit: per 32-code block, words 0/1 the 2-bit plane, word 2 the 1-bit plane
    static_assert(NM % 4 == 0, "3-bit shares are whole 32-code blocks");
#pragma unroll
    for (int m = 0; m < NM; m++) {
      const int blk = 3 * (m / 4);
      uint32_t lo[4], hi[4];
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const int p = 4 * (m % 4) + j;   // output register: block codes 2p, 2p+1
        lo[j] = andor(cw[blk + (p >> 3)] >> (2 * (p & 7)), 0x00030003u, vm);
        hi[j] = andor(cw[blk + 2] >> p, 0x00010001u, vh);
      }
      wf[0][m] = u32x4{lo[0], lo[1], lo[2], lo[3]};
      wf[1][m] = u32x4{hi[0], hi[1], hi[2], hi[3]};
    }
  }
}

__device__ __forceinline__ float silu_mul(float g, float u) {
  return g / (1.0f + __expf(-g)) * u;
}

// ------------------------------------------------------------------ buffer loads
// Every load of the streaming loop is a raw buffer load through a
// range-checked resource.  A lane whose offset lies past the resource reads
// zeros without touching memory, so dead rows, groups past the end of a K
// slice and padding tokens need no branch around their loads: the loop stays
// straight-line and the compiler's wait counts keep every prefetch stage in
// flight (a branch around a load makes it drain all outstanding loads).
constexpr uint32_t kOOB = 0x80000000u;   // past every resource: sizes are < 2^31

typedef __amdgpu_buffer_rsrc_t Rsrc;

// Values that are the same in every lane but were loaded from global memory
// live in vector registers; a buffer resource built from them would need a
// loop over lanes at every load.  These move such values to scalar registers.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint32_t uni(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(v)));
}
__device__ __forceinline__ int64_t uni(int64_t v) {
  const uint64_t u = static_cast<uint64_t>(v);
  const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(u)));
  const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(u >> 32)));
  return static_cast<int64_t>(lo | (hi << 32));
}

__device__ __forceinline__ Rsrc make_rsrc(const void* p, uint32_t bytes) {
  // word 3 = 0x00020000: 32-bit data format, raw (unswizzled) addressing
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}

// Loads at byte offset off + soff of resource r; the range check applies to
// `off`, so kOOB there reads zeros whatever the scalar offset `soff`.
__device__ __forceinline__ u32x4 bload4(Rsrc r, uint32_t off, uint32_t soff = 0) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, 0);
}

template <int NW>
__device__ __forceinline__ void bload(uint32_t (&cw)[NW], Rsrc r, uint32_t off, uint32_t soff) {
  if constexpr (NW == 12) {
#pragma unroll
    for (int c = 0; c < 3; c++) {
      const u32x4 a = bload4(r, off == kOOB ? kOOB : off + 16u * c, soff);
#pragma unroll
      for (int i = 0; i < 4; i++) cw[4 * c + i] = a[i];
    }
  } else if constexpr (NW == 16 || NW == 6) {
    // four 16-byte loads, or three 8-byte loads (12-byte shares are 8-byte aligned)
    constexpr int P = NW == 16 ? 4 : 2;
#pragma unroll
    for (int c = 0; c < NW / P; c++) {
      const uint32_t o = off == kOOB ? kOOB : off + 4u * P * c;
      if constexpr (P == 4) {
        const u32x4 a = bload4(r, o, soff);
#pragma unroll
        for (int i = 0; i < 4; i++) cw[4 * c + i] = a[i];
      } else {
        const auto a = __builtin_amdgcn_raw_buffer_load_b64(r, o, soff, 0);
        cw[2 * c] = a[0];
        cw[2 * c + 1] = a[1];
      }
    }
  } else if constexpr (NW == 8) {
    const u32x4 a = bload4(r, off, soff);
    const u32x4 b = bload4(r, off == kOOB ? kOOB : off + 16u, soff);
#pragma unroll
    for (int i = 0; i < 4; i++) {
      cw[i] = a[i];
      cw[4 + i] = b[i];
    }
  } else if constexpr (NW == 4) {
    const u32x4 a = bload4(r, off, soff);
#pragma unroll
    for (int i = 0; i < 4; i++) cw[i] = a[i];
  } else if constexpr (NW == 3) {
    const auto a = __builtin_amdgcn_raw_buffer_load_b96(r, off, soff, 0);
    cw[0] = a[0]; cw[1] = a[1]; cw[2] = a[2];
  } else if constexpr (NW == 2) {
    const auto a = __builtin_amdgcn_raw_buffer_load_b64(r, off, soff, 0);
    cw[0] = a[0]; cw[1] = a[1];
  } else {
    cw[0] = __builtin_amdgcn_raw_buffer_load_b32(r, off, soff, 0);
  }
}

// Vector-memory instructions bload<NW> issues.
template <int NW>
constexpr int kCodeLoads = NW == 16 ? 4 : ((NW == 6 || NW == 12) ? 3 : (NW == 8 ? 2 : 1));

// Direct-to-LDS load of 16 bytes per lane: lane l of the wave writes
// lds + 16*l (lds wave-uniform); a lane whose offset lies past the resource
// writes zeros.
__device__ __forceinline__ void lds_dma16(Rsrc r, void* lds, uint32_t off, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, off, soff, 0, 0);
}

// ------------------------------------------------------------------ streaming kernel
// One workgroup = kWavesOf<NK> waves on one expert and one source class of its rows.
// Each wave owns 16*RT consecutive positions of the expert's row order for
// each of NK weight kinds (NK = 2: the gate and up rows of the same neurons;
// NK = 1: down rows = output channels).  Within a class every kind has one
// source for all rows -- the expert's base codes at bit-width B, or the
// cached 8-bit copies -- so the loads are wave-uniform in shape and the code
// registers are sized for that width (template BG / BU).  The packed codes of
// the next kStages<BG, BU> groups are in flight in registers while the current group
// is dequantized and contracted; the activations of the workgroup's token
// tile (NT*16 rows) are staged in LDS two groups at a time (double-buffered,
// one barrier per two groups), so every wave reads them from LDS.

// Waves per workgroup: four for gate/up; eight for down, whose tile of
// activations (h) is then shared by twice the rows (measured: the down
// launch 7 % faster, gate/up not).
template <int NK>
constexpr int kWavesOf = NK == 1 ? 8 : 4;
// Groups of codes in flight per wave: four, or two when a kind streams 8- or
// 6-bit codes (about the same bytes in flight in half the registers).  The activations
// of chunk c+2 are loaded while chunk c is contracted, so that waiting for
// them (vector loads complete in order) never waits for a code load the loop
// does not already need: with two-group chunks that holds for up to four
// groups in flight.
template <int BG, int BU>
constexpr int kStages = (BG == 8 || BU == 8 || BG == 6 || BU == 6) ? 2 : 4;

// Work of one launch over experts e0 .. e0+n_e-1.  Every workgroup covers
// kWavesOf<NK>*16 row positions of one source class of one expert.  Workgroups
// [0, n_e*n_sw) take the switched classes (n_sw per expert, an upper bound
// on what its copies can need; those beyond the expert's actual class sizes
// exit at once); the rest take class 0, per_e workgroups per expert, experts
// in the order `order` (widest bit-width first).
struct WgMap {
  int e0, n_e;
  int n_sw;
  int per_e;
  int16_t order[MOE_MAX_EXPERTS];
  int8_t bits[MOE_MAX_EXPERTS];   // bits[e - e0]
};

// Metadata a workgroup loads in its prologue, all issued before any is
// waited for (a chain of dependent loads at the start of every workgroup
// costs more than the loads themselves).
struct Pre {
  int64_t code_off[2], sz_off[2];   // per kind of the launch
  int row0;                         // class 0: this lane's row of the order
  int tt, n_tt;                     // token tile of the workgroup, when the tiles are split over workgroups
};

template <int NM, int B>
constexpr int kWords = NM * B / 4;   // code words per lane per group

template <int NM, int RT, int BG, int BU>
struct Stage {
  uint32_t cg[RT][(kWords<NM, BG>)];
  uint32_t cu[RT][(kWords<NM, BU>)];   // unused for NK = 1
};

// Source of one kind for a workgroup: resources over the expert's codes and
// {scale, zero} words (or the copies), the per-group stride of the {s, z}
// words and the lane's byte offsets (kOOB for lanes past the rows of the
// class).  The per-group advance goes into the scalar offset of the loads.
template <int RT>
struct Src {
  Rsrc code, sz;
  uint32_t sz_gstride;     // bytes between consecutive groups' {s, z} words
  uint32_t coff[RT];       // byte offset of the lane's code share of group 0
  uint32_t soff[RT];       // byte offset of the row's {s, z} word of group 0
};

template <int NM, int B, int RT>
__device__ __forceinline__ void load_kind(uint32_t (&cw)[RT][(kWords<NM, B>)], const Src<RT>& s, int gi,
                                          bool gv) {
  constexpr uint32_t gcb = NM * 32 * B / 8;   // code bytes per row and group
  const uint32_t cadv = gv ? static_cast<uint32_t>(gi) * gcb : 0u;
#pragma unroll
  for (int rt = 0; rt < RT; rt++) bload<kWords<NM, B>>(cw[rt], s.code, gv ? s.coff[rt] : kOOB, cadv);
}

// {s, z} words of the four groups [gb, gb+4): lane (r16, kq) loads row r16's
// word of group gb + kq (zero past g1), one load per kind and row tile for
// four groups; each group then reads its word from lane r16 + 16*(g - gb).
template <int RT, int NK>
__device__ __forceinline__ void load_sz4(uint32_t (&szb)[RT][2], const Src<RT> (&src)[2], int gb, int g1,
                                         int kq) {
  const bool ok = gb + kq < g1;
#pragma unroll
  for (int kk = 0; kk < NK; kk++) {
    const uint32_t sadv = gb < g1 ? static_cast<uint32_t>(gb) * src[kk].sz_gstride : 0u;
#pragma unroll
    for (int rt = 0; rt < RT; rt++) {
      const uint32_t so = src[kk].soff[rt];
      const uint32_t voff = (ok && so != kOOB) ? so + static_cast<uint32_t>(kq) * src[kk].sz_gstride : kOOB;
      szb[rt][kk] = __builtin_amdgcn_raw_buffer_load_b32(src[kk].sz, voff, sadv, 0);
    }
  }
}

template <int NM, int RT, int NK, int BG, int BU>
__device__ __forceinline__ void load_stage(Stage<NM, RT, BG, BU>& st, const Src<RT> (&src)[2], int gi,
                                           bool gv) {
  load_kind<NM, BG, RT>(st.cg, src[0], gi, gv);
  if constexpr (NK == 2) load_kind<NM, BU, RT>(st.cu, src[1], gi, gv);
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
template <int NM, int NT, int Bk>
__device__ __forceinline__ void contract_kind(const uint32_t (&cw)[(kWords<NM, Bk>)], uint32_t szw,
                                              const u32x4 (&af)[NT][NM], uint32_t vm, uint32_t vh,
                                              f32x4 (&tmp)[NT], float& sc, float& zz) {
  u32x4 wf[kPlanes<Bk>][NM];
  dequant_b<Bk, NM, kWords<NM, Bk>>(cw, wf, vm, vh);
  sc = fp16_bits_to_f32(szw & 0xFFFFu);
  zz = fp16_bits_to_f32(szw >> 16) + kOffset<Bk>;
#pragma unroll
  for (int nt = 0; nt < NT; nt++) {
    f32x4 t = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < NM; m++)
#pragma unroll
      for (int pl = 0; pl < kPlanes<Bk>; pl++) t = mfma16(af[nt][m], wf[pl][m], t);
    tmp[nt] = t;
  }
}

template <int NM, int NT, int RT, int NK, int BG, int BU>
__device__ __forceinline__ void compute_group(const Stage<NM, RT, BG, BU>& st, const uint32_t (&szw)[RT][2],
                                              const u32x4 (&af)[NT][NM], const f32x4 (&X)[NT],
                                              uint32_t vm, uint32_t vh, f32x4 (&acc)[RT][NK][NT]) {
  f32x4 tmp[RT][NK][NT];
  float sc[RT][NK], zz[RT][NK];
#pragma unroll
  for (int rt = 0; rt < RT; rt++) {
    contract_kind<NM, NT, BG>(st.cg[rt], szw[rt][0], af, vm, vh, tmp[rt][0], sc[rt][0], zz[rt][0]);
    if constexpr (NK == 2)
      contract_kind<NM, NT, BU>(st.cu[rt], szw[rt][1], af, vm, vh, tmp[rt][1], sc[rt][1], zz[rt][1]);
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

// Groups per LDS chunk of activations.  (Four-group chunks halve the
// barriers but double the tile's LDS, which limits the occupancy of the
// down projection; two measured faster.)
constexpr int kChunk = 2;

template <int NM, int NT>
struct XTile {
  static constexpr int g = NM * 32;
  static constexpr int CG = kChunk;
  static constexpr int KC = CG * g;   // K columns per LDS chunk
  static constexpr int TOK = NT * 16;
  static constexpr int LDW = KC + 8;  // row stride in bf16 (16-byte pad)
  uint16_t x[2][TOK][LDW];
  float xs[2][CG][TOK];
};

// The rows at order positions [pos0, pos1) of expert e (lanes past pos1
// idle), class cls (bit kk set: kind kk reads the 8-bit copies), token tile
// passes over the expert's segment, K groups [g0, g1) of split sp.
template <int NM, int NT, int RT, int NK, int BG, int BU>
__device__ __forceinline__ void stream_body(const FfnArgs& a, XTile<NM, NT>& tl, const Pre& pre, int e,
                                            int cls, int pos0, int pos1, int R, int sp, int n_split) {
  constexpr int kThreads = 64 * kWavesOf<NK>;
  constexpr int g = NM * 32;
  constexpr int KC = XTile<NM, NT>::KC;
  constexpr int TOK = XTile<NM, NT>::TOK;
  constexpr int PIECES = TOK * KC / 8;   // 16-byte pieces per chunk
  constexpr int PPT = (PIECES + kThreads - 1) / kThreads;
  static_assert(PIECES % kThreads == 0 || PIECES < kThreads, "chunk must split evenly over the workgroup");
  constexpr int S = kStages<BG, BU>;
  constexpr int CG = XTile<NM, NT>::CG;
  static_assert((S == 2 || S == 4) && CG == 2, "the loop body below handles two two-group chunks");
  static_assert(CG * TOK <= kThreads, "one thread per group-sum entry of a chunk");
  const int tid = threadIdx.x;
  const int wv = tid >> 6;
  const int lane = tid & 63;
  const int r16 = lane & 15;
  const int kq = lane >> 4;
  const int seg0 = uni(a.offsets[e]);
  const int seg1 = uni(a.offsets[e + 1]);
  const bool routed = e < a.E;
  const bool down = NK == 1;
  const int K = down ? (routed ? a.f : a.fs) : a.d;
  const int G = K / g;
  const int g0 = sp * G / n_split;
  const int g1 = (sp + 1) * G / n_split;
  const int be = BG == BU ? BG : (cls == 1 ? BU : BG);   // the base width of the expert
  const int kind0 = down ? 2 : 0;
  const int32_t* order = down ? a.order_dn : a.order_gu;

  int row_id[RT];
  bool live[RT];
#pragma unroll
  for (int rt = 0; rt < RT; rt++) {
    const int pos = pos0 + wv * 16 * RT + rt * 16 + r16;
    live[rt] = pos < pos1;
    const int prow = (RT == 1 && cls == 0) ? pre.row0 : order[static_cast<int64_t>(e) * R + pos];
    row_id[rt] = live[rt] ? (routed ? prow : pos) : 0;
  }
  Src<RT> src[2];
#pragma unroll
  for (int kk = 0; kk < NK; kk++) {
    // scalar selects first, one resource each: a resource chosen by a branch
    // would be merged in vector registers and force a loop per load
    const KindDev& kd = a.kd[kind0 + kk];
    const bool copy = (cls >> kk) & 1;
    const uint32_t row_bytes = 4u * static_cast<uint32_t>(code_row_words(K, be));
    const uint32_t words = static_cast<uint32_t>(g) * be / 128;   // per lane per group
    const void* cptr = copy ? static_cast<const void*>(kd.copy_codes)
                            : static_cast<const void*>(kd.codes + uni(pre.code_off[kk]));
    const void* sptr = copy ? static_cast<const void*>(kd.copy_sz)
                            : static_cast<const void*>(kd.sz + uni(pre.sz_off[kk]));
    const uint32_t cbytes = copy ? a.copy_bytes[kind0 + kk] : static_cast<uint32_t>(R) * row_bytes;
    const uint32_t sbytes = copy ? a.copy_sz_bytes[kind0 + kk] : static_cast<uint32_t>(R) * G * 4u;
    Src<RT>& s = src[kk];
    s.code = make_rsrc(cptr, cbytes);
    s.sz = make_rsrc(sptr, sbytes);
    s.sz_gstride = copy ? 4u : static_cast<uint32_t>(R) * 4u;
#pragma unroll
    for (int rt = 0; rt < RT; rt++) {
      const int slot = (copy && live[rt]) ? kd.row_slot[static_cast<int64_t>(e) * R + row_id[rt]] : -1;
      const uint32_t c_base = live[rt] ? row_id[rt] * row_bytes + kq * words * 4u : kOOB;
      const uint32_t s_base = live[rt] ? row_id[rt] * 4u : kOOB;
      const uint32_t c_copy =
          slot >= 0 ? static_cast<uint32_t>(slot) * 4u * static_cast<uint32_t>(code_row_words(K, 8)) + kq * (g / 4)
                    : kOOB;
      const uint32_t s_copy = slot >= 0 ? static_cast<uint32_t>(slot) * G * 4u : kOOB;
      s.coff[rt] = copy ? c_copy : c_base;
      s.soff[rt] = copy ? s_copy : s_base;
    }
  }
  const float* xsum = down ? a.hsum : a.xsum;
  const Rsrc xr = make_rsrc(down ? a.h : a.x, down ? a.h_bytes : a.x_bytes);
  const Rsrc xsr = make_rsrc(xsum, down ? a.hsum_bytes : a.xsum_bytes);

  // token tiles pre.tt, pre.tt + n_tt, ... of the segment (all of them
  // when the launch has one workgroup set per row block)
  for (int t0 = seg0 + pre.tt * TOK; t0 < seg1; t0 += pre.n_tt * TOK) {
    // piece q = tid + kThreads*i of a chunk: token row q / (KC/8), column (q % (KC/8))*8
    uint32_t arow[PPT];   // byte offset of the token's row, kOOB when absent
#pragma unroll
    for (int i = 0; i < PPT; i++) {
      const int p = t0 + (tid + kThreads * i) / (KC / 8);
      arow[i] = p < seg1 && tid + kThreads * i < PIECES ? static_cast<uint32_t>(2 * (down ? h_row(a, p)
                                                          : static_cast<int64_t>(a.perm[p]) * K))
                         : kOOB;
    }
    const int acol = (tid % (KC / 8)) * 8;   // same column for every piece of a thread
#pragma unroll
    for (int i = 0; i < PPT; i++)
      if (arow[i] != kOOB) arow[i] += 2u * acol;
    const int xs_g = tid / TOK, xs_j = tid % TOK;   // xsum entry of threads < CG*TOK
    const uint32_t xs_off = tid < CG * TOK && t0 + xs_j < seg1
                                ? 4u * static_cast<uint32_t>(xs_g * a.rows + t0 + xs_j) : kOOB;
    // chunk [gc, gc+CG): the chunk's first column / group goes into the scalar offset
    auto stage_x = [&](u32x4 (&v)[PPT], float& xsv, int gc) {
      const bool live_c = gc < g1;
      const uint32_t xadv = live_c ? 2u * static_cast<uint32_t>(gc * g) : 0u;
      const uint32_t sadv = live_c ? 4u * static_cast<uint32_t>(gc * a.rows) : 0u;
      const bool in_k = gc + acol / g < g1;   // the chunk's later groups may not exist
#pragma unroll
      for (int i = 0; i < PPT; i++) v[i] = bload4(xr, in_k ? arow[i] : kOOB, xadv);
      const bool ok = gc + xs_g < g1;
      xsv = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xsr, ok ? xs_off : kOOB, sadv, 0));
    };
    auto write_x = [&](const u32x4 (&v)[PPT], float xsv, int buf) {
#pragma unroll
      for (int i = 0; i < PPT; i++)
        if (PIECES >= kThreads || tid < PIECES)
          *reinterpret_cast<u32x4*>(&tl.x[buf][(tid + kThreads * i) / (KC / 8)][acol]) = v[i];
      if (tid < CG * TOK) tl.xs[buf][xs_g][xs_j] = xsv;
    };

    f32x4 acc[RT][NK][NT];
#pragma unroll
    for (int rt = 0; rt < RT; rt++)
#pragma unroll
      for (int kk = 0; kk < NK; kk++)
#pragma unroll
        for (int nt = 0; nt < NT; nt++) acc[rt][kk][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // dequantization constants, kept in vector registers (see dequant_b)
    uint32_t vm = kMagic, vh = kHighMagic<BG, BU>;
    asm volatile("" : "+v"(vm), "+v"(vh));
    Stage<NM, RT, BG, BU> st[S];
#pragma unroll
    for (int s = 0; s < S; s++) load_stage<NM, RT, NK, BG, BU>(st[s], src, g0 + s, g0 + s < g1);
    u32x4 vx[CG == 2 ? 2 : 1][PPT];   // activations of the next chunk(s)
    float vxs[CG == 2 ? 2 : 1];
    uint32_t szc[RT][2], szn[RT][2];   // {s, z} words of this and the next four groups
    load_sz4<RT, NK>(szc, src, g0, g1, kq);
    stage_x(vx[0], vxs[0], g0);
    write_x(vx[0], vxs[0], 0);
    if constexpr (CG == 2) stage_x(vx[1], vxs[1], g0 + 2);
    __syncthreads();
    auto group = [&](Stage<NM, RT, BG, BU>& s, int buf, int gg, int gi, int i4) {
      if (gi < g1) {   // wave-uniform; the loads below are unconditional
        uint32_t szw[RT][2];
#pragma unroll
        for (int rt = 0; rt < RT; rt++)
#pragma unroll
          for (int kk = 0; kk < NK; kk++)
            szw[rt][kk] = static_cast<uint32_t>(__shfl(static_cast<int>(szc[rt][kk]), r16 + 16 * i4));
        u32x4 af[NT][NM];
        f32x4 X[NT];
#pragma unroll
        for (int nt = 0; nt < NT; nt++) {
#pragma unroll
          for (int m = 0; m < NM; m++)
            af[nt][m] = *reinterpret_cast<const u32x4*>(&tl.x[buf][nt * 16 + r16][gg * g + kq * (g / 4) + 8 * m]);
          X[nt] = *reinterpret_cast<const f32x4*>(&tl.xs[buf][gg][nt * 16 + 4 * kq]);
        }
        compute_group<NM, NT, RT, NK, BG, BU>(s, szw, af, X, vm, vh, acc);
      }
      load_stage<NM, RT, NK, BG, BU>(s, src, gi + S, gi + S < g1);
    };
    for (int gc = g0; gc < g1; gc += 4) {
#pragma unroll
      for (int c = 0; c < 2; c++) {   // chunk c of the iteration sits in LDS buffer c
        // vx[c] held chunk gc+2c (written to LDS already); reuse it for gc+2c+4
        stage_x(vx[c], vxs[c], gc + 2 * c + 4);
        group(st[(2 * c) % S], c, 0, gc + 2 * c, 2 * c);
        if (c == 0) load_sz4<RT, NK>(szn, src, gc + 4, g1, kq);
        group(st[(2 * c + 1) % S], c, 1, gc + 2 * c + 1, 2 * c + 1);
        write_x(vx[c ^ 1], vxs[c ^ 1], c ^ 1);   // chunk gc+2c+2, loaded one chunk ago
        __syncthreads();
      }
#pragma unroll
      for (int rt = 0; rt < RT; rt++)
#pragma unroll
        for (int kk = 0; kk < NK; kk++) szc[rt][kk] = szn[rt][kk];
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


template <int NM, int NT, int NK, int B>
__device__ __forceinline__ void dispatch_class(const FfnArgs& a, XTile<NM, NT>& tl, const Pre& pre, int e,
                                               int cls, int pos0, int pos1, int R, int sp, int n_split) {
  if constexpr (NK == 1) {
    if (cls == 0) stream_body<NM, NT, 1, 1, B, B>(a, tl, pre, e, 0, pos0, pos1, R, sp, n_split);
    else stream_body<NM, NT, 1, 1, 8, 8>(a, tl, pre, e, 1, pos0, pos1, R, sp, n_split);
  } else {
    if (cls == 0) stream_body<NM, NT, 1, 2, B, B>(a, tl, pre, e, 0, pos0, pos1, R, sp, n_split);
    else if (cls == 1) stream_body<NM, NT, 1, 2, 8, B>(a, tl, pre, e, 1, pos0, pos1, R, sp, n_split);
    else if (cls == 2) stream_body<NM, NT, 1, 2, B, 8>(a, tl, pre, e, 2, pos0, pos1, R, sp, n_split);
    else stream_body<NM, NT, 1, 2, 8, 8>(a, tl, pre, e, 3, pos0, pos1, R, sp, n_split);
  }
}

// One launch serves every class of a set of experts: the switched-class
// workgroups come first in the grid, then the class-0 workgroups, widest
// bit-width first.
template <int NM, int NT, int NK>
__global__ void __launch_bounds__(64 * kWavesOf<NK>) __attribute__((amdgpu_waves_per_eu(2)))
ffn_stream_kernel(FfnArgs a, WgMap map, int n_split, int n_tt) {
  __shared__ __attribute__((aligned(16))) XTile<NM, NT> tl;
  constexpr int rows = kWavesOf<NK> * 16;
  const int tt = blockIdx.x % n_tt;
  const int wgi = blockIdx.x / n_tt / n_split;
  const int sp = blockIdx.x / n_tt % n_split;
  const int n_swg = map.n_e * map.n_sw;
  int e, cls, blk;
  if (wgi < n_swg) {
    e = map.e0 + wgi / map.n_sw;
    blk = wgi % map.n_sw;
    cls = 0;
  } else {
    const int j = wgi - n_swg;
    e = map.e0 + map.order[j / map.per_e];
    blk = j % map.per_e;
    cls = 0;
  }
  const bool routed = e < a.E;
  const int R = NK == 1 ? a.d : (routed ? a.f : a.fs);
  const int kind0 = NK == 1 ? 2 : 0;
  // issue every metadata load of the workgroup before waiting for any of them
  const int32_t* ccp = a.class_cnt + (NK == 1 ? 4 * a.E : 0) + 4 * (routed ? e : 0);
  const int o0 = a.offsets[e], o1 = a.offsets[e + 1];
  int cnt[4];
#pragma unroll
  for (int c = 0; c < 4; c++) cnt[c] = ccp[c];
  Pre pre;
  pre.tt = tt;
  pre.n_tt = n_tt;
#pragma unroll
  for (int kk = 0; kk < NK; kk++) {
    pre.code_off[kk] = a.kd[kind0 + kk].code_off[e];
    pre.sz_off[kk] = a.kd[kind0 + kk].sz_off[e];
  }
  const int32_t* order = NK == 1 ? a.order_dn : a.order_gu;
  pre.row0 = (routed && wgi >= n_swg)
                 ? order[static_cast<int64_t>(e) * R + blk * rows + (threadIdx.x >> 6) * 16 + (threadIdx.x & 15)]
                 : 0;
  if (uni(o1) <= uni(o0)) return;
  int start = 0, count = R;
  if (routed) {
#pragma unroll
    for (int c = 0; c < 4; c++) cnt[c] = uni(cnt[c]);
    if (wgi < n_swg) {   // find the switched class of this workgroup
      start = cnt[0];
      cls = 4;
      for (int c = 1; c < (NK == 1 ? 2 : 4); c++) {
        const int nwg = (cnt[c] + rows - 1) / rows;
        if (blk < nwg) {
          cls = c;
          break;
        }
        blk -= nwg;
        start += cnt[c];
      }
      if (cls == 4) return;
    }
    count = cnt[cls];
  }
  const int pos0 = start + blk * rows;
  if (blk * rows >= count) return;
  const int pos1 = min(pos0 + rows, start + count);
  const int B = map.bits[e - map.e0];
  if constexpr (NT == 2) {
    // an expert with at most 16 tokens needs one 16-token tile: half the
    // contraction and epilogue work of the 32-token tile (same LDS)
    if (uni(o1) - uni(o0) <= 16) {
      auto& t1 = *reinterpret_cast<XTile<NM, 1>*>(&tl);
      if (B == 8) dispatch_class<NM, 1, NK, 8>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      else if (B == 4) dispatch_class<NM, 1, NK, 4>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      else if (B == 2) dispatch_class<NM, 1, NK, 2>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      else if constexpr (NM == 4) {
        if (B == 6) dispatch_class<NM, 1, NK, 6>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
        else dispatch_class<NM, 1, NK, 3>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      }
      return;
    }
  }
  if (B == 8) dispatch_class<NM, NT, NK, 8>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  else if (B == 4) dispatch_class<NM, NT, NK, 4>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  else if (B == 2) dispatch_class<NM, NT, NK, 2>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  else if constexpr (NM == 4) {
    if (B == 6) dispatch_class<NM, NT, NK, 6>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
    else dispatch_class<NM, NT, NK, 3>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  }
}

// ------------------------------------------------------------------ tile kernel
// For experts with many tokens (prefill, shared experts), where the
// contraction is MFMA-bound: a workgroup computes a tile of kTileTok tokens x
// kTileRowsOf<NK> row positions with v_mfma_f32_32x32x16_f16.  This is
// the paper's formulation of the dequantized product (Sec. V-B: dequantize to
// a 16-bit operand, then matrix-core multiply): the weight operand is
// fp16(s * (q - z)) -- one rounding per weight -- and the activations enter
// as fp16 (the bf16 activations and hidden values convert exactly while
// their magnitude stays below 65504).  The scale is thus inside the operand
// and the accumulation runs over the whole K with no per-group epilogue.
//
// Dequantization: a code q OR-ed into the mantissa of fp16 1024.0 gives
// exactly 1024 + q (q < 1024); one packed fp16 subtraction of 1024 + z makes
// q - z exactly, one packed fp16 multiplication by s rounds the product.
//
// Eight waves per workgroup, two per SIMD.  Each wave owns 32 rows of one
// kind (gate/up: waves 0-3 the gate rows, 4-7 the up rows of the tile's 128
// positions; down: 256 rows) and all kTileTok tokens (four 32-token blocks),
// so every dequantized B fragment feeds four MFMAs.  Lane l holds row l % 32
// and the K-half l/32 of each group (group code g/2*half + 8*s + j feeds
// K-step s, slot j); accumulator element r of lane l is token
// 8*(r/4) + 4*(l/32) + r%4 of the block.  The activations of one group for
// the whole tile are staged in LDS by direct-to-LDS loads, two groups ahead
// (three stages), with the XOR swizzle of the streaming kernel; the packed
// codes of the next three groups are in flight in registers.  The SiLU-GLU
// epilogue meets the gate and up sums of a row through LDS.
//
// Work items (expert, row block, token tile) come from a prefix table a small
// plan kernel builds from the routing offsets and class counts, and are
// spread over a persistent grid so that the workgroups of one XCD (hardware
// places workgroup b on XCD b % 8) take consecutive items.  Within an expert
// the items run in super-tiles of kSuper row blocks x kSuper token tiles, so
// that the workgroups one XCD runs together share both their code rows and
// their activation rows through that XCD's L2.

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x16 mfma32h(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                 0, 0);
}

constexpr int kTileTok = 128;   // tokens per workgroup tile (four 32-token blocks)

// Row positions per workgroup tile: eight waves of 32 rows, gate/up split
// over the waves by kind (128 rows of both kinds) or down (256 rows).
template <int NK>
constexpr int kTileRowsOf = NK == 2 ? 128 : 256;

constexpr int kTileWaves = 8;

constexpr int kXcds = 8;
constexpr int kSuper = 8;
constexpr uint32_t kMagic16 = 0x64006400u;   // two fp16 1024.0

// LDS of the tile kernel: three stages of kTileTok token rows x g columns of
// fp16 activations in 16-byte slots (slot s: token s / (g/8), column chunk
// (s % (g/8)) ^ (token % (g/8))).
template <int NM2>
struct HTile {
  static constexpr int g = NM2 * 16;
  static constexpr int SPT = g / 8;
  static constexpr int SLOTS = kTileTok * SPT;
  union {
    u32x4 a[3][SLOTS];
    float xch[4 * 4 * 16 * 64];   // gate/up epilogue: the up sums of four 32-row blocks
  };
};

// Experts e0 .. e0+n_e-1 of one tile launch; bits[e - e0].
struct TileMap {
  int e0, n_e;
  int8_t bits[MOE_MAX_EXPERTS];
};

// Items of expert e: (row blocks over its classes) x (token tiles); the
// exclusive prefix over the launch's experts goes to prefix[0 .. n_e].
template <int NK>
__global__ void __launch_bounds__(256) tile_plan_kernel(FfnArgs a, TileMap map, int32_t* __restrict__ prefix) {
  __shared__ int cnt[MOE_MAX_EXPERTS];
  const int i = threadIdx.x;
  int items = 0;
  if (i < map.n_e) {
    const int e = map.e0 + i;
    const int n_tok = a.offsets[e + 1] - a.offsets[e];
    const int tiles = (n_tok + kTileTok - 1) / kTileTok;
    int blocks = 0;
    if (e < a.E) {
      const int32_t* cc = a.class_cnt + (NK == 1 ? 4 * a.E : 0) + 4 * e;
      for (int c = 0; c < (NK == 1 ? 2 : 4); c++) blocks += (cc[c] + kTileRowsOf<NK> - 1) / kTileRowsOf<NK>;
    } else {
      blocks = ((NK == 1 ? a.d : a.fs) + kTileRowsOf<NK> - 1) / kTileRowsOf<NK>;
    }
    items = tiles * blocks;
  }
  if (i < MOE_MAX_EXPERTS) cnt[i] = items;
  __syncthreads();
  if (i == 0) {
    int acc = 0;
    for (int j = 0; j < map.n_e; j++) {
      const int v = cnt[j];
      prefix[j] = acc;
      acc += v;
    }
    prefix[map.n_e] = acc;
  }
}

// One lane's source of one kind: resources, {s, z} group stride and offsets.
struct TSrc {
  Rsrc code, sz;
  uint32_t sz_gstride, coff, soff;
};

// Packed-code words of one lane's half of a group (g/2 codes).
template <int NM2, int B>
constexpr int kHalfWords = NM2 * 16 / 2 * B / 32;

// fp16 pair (1024 + q_lo, 1024 + q_hi) from two codes at bit offset sh of
// each half-word (b <= 8 bits wide, masked by m).
__device__ __forceinline__ uint32_t unpack16(uint32_t w, int sh, uint32_t m, uint32_t vm) {
  return ((w >> sh) & m) | vm;
}

// B fragment of K-step s: 8 fp16 weights s*(q - z) of this lane's row.
template <int NM2, int B>
__device__ __forceinline__ u32x4 dequant_h(const uint32_t (&cw)[(kHalfWords<NM2, B>)], int s, f16x2 zneg, f16x2 sc,
                                           uint32_t vm) {
  uint32_t r[4];
  if constexpr (B == 4) {
    const uint32_t w = cw[s];
#pragma unroll
    for (int i = 0; i < 4; i++) r[i] = unpack16(w, 4 * i, 0x000F000Fu, vm);
  } else if constexpr (B == 8) {
    const uint32_t w0 = cw[2 * s], w1 = cw[2 * s + 1];   // bytes (c0, c2, c1, c3)
    r[0] = unpack16(w0, 0, 0x00FF00FFu, vm);
    r[1] = unpack16(w0, 8, 0x00FF00FFu, vm);
    r[2] = unpack16(w1, 0, 0x00FF00FFu, vm);
    r[3] = unpack16(w1, 8, 0x00FF00FFu, vm);
  } else if constexpr (B == 2) {
    const uint32_t w = cw[s >> 1];
    const int o = (s & 1) * 8;
#pragma unroll
    for (int i = 0; i < 4; i++) r[i] = unpack16(w, o + 2 * i, 0x00030003u, vm);
  } else if constexpr (B == 6) {  // per 32-code block: words 0-3 bits 0..3, words 4-5 bits 4..5
    const int blk = 6 * (s >> 2);
    const int q = s & 3;   // octet within the block
    const uint32_t lo = cw[blk + q], hi = cw[blk + 4 + (q >> 1)];
    const int o = (q & 1) * 8;
#pragma unroll
    for (int i = 0; i < 4; i++)
      r[i] = (((lo >> (4 * i)) & 0x000F000Fu) | (((hi >> (o + 2 * i)) & 0x00030003u) << 4)) | vm;
  } else {  // 3-bit: per 32-code block words (low plane 0-15, low plane 16-31, high plane)
    const int blk = 3 * (s >> 2);
    const int q = s & 3;   // octet within the block
    const uint32_t lo = cw[blk + (q >> 1)], hi = cw[blk + 2];
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int pi = 4 * q + i;   // pair index within the block
      r[i] = (((lo >> (2 * (pi & 7))) & 0x00030003u) | (((hi >> pi) & 0x00010001u) << 2)) | vm;
    }
  }
  u32x4 out;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const f16x2 d = __builtin_bit_cast(f16x2, r[i]) + zneg;   // q - z, exact
    out[i] = __builtin_bit_cast(uint32_t, d * sc);            // s * (q - z), rounded once
  }
  return out;
}

// {s, z} word -> packed (-(1024 + z), -(1024 + z)) and (s, s).
__device__ __forceinline__ void sz_pair(uint32_t w, f16x2& zneg, f16x2& sc) {
  const _Float16 s16 = __builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xFFFFu));
  const _Float16 z16 = __builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16));
  const _Float16 zn = -(z16 + static_cast<_Float16>(1024.0f));   // exact: integer <= 1279
  zneg = f16x2{zn, zn};
  sc = f16x2{s16, s16};
}

template <int NM2, int BW>
struct HCodes {
  uint32_t cw[(kHalfWords<NM2, BW>)];
  uint32_t szw;
};

template <int NM2, int BW>
__device__ __forceinline__ void hload(HCodes<NM2, BW>& st, const TSrc& sr, int gi, bool gv) {
  constexpr uint32_t gcb = NM2 * 16 * BW / 8;   // code bytes per row and group
  bload<kHalfWords<NM2, BW>>(st.cw, sr.code, gv ? sr.coff : kOOB, gv ? gi * gcb : 0u);
  st.szw = __builtin_amdgcn_raw_buffer_load_b32(sr.sz, gv ? sr.soff : kOOB, gv ? gi * sr.sz_gstride : 0u, 0);
}

template <int N>
__device__ __forceinline__ void hwait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Barrier without __syncthreads()' fences (those would drain the in-flight
// code loads); the LDS stages are ordered by the explicit waits around it.
__device__ __forceinline__ void tile_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// silu(g) * u with a hardware reciprocal: h is rounded to bf16 right after,
// far coarser than the reciprocal's error.
__device__ __forceinline__ float silu_mul_fast(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

// Activation stages in flight: the stage of group gi+2 is loaded while group
// gi is contracted; three LDS stages.
constexpr int kAStages = 3;

// One wave's share of a tile item: 32 rows (position block rb) of weight kind
// kk, whose source has width BW (the expert's base width, or 8 for the
// cached copies of a switched class), against all kTileTok tokens.
template <int NM2, int NK, int BW, int TB>
__device__ __forceinline__ void tile_wave(const FfnArgs& a, HTile<NM2>& tl, int e, bool copy, int be, int kk,
                                          int rb, int pos0, int pos1, int R, int t0, int t1) {
  constexpr int g = NM2 * 16;
  constexpr int SPT = HTile<NM2>::SPT;
  // activation slots of the tile's TB token blocks, and loads per thread and
  // stage (slots past them are written with zeros)
  constexpr int SL = TB * 32 * SPT;
  constexpr int NLD = (SL + 64 * kTileWaves - 1) / (64 * kTileWaves);
  constexpr bool down = NK == 1;
  // vector-memory instructions of one group's code and {s, z} loads
  constexpr int LC = kCodeLoads<(kHalfWords<NM2, BW>)> + 1;
  const int tid = threadIdx.x;
  const int wv = tid >> 6, lane = tid & 63;
  const int n = lane & 31, kh = lane >> 5;
  const bool routed = e < a.E;
  const int K = down ? (routed ? a.f : a.fs) : a.d;
  const int G = K / g;
  const int kind0 = down ? 2 : 0;
  const int32_t* order = down ? a.order_dn : a.order_gu;
  const int pos = pos0 + 32 * rb + n;
  const bool live = pos < pos1;
  const int row = live ? (routed ? order[static_cast<int64_t>(e) * R + pos] : pos) : 0;

  TSrc src;
  {
    const KindDev& kd = a.kd[kind0 + kk];
    const uint32_t row_bytes = 4u * static_cast<uint32_t>(code_row_words(K, be));
    const uint32_t crow_bytes = 4u * static_cast<uint32_t>(code_row_words(K, 8));
    const void* cptr = copy ? static_cast<const void*>(kd.copy_codes)
                            : static_cast<const void*>(kd.codes + uni(kd.code_off[e]));
    const void* sptr = copy ? static_cast<const void*>(kd.copy_sz)
                            : static_cast<const void*>(kd.sz + uni(kd.sz_off[e]));
    const uint32_t cbytes = copy ? a.copy_bytes[kind0 + kk] : static_cast<uint32_t>(R) * row_bytes;
    const uint32_t sbytes = copy ? a.copy_sz_bytes[kind0 + kk] : static_cast<uint32_t>(R) * G * 4u;
    src.code = make_rsrc(cptr, cbytes);
    src.sz = make_rsrc(sptr, sbytes);
    src.sz_gstride = copy ? 4u : static_cast<uint32_t>(R) * 4u;
    const int slot = (copy && live) ? kd.row_slot[static_cast<int64_t>(e) * R + row] : -1;
    const uint32_t c_base = live ? row * row_bytes + kh * (g / 2) * be / 8 : kOOB;
    const uint32_t s_base = live ? row * 4u : kOOB;
    const uint32_t c_copy = slot >= 0 ? static_cast<uint32_t>(slot) * crow_bytes + kh * (g / 2) : kOOB;
    const uint32_t s_copy = slot >= 0 ? static_cast<uint32_t>(slot) * G * 4u : kOOB;
    src.coff = copy ? c_copy : c_base;
    src.soff = copy ? s_copy : s_base;
  }
  // fp16 activations: gathered x rows (gate/up) or h rows (down), row p of the
  // permuted order; slot i of this thread's loads
  const Rsrc xr = make_rsrc(down ? static_cast<const void*>(a.h) : static_cast<const void*>(a.x16),
                            down ? a.h_bytes : a.x16_bytes);
  uint32_t aoff[NLD];
#pragma unroll
  for (int i = 0; i < NLD; i++) {
    const int sl = tid + 64 * kTileWaves * i;
    const int t = sl / SPT;
    const int c = (sl % SPT) ^ (t % SPT);
    const int p = t0 + t;
    aoff[i] = (sl < SL && p < t1)
                  ? static_cast<uint32_t>(2 * (down ? h_row(a, p) : static_cast<int64_t>(a.perm[p]) * K) + 16 * c)
                  : kOOB;
  }
  auto stage_a = [&](int buf, int gi) {
    const bool gv = gi < G;
    const uint32_t adv = gv ? 2u * static_cast<uint32_t>(gi * g) : 0u;
#pragma unroll
    for (int i = 0; i < NLD; i++)
      lds_dma16(xr, &tl.a[buf][64 * kTileWaves * i + 64 * wv], gv ? aoff[i] : kOOB, adv);
  };

  // the OR operand of the unpacking in a vector register (one v_and_or_b32)
  uint32_t vm = kMagic16;
  asm volatile("" : "+v"(vm));
  f32x16 acc[TB];
#pragma unroll
  for (int tb = 0; tb < TB; tb++) acc[tb] = f32x16{};

  HCodes<NM2, BW> cs[3];
  stage_a(0, 0);
  hload<NM2, BW>(cs[0], src, 0, 0 < G);
  stage_a(1, 1);
  hload<NM2, BW>(cs[1], src, 1, 1 < G);
  hload<NM2, BW>(cs[2], src, 2, 2 < G);
  hwait_vm<2 * LC + NLD>();   // activations of group 0 have landed (this wave's share)
  tile_barrier();             // ... every wave's share

  auto group = [&](HCodes<NM2, BW>& c, int buf, int gi) {
    stage_a((buf + 2) % kAStages, gi + 2);   // that stage was last read for group gi-1 (barrier since)
    if (gi < G) {   // workgroup-uniform (G is odd for some shapes)
      f16x2 zn, sc;
      sz_pair(c.szw, zn, sc);
#pragma unroll
      for (int s = 0; s < NM2; s++) {
        u32x4 af[TB];
#pragma unroll
        for (int tb = 0; tb < TB; tb++) {
          const int t = tb * 32 + n;
          af[tb] = tl.a[buf][t * SPT + ((kh * NM2 + s) ^ (t % SPT))];
        }
        const u32x4 bf = dequant_h<NM2, BW>(c.cw, s, zn, sc, vm);
#pragma unroll
        for (int tb = 0; tb < TB; tb++) acc[tb] = mfma32h(af[tb], bf, acc[tb]);
      }
    }
    hload<NM2, BW>(c, src, gi + 3, gi + 3 < G);
    hwait_vm<2 * LC + NLD>();   // everything but the last two code loads and the newest stage: group gi+1's
    tile_barrier();
  };
  for (int gi = 0; gi < G; gi += 3) {
    group(cs[0], 0, gi);
    group(cs[1], 1, gi + 1);
    group(cs[2], 2, gi + 2);
  }
  hwait_vm<0>();

  // outputs: tokens t0 + 32*tb + 8*(r/4) + 4*kh + r%4, row `row`
  if constexpr (NK == 2) {
    // the up waves hand their sums to the gate waves of the same rows through
    // the (now idle) activation stages; same lane layout on both sides
    float* xch = tl.xch;
    tile_barrier();   // every wave is done reading the activation stages
    if (kk == 1) {
#pragma unroll
      for (int tb = 0; tb < TB; tb++)
#pragma unroll
        for (int r = 0; r < 16; r++) xch[((rb * 4 + tb) * 16 + r) * 64 + lane] = acc[tb][r];
    }
    tile_barrier();
    if (kk == 0) {
      // rows of one item are all routed or all shared: one h row width
      const int hw = t0 < a.Tk ? a.f : a.fs;
      uint16_t* hbase = a.h + h_row(a, t0 + 4 * kh) + row;
#pragma unroll
      for (int tb = 0; tb < TB; tb++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
          const int dt = tb * 32 + 8 * (r / 4) + (r % 4);
          const float u = xch[((rb * 4 + tb) * 16 + r) * 64 + lane];
          if (live && t0 + 4 * kh + dt < t1) {
            // h = bf16(silu(g) * u), stored as its (exact) fp16 value
            const float hb = __uint_as_float(bf16_rne(silu_mul_fast(acc[tb][r], u)) << 16);
            hbase[dt * hw] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(hb));
          }
        }
    }
  } else {
    float* obase = a.o + static_cast<int64_t>(t0 + 4 * kh) * R + row;
#pragma unroll
    for (int tb = 0; tb < TB; tb++)
#pragma unroll
      for (int r = 0; r < 16; r++) {
        const int dt = tb * 32 + 8 * (r / 4) + (r % 4);
        if (live && t0 + 4 * kh + dt < t1) obase[dt * R] = acc[tb][r];
      }
    // the other split slices of these rows (the combine adds every slice)
    for (int sp = 1; sp < a.n_split_out; sp++) {
      float* ob = obase + static_cast<int64_t>(sp) * a.split_stride;
#pragma unroll
      for (int tb = 0; tb < TB; tb++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
          const int dt = tb * 32 + 8 * (r / 4) + (r % 4);
          if (live && t0 + 4 * kh + dt < t1) ob[dt * R] = 0.f;
        }
    }
  }
}

// Waves 0-3 take the gate rows and waves 4-7 the up rows of the tile's 128
// positions, or all eight waves take 32 of the 256 down rows; a kind whose
// class bit is set reads the 8-bit copies.
template <int NM2, int NK, int B>
__device__ __forceinline__ void tile_dispatch(const FfnArgs& a, HTile<NM2>& tl, int e, int cls, int pos0,
                                              int pos1, int R, int t0, int t1) {
  // the wave index through readfirstlane: the kind, the class bit and the
  // buffer descriptors chosen by them are then scalar values, so no load is
  // wrapped in a loop over the distinct descriptors of the wave's lanes
  const int wv = uni(static_cast<int>(threadIdx.x >> 6));
  const int kk = NK == 2 ? wv / 4 : 0;
  const int rb = NK == 2 ? wv % 4 : wv;
  const bool copy = (cls >> kk) & 1;
  // the expert's base width: class 1 or 2 has one kind on copies, whose
  // template width is 8 even though the base width is B.  The token tile of
  // the item (an expert's last tile is partial) picks one, two or four
  // 32-token blocks.
  const int nt = t1 - t0;
  if (nt <= 32) {
    if (copy) tile_wave<NM2, NK, 8, 1>(a, tl, e, true, B, kk, rb, pos0, pos1, R, t0, t1);
    else tile_wave<NM2, NK, B, 1>(a, tl, e, false, B, kk, rb, pos0, pos1, R, t0, t1);
  } else if (nt <= 64) {
    if (copy) tile_wave<NM2, NK, 8, 2>(a, tl, e, true, B, kk, rb, pos0, pos1, R, t0, t1);
    else tile_wave<NM2, NK, B, 2>(a, tl, e, false, B, kk, rb, pos0, pos1, R, t0, t1);
  } else {
    if (copy) tile_wave<NM2, NK, 8, 4>(a, tl, e, true, B, kk, rb, pos0, pos1, R, t0, t1);
    else tile_wave<NM2, NK, B, 4>(a, tl, e, false, B, kk, rb, pos0, pos1, R, t0, t1);
  }
}

// Eight waves, two per SIMD: a wave's 64 accumulator registers leave room for
// a second wave, which hides the first one's load and LDS latencies.
template <int NM2, int NK>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2)))
ffn_tile_kernel(FfnArgs a, TileMap map, const int32_t* __restrict__ prefix) {
  __shared__ __attribute__((aligned(16))) HTile<NM2> tl;
  __shared__ int pre[MOE_MAX_EXPERTS + 1];
  for (int i = threadIdx.x; i <= map.n_e; i += blockDim.x) pre[i] = prefix[i];
  __syncthreads();
  const int total = pre[map.n_e];
  const int G = gridDim.x;   // a multiple of kXcds
  const int per = G / kXcds;
  const int xcd = blockIdx.x % kXcds, loc = blockIdx.x / kXcds;
  for (int it = 0;; it++) {
    const int item = it * G + xcd * per + loc;
    if (item >= total) break;
    int lo = 0, hi = map.n_e - 1;   // last expert whose prefix is <= item
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (pre[mid] <= item) lo = mid; else hi = mid - 1;
    }
    const int e = map.e0 + lo;
    const int local = item - pre[lo];
    const int seg0 = uni(a.offsets[e]), seg1 = uni(a.offsets[e + 1]);
    const int tiles = (seg1 - seg0 + kTileTok - 1) / kTileTok;
    const bool routed = e < a.E;
    const int R = NK == 1 ? a.d : (routed ? a.f : a.fs);
    // (row block, token tile) of the local index: super-rows of kSuper row
    // blocks, token tiles outer and row blocks inner within a super-row
    int n_rb = 0;
    if (routed) {
      const int32_t* cc = a.class_cnt + (NK == 1 ? 4 * a.E : 0) + 4 * e;
      for (int c = 0; c < (NK == 1 ? 2 : 4); c++) n_rb += (uni(cc[c]) + kTileRowsOf<NK> - 1) / kTileRowsOf<NK>;
    } else {
      n_rb = (R + kTileRowsOf<NK> - 1) / kTileRowsOf<NK>;
    }
    const int full = (n_rb / kSuper) * kSuper * tiles;
    int rb, tt;
    if (local < full) {
      const int sr = local / (kSuper * tiles), rem = local - sr * kSuper * tiles;
      tt = rem / kSuper;
      rb = sr * kSuper + rem % kSuper;
    } else {
      const int h = n_rb % kSuper, rem = local - full;
      tt = rem / h;
      rb = (n_rb / kSuper) * kSuper + rem % h;
    }
    int cls = 0, start = 0, count = R;
    if (routed) {
      const int32_t* cc = a.class_cnt + (NK == 1 ? 4 * a.E : 0) + 4 * e;
      for (int c = 0; c < (NK == 1 ? 2 : 4); c++) {
        const int cn = uni(cc[c]);
        const int nb = (cn + kTileRowsOf<NK> - 1) / kTileRowsOf<NK>;
        if (rb < nb) {
          cls = c;
          count = cn;
          break;
        }
        rb -= nb;
        start += cn;
      }
    }
    const int pos0 = start + rb * kTileRowsOf<NK>;
    const int pos1 = min(pos0 + kTileRowsOf<NK>, start + count);
    const int t0 = seg0 + tt * kTileTok, t1 = min(t0 + kTileTok, seg1);
    const int B = map.bits[e - map.e0];
    if (B == 8) tile_dispatch<NM2, NK, 8>(a, tl, e, cls, pos0, pos1, R, t0, t1);
    else if (B == 4) tile_dispatch<NM2, NK, 4>(a, tl, e, cls, pos0, pos1, R, t0, t1);
    else if (B == 2) tile_dispatch<NM2, NK, 2>(a, tl, e, cls, pos0, pos1, R, t0, t1);
    else if constexpr (NM2 % 4 == 0) {
      if (B == 6) tile_dispatch<NM2, NK, 6>(a, tl, e, cls, pos0, pos1, R, t0, t1);
      else tile_dispatch<NM2, NK, 3>(a, tl, e, cls, pos0, pos1, R, t0, t1);
    }
    tile_barrier();   // the LDS stages are reused by the next item
  }
}

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
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const uint32_t lo = __builtin_bit_cast(uint16_t, static_cast<_Float16>(bf16_lo(v[i])));
    const uint32_t hi = __builtin_bit_cast(uint16_t, static_cast<_Float16>(bf16_hi(v[i])));
    o[i] = lo | (hi << 16);
  }
  *reinterpret_cast<u32x4*>(const_cast<uint16_t*>(a.x16) + static_cast<int64_t>(p) * a.d + c) = o;
}

size_t align256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

struct Plan {
  int n_split;
  int nt_routed, nt_shared;   // token tiles of the streaming kernel, 0: tile kernel
  int tt_routed, tt_shared;   // workgroup sets per row block, each taking every n-th 32-token tile
  size_t xsum_bytes, h_bytes, hsum_bytes, tile_bytes, x16_bytes, total;
};

// Shared experts with up to this many tokens stream, one workgroup set per
// 32-token tile (measured on the Qwen-shaped layer, 512 tokens: step 440 ->
// 389 us against the tile kernel's few items).
constexpr int kSharedSplitMax = 512;
// Routed experts expecting up to this many tokens stream too, with
// workgroup sets taking every n_tt-th 32-token tile of the expert.
constexpr int kRoutedSplitMax = 96;

// Streaming kernel for up to 28 expected tokens per expert (one or two
// 16-token MFMA tiles, weights streamed once); beyond, make_plan spreads the
// 32-token tiles of mid-sized experts over workgroup sets, and the rest go to
// the tile kernel.
int pick_nt(double tokens) {
  if (tokens <= 12.0) return 1;
  if (tokens <= 28.0) return 2;
  return 0;
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
  p.nt_routed = pick_nt(static_cast<double>(Tk) / E);
  p.tt_routed = 1;
  if (p.nt_routed == 0 && Tk <= static_cast<int64_t>(kRoutedSplitMax) * E) {
    // a few dozen tokens per expert: 32-token tiles over several workgroup
    // sets (one more than the mean needs, for skewed loads)
    p.nt_routed = 2;
    p.tt_routed = static_cast<int>(cdiv(cdiv(Tk, E), 32)) + 1;
  }
  p.nt_shared = pick_nt(static_cast<double>(T));
  p.tt_shared = 1;
  if (p.nt_shared == 0 && T <= kSharedSplitMax) {
    // shared experts at a few dozen to a few hundred tokens: 32-token tiles,
    // each on its own workgroups (the expert's weights are re-read from L2
    // per tile), rather than the tile kernel's few 128-token items
    p.nt_shared = 2;
    p.tt_shared = static_cast<int>(cdiv(T, 32));
  }
  // split-K slices of the down projection only where the routed experts
  // stream (few tokens, too few output rows to fill the machine)
  p.n_split = p.nt_routed == 0 ? 1 : std::max(ns, 1);
  const int64_t hcols = Tk * L->d_ff + static_cast<int64_t>(S) * T * L->d_ff_shared;
  p.xsum_bytes = align256(sizeof(float) * static_cast<size_t>(rows) * (L->d_model / g));
  p.h_bytes = align256(sizeof(uint16_t) * static_cast<size_t>(hcols));
  p.hsum_bytes = align256(sizeof(float) * static_cast<size_t>(rows) * (fmax / g));
  p.tile_bytes = align256(sizeof(int32_t) * 4 * (MOE_MAX_EXPERTS + 1));
  const bool tiled = p.nt_routed == 0 || (S > 0 && p.nt_shared == 0);
  p.x16_bytes = tiled ? align256(sizeof(uint16_t) * static_cast<size_t>(T) * L->d_model) : 0;
  p.total = p.xsum_bytes + p.h_bytes + p.hsum_bytes + p.tile_bytes + p.x16_bytes + 256;
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
  if (!L->bits || !L->bits_host || !L->order_gu || !L->order_dn || !L->class_cnt) return MOE_ERR_ARG;
  // buffer resources address each expert's codes and {scale, zero} words with
  // 32-bit byte offsets below 2^31
  const int64_t fm = std::max<int64_t>(L->d_ff, S > 0 ? L->d_ff_shared : 0);
  if (fm * 4 * code_row_words(std::max<int64_t>(fm, L->d_model), 8) >= (int64_t{1} << 31))
    return MOE_ERR_ARG;
  for (int e = 0; e < E + S; e++) {
    if (!valid_bits(L->bits_host[e])) return MOE_ERR_BITS;
    if ((L->bits_host[e] == 3 || L->bits_host[e] == 6) && L->group != 128) return MOE_ERR_ARG;
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

// Work map of one launch (routed experts, or the shared experts).  The
// switched-class workgroups per routed expert bound what its copies can need:
// classes 1..3 of gate/up hold at most n_gate + n_up rows in three classes,
// class 1 of down at most n_down rows.
WgMap stream_map(const moe_layer_t* L, bool shared, bool down) {
  WgMap m{};
  const int rows = (down ? kWavesOf<1> : kWavesOf<2>) * 16;
  const int E = L->n_experts;
  if (shared) {
    m.e0 = E;
    m.n_e = L->n_shared;
    m.n_sw = 0;
    m.per_e = (down ? L->d_model : L->d_ff_shared) / rows;
    for (int i = 0; i < L->n_shared; i++) {
      m.order[i] = static_cast<int16_t>(i);
      m.bits[i] = static_cast<int8_t>(L->bits_host[E + i]);
    }
    return m;
  }
  const int R = down ? L->d_model : L->d_ff;
  m.e0 = 0;
  m.n_e = E;
  m.per_e = R / rows;
  std::vector<int> nc[2];
  for (int kk = 0; kk < (down ? 1 : 2); kk++) {
    const moe_kind_desc_t& k = L->kind[down ? 2 : kk];
    nc[kk].assign(E, 0);
    for (int s = 0; s < k.n_slots; s++) {
      const int e = k.copy_hdr_host ? k.copy_hdr_host[2 * s] : -1;
      if (e >= 0 && e < E) nc[kk][e]++;
      else std::fill(nc[kk].begin(), nc[kk].end(), R);   // headers unknown: any row
    }
    for (int e = 0; e < E; e++) nc[kk][e] = std::min(nc[kk][e], R);
  }
  int n_sw = 0;
  for (int e = 0; e < E; e++) {
    const int64_t need = down ? cdiv(nc[0][e], rows)
                              : (nc[0][e] + nc[1][e] > 0 ? cdiv(nc[0][e] + nc[1][e], rows) + 2 : 0);
    n_sw = std::max<int>(n_sw, static_cast<int>(std::min<int64_t>(need, cdiv(R, rows) + 3)));
  }
  m.n_sw = n_sw;
  for (int e = 0; e < E; e++) m.bits[e] = static_cast<int8_t>(L->bits_host[e]);
  int n = 0;
  for (int b : {8, 6, 4, 3, 2})
    for (int e = 0; e < E; e++)
      if (L->bits_host[e] == b) m.order[n++] = static_cast<int16_t>(e);
  return m;
}

TileMap tile_map(const moe_layer_t* L, bool shared) {
  TileMap m{};
  m.e0 = shared ? L->n_experts : 0;
  m.n_e = shared ? L->n_shared : L->n_experts;
  for (int i = 0; i < m.n_e; i++) m.bits[i] = static_cast<int8_t>(L->bits_host[m.e0 + i]);
  return m;
}

// Persistent tile grid: one workgroup per compute unit (the tile kernel runs
// one wave per SIMD), a multiple of the XCD count.
int tile_grid() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] == 0) {
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu <= 0) cu = 256;
    cached[dev] = std::max(kXcds, cu / kXcds * kXcds);
  }
  return cached[dev];
}

// One kernel launch of a stage; `start` / `stop` (may be null) are HIP events
// that take the dispatch's own begin / end timestamps.
using Launch = std::function<void(hipEvent_t start, hipEvent_t stop)>;

template <typename F, typename... A>
void klaunch(F kernel, dim3 grid, dim3 block, hipStream_t s, hipEvent_t start, hipEvent_t stop,
             A... args) {
  if (start || stop) hipExtLaunchKernelGGL(kernel, grid, block, 0, s, start, stop, 0, args...);
  else hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}

// Issues a stage's launches in order: the first carries `start`, the last
// `stop`.  An empty stage records the events as plain stream markers.
void issue(const std::vector<Launch>& v, hipEvent_t start, hipEvent_t stop, hipStream_t s) {
  if (v.empty()) {
    if (start) (void)hipEventRecord(start, s);
    if (stop) (void)hipEventRecord(stop, s);
    return;
  }
  for (size_t i = 0; i < v.size(); i++)
    v[i](i == 0 ? start : nullptr, i + 1 == v.size() ? stop : nullptr);
}

template <int NM>
void launch_all(const FfnArgs& a, const Plan& p, const moe_layer_t* L, int T, hipStream_t s,
                hipEvent_t* ev, int n_ev) {
  constexpr int g = NM * 32;
  const int S = a.S;
  auto event = [&](int i) -> hipEvent_t { return (ev && i < n_ev) ? ev[i] : nullptr; };
  std::vector<Launch> xsum, gate_up, hsum, down;
  // activation preparation per row range: group sums [d/g][rows] for the
  // streaming kernel, fp16 copies for the tile kernel
  bool x16_done = false;
  auto prep = [&](int p0, int p1, bool tiled) {
    if (p1 <= p0) return;
    if (tiled) {   // one fp16 copy of the T token rows serves every tiled range
      if (x16_done) return;
      x16_done = true;
      const int64_t n = static_cast<int64_t>(T) * (a.d / 8);
      xsum.push_back([=, &a](hipEvent_t e0, hipEvent_t e1) {
        klaunch(gather_f16_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), s, e0, e1, a, T);
      });
    } else {
      const int64_t n = static_cast<int64_t>(p1 - p0) * (a.d / g) * (g / 8);
      xsum.push_back([=, &a](hipEvent_t e0, hipEvent_t e1) {
        klaunch(group_sum_kernel<NM>, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), s, e0, e1,
                a, a.x, a.perm, static_cast<int64_t>(a.d), p0, p1, a.d, p1, a.d, const_cast<float*>(a.xsum));
      });
    }
  };
  if (p.nt_routed != 0 && (S == 0 || p.nt_shared != 0)) {
    prep(0, a.rows, false);   // every row streams: one launch of group sums
  } else {
    prep(0, a.Tk, p.nt_routed == 0);
    if (S > 0) prep(a.Tk, a.rows, p.nt_shared == 0);
  }
  int32_t* prefix = a.tile_prefix;
  auto add = [&](std::vector<Launch>& v, auto nk, bool shared, int nt, int nsplit) {
    constexpr int NK = decltype(nk)::value;
    if (nt == 0) {  // tile path: plan kernel, then the persistent tile kernel
      const TileMap m = tile_map(L, shared);
      const int32_t* pf = prefix;
      prefix += MOE_MAX_EXPERTS + 1;
      if (m.n_e == 0) return;
      v.push_back([=, &a](hipEvent_t e0, hipEvent_t e1) {
        klaunch(tile_plan_kernel<NK>, dim3(1), dim3(256), s, e0, e1, a, m, const_cast<int32_t*>(pf));
      });
      v.push_back([=, &a](hipEvent_t e0, hipEvent_t e1) {
        klaunch(ffn_tile_kernel<2 * NM, NK>, dim3(static_cast<unsigned>(tile_grid())), dim3(64 * kTileWaves), s,
                e0, e1, a, m, pf);
      });
      return;
    }
    const WgMap m = stream_map(L, shared, NK == 1);
    const int64_t n_wg = static_cast<int64_t>(m.n_e) * (m.n_sw + m.per_e);
    if (n_wg == 0) return;
    const int n_tt = shared ? p.tt_shared : p.tt_routed;
    const dim3 grid(static_cast<unsigned>(n_wg * nsplit * n_tt));
    v.push_back([=, &a](hipEvent_t e0, hipEvent_t e1) {
      const dim3 block(64 * kWavesOf<NK>);
      if (nt == 1) klaunch(ffn_stream_kernel<NM, 1, NK>, grid, block, s, e0, e1, a, m, nsplit, n_tt);
      else klaunch(ffn_stream_kernel<NM, 2, NK>, grid, block, s, e0, e1, a, m, nsplit, n_tt);
    });
  };
  using two = std::integral_constant<int, 2>;
  using one = std::integral_constant<int, 1>;
  add(gate_up, two{}, false, p.nt_routed, 1);
  if (S > 0) add(gate_up, two{}, true, p.nt_shared, 1);
  {  // group sums of h, [max(f,fs)/g][rows], for the rows the streaming kernel reads
    // (routed rows f wide, shared rows fs wide; one launch when both stream)
    auto hs = [&](int p0, int p1) {
      const int64_t n = static_cast<int64_t>(p1 - p0) * (std::max(a.f, a.fs) / g) * (g / 8);
      hsum.push_back([=, &a](hipEvent_t e0, hipEvent_t e1) {
        klaunch(group_sum_kernel<NM>, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), s, e0, e1,
                a, static_cast<const uint16_t*>(a.h), static_cast<const int32_t*>(nullptr),
                int64_t{0}, p0, p1, a.f, a.Tk, a.fs, a.hsum);
      });
    };
    const bool rs = p.nt_routed != 0 && a.Tk > 0, ss = S > 0 && p.nt_shared != 0;
    if (rs && ss) hs(0, a.rows);
    else if (rs) hs(0, a.Tk);
    else if (ss) hs(a.Tk, a.rows);
  }
  add(down, one{}, false, p.nt_routed, p.n_split);
  if (S > 0) add(down, one{}, true, p.nt_shared, p.n_split);
  issue(xsum, event(0), nullptr, s);
  issue(gate_up, event(1), event(2), s);
  issue(hsum, nullptr, nullptr, s);
  issue(down, event(3), event(4), s);
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
  a.class_cnt = L->class_cnt;
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
  a.tile_prefix = reinterpret_cast<int32_t*>(w + p.xsum_bytes + p.h_bytes + p.hsum_bytes);
  a.x16 = reinterpret_cast<const uint16_t*>(w + p.xsum_bytes + p.h_bytes + p.hsum_bytes + p.tile_bytes);
  a.n_split_out = p.n_split;
  a.o = o;
  a.split_stride = static_cast<int64_t>(T) * (k + L->n_shared) * L->d_model;
  {  // sizes of the buffer resources; every one must stay below 2^31 bytes
    const int64_t lim = int64_t{1} << 31;
    const int64_t xb = static_cast<int64_t>(T) * L->d_model * 2;
    if (xb >= lim || static_cast<int64_t>(p.h_bytes) >= lim || static_cast<int64_t>(p.xsum_bytes) >= lim ||
        static_cast<int64_t>(p.hsum_bytes) >= lim || static_cast<int64_t>(p.x16_bytes) >= lim)
      return MOE_ERR_ARG;
    a.x16_bytes = static_cast<uint32_t>(p.x16_bytes);
    a.x_bytes = static_cast<uint32_t>(xb);
    a.h_bytes = static_cast<uint32_t>(p.h_bytes);
    a.xsum_bytes = static_cast<uint32_t>(p.xsum_bytes);
    a.hsum_bytes = static_cast<uint32_t>(p.hsum_bytes);
    for (int kd = 0; kd < 3; kd++) {
      const int64_t K = kd == MOE_KIND_DOWN ? L->d_ff : L->d_model;
      const int64_t cb = static_cast<int64_t>(L->kind[kd].n_slots) * 4 * code_row_words(K, 8);
      const int64_t sb = static_cast<int64_t>(L->kind[kd].n_slots) * (K / L->group) * 4;
      if (cb >= lim || sb >= lim) return MOE_ERR_ARG;
      a.copy_bytes[kd] = static_cast<uint32_t>(cb);
      a.copy_sz_bytes[kd] = static_cast<uint32_t>(sb);
    }
  }
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
