// ffn_tile.hip -- the tile kernel of moe_expert_ffn_mixed, for experts with
// many tokens (prefill sizes), and its work-plan kernel.
#include "ffn_common.hpp"

namespace moe {
namespace ffn {

// ------------------------------------------------------------------ tile kernel
// For experts with many tokens (prefill, shared experts), where the
// contraction is MFMA-bound: a workgroup computes a tile of kTileTok tokens x
// eight waves' row positions with v_mfma_f32_32x32x16_f16.  This is
// the paper's formulation of the dequantized product (Sec. V-B: dequantize to
// a 16-bit operand, then matrix-core multiply): the weight operand is
// fp16(s * (q - z)) -- one rounding per weight -- and the activations enter
// as fp16 (the bf16 activations and hidden values convert exactly while
// their magnitude lies in [2^-17, 65504]; a value beyond 65504 sets the
// call's status word to MOE_ERR_RANGE).  The scale is thus inside the operand
// and the accumulation runs over the whole K with no per-group epilogue.
//
// Dequantization: a code q OR-ed into the mantissa of fp16 1024.0 gives
// exactly 1024 + q (q < 1024; 8-bit codes: one byte permute against bytes of
// 0x64 per pair).  A code sitting higher in the word is OR-ed into a smaller
// magic M whose mantissa unit falls on its lowest bit (64.0 for a 4-bit code
// at bit 4; 256.0, 64.0, 16.0 for 2-bit codes, and the low two bits of 3-bit
// codes, at bits 2, 4, 6), which reads M + q with no shift.  One packed fp16 subtraction of M + z makes q - z
// exactly, one packed fp16 multiplication by s rounds the product.
//
// Eight waves per workgroup, two per SIMD.  Each wave owns two weight rows
// per lane column -- the gate and the up row of 32 positions (gate/up), or
// two blocks of 32 positions 32 apart (down) -- and all kTileTok tokens
// (four 32-token blocks): every activation fragment read from LDS feeds two
// MFMAs and every dequantized weight fragment four.  Lane l holds position
// l % 32 and the K-half l/32 of each group (group code g/2*half + 8*s + j
// feeds K-step s, slot j); accumulator element r of lane l is token
// 8*(r/4) + 4*(l/32) + r%4 of the block.  The activations of one group for
// the whole tile are staged in LDS by direct-to-LDS loads, NS-1 groups ahead,
// with the XOR swizzle of the streaming kernel; the packed codes of the next
// NS groups are in flight in registers (NS = 3 stages, or 2 where the codes of
// a group take many registers or the item mixes source classes).  Gate/up
// applies SiLU-GLU to its own two accumulators.
//
// An expert's row positions are cut into waves class by class (each source
// class of the row order -- base codes, or copies for the gate, the up or both
// rows -- starts a new wave), and eight consecutive waves form a row block;
// a wave's class picks its sources, so a small class costs one wave, not a
// workgroup.  Work items (expert, row block, token tile; a down item also
// takes a K slice and writes its own slice of o, which the combine adds) come
// from a prefix table a small plan kernel builds from the routing offsets and
// class counts, and are spread over a persistent grid so that the workgroups
// of one XCD (hardware places workgroup b on XCD b % 8) take consecutive
// items.  Within an expert the items run in super-tiles of kSuper row blocks
// x kSuper token tiles, so that the workgroups one XCD runs together share
// both their code rows and their activation rows through that XCD's L2.

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x16 mfma32h(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                 0, 0);
}

constexpr uint32_t kHigh64 = 0x64646464u;    // the high byte of fp16 1024.0, in every byte

// One LDS stage of the tile kernel: kTileTok token rows x g columns of fp16
// activations in 16-byte slots (slot s: token s / (g/8), column chunk
// (s % (g/8)) ^ (token % (g/8))).
template <int NM2>
struct TileStage {
  static constexpr int g = NM2 * 16;
  static constexpr int SPT = g / 8;
  static constexpr int SLOTS = kTileTok * SPT;
};

// The stages are three separate __shared__ arrays: the compiler then knows
// that the direct-to-LDS loads into one stage do not write what the waves
// read from another, and waits for none of them before its reads.
struct TileLds {
  u32x4* s0;
  u32x4* s1;
  u32x4* s2;
};

__device__ __forceinline__ u32x4* stage_of(const TileLds& l, int b) { return b == 0 ? l.s0 : (b == 1 ? l.s1 : l.s2); }

// Waves of expert e: class c of its row order (routed experts; a shared
// expert is one class of R rows) takes ceil(count / kTileWaveRows) waves,
// classes in order.  pre[c] = first wave of class c (pre[NC] = the total),
// beg[c] / cnt[c] = its positions.  UNI: e is the same in every lane (the
// counts then go through readfirstlane, so they are scalar values).
template <int NK>
struct TileWaves {
  static constexpr int NC = NK == 1 ? 2 : 4;
  int pre[NC + 1], beg[NC], cnt[NC];
};

template <int NK, bool UNI>
__device__ __forceinline__ TileWaves<NK> tile_waves(const FfnArgs& a, int e, int R) {
  constexpr int NC = TileWaves<NK>::NC;
  TileWaves<NK> w;
  w.pre[0] = 0;
  int start = 0;
#pragma unroll
  for (int c = 0; c < NC; c++) {
    int cn = e < a.E ? a.class_cnt[(NK == 1 ? 4 * a.E : 0) + 4 * e + c] : (c == 0 ? R : 0);
    if constexpr (UNI) cn = uni(cn);
    w.beg[c] = start;
    w.cnt[c] = cn;
    w.pre[c + 1] = w.pre[c] + (cn + kTileWaveRows<NK> - 1) / kTileWaveRows<NK>;
    start += cn;
  }
  return w;
}

// Items of expert e: (row blocks of eight waves) x (token tiles) x (K
// slices); the exclusive prefix over the launch's experts goes to
// prefix[0 .. n_e].
template <int NK>
__global__ void __launch_bounds__(256) tile_plan_kernel(FfnArgs a, TileMap map, int32_t* __restrict__ prefix) {
  __shared__ int cnt[MOE_MAX_EXPERTS];
  const int i = threadIdx.x;
  int items = 0;
  if (i < map.n_e) {
    const int e = map.e0 + i;
    const int n_tok = a.offsets[e + 1] - a.offsets[e];
    const int tiles = (n_tok + kTileTok - 1) / kTileTok;
    const int R = NK == 1 ? a.d : (e < a.E ? a.f : a.fs);
    const TileWaves<NK> w = tile_waves<NK, false>(a, e, R);
    items = tiles * ((w.pre[TileWaves<NK>::NC] + kTileWaves - 1) / kTileWaves) * map.n_split;
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

// Magic fp16 pairs M whose mantissa unit is 1 at the bit offset of a code
// field: 1024.0 (bits 0..), 256.0 (2..), 64.0 (4..), 16.0 (6..).  A code q
// OR-ed into the field then reads exactly M + q.
constexpr uint32_t kMagicAt[4] = {0x64006400u, 0x5C005C00u, 0x54005400u, 0x4C004C00u};
constexpr float kMagicVal[4] = {1024.0f, 256.0f, 64.0f, 16.0f};

// Magic of component i (weights 2i, 2i+1) of a K-step: 4-bit codes sit at
// bits 0 and 4 of a byte (1024, 64), 2-bit codes and the low two bits of
// 3-bit codes at bits 0, 2, 4, 6 (1024, 256, 64, 16; a 3-bit code's high bit
// goes two bits above its low field); the other widths use 1024 throughout.
template <int B>
constexpr int kMagicOf(int i) {
  return (B == 2 || B == 3) ? i : (B == 4 ? 2 * (i & 1) : 0);
}

// Component i (weights 2i, 2i+1) of the B fragment of K-step s: two fp16
// weights s*(q - z) of this lane's row.  zn[i] = -(M + z) for the magic M of
// component i, mg the magics in registers.
template <int NM2, int B>
__device__ __forceinline__ uint32_t dequant_h1(const uint32_t (&cw)[(kHalfWords<NM2, B>)], int s, int i,
                                               const f16x2 (&zn)[4], f16x2 sc, const uint32_t (&mg)[4]) {
  if constexpr (B == 16) {
    // unquantized bf16 weights to fp16, rounding toward zero: exact for every
    // bf16 magnitude in [2^-17, 65504] (its last significand bit is >= 2^-24,
    // the fp16 subnormal spacing); larger magnitudes clamp to 65504
    const uint32_t w = cw[4 * s + i];
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(bf16_lo(w), bf16_hi(w)));
  }
  uint32_t r;
  if constexpr (B == 4) {
    // codes at bits 0-3 and 4-7 of each half's low byte (i = 0, 1) and high
    // byte (i = 2, 3): one shift per K-step word
    const uint32_t w = i < 2 ? cw[s] : cw[s] >> 8;
    r = (w & ((i & 1) ? 0x00F000F0u : 0x000F000Fu)) | mg[kMagicOf<4>(i)];
  } else if constexpr (B == 8) {
    // bytes (c0, c2, c1, c3): one byte permute with 0x64 bytes per pair gives
    // (0x64 << 8 | q) = 1024 + q in both halves
    r = __builtin_amdgcn_perm(kHigh64, cw[2 * s + (i >> 1)], (i & 1) ? 0x04030401u : 0x04020400u);
  } else if constexpr (B == 2) {
    // codes at bits 2i, 2i+1 of each half's low byte (even K-steps) or high
    // byte (odd K-steps)
    const uint32_t w = (s & 1) ? cw[s >> 1] >> 8 : cw[s >> 1];
    r = (w & (0x00030003u << (2 * i))) | mg[kMagicOf<2>(i)];
  } else if constexpr (B == 6) {  // per 32-code block: words 0-3 bits 0..3, words 4-5 bits 4..5
    const int blk = 6 * (s >> 2);
    const int q = s & 3;   // octet within the block
    const uint32_t lo = cw[blk + q], hi = cw[blk + 4 + (q >> 1)];
    const int o = (q & 1) * 8;
    r = (((lo >> (4 * i)) & 0x000F000Fu) | (((hi >> (o + 2 * i)) & 0x00030003u) << 4)) | mg[0];
  } else {  // 3-bit: per 32-code block words (low plane 0-15, low plane 16-31, high plane)
    // pair pi = 4q + i: low bits at bits 2*(pi & 7) of its low-plane word
    // (odd octets: the upper byte, shifted down once), high bit at bit pi of
    // the high plane, moved to two bits above the low field
    const int blk = 3 * (s >> 2);
    const int q = s & 3;   // octet within the block
    const uint32_t lo = (q & 1) ? cw[blk + (q >> 1)] >> 8 : cw[blk + (q >> 1)];
    const uint32_t hi = cw[blk + 2];
    const int sh = 4 * q + i - (2 * i + 2);   // high bit: from bit 4q + i to bit 2i + 2
    const uint32_t hs = sh >= 0 ? hi >> sh : hi << -sh;
    r = (lo & (0x00030003u << (2 * i))) | (hs & (0x00010001u << (2 * i + 2))) | mg[kMagicOf<3>(i)];
  }
  const f16x2 d = __builtin_bit_cast(f16x2, r) + zn[i];   // q - z, exact
  return __builtin_bit_cast(uint32_t, d * sc);              // s * (q - z), rounded once
}

// {s, z} word -> zn[i] = packed -(M + z) for component i's magic M (exact:
// integers <= 1279) and (s, s).
template <int B>
__device__ __forceinline__ void sz_pair(uint32_t w, f16x2 (&zn)[4], f16x2& sc) {
  const _Float16 s16 = __builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xFFFFu));
  const _Float16 z16 = __builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16));
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const _Float16 v = -(z16 + static_cast<_Float16>(kMagicVal[kMagicOf<B>(i)]));
    zn[i] = f16x2{v, v};
  }
  sc = f16x2{s16, s16};
}

template <int NM2, int BW>
struct HCodes {
  uint32_t cw[(kHalfWords<NM2, BW>)];
  uint32_t szw;
};

// Vector-memory instructions of one row's group in hload: the code loads and,
// except for unquantized weights (whose {s, z} word the dequantization does
// not read), the {s, z} load.  The waits of the tile kernel count these
// exactly: a load the compiler could drop as unused must not be issued.
template <int NM2, int BW>
constexpr int kGroupLoads = kCodeLoads<(kHalfWords<NM2, BW>)> + (BW == 16 ? 0 : 1);

template <int NM2, int BW>
__device__ __forceinline__ void hload(HCodes<NM2, BW>& st, const TSrc& sr, int gi, bool gv) {
  constexpr uint32_t gcb = NM2 * 16 * BW / 8;   // code bytes per row and group
  bload<kHalfWords<NM2, BW>>(st.cw, sr.code, gv ? sr.coff : kOOB, gv ? gi * gcb : 0u);
  if constexpr (BW == 16) st.szw = 0u;
  else st.szw = __builtin_amdgcn_raw_buffer_load_b32(sr.sz, gv ? sr.soff : kOOB, gv ? gi * sr.sz_gstride : 0u, 0);
}

// Wait until at most N vector-memory instructions are in flight.  Loads
// complete in issue order, so this makes every load issued before the last N
// complete.  The comment names the stage count and whether the wait ends the
// prologue, for the check of these counts against the compiled code
// (tests/test_tile_waits.py).
template <int N, int NS, int PRO>
__device__ __forceinline__ void hwait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  asm volatile("s_waitcnt vmcnt(%0) ; tile-wait ns=%1 pro=%2" ::"n"(N), "n"(NS), "n"(PRO) : "memory");
}

// Barrier without __syncthreads()' fences (those would drain the in-flight
// code loads); the LDS stages are ordered by the explicit waits around it.
__device__ __forceinline__ void tile_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// silu(g) * u with a hardware reciprocal: h is rounded to bf16 right after,
// far coarser than the reciprocal's error.
__device__ __forceinline__ float silu_mul_fast(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

// Stages of a tile item: 3 (codes of three groups and activations of two
// groups in flight) where the two sources' codes of a group take at most 16
// registers, else 2 (the accumulators of both sources leave no room).
template <int NM2, int BW0, int BW1>
constexpr int kTileStages =
    (kTileLdsStages == 3 && (kHalfWords<NM2, BW0>) + (kHalfWords<NM2, BW1>) <= 16) ? 3 : 2;

// Buffer source of one weight row of kind `kind`: the expert's own codes of
// width be, or the cached 8-bit copy of the row (copy).
template <int NM2>
__device__ __forceinline__ TSrc tile_src(const FfnArgs& a, int kind, bool copy, int be, int e, int R, int K, int row,
                                         bool live, int kh) {
  constexpr int g = NM2 * 16;
  const int G = K / g;
  const KindDev& kd = a.kd[kind];
  const uint32_t row_bytes = 4u * static_cast<uint32_t>(code_row_words(K, be));
  const uint32_t crow_bytes = 4u * static_cast<uint32_t>(code_row_words(K, 8));
  const void* cptr = copy ? static_cast<const void*>(kd.copy_codes)
                          : static_cast<const void*>(kd.codes + uni(kd.code_off[e]));
  const void* sptr = copy ? static_cast<const void*>(kd.copy_sz)
                          : static_cast<const void*>(kd.sz + uni(kd.sz_off[e]));
  const uint32_t cbytes = copy ? a.copy_bytes[kind] : static_cast<uint32_t>(R) * row_bytes;
  const uint32_t sbytes = copy ? a.copy_sz_bytes[kind] : static_cast<uint32_t>(R) * G * 4u;
  TSrc src;
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
  return src;
}

// One wave's share of a tile item against all of the item's tokens (TB
// 32-token blocks), over its positions [wpos, wend) of the expert's row
// order (one class; wpos >= wend for a wave past the expert's last class):
// gate/up takes the gate row (source 0) and the up row (source 1) of 32
// positions; down takes two blocks of 32 positions, wpos and wpos + 32.
// Source j has width BWj (the expert's base width be, or 8 where it reads the
// cached copies of a switched class, copyj).  NS, the item's stage count, is
// the same in every wave of the workgroup.
template <int NM2, int NK, int NS, int BW0, int BW1, int TB>
__device__ __forceinline__ void tile_item(const FfnArgs& a, const TileLds& lds, int e, bool copy0, bool copy1, int be,
                                          int wpos, int wend, int R, int t0, int t1, int sp, int n_split) {
  constexpr int g = NM2 * 16;
  constexpr int SPT = TileStage<NM2>::SPT;
  // activation slots of the tile's TB token blocks, and loads per thread and
  // stage (slots past them are written with zeros)
  constexpr int SL = TB * 32 * SPT;
  constexpr int NLD = (SL + 64 * kTileWaves - 1) / (64 * kTileWaves);
  constexpr bool down = NK == 1;
  static_assert(NS == 2 || (NS == 3 && kTileStages<NM2, BW0, BW1> == 3), "register budget of the code stages");
  // vector-memory instructions of one group's code and {s, z} loads (both
  // sources), and the loads that may stay in flight once the codes and the
  // activation stage of the next group have landed
  constexpr int LCG = kGroupLoads<NM2, BW0> + kGroupLoads<NM2, BW1>;
  constexpr int WAITN = NS == 3 ? 2 * LCG + NLD : LCG;
  const int tid = threadIdx.x;
  const int wv = uni(static_cast<int>(tid >> 6));
  const int lane = tid & 63;
  const int n = lane & 31, kh = lane >> 5;
  const bool routed = e < a.E;
  const int K = down ? (routed ? a.f : a.fs) : a.d;
  // the item's groups of K: [g0, g1), slice sp of n_split
  const int g0 = sp * (K / g) / n_split, g1 = (sp + 1) * (K / g) / n_split;
  const int32_t* order = down ? a.order_dn : a.order_gu;
  const bool wlive = wpos < wend;   // wave-uniform: a wave without positions only stages and waits
  const int q0 = wpos + n, q1 = down ? q0 + 32 : q0;
  const bool live0 = q0 < wend, live1 = q1 < wend;
  const int row0 = live0 ? (routed ? order[static_cast<int64_t>(e) * R + q0] : q0) : 0;
  const int row1 = down ? (live1 ? (routed ? order[static_cast<int64_t>(e) * R + q1] : q1) : 0) : row0;
  const TSrc src0 = tile_src<NM2>(a, down ? 2 : 0, copy0, be, e, R, K, row0, live0, kh);
  const TSrc src1 = tile_src<NM2>(a, down ? 2 : 1, copy1, be, e, R, K, row1, live1, kh);

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
    const bool gv = gi < g1;
    const uint32_t adv = gv ? 2u * static_cast<uint32_t>(gi * g) : 0u;
    u32x4* st = stage_of(lds, buf);
#pragma unroll
    for (int i = 0; i < NLD; i++) lds_dma16(xr, &st[64 * kTileWaves * i + 64 * wv], gv ? aoff[i] : kOOB, adv);
  };

  // the OR operands of the unpacking in vector registers (one v_and_or_b32
  // each); only the magics the two widths use
  uint32_t mg[4];
#pragma unroll
  for (int m = 0; m < 4; m++) {
    mg[m] = kMagicAt[m];
    const bool used = m == 0 || (m == 2 && (BW0 == 4 || BW1 == 4)) || BW0 == 2 || BW1 == 2 || BW0 == 3 ||
                      BW1 == 3;
    if (used) asm volatile("" : "+v"(mg[m]));
  }
  f32x16 acc0[TB], acc1[TB];
#pragma unroll
  for (int tb = 0; tb < TB; tb++) {
    acc0[tb] = f32x16{};
    acc1[tb] = f32x16{};
  }

  HCodes<NM2, BW0> c0[NS];
  HCodes<NM2, BW1> c1[NS];
  auto load = [&](HCodes<NM2, BW0>& x0, HCodes<NM2, BW1>& x1, int gi) {
    hload<NM2, BW0>(x0, src0, gi, gi < g1);
    hload<NM2, BW1>(x1, src1, gi, gi < g1);
  };
  stage_a(0, g0);
  load(c0[0], c1[0], g0);
  if constexpr (NS == 3) stage_a(1, g0 + 1);
  load(c0[1], c1[1], g0 + 1);
  if constexpr (NS == 3) load(c0[2], c1[2], g0 + 2);
  hwait_vm<WAITN, NS, 1>();   // codes and activations of group 0 have landed (this wave's share)
  tile_barrier();      // ... every wave's share

  auto group = [&](HCodes<NM2, BW0>& x0, HCodes<NM2, BW1>& x1, int buf, int gi) {
    // that stage was last read for group gi-1 (barrier since)
    stage_a((buf + NS - 1) % NS, gi + NS - 1);
    if (gi < g1 && wlive) {   // workgroup-uniform g1 (odd group counts), wave-uniform wlive
      const u32x4* st = stage_of(lds, buf);
      // the slot of K-step s and token block tb is a0 ^ s plus 32*SPT*tb
      // (n % SPT is the swizzle of every token block, and s < NM2 touches
      // only the low bits of kh*NM2); a0 passes through an empty asm so the
      // eight K-step addresses are formed here, not kept live over the loop
      uint32_t a0 = static_cast<uint32_t>(n * SPT + ((kh * NM2) ^ (n % SPT)));
      asm volatile("" : "+v"(a0));
      f16x2 zn0[4], sc0, zn1[4], sc1;
      sz_pair<BW0>(x0.szw, zn0, sc0);
      sz_pair<BW1>(x1.szw, zn1, sc1);
      // Software pipeline over the K-steps, fixed by scheduling fences (the
      // compiler would otherwise move each LDS read next to its first MFMA
      // and wait for it there): each MFMA of source 0 is issued with a
      // quarter of source 1's fragment; each MFMA of source 1 with the next
      // K-step's read into the activation register it has just read last
      // and a quarter of source 0's next fragment.
      u32x4 af[TB], b0, b1;
#pragma unroll
      for (int tb = 0; tb < TB; tb++) af[tb] = st[a0 + 32 * SPT * tb];
#pragma unroll
      for (int i = 0; i < 4; i++) b0[i] = dequant_h1<NM2, BW0>(x0.cw, 0, i, zn0, sc0, mg);
#pragma unroll
      for (int s = 0; s < NM2; s++) {
        const uint32_t an = a0 ^ static_cast<uint32_t>(s + 1);
#pragma unroll
        for (int tb = 0; tb < TB; tb++) {
          acc0[tb] = mfma32h(af[tb], b0, acc0[tb]);
#pragma unroll
          for (int i = tb; i < 4; i += TB) b1[i] = dequant_h1<NM2, BW1>(x1.cw, s, i, zn1, sc1, mg);
          __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int tb = 0; tb < TB; tb++) {
          acc1[tb] = mfma32h(af[tb], b1, acc1[tb]);
          if (s + 1 < NM2) {
            af[tb] = st[an + 32 * SPT * tb];
#pragma unroll
            for (int i = tb; i < 4; i += TB) b0[i] = dequant_h1<NM2, BW0>(x0.cw, s + 1, i, zn0, sc0, mg);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    load(x0, x1, gi + NS);
    hwait_vm<WAITN, NS, 0>();   // everything but the newer loads: group gi+1's codes and activations
    tile_barrier();
  };
  for (int gi = g0; gi < g1; gi += NS) {
    group(c0[0], c1[0], 0, gi);
    group(c0[1], c1[1], 1, gi + 1);
    if constexpr (NS == 3) group(c0[2], c1[2], 2, gi + 2);
  }
  hwait_vm<0, 0, 0>();
  if (!wlive) return;

  // outputs: tokens t0 + 32*tb + 8*(r/4) + 4*kh + r%4, stored through a
  // buffer resource over the tile's rows (the token's part of the offset is
  // the scalar offset; a lane's offset is kOOB past its class or, in a
  // partial tile, past the segment, which drops the store)
  const int lim = t1 - t0 - 4 * kh;   // the lane's tokens t0 + 4*kh + dt exist for dt < lim
  const bool full = t1 - t0 == 32 * TB;   // workgroup-uniform
  if constexpr (!down) {
    // rows of one item are all routed or all shared: one h row width
    const int hw = t0 < a.Tk ? a.f : a.fs;
    const Rsrc hr = make_rsrc(a.h + h_row(a, t0), static_cast<uint32_t>(kTileTok * hw * 2));
    const uint32_t off = live0 ? 2u * static_cast<uint32_t>(4 * kh * hw + row0) : kOOB;
    uint32_t hmax = 0u;   // running maximum of the fp16 magnitudes (bit patterns), per half
#pragma unroll
    for (int tb = 0; tb < TB; tb++)
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const int dt = tb * 32 + 8 * (r / 4) + (r % 4);   // element r + 1 is token dt + 1
        // h = bf16(silu(g) * u) (round to nearest even), stored as its fp16
        // value: exact unless below 2^-17 in magnitude or beyond fp16's range
        const f32x2 v = {silu_mul_fast(acc0[tb][r], acc1[tb][r]), silu_mul_fast(acc0[tb][r + 1], acc1[tb][r + 1])};
        const uint32_t hb = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
        const f32x2 hv = {bf16_lo(hb), bf16_hi(hb)};
        const uint32_t h16 = __builtin_bit_cast(uint32_t, __builtin_convertvector(hv, f16x2));
        hmax = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2, hmax),
                                                                      __builtin_bit_cast(u16x2, h16 & 0x7FFF7FFFu)));
        const uint32_t o0 = (full || dt < lim) ? off : kOOB, o1 = (full || dt + 1 < lim) ? off : kOOB;
        __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(h16), hr, o0, static_cast<uint32_t>(dt * hw * 2), 0);
        __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(h16 >> 16), hr, o1,
                                              static_cast<uint32_t>((dt + 1) * hw * 2), 0);
      }
    // fp16 infinity or NaN (0x7C00 and above) where a stored value did not fit;
    // values a lane does not store come from zero accumulators or rows past
    // the segment, whose h is never read, so they take part in the check too
    if (live0 && ((hmax & 0xFFFFu) >= 0x7C00u || (hmax >> 16) >= 0x7C00u) && a.status) *a.status = MOE_ERR_RANGE;
  } else {
    // slice sp of o (the combine adds the slices)
    const Rsrc orc = make_rsrc(a.o + sp * a.split_stride + static_cast<int64_t>(t0) * R,
                               static_cast<uint32_t>(kTileTok * R * 4));
    const uint32_t off0 = live0 ? 4u * static_cast<uint32_t>(4 * kh * R + row0) : kOOB;
    const uint32_t off1 = live1 ? 4u * static_cast<uint32_t>(4 * kh * R + row1) : kOOB;
#pragma unroll
    for (int tb = 0; tb < TB; tb++)
#pragma unroll
      for (int r = 0; r < 16; r++) {
        const int dt = tb * 32 + 8 * (r / 4) + (r % 4);
        const bool ok = full || dt < lim;
        const uint32_t so = static_cast<uint32_t>(dt * R * 4);
        // through float temporaries: a bit cast of a vector element itself
        // takes element 0 in this compiler
        const float v0 = acc0[tb][r], v1 = acc1[tb][r];
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v0), orc, ok ? off0 : kOOB, so, 0);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v1), orc, ok ? off1 : kOOB, so, 0);
      }
  }
}

// The wave's class picks each source's width: gate/up class bit j set =
// kind j reads the 8-bit copies; down class 1 = copies.  The item's stage
// count: the narrow widths' three stages where every wave of the item is of
// class 0, else two.  The token tile of the item (an expert's last tile is
// partial) picks one, two or four 32-token blocks.
template <int NM2, int NK, int B>
__device__ __forceinline__ void tile_dispatch(const FfnArgs& a, const TileLds& lds, int e, int cls, bool base_item,
                                              int wpos, int wend, int R, int t0, int t1, int sp, int n_split) {
  const int nt = t1 - t0;
  auto by_tb = [&](auto ns, auto w0, auto w1, bool c0, bool c1) {
    constexpr int NS = decltype(ns)::value, W0 = decltype(w0)::value, W1 = decltype(w1)::value;
    if (nt <= 32) tile_item<NM2, NK, NS, W0, W1, 1>(a, lds, e, c0, c1, B, wpos, wend, R, t0, t1, sp, n_split);
    else if (nt <= 64) tile_item<NM2, NK, NS, W0, W1, 2>(a, lds, e, c0, c1, B, wpos, wend, R, t0, t1, sp, n_split);
    else tile_item<NM2, NK, NS, W0, W1, 4>(a, lds, e, c0, c1, B, wpos, wend, R, t0, t1, sp, n_split);
  };
  using WB = std::integral_constant<int, B>;
  using W8 = std::integral_constant<int, 8>;
  using S2 = std::integral_constant<int, 2>;
  using SB = std::integral_constant<int, kTileStages<NM2, B, B>>;
  if (cls == 0) {
    if (base_item) by_tb(SB{}, WB{}, WB{}, false, false);
    else by_tb(S2{}, WB{}, WB{}, false, false);
  } else if constexpr (NK == 1 || B == 8) {
    by_tb(S2{}, W8{}, W8{}, (cls & 1) != 0, NK == 1 || (cls & 2) != 0);
  } else {
    if (cls == 1) by_tb(S2{}, W8{}, WB{}, true, false);
    else if (cls == 2) by_tb(S2{}, WB{}, W8{}, false, true);
    else by_tb(S2{}, W8{}, W8{}, true, true);
  }
}

// Eight waves, two per SIMD: a wave's accumulators (two sources x four token
// blocks, 128 registers) leave room for a second wave, which hides the
// first one's load and LDS latencies.
template <int NM2, int NK>
__global__ void __launch_bounds__(64 * kTileWaves) __attribute__((amdgpu_waves_per_eu(2)))
ffn_tile_kernel(FfnArgs a, TileMap map, const int32_t* __restrict__ prefix) {
  __shared__ __attribute__((aligned(16))) u32x4 st0[TileStage<NM2>::SLOTS];
  __shared__ __attribute__((aligned(16))) u32x4 st1[TileStage<NM2>::SLOTS];
  __shared__ __attribute__((aligned(16))) u32x4 st2[kTileLdsStages == 3 ? TileStage<NM2>::SLOTS : 1];
  __shared__ int pre[MOE_MAX_EXPERTS + 1];
  const TileLds lds{st0, st1, st2};
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
    int local = item - pre[lo];
    const int seg0 = uni(a.offsets[e]), seg1 = uni(a.offsets[e + 1]);
    const int tiles = (seg1 - seg0 + kTileTok - 1) / kTileTok;
    const bool routed = e < a.E;
    const int R = NK == 1 ? a.d : (routed ? a.f : a.fs);
    // the expert's waves, class after class; eight waves per row block
    const TileWaves<NK> w = tile_waves<NK, true>(a, e, R);
    constexpr int NC = TileWaves<NK>::NC;
    const int n_w = w.pre[NC];
    const int n_rb = (n_w + kTileWaves - 1) / kTileWaves;
    // (K slice, row block, token tile) of the local index: slices outermost;
    // within a slice super-rows of kSuper row blocks, token tiles outer and
    // row blocks inner within a super-row
    const int sp = local / (n_rb * tiles);
    local -= sp * n_rb * tiles;
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
    // this wave's class and positions; the item runs three stages only when
    // all of its waves are of class 0
    const int gw = rb * kTileWaves + uni(static_cast<int>(threadIdx.x >> 6));
    int cls = 0;
#pragma unroll
    for (int c = 1; c < NC; c++) cls += gw >= w.pre[c] ? 1 : 0;
    const bool dead = gw >= n_w;
    const int wpos = dead ? 0 : w.beg[cls] + (gw - w.pre[cls]) * kTileWaveRows<NK>;
    const int wend = dead ? 0 : min(wpos + kTileWaveRows<NK>, w.beg[cls] + w.cnt[cls]);
    if (dead) cls = 0;
    const bool base_item = min((rb + 1) * kTileWaves, n_w) <= w.pre[1];
    const int t0 = seg0 + tt * kTileTok, t1 = min(t0 + kTileTok, seg1);
    const int B = map.bits[e - map.e0];
    if (B == 8) tile_dispatch<NM2, NK, 8>(a, lds, e, cls, base_item, wpos, wend, R, t0, t1, sp, map.n_split);
    else if (NM2 == 4 && B == 16) {   // unquantized experts need group 64
      if constexpr (NM2 == 4)
        tile_dispatch<NM2, NK, 16>(a, lds, e, cls, base_item, wpos, wend, R, t0, t1, sp, map.n_split);
    } else if (B == 4) tile_dispatch<NM2, NK, 4>(a, lds, e, cls, base_item, wpos, wend, R, t0, t1, sp, map.n_split);
    else if (B == 2) tile_dispatch<NM2, NK, 2>(a, lds, e, cls, base_item, wpos, wend, R, t0, t1, sp, map.n_split);
    else if constexpr (NM2 % 4 == 0) {
      if (B == 6) tile_dispatch<NM2, NK, 6>(a, lds, e, cls, base_item, wpos, wend, R, t0, t1, sp, map.n_split);
      else tile_dispatch<NM2, NK, 3>(a, lds, e, cls, base_item, wpos, wend, R, t0, t1, sp, map.n_split);
    }
    tile_barrier();   // the LDS stages are reused by the next item
  }
}

// Instantiations: every group size by default; a build may compile this file
// once per group size (MOE_FFN_NM = 2 or 4, that is 64 or 128).
#if !defined(MOE_FFN_NM) || MOE_FFN_NM == 2
template __global__ void tile_plan_kernel<1>(FfnArgs, TileMap, int32_t*);
template __global__ void tile_plan_kernel<2>(FfnArgs, TileMap, int32_t*);
template __global__ void ffn_tile_kernel<4, 1>(FfnArgs, TileMap, const int32_t*);
template __global__ void ffn_tile_kernel<4, 2>(FfnArgs, TileMap, const int32_t*);
#endif
#if !defined(MOE_FFN_NM) || MOE_FFN_NM == 4
template __global__ void ffn_tile_kernel<8, 1>(FfnArgs, TileMap, const int32_t*);
template __global__ void ffn_tile_kernel<8, 2>(FfnArgs, TileMap, const int32_t*);
#endif

}  // namespace ffn
}  // namespace moe
