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
#include "ffn_common.hpp"

namespace moe {
namespace ffn {

// ------------------------------------------------------------------ streaming kernel
// One workgroup = kWavesOf<NK> waves on one expert and one source class of its rows.
// Each wave owns 16*RT consecutive positions of the expert's row order for
// each of NK weight kinds (NK = 2: the gate and up rows of the same neurons;
// NK = 1: down rows = output channels).  Within a class every kind has one
// source for all rows -- the expert's base codes at bit-width B, or the
// cached 8-bit copies -- so the loads are wave-uniform in shape and the code
// registers are sized for that width (template BG / BU).  The packed codes of
// the next kStages<RT, BG, BU> groups are in flight in registers while the current group
// is dequantized and contracted; the activations of the workgroup's token
// tile (NT*16 rows) are staged in LDS two groups at a time (double-buffered,
// one barrier per two groups), so every wave reads them from LDS.

// Groups of codes in flight per wave: four, or two when a kind streams 8- or
// 6-bit codes (about the same bytes in flight in half the registers).  The activations
// of chunk c+2 are loaded while chunk c is contracted, so that waiting for
// them (vector loads complete in order) never waits for a code load the loop
// does not already need: with two-group chunks that holds for up to four
// groups in flight.
// With two or four row tiles per wave (narrow codes) two groups in flight
// already hold as many bytes as four groups of one row tile.
template <int RT, int BG, int BU>
constexpr int kStages = (RT >= 2 || BG >= 8 || BU >= 8 || BG == 6 || BU == 6) ? 2 : 4;


// Metadata a workgroup loads in its prologue, all issued before any is
// waited for (a chain of dependent loads at the start of every workgroup
// costs more than the loads themselves).
struct Pre {
  int64_t code_off[2], sz_off[2];   // per kind of the launch
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

// The row tiles of a wave are contracted in turn, software-pipelined: the
// MFMAs of row tile rt are issued before the scale/zero epilogue of tile
// rt - 1, so the matrix cores work on one tile while the epilogue of the
// previous one runs, and only two tiles' partial sums are live at once.
template <int NM, int NT, int RT, int NK, int BG, int BU>
__device__ __forceinline__ void compute_group(const Stage<NM, RT, BG, BU>& st, const uint32_t (&szw)[RT][2],
                                              const u32x4 (&af)[NT][NM], const f32x4 (&X)[NT],
                                              uint32_t vm, uint32_t vh, f32x4 (&acc)[RT][NK][NT]) {
  f32x4 tmp[2][NK][NT];
  float sc[2][NK], zz[2][NK];
#pragma unroll
  for (int rt = 0; rt <= RT; rt++) {
    if (rt < RT) {
      const int b = rt & 1;
      contract_kind<NM, NT, BG>(st.cg[rt], szw[rt][0], af, vm, vh, tmp[b][0], sc[b][0], zz[b][0]);
      if constexpr (NK == 2)
        contract_kind<NM, NT, BU>(st.cu[rt], szw[rt][1], af, vm, vh, tmp[b][1], sc[b][1], zz[b][1]);
    }
    if (rt > 0) {
      const int b = (rt - 1) & 1;
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < NK; kk++)
#pragma unroll
        for (int nt = 0; nt < NT; nt++)
#pragma unroll
          for (int i = 0; i < 4; i++)
            acc[rt - 1][kk][nt][i] = __fmaf_rn(sc[b][kk], __fmaf_rn(-zz[b][kk], X[nt][i], tmp[b][kk][nt][i]),
                                               acc[rt - 1][kk][nt][i]);
    }
  }
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
  constexpr int S = kStages<RT, BG, BU>;
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
    // positions past the class (pos >= pos1) are not read: for the last
    // expert's last class they would lie past the end of the order table
    const int prow = (live[rt] && routed) ? order[static_cast<int64_t>(e) * R + pos] : 0;
    row_id[rt] = live[rt] ? (routed ? prow : pos) : 0;
  }
  // a wave whose rows all lie past the class (the last workgroup of an
  // expert whose rows do not fill it) still stages activations and meets the
  // barriers, but contracts nothing
  const bool wave_live = uni(pos0 + wv * 16 * RT) < pos1;
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
      if (gi < g1 && wave_live) {   // wave-uniform; the loads below are unconditional
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


// Class 0 (both kinds on the expert's base codes) takes stream_rt(B) row
// tiles per wave; the switched classes (one or both kinds on the 8-bit
// copies) one.
template <int NM, int NT, int NK, int B>
__device__ __forceinline__ void dispatch_class(const FfnArgs& a, XTile<NM, NT>& tl, const Pre& pre, int e,
                                               int cls, int pos0, int pos1, int R, int sp, int n_split) {
  constexpr int RT0 = stream_rt(B);
  if constexpr (NK == 1) {
    if (cls == 0) stream_body<NM, NT, RT0, 1, B, B>(a, tl, pre, e, 0, pos0, pos1, R, sp, n_split);
    else stream_body<NM, NT, 1, 1, 8, 8>(a, tl, pre, e, 1, pos0, pos1, R, sp, n_split);
  } else {
    if (cls == 0) stream_body<NM, NT, RT0, 2, B, B>(a, tl, pre, e, 0, pos0, pos1, R, sp, n_split);
    else if (cls == 1) stream_body<NM, NT, 1, 2, 8, B>(a, tl, pre, e, 1, pos0, pos1, R, sp, n_split);
    else if (cls == 2) stream_body<NM, NT, 1, 2, B, 8>(a, tl, pre, e, 2, pos0, pos1, R, sp, n_split);
    else stream_body<NM, NT, 1, 2, 8, 8>(a, tl, pre, e, 3, pos0, pos1, R, sp, n_split);
  }
}

// Local index l of a workgroup inside a run of nblk row blocks with m
// variants each (token-tile sets x K slices) -> (block, variant).  Blocks
// go in chunks of 8 with the variant outside the block inside a chunk, so
// the variants of one block are 8 workgroups apart: the hardware places
// workgroup b on XCD b % 8, so they run on one XCD and share its L2 (the
// block's codes are read from HBM once).
__device__ __forceinline__ void block_variant(int l, int nblk, int m, int& blk, int& v) {
  const int c = l / (8 * m);
  const int r = l - c * 8 * m;
  const int nb = min(8, nblk - 8 * c);
  v = r / nb;
  blk = 8 * c + (r - v * nb);
}

// One launch serves every streamed expert of a stage: the switched-class
// workgroups of the routed experts first (n_sw per expert, an upper bound on
// what its copies can need; those past its actual class sizes exit at once),
// then the class-0 workgroups of the entries of the map (shared experts,
// then routed experts widest first), each entry's row blocks sized by its
// bit-width so that every workgroup streams about the same bytes.
template <int NM, int NT, int NK>
__global__ void __launch_bounds__(64 * kWavesOf<NK>) __attribute__((amdgpu_waves_per_eu(2)))
ffn_stream_kernel(FfnArgs a, WgMap map) {
  __shared__ __attribute__((aligned(16))) XTile<NM, NT> tl;
  constexpr int rows1 = kWavesOf<NK> * 16;   // rows of one row tile per wave
  const int bid = blockIdx.x;
  const int n_swg = map.n_r * map.n_sw * map.m_r;
  int e, blk, v;
  const bool sw = bid < n_swg;
  if (sw) {
    const int per = map.n_sw * map.m_r;
    e = bid / per;
    block_variant(bid - e * per, map.n_sw, map.m_r, blk, v);
  } else {
    const int w = bid - n_swg;
    int lo = 0, hi = map.n_ent - 1;   // last entry whose start is <= w
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (map.ent_start[mid] <= w) lo = mid; else hi = mid - 1;
    }
    e = map.ent_e[lo];
    const int m = e < a.E ? map.m_r : map.m_s;
    block_variant(w - map.ent_start[lo], (map.ent_start[lo + 1] - map.ent_start[lo]) / m, m, blk, v);
  }
  const bool routed = e < a.E;
  const int n_tt = routed ? map.tt_r : map.tt_s;
  const int tt = v % n_tt, sp = v / n_tt;
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
  if (uni(o1) <= uni(o0)) return;
  const int B = map.bits[e];
  int cls = 0, start = 0, count = R, rows = rows1 * stream_rt(B);
  if (routed) {
#pragma unroll
    for (int c = 0; c < 4; c++) cnt[c] = uni(cnt[c]);
    count = cnt[0];
    if (sw) {   // find the switched class of this workgroup
      rows = rows1;
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
      count = cnt[cls];
    }
  }
  const int pos0 = start + blk * rows;
  if (blk * rows >= count) return;
  const int pos1 = min(pos0 + rows, start + count);
  const int n_split = map.n_split;
  if constexpr (NT == 2) {
    // an expert with at most 16 tokens needs one 16-token tile: half the
    // contraction and epilogue work of the 32-token tile (same LDS)
    if (uni(o1) - uni(o0) <= 16) {
      auto& t1 = *reinterpret_cast<XTile<NM, 1>*>(&tl);
      if (B == 8) dispatch_class<NM, 1, NK, 8>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      else if (NM == 2 && B == 16) {   // unquantized experts need group 64
        if constexpr (NM == 2) dispatch_class<NM, 1, NK, 16>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      } else if (B == 4) dispatch_class<NM, 1, NK, 4>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      else if (B == 2) dispatch_class<NM, 1, NK, 2>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      else if constexpr (NM == 4) {
        if (B == 6) dispatch_class<NM, 1, NK, 6>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
        else dispatch_class<NM, 1, NK, 3>(a, t1, pre, e, cls, pos0, pos1, R, sp, n_split);
      }
      return;
    }
  }
  if (B == 8) dispatch_class<NM, NT, NK, 8>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  else if (NM == 2 && B == 16) {   // unquantized experts need group 64
    if constexpr (NM == 2) dispatch_class<NM, NT, NK, 16>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  } else if (B == 4) dispatch_class<NM, NT, NK, 4>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  else if (B == 2) dispatch_class<NM, NT, NK, 2>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  else if constexpr (NM == 4) {
    if (B == 6) dispatch_class<NM, NT, NK, 6>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
    else dispatch_class<NM, NT, NK, 3>(a, tl, pre, e, cls, pos0, pos1, R, sp, n_split);
  }
}

// Instantiations: every group size by default; a build may compile this file
// once per group size (MOE_FFN_NM = 2 or 4, that is 64 or 128) to spread the
// work over several compiler processes.
#if !defined(MOE_FFN_NM) || MOE_FFN_NM == 2
template __global__ void ffn_stream_kernel<2, 1, 1>(FfnArgs, WgMap);
template __global__ void ffn_stream_kernel<2, 1, 2>(FfnArgs, WgMap);
template __global__ void ffn_stream_kernel<2, 2, 1>(FfnArgs, WgMap);
template __global__ void ffn_stream_kernel<2, 2, 2>(FfnArgs, WgMap);
#endif
#if !defined(MOE_FFN_NM) || MOE_FFN_NM == 4
template __global__ void ffn_stream_kernel<4, 1, 1>(FfnArgs, WgMap);
template __global__ void ffn_stream_kernel<4, 1, 2>(FfnArgs, WgMap);
template __global__ void ffn_stream_kernel<4, 2, 1>(FfnArgs, WgMap);
template __global__ void ffn_stream_kernel<4, 2, 2>(FfnArgs, WgMap);
#endif

}  // namespace ffn
}  // namespace moe
