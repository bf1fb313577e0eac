// ffn_common.hpp -- types, constants and device helpers shared by the
// expert-FFN kernels (ffn_stream.hip: the streaming kernel for experts with
// few tokens and the activation preparation kernels; ffn_tile.hip: the tile
// kernel for experts with many tokens) and their host code (ffn.hip).
#pragma once

#include "common.hpp"

namespace moe {
namespace ffn {


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
  int n_split_out;     // K slices of the down projection: slices of o the combine adds
  int32_t* tile_prefix;   // workspace: 4 x (MOE_MAX_EXPERTS + 1) item prefixes
  const uint16_t* x16;  // [T][d] fp16 copy of x (tile kernel; row of permuted row p: perm[p])
  int32_t* status;      // device status word or null: MOE_ERR_RANGE when an fp16 operand overflows
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
constexpr float kOffset = (B == 8 || B == 16) ? 0.f : (B == 3 ? 640.f : (B == 6 ? 2176.f : 128.f));

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
  } else if constexpr (B == 16) {   // unquantized bf16 weights: the operand as stored
#pragma unroll
    for (int m = 0; m < NM; m++) wf[0][m] = u32x4{cw[4 * m], cw[4 * m + 1], cw[4 * m + 2], cw[4 * m + 3]};
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

// ------------------------------------------------------------------ launch maps
// Waves per workgroup: four for gate/up; eight for down, whose tile of
// activations (h) is then shared by twice the rows (measured: the down
// launch 7 % faster, gate/up not).
template <int NK>
constexpr int kWavesOf = NK == 1 ? 8 : 4;

// Row tiles of 16 rows per wave for a class whose rows all read base codes
// of width b, shared by the kernel and the host's work map.  Measured on
// MI355X: two row tiles per wave at 3 and 4 bits and three at 2 bits
// (workgroups streaming about as many bytes as an 8-bit one) left a layer of
// one width unchanged and the mixed layers slower (fewer, equal workgroups
// leave a partial last round), so every width takes one.
__host__ __device__ constexpr int stream_rt(int b) { return b > 0 ? 1 : 1; }

// Work map of one streaming launch.  Workgroups [0, n_r*n_sw*m_r) take the
// switched classes of routed experts 0..n_r-1 (n_sw row blocks of one row
// tile per wave per expert, m_r variants each); the rest are the class-0
// row blocks of the entries ent_e[0..n_ent), entry i owning workgroups
// [ent_start[i], ent_start[i+1]) after the switched section: its row blocks
// (kWavesOf<NK> * 16 * stream_rt(bits) rows each) times its variants (m_r
// for routed, m_s for shared experts).  A variant is a token-tile set
// (tt_r / tt_s sets, each taking every n-th 32-token tile of the expert)
// and a K slice (n_split).
struct WgMap {
  int n_r, n_sw, m_r, m_s, tt_r, tt_s, n_split, n_ent;
  int32_t ent_start[MOE_MAX_EXPERTS + 1];
  int16_t ent_e[MOE_MAX_EXPERTS];
  int8_t bits[MOE_MAX_EXPERTS];   // bit-width of expert e (routed and shared)
};

constexpr int kTileTok = 128;   // tokens per workgroup tile (four 32-token blocks)

// Row positions per wave of the tile kernel: the gate and the up row of 32
// positions, or 64 down rows.  A workgroup's item is eight such waves.
template <int NK>
constexpr int kTileWaveRows = NK == 2 ? 32 : 64;

// Workgroups of the tile kernel resident per compute unit, and its waves per
// workgroup (two waves per SIMD in all) and LDS stages (three stages of one
// workgroup or two of each of two fit the 160 KB of LDS).
constexpr int kTileWgPerCu = 1;
constexpr int kTileWaves = 8 / kTileWgPerCu;
constexpr int kTileLdsStages = kTileWgPerCu == 1 ? 3 : 2;

constexpr int kXcds = 8;
constexpr int kSuper = 8;

// Experts e0 .. e0+n_e-1 of one tile launch; bits[e - e0].
struct TileMap {
  int e0, n_e;
  int n_split;   // K slices per item (down projection; 1 for gate/up)
  int8_t bits[MOE_MAX_EXPERTS];
};

// ------------------------------------------------------------------ kernels
// Defined in ffn_stream.hip and ffn_tile.hip; launched by the host code of
// ffn.hip.
template <int NM, int NT, int NK>
__global__ void __launch_bounds__(64 * kWavesOf<NK>) __attribute__((amdgpu_waves_per_eu(2)))
ffn_stream_kernel(FfnArgs a, WgMap map);

template <int NM>
__global__ void __launch_bounds__(256)
group_sum_kernel(FfnArgs a, const uint16_t* __restrict__ in, const int32_t* __restrict__ perm,
                 int64_t ld, int p0, int p1, int K, int p_split, int K2, float* __restrict__ out);

__global__ void __launch_bounds__(256) gather_f16_kernel(FfnArgs a, int T);

template <int NK>
__global__ void __launch_bounds__(256) tile_plan_kernel(FfnArgs a, TileMap map, int32_t* __restrict__ prefix);

template <int NM2, int NK>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2)))
ffn_tile_kernel(FfnArgs a, TileMap map, const int32_t* __restrict__ prefix);

}  // namespace ffn
}  // namespace moe
