// pack.hip -- moe_quant_pack: group-wise asymmetric uniform quantization of
// fp32 rows and packing of the codes into 32-bit words; moe_requant_channels:
// the same quantizer applied to cached 16-bit channels, written into the
// 8-bit copy slots the FFN reads.
//
// Sec. IV-A (each expert quantized uniformly at its precision), Sec. V-B
// (several low-bit codes loaded as one 32-bit word) and Sec. IV-B
// (requantization of the cached channels for a new dataset).  The quantizer and the
// word layout are defined in moe_quant.h; parameter math is binary64, which
// gfx950 rounds exactly as IEEE requires, so the codes are reproducible bit
// for bit on any IEEE host.
#include "common.hpp"

namespace moe {
namespace {

// Smallest binary16 >= s for a finite s > 0, by truncating the binary64
// significand and bumping the last kept bit when anything was cut off.
// Returns 0x7C00 (+inf) past 65504.
__device__ uint32_t fp16_ceil_bits(double s) {
  const uint64_t b = static_cast<uint64_t>(__double_as_longlong(s));
  const int e = static_cast<int>((b >> 52) & 0x7FF) - 1023;
  const uint64_t frac = b & ((1ull << 52) - 1);
  if (e < -24) return 1u;  // below the smallest subnormal 2^-24
  if (e < -14) {           // subnormal grid k * 2^-24, k = ceil(s * 2^24)
    const uint64_t full = (1ull << 52) | frac;
    const int sh = 52 - (e + 24);
    uint64_t k = full >> sh;
    if (full & ((1ull << sh) - 1)) k++;
    return static_cast<uint32_t>(k);  // k == 1024 is the pattern of 2^-14
  }
  if (e > 15) return 0x7C00u;
  uint32_t h = static_cast<uint32_t>(((e + 15) << 10) | (frac >> 42));
  if (frac & ((1ull << 42) - 1)) h++;  // may carry into the exponent, up to +inf
  return h;
}

// Value of an fp16 bit pattern as binary64 (exact).
__device__ double fp16_to_f64(uint32_t h) { return static_cast<double>(fp16_bits_to_f32(h)); }

// binary16 pattern of an integer 0 <= z <= 255 (exact).
__device__ uint32_t fp16_of_small_int(int z) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(static_cast<float>(z)));
}

// Bit position of local code i in a word of the b-bit half-split order.
__device__ __forceinline__ int hs_pos(int i, int b) { return (i >> 1) * b + 16 * (i & 1); }

// One thread per (list row, group).
__global__ void __launch_bounds__(256)
pack_kernel(const float* __restrict__ w, int64_t ld_w, int K, int bits, int group,
            const int32_t* __restrict__ rows, int n, uint32_t* __restrict__ codes,
            int64_t ld_codes, uint32_t* __restrict__ sz, int64_t sz_rs, int64_t sz_gs,
            int32_t* status) {
  const int G = K / group;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= static_cast<int64_t>(n) * G) return;
  const int i = static_cast<int>(id / G);
  const int j = static_cast<int>(id % G);
  const int r = rows ? rows[i] : i;
  const float* wg = w + static_cast<int64_t>(r) * ld_w + static_cast<int64_t>(j) * group;

  if (bits == 16) {   // unquantized: the bf16 value of each weight, scale 1 and zero 0
    uint32_t* out = codes + static_cast<int64_t>(i) * ld_codes + static_cast<int64_t>(j) * (group / 2);
    for (int t = 0; t < group / 2; t++)
      out[t] = bf16_rne(wg[2 * t]) | (bf16_rne(wg[2 * t + 1]) << 16);
    sz[static_cast<int64_t>(i) * sz_rs + static_cast<int64_t>(j) * sz_gs] = 0x3C00u;
    return;
  }
  double mn = 0.0, mx = 0.0;
  for (int c = 0; c < group; c++) {
    const double v = static_cast<double>(wg[c]);
    mn = v < mn ? v : mn;
    mx = v > mx ? v : mx;
  }
  const int qmax = (1 << bits) - 1;
  const double s = (mx - mn) / static_cast<double>(qmax);
  const uint32_t sb = (s == 0.0) ? 0x3C00u : fp16_ceil_bits(s);
  if (sb == 0x7C00u && status) *status = MOE_ERR_RANGE;
  const double sf = fp16_to_f64(sb);
  int z = static_cast<int>(rint(-mn / sf));
  z = z < 0 ? 0 : z;
  sz[static_cast<int64_t>(i) * sz_rs + static_cast<int64_t>(j) * sz_gs] =
      sb | (fp16_of_small_int(z) << 16);

  auto code = [&](int c) -> uint32_t {
    double t = rint(static_cast<double>(wg[c]) / sf) + static_cast<double>(z);
    t = t < 0.0 ? 0.0 : (t > static_cast<double>(qmax) ? static_cast<double>(qmax) : t);
    return static_cast<uint32_t>(t);
  };

  uint32_t* out = codes + static_cast<int64_t>(i) * ld_codes +
                  static_cast<int64_t>(j) * (group * bits / 32);
  if (bits == 6) {   // per 32-code block: bits 0..3 in four 4-bit words, bits 4..5 in two 2-bit words
    for (int blk = 0; blk < group / 32; blk++) {
      uint32_t w[6] = {0, 0, 0, 0, 0, 0};
      for (int l = 0; l < 32; l++) {
        const uint32_t q = code(blk * 32 + l);
        w[l >> 3] |= (q & 15u) << hs_pos(l & 7, 4);
        w[4 + (l >> 4)] |= (q >> 4) << hs_pos(l & 15, 2);
      }
      for (int i = 0; i < 6; i++) out[6 * blk + i] = w[i];
    }
  } else if (bits != 3) {
    const int per = 32 / bits;
    for (int t = 0; t < group / per; t++) {
      uint32_t word = 0;
      for (int l = 0; l < per; l++) word |= code(t * per + l) << hs_pos(l, bits);
      out[t] = word;
    }
  } else {
    for (int blk = 0; blk < group / 32; blk++) {
      uint32_t lo0 = 0, lo1 = 0, hi = 0;
      for (int l = 0; l < 32; l++) {
        const uint32_t q = code(blk * 32 + l);
        if (l < 16)
          lo0 |= (q & 3u) << hs_pos(l, 2);
        else
          lo1 |= (q & 3u) << hs_pos(l - 16, 2);
        hi |= ((q >> 2) & 1u) << hs_pos(l, 1);
      }
      out[3 * blk] = lo0;
      out[3 * blk + 1] = lo1;
      out[3 * blk + 2] = hi;
    }
  }
}


// Per-expert target precision of a requantization, passed by value
// (0 = the expert's slots are left as they are).
struct ExpertBits {
  uint8_t b[MOE_MAX_EXPERTS];
};

// Groups per wave of the requantization: their loads are all issued before
// the first group is reduced.
constexpr int kRqGroups = 4;

// One wave per (copy slot, kRqGroups groups).  Lane l holds group/64
// consecutive fp16 values of each group of the cached row; the range, scale,
// zero and codes follow the same
// binary64 quantizer as pack_kernel, so a row requantized at b bits carries
// exactly the codes moe_quant_pack gives for its binary16 values.  The b-bit
// codes are stored in the 8-bit copy format: each byte holds one code, bytes
// of a word in the 8-bit half-split order.
__global__ void __launch_bounds__(256)
requant_kernel(const uint16_t* __restrict__ cache, int64_t ld_cache, int K, int group,
               const int32_t* __restrict__ hdr, int n_slots, ExpertBits eb,
               uint32_t* __restrict__ codes, int64_t ld_codes, uint32_t* __restrict__ sz,
               int32_t* status) {
  const int G = K / group;
  const int GB = (G + kRqGroups - 1) / kRqGroups;
  const int wv = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t id = static_cast<int64_t>(blockIdx.x) * 4 + wv;
  if (id >= static_cast<int64_t>(n_slots) * GB) return;  // whole waves leave together
  const int s = static_cast<int>(id / GB);
  const int j0 = static_cast<int>(id % GB) * kRqGroups;
  const int bits = eb.b[hdr[2 * s]];
  if (bits == 0) return;
  const int per = group / 64;  // 1 or 2 values per lane
  const uint16_t* row = cache + static_cast<int64_t>(s) * ld_cache + lane * per;
  uint32_t raw[kRqGroups];
#pragma unroll
  for (int q = 0; q < kRqGroups; q++) {
    const uint16_t* src = row + static_cast<int64_t>(j0 + q) * group;
    raw[q] = j0 + q >= G ? 0u
                         : (per == 2 ? *reinterpret_cast<const uint32_t*>(src) : static_cast<uint32_t>(*src));
  }
#pragma unroll
  for (int q = 0; q < kRqGroups; q++) {
    const int j = j0 + q;
    if (j >= G) break;   // wave-uniform
    const double v0 = fp16_to_f64(raw[q] & 0xFFFFu);
    const double v1 = per == 2 ? fp16_to_f64(raw[q] >> 16) : v0;
    double mn = v0 < v1 ? v0 : v1;
    double mx = v0 > v1 ? v0 : v1;
    mn = mn < 0.0 ? mn : 0.0;
    mx = mx > 0.0 ? mx : 0.0;
    for (int m = 1; m < 64; m <<= 1) {
      const double a = __shfl_xor(mn, m);
      const double b = __shfl_xor(mx, m);
      mn = a < mn ? a : mn;
      mx = b > mx ? b : mx;
    }
    const int qmax = (1 << bits) - 1;
    const double sc = (mx - mn) / static_cast<double>(qmax);
    const uint32_t sb = (sc == 0.0) ? 0x3C00u : fp16_ceil_bits(sc);
    const double sf = fp16_to_f64(sb);
    int z = static_cast<int>(rint(-mn / sf));
    z = z < 0 ? 0 : z;
    auto code = [&](double v) -> uint32_t {
      double t = rint(v / sf) + static_cast<double>(z);
      t = t < 0.0 ? 0.0 : (t > static_cast<double>(qmax) ? static_cast<double>(qmax) : t);
      return static_cast<uint32_t>(t);
    };
    // word t holds codes 4t..4t+3 at bits 0, 16, 8, 24
    const uint32_t c0 = code(v0);
    uint32_t word;
    if (per == 2) {  // lane l holds codes 2l (bits 0) and 2l+1 (bits 16) of the group
      const uint32_t pair = c0 | (code(v1) << 16);
      const uint32_t a = static_cast<uint32_t>(__shfl(static_cast<int>(pair), (2 * lane) & 63));
      const uint32_t b = static_cast<uint32_t>(__shfl(static_cast<int>(pair), (2 * lane + 1) & 63));
      word = a | (b << 8);
    } else {  // lane l holds code l
      uint32_t c[4];
      for (int l = 0; l < 4; l++)
        c[l] = static_cast<uint32_t>(__shfl(static_cast<int>(c0), (4 * lane + l) & 63));
      word = c[0] | (c[1] << 16) | (c[2] << 8) | (c[3] << 24);
    }
    uint32_t* out = codes + static_cast<int64_t>(s) * ld_codes + static_cast<int64_t>(j) * (group / 4);
    if (lane < group / 4) out[lane] = word;
    if (lane == 0) {
      sz[static_cast<int64_t>(s) * G + j] = sb | (fp16_of_small_int(z) << 16);
      if (sb == 0x7C00u && status) *status = MOE_ERR_RANGE;
    }
  }
}

}  // namespace
}  // namespace moe

extern "C" int moe_quant_pack(const float* w, int64_t ld_w, int32_t R, int32_t K,
                              int32_t bits, int32_t group, const int32_t* rows, int32_t n,
                              uint32_t* codes, int64_t ld_codes, uint32_t* sz,
                              int64_t sz_row_stride, int64_t sz_group_stride,
                              int32_t* status, void* stream) {
  using namespace moe;
  if (!valid_expert_bits(bits)) return MOE_ERR_BITS;
  if (!w || !codes || !sz || R <= 0 || K <= 0 || n < 0) return MOE_ERR_ARG;
  if (!(group == 64 || group == 128) || K % group || K % 32) return MOE_ERR_ARG;
  if ((bits == 3 || bits == 6) && group != 128) return MOE_ERR_ARG;
  if (ld_w < K || ld_codes < static_cast<int64_t>(K) * bits / 32) return MOE_ERR_ARG;
  if (!rows && n > R) return MOE_ERR_ARG;
  if (!aligned16(codes) || (ld_codes * 4) % 16) return MOE_ERR_ALIGN;
  if (n == 0) return MOE_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t total = static_cast<int64_t>(n) * (K / group);
  const int threads = 256;
  hipLaunchKernelGGL(pack_kernel, dim3(static_cast<unsigned>(cdiv(total, threads))),
                     dim3(threads), 0, s, w, ld_w, K, bits, group, rows, n, codes, ld_codes,
                     sz, sz_row_stride, sz_group_stride, status);
  return launch_status(s);
}

extern "C" int moe_requant_channels(moe_layer_t* L, int32_t kind, const uint16_t* cache,
                                    int64_t ld_cache, const int32_t* expert_bits,
                                    int32_t* status, void* stream) {
  using namespace moe;
  if (!L || kind < 0 || kind > 2 || !expert_bits) return MOE_ERR_ARG;
  const int E = L->n_experts;
  if (E <= 0 || E + L->n_shared > MOE_MAX_EXPERTS) return MOE_ERR_ARG;
  if (!(L->group == 64 || L->group == 128)) return MOE_ERR_ARG;
  const int K = kind == MOE_KIND_DOWN ? L->d_ff : L->d_model;
  if (K <= 0 || K % L->group || K % 128) return MOE_ERR_ARG;
  ExpertBits eb{};
  for (int e = 0; e < E; e++) {
    const int b = expert_bits[e];
    if (b != 0 && !valid_bits(b)) return MOE_ERR_BITS;
    eb.b[e] = static_cast<uint8_t>(b);
  }
  const moe_kind_desc_t& D = L->kind[kind];
  if (D.n_slots < 0) return MOE_ERR_ARG;
  if (D.n_slots == 0) return MOE_OK;
  if (!cache || ld_cache < K || (ld_cache % 2) || (reinterpret_cast<uintptr_t>(cache) & 3u))
    return MOE_ERR_ARG;
  if (!D.copy_codes || !D.copy_sz || !D.copy_hdr || !D.copy_hdr_host) return MOE_ERR_ARG;
  for (int sl = 0; sl < D.n_slots; sl++) {
    const int e = D.copy_hdr_host[2 * sl];
    if (e < 0 || e >= E) return MOE_ERR_SLOT;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t waves = static_cast<int64_t>(D.n_slots) * cdiv(K / L->group, kRqGroups);
  hipLaunchKernelGGL(requant_kernel, dim3(static_cast<unsigned>(cdiv(waves, 4))), dim3(256), 0, s,
                     cache, ld_cache, K, L->group, D.copy_hdr, D.n_slots, eb,
                     const_cast<uint32_t*>(D.copy_codes), code_row_words(K, 8),
                     const_cast<uint32_t*>(D.copy_sz), status);
  return launch_status(s);
}

extern "C" const char* moe_status_str(int status) {
  switch (status) {
    case MOE_OK: return "ok";
    case MOE_ERR_ARG: return "invalid argument";
    case MOE_ERR_BITS: return "bit-width not in {2,3,4,6,8} (or 16 where allowed)";
    case MOE_ERR_ALIGN: return "pointer or stride not 16-byte aligned";
    case MOE_ERR_WORKSPACE: return "workspace missing or too small";
    case MOE_ERR_SLOT: return "bad switch slot list";
    case MOE_ERR_RANGE: return "fp16 scale overflow";
    case MOE_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

extern "C" int64_t moe_code_row_words(int32_t K, int32_t bits) {
  if (!moe::valid_expert_bits(bits) || K <= 0 || K % 128) return 0;
  return moe::code_row_words(K, bits);
}
