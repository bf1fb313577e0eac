// ffn.hip -- host side of moe_expert_ffn_mixed: argument validation, the
// launch plan (which kernel serves which experts, workspace layout, split
// of the down projection) and the launches.  The kernels live in
// ffn_stream.hip and ffn_tile.hip.
#include <algorithm>
#include <functional>
#include <mutex>
#include <type_traits>
#include <vector>

#include <hip/hip_ext.h>

#include "ffn_common.hpp"

namespace moe {
namespace ffn {
namespace {

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
// workgroup sets taking every n_tt-th 32-token tile of the expert -- where the
// experts are narrow (d_ff below kTileWideFf; DeepSeek-shaped layer, d_ff
// 1408: the tile kernel is 13 % slower at 36 tokens per expert, even at 48,
// 10-25 % faster from 56).  Wide experts give the tile kernel enough row
// blocks to fill its grid at any token count, and there it is faster from 29
// tokens per expert (Mixtral-shaped layer, 32 to 96 tokens per expert: FFN
// 13-32 % faster).
constexpr int kRoutedSplitMax = 48;
constexpr int kTileWideFf = 4096;

// Persistent tile grid: kTileWgPerCu workgroups per compute unit (two waves
// per SIMD in all), a multiple of the XCD count.
int tile_grid() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] == 0) {
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu <= 0) cu = 256;
    cached[dev] = kTileWgPerCu * std::max(kXcds, cu / kXcds * kXcds);
  }
  return cached[dev];
}

// Split-K of the tile kernel's down projection: slices (at most
// kTileSplitMax, each at least kTileSplitMinGroups groups of K) until the
// estimated items reach kTileItemsPerWg per workgroup of the grid.
constexpr int kTileSplitMax = 8;
constexpr int kTileItemsPerWg = 4;
constexpr int kTileSplitMinGroups = 8;

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
  if (p.nt_routed == 0 && Tk <= static_cast<int64_t>(kRoutedSplitMax) * E && L->d_ff < kTileWideFf) {
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
  // split-K slices of the down projection: where the routed experts stream
  // (few tokens, too few output rows to fill the machine), and where the
  // tile kernel's down items (token tiles x row blocks) are too few for its
  // persistent grid: with a few long items per workgroup, the last round
  // of items leaves most workgroups idle
  p.n_split = std::max(ns, 1);
  if (p.nt_routed == 0) {
    const int64_t rb = cdiv(L->d_model, kTileWaves * kTileWaveRows<1>);
    int64_t items = (cdiv(Tk, kTileTok) + E / 2) * rb;   // Zipf-skewed segments: about E/2 extra partial tiles
    if (S > 0 && p.nt_shared == 0) items += S * cdiv(T, kTileTok) * rb;
    const int gdown = fmin / g;
    int nsd = 1;
    while (nsd < kTileSplitMax && items * nsd < static_cast<int64_t>(kTileItemsPerWg) * tile_grid() &&
           gdown / (nsd + 1) >= kTileSplitMinGroups)
      nsd++;
    p.n_split = nsd;
  }
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
    if (!valid_expert_bits(L->bits_host[e])) return MOE_ERR_BITS;
    if (L->bits_host[e] == 16 && L->group != 64) return MOE_ERR_ARG;   // unquantized experts: group 64
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

// Work map of the streaming launch of one stage, over the routed experts
// (routed) and/or the shared experts (shared).  The switched-class
// workgroups per routed expert bound what its copies can need: classes 1..3
// of gate/up hold at most n_gate + n_up rows in three classes, class 1 of
// down at most n_down rows.  Class-0 entries: shared experts first, then
// the routed experts widest first.
WgMap stream_map(const moe_layer_t* L, const Plan& p, bool routed, bool shared, bool down, int n_split) {
  WgMap m{};
  const int rows1 = (down ? kWavesOf<1> : kWavesOf<2>) * 16;
  const int E = L->n_experts, S = L->n_shared;
  m.n_split = n_split;
  m.tt_r = std::max(p.tt_routed, 1);
  m.tt_s = std::max(p.tt_shared, 1);
  m.m_r = m.tt_r * n_split;
  m.m_s = m.tt_s * n_split;
  for (int e = 0; e < E + S; e++) m.bits[e] = static_cast<int8_t>(L->bits_host[e]);
  if (routed) {
    const int R = down ? L->d_model : L->d_ff;
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
      const int64_t need = down ? cdiv(nc[0][e], rows1)
                                : (nc[0][e] + nc[1][e] > 0 ? cdiv(nc[0][e] + nc[1][e], rows1) + 2 : 0);
      n_sw = std::max<int>(n_sw, static_cast<int>(std::min<int64_t>(need, cdiv(R, rows1) + 3)));
    }
    m.n_r = n_sw > 0 ? E : 0;
    m.n_sw = n_sw;
  }
  int n = 0;
  int32_t start = 0;
  auto entry = [&](int e) {
    const int R = down ? L->d_model : (e < E ? L->d_ff : L->d_ff_shared);
    const int64_t nblk = cdiv(R, rows1 * stream_rt(L->bits_host[e]));
    m.ent_e[n] = static_cast<int16_t>(e);
    m.ent_start[n] = start;
    start += static_cast<int32_t>(nblk * (e < E ? m.m_r : m.m_s));
    n++;
  };
  if (shared)
    for (int s = 0; s < S; s++) entry(E + s);
  if (routed)
    for (int b : {16, 8, 6, 4, 3, 2})
      for (int e = 0; e < E; e++)
        if (L->bits_host[e] == b) entry(e);
  m.ent_start[n] = start;
  m.n_ent = n;
  return m;
}

int64_t stream_grid(const WgMap& m) {
  return static_cast<int64_t>(m.n_r) * m.n_sw * m.m_r + (m.n_ent > 0 ? m.ent_start[m.n_ent] : 0);
}

TileMap tile_map(const moe_layer_t* L, int e0, int n_e, int n_split) {
  TileMap m{};
  m.e0 = e0;
  m.n_e = n_e;
  m.n_split = n_split;
  for (int i = 0; i < m.n_e; i++) m.bits[i] = static_cast<int8_t>(L->bits_host[m.e0 + i]);
  return m;
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
  // tile path: plan kernel, then the persistent tile kernel, over the experts
  // that take it -- routed, shared, or both in one launch (routed first), so
  // that one persistent grid balances all of their items
  const bool tile_r = p.nt_routed == 0, tile_s = S > 0 && p.nt_shared == 0;
  auto add_tile = [&](std::vector<Launch>& v, auto nk) {
    constexpr int NK = decltype(nk)::value;
    if (!tile_r && !tile_s) return;
    const int e0 = tile_r ? 0 : a.E, n_e = (tile_r ? a.E : 0) + (tile_s ? S : 0);
    const TileMap m = tile_map(L, e0, n_e, NK == 1 ? p.n_split : 1);
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
  };
  // streaming path: one launch for every expert set that streams
  auto add_stream = [&](std::vector<Launch>& v, auto nk, int nsplit) {
    constexpr int NK = decltype(nk)::value;
    const bool r = p.nt_routed != 0, sh = S > 0 && p.nt_shared != 0;
    if (!r && !sh) return;
    const WgMap m = stream_map(L, p, r, sh, NK == 1, nsplit);
    const int64_t n_wg = stream_grid(m);
    if (n_wg == 0) return;
    const int nt = std::max(r ? p.nt_routed : 0, sh ? p.nt_shared : 0);
    const dim3 grid(static_cast<unsigned>(n_wg));
    v.push_back([=, &a](hipEvent_t e0, hipEvent_t e1) {
      const dim3 block(64 * kWavesOf<NK>);
      if (nt == 1) klaunch(ffn_stream_kernel<NM, 1, NK>, grid, block, s, e0, e1, a, m);
      else klaunch(ffn_stream_kernel<NM, 2, NK>, grid, block, s, e0, e1, a, m);
    });
  };
  using two = std::integral_constant<int, 2>;
  using one = std::integral_constant<int, 1>;
  add_tile(gate_up, two{});
  add_stream(gate_up, two{}, 1);
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
  add_tile(down, one{});
  add_stream(down, one{}, p.n_split);
  issue(xsum, event(0), nullptr, s);
  issue(gate_up, event(1), event(2), s);
  issue(hsum, nullptr, nullptr, s);
  issue(down, event(3), event(4), s);
}

}  // namespace
}  // namespace ffn
}  // namespace moe

extern "C" int moe_ffn_plan(const moe_layer_t* L, int32_t T, int32_t k, int32_t* n_split,
                            size_t* ws_bytes) {
  using namespace moe::ffn;
  const int st = validate_layer(L);
  if (st != MOE_OK) return st;
  if (T < 0 || k < 1 || k > L->n_experts) return MOE_ERR_ARG;
  const Plan p = make_plan(L, T, k);
  if (n_split) *n_split = p.n_split;
  if (ws_bytes) *ws_bytes = p.total;
  return MOE_OK;
}

namespace moe {
namespace ffn {
namespace {
int ffn_entry(const moe_layer_t* L, const uint16_t* x, int32_t T, int32_t k,
              const int32_t* offsets, const int32_t* perm_token, float* o, void* ws,
              size_t ws_bytes, int32_t* status, void* stream, void* const* events,
              int32_t n_events) {
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
  a.status = status;
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
}  // namespace ffn
}  // namespace moe

extern "C" int moe_expert_ffn_mixed(const moe_layer_t* L, const uint16_t* x, int32_t T, int32_t k,
                                    const int32_t* offsets, const int32_t* perm_token, float* o,
                                    void* ws, size_t ws_bytes, int32_t* status, void* stream) {
  return moe::ffn::ffn_entry(L, x, T, k, offsets, perm_token, o, ws, ws_bytes, status, stream, nullptr, 0);
}

extern "C" int moe_expert_ffn_mixed_ev(const moe_layer_t* L, const uint16_t* x, int32_t T,
                                       int32_t k, const int32_t* offsets,
                                       const int32_t* perm_token, float* o, void* ws,
                                       size_t ws_bytes, int32_t* status, void* stream,
                                       void* const* events, int32_t n_events) {
  if (n_events < 0 || (n_events > 0 && !events)) return MOE_ERR_ARG;
  return moe::ffn::ffn_entry(L, x, T, k, offsets, perm_token, o, ws, ws_bytes, status, stream, events,
                        n_events);
}

// ------------------------------------------------------------------ no-allocation variant
// The workspace of moe_expert_ffn_mixed_noalloc: one fixed array per GPU,
// loaded with the library's code object, so the call needs no allocation.
// Host code never uses the array's name as an address (on the host it is a
// stand-in, not the device address): the device address comes from
// hipGetSymbolAddress, taken once per device with that device current.
static __device__ __align__(256) unsigned char scratch[MOE_NOALLOC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[64] = {nullptr};

// Device address of this device's scratch array, or null on failure.
void* scratch_address() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

extern "C" int moe_expert_ffn_mixed_noalloc(const moe_layer_t* L, const uint16_t* x, int32_t T,
                                            int32_t k, const int32_t* offsets,
                                            const int32_t* perm_token, float* o, int32_t* status,
                                            void* stream) {
  using namespace moe::ffn;
  int st = validate_layer(L);
  if (st != MOE_OK) return st;
  if (T < 0 || k < 1 || k > L->n_experts || k > MOE_MAX_TOPK) return MOE_ERR_ARG;
  if (T == 0) return MOE_OK;
  const Plan p = make_plan(L, T, k);
  // the plan's workspace (already including its 256 bytes of alignment slack)
  // must fit the fixed array
  if (p.total > static_cast<size_t>(MOE_NOALLOC_SCRATCH_BYTES)) return MOE_ERR_WORKSPACE;
  void* ws = scratch_address();
  if (!ws) return MOE_ERR_HIP;
  return moe::ffn::ffn_entry(L, x, T, k, offsets, perm_token, o, ws, MOE_NOALLOC_SCRATCH_BYTES, status,
                             stream, nullptr, 0);
}
