// switch.hip -- moe_set_channel_switch: install a set of cached 8-bit copies.
//
// Sec. IV-B "Channel Weights Replacement based on Caching": a cached channel
// replaces the quantized channel whose (expert, channel) index it carries.
// Sec. V-A "Data Format in the Channel Cache": the expert and channel indexes
// are stored as headers of the cache entries so the target is found directly.
// Here the headers are scattered into a per-(expert, row) table (row_slot), so
// the FFN finds a row's source with one load; no weights move and nothing is
// requantized.  The visiting order of rows (order_gu / order_dn) is rebuilt
// as a stable partition by precision source, which keeps most 16-row tiles of
// the FFN uniform in bit-width.
#include <vector>

#include "common.hpp"

namespace moe {
namespace {

__global__ void __launch_bounds__(256) fill_kernel(int32_t* p, int64_t n, int32_t v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void __launch_bounds__(256)
scatter_slots_kernel(const int32_t* __restrict__ list, int n, const int32_t* __restrict__ hdr,
                     int R, int32_t* __restrict__ row_slot) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int s = list[i];
  const int e = hdr[2 * s];
  const int r = hdr[2 * s + 1];
  row_slot[static_cast<int64_t>(e) * R + r] = s;
}

// One workgroup (4 waves) per routed expert.  Class of row i:
// bit 0 = row_slot_a[i] >= 0, bit 1 = row_slot_b[i] >= 0 (b may be NULL).
// order lists class 0 rows ascending, then class 1, 2, 3; class_cnt[4e + c]
// receives the size of class c.
__global__ void __launch_bounds__(256)
order_kernel(const int32_t* __restrict__ rs_a, const int32_t* __restrict__ rs_b, int R,
             int32_t* __restrict__ order, int32_t* __restrict__ class_cnt) {
  __shared__ int cnt[4];
  __shared__ int wave_cnt[4][4];
  __shared__ int start[4];
  const int e = blockIdx.x;
  const int tid = threadIdx.x;
  const int wv = tid >> 6;
  const int lane = tid & 63;
  rs_a += static_cast<int64_t>(e) * R;
  if (rs_b) rs_b += static_cast<int64_t>(e) * R;
  order += static_cast<int64_t>(e) * R;
  if (tid < 4) cnt[tid] = 0;
  __syncthreads();
  int local[4] = {0, 0, 0, 0};
  for (int i = tid; i < R; i += blockDim.x) {
    const int c = (rs_a[i] >= 0 ? 1 : 0) | ((rs_b && rs_b[i] >= 0) ? 2 : 0);
    local[c]++;
  }
  for (int c = 0; c < 4; c++) atomicAdd(&cnt[c], local[c]);
  __syncthreads();
  if (tid < 4) class_cnt[4 * e + tid] = cnt[tid];
  if (tid == 0) {
    start[0] = 0;
    for (int c = 1; c < 4; c++) start[c] = start[c - 1] + cnt[c - 1];
  }
  __syncthreads();
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  for (int base = 0; base < R; base += blockDim.x) {
    const int i = base + tid;
    const bool live = i < R;
    const int c = live ? ((rs_a[i] >= 0 ? 1 : 0) | ((rs_b && rs_b[i] >= 0) ? 2 : 0)) : -1;
    int rank = 0;
    for (int cc = 0; cc < 4; cc++) {
      const uint64_t m = __ballot(c == cc);
      if (lane == 0) wave_cnt[wv][cc] = __popcll(m);
      if (c == cc) rank = __popcll(m & below);
    }
    __syncthreads();
    if (live) {
      int pos = start[c] + rank;
      for (int w2 = 0; w2 < wv; w2++) pos += wave_cnt[w2][c];
      order[pos] = i;
    }
    __syncthreads();
    if (tid < 4) {
      int add = 0;
      for (int w2 = 0; w2 < 4; w2++) add += wave_cnt[w2][tid];
      start[tid] += add;
    }
    __syncthreads();
  }
}

int rows_of_kind(const moe_layer_t* L, int kind) {
  return kind == MOE_KIND_DOWN ? L->d_model : L->d_ff;
}

}  // namespace
}  // namespace moe

extern "C" int moe_set_channel_switch(moe_layer_t* L, int32_t kind, const int32_t* slots_on,
                                      int32_t n_on, void* stream) {
  using namespace moe;
  if (!L || L->n_experts <= 0 || L->d_model <= 0 || L->d_ff <= 0) return MOE_ERR_ARG;
  if (!L->order_gu || !L->order_dn || !L->class_cnt) return MOE_ERR_ARG;
  for (int kd = 0; kd < 3; kd++)
    if (!L->kind[kd].row_slot) return MOE_ERR_ARG;
  if (kind < -1 || kind > 2) return MOE_ERR_ARG;
  if (kind == -1 && n_on != 0) return MOE_ERR_ARG;
  const int E = L->n_experts;
  hipStream_t s = static_cast<hipStream_t>(stream);

  if (kind >= 0) {
    const moe_kind_desc_t& K = L->kind[kind];
    const int R = rows_of_kind(L, kind);
    if (n_on < 0 || n_on > K.n_slots) return MOE_ERR_SLOT;
    if (n_on > 0 && (!slots_on || !K.copy_hdr || !K.copy_hdr_host || !L->staging))
      return MOE_ERR_ARG;
    // duplicate slots and two slots on one (expert, row): one flag per slot
    // and one per row of the kind (E*R bytes, reused across calls)
    static thread_local std::vector<uint8_t> seen, rows;
    seen.assign(static_cast<size_t>(K.n_slots), 0);
    rows.assign(static_cast<size_t>(E) * R, 0);
    for (int i = 0; i < n_on; i++) {
      const int sl = slots_on[i];
      if (sl < 0 || sl >= K.n_slots || seen[sl]) return MOE_ERR_SLOT;
      seen[sl] = 1;
      const int e = K.copy_hdr_host[2 * sl];
      const int r = K.copy_hdr_host[2 * sl + 1];
      if (e < 0 || e >= E || r < 0 || r >= R) return MOE_ERR_SLOT;
      uint8_t& f = rows[static_cast<size_t>(e) * R + r];
      if (f) return MOE_ERR_SLOT;
      f = 1;
    }
    if (n_on > 0 &&
        hipMemcpyAsync(L->staging, slots_on, sizeof(int32_t) * n_on, hipMemcpyHostToDevice, s) !=
            hipSuccess)
      return MOE_ERR_HIP;
    const int64_t n = static_cast<int64_t>(E) * R;
    hipLaunchKernelGGL(fill_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0, s,
                       K.row_slot, n, -1);
    if (n_on > 0)
      hipLaunchKernelGGL(scatter_slots_kernel, dim3(static_cast<unsigned>(cdiv(n_on, 256))),
                         dim3(256), 0, s, L->staging, n_on, K.copy_hdr, R, K.row_slot);
  } else {
    for (int kd = 0; kd < 3; kd++) {
      const int64_t n = static_cast<int64_t>(E) * rows_of_kind(L, kd);
      hipLaunchKernelGGL(fill_kernel, dim3(static_cast<unsigned>(cdiv(n, 256))), dim3(256), 0, s,
                         L->kind[kd].row_slot, n, -1);
    }
  }
  if (kind != MOE_KIND_DOWN)
    hipLaunchKernelGGL(order_kernel, dim3(E), dim3(256), 0, s, L->kind[0].row_slot,
                       static_cast<const int32_t*>(L->kind[1].row_slot), L->d_ff, L->order_gu,
                       L->class_cnt);
  if (kind == MOE_KIND_DOWN || kind == -1)
    hipLaunchKernelGGL(order_kernel, dim3(E), dim3(256), 0, s, L->kind[2].row_slot,
                       static_cast<const int32_t*>(nullptr), L->d_model, L->order_dn,
                       L->class_cnt + 4 * E);
  return launch_status(s);
}
