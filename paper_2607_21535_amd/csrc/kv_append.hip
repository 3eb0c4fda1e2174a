// Draft KV append (dense cache or compact ring) and the selection export.
//
// The draft forward of each draft token writes that token's K/V row before
// the token attends (Windowed-MTP Section 3, per-step latency model).  For the
// compact ring (Section 4 and Section 6 "Memory"; the ring comment of the
// Appendix A pseudocode) logical position p goes to slot p below the sink and
// to sink + (p - sink) mod R_w above it.  Lengths stay on the device: each
// workgroup owns one sequence, reads lens[b], copies its rows with 16-byte
// accesses and, after a barrier, advances lens[b] -- so a captured graph can
// replay append + attention steps without host involvement.

#include "../../include/wmtp.h"
#include "common.h"
#include "index_map.h"
#include "launch.h"

#include <climits>

namespace wmtp {
namespace {

struct AppendArgs {
  uint16_t* k;
  uint16_t* v;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const int32_t* n_new;
  int32_t* lens;
  int32_t* err;
  int B, Hkv, d;
  int64_t rows;
  int sink, R_w, n_max;
};

template <bool RING>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
  const int b = blockIdx.x;
  const int64_t cap = RING ? static_cast<int64_t>(INT_MAX) : a.rows;
  const bool report = threadIdx.x == 0;

  int L0 = a.lens[b];
  if (L0 < 0 || L0 > cap) {
    if (report) raise_error(a.err, WMTP_DERR_LEN_RANGE);
    L0 = L0 < 0 ? 0 : static_cast<int>(cap);
  }
  int n = a.n_new[b];
  if (n < 0 || n > a.n_max) {
    if (report) raise_error(a.err, WMTP_DERR_NNEW_RANGE);
    n = n < 0 ? 0 : a.n_max;
  }
  int n_take = n;  // rows that get a position
  if (static_cast<int64_t>(L0) + n > cap) {
    if (report) raise_error(a.err, RING ? WMTP_DERR_LEN_RANGE : WMTP_DERR_CAPACITY);
    n_take = static_cast<int>(cap - L0);
  }
  const int S_new = L0 + n_take;

  // Rows i (position L0 + i) to write.  Ring: the sink positions, and the
  // positions that are still resident after the append (the last R_w); the
  // two ranges hit distinct slots, so no two threads write one slot.
  int a_end = n_take, b_begin = n_take;
  if (RING) {
    a_end = min(max(a.sink - L0, 0), n_take);
    b_begin = max(a_end, S_new - a.R_w - L0);
  }
  const int n_a = a_end;
  const int n_rows = n_a + (n_take - b_begin);

  const int units = a.Hkv * a.d / 8;  // 16-byte units per row
  const int64_t row_elems = static_cast<int64_t>(a.Hkv) * a.d;
  const int64_t dst_seq = static_cast<int64_t>(b) * a.rows * row_elems;
  const int64_t src_seq = static_cast<int64_t>(b) * a.n_max * row_elems;
  const int64_t total = static_cast<int64_t>(n_rows) * units;
  for (int64_t u = threadIdx.x; u < total; u += blockDim.x) {
    const int r = static_cast<int>(u / units);
    const int off = static_cast<int>(u % units) * 8;
    const int i = r < n_a ? r : b_begin + (r - n_a);
    const int p = L0 + i;
    const int slot = RING ? (p < a.sink ? p : a.sink + (p - a.sink) % a.R_w) : p;
    const int64_t src = src_seq + static_cast<int64_t>(i) * row_elems + off;
    const int64_t dst = dst_seq + static_cast<int64_t>(slot) * row_elems + off;
    *reinterpret_cast<u32x4*>(a.k + dst) = *reinterpret_cast<const u32x4*>(a.k_new + src);
    *reinterpret_cast<u32x4*>(a.v + dst) = *reinterpret_cast<const u32x4*>(a.v_new + src);
  }
  __syncthreads();  // every thread has read lens[b] before it changes
  if (threadIdx.x == 0) a.lens[b] = S_new;
}

// The export runs the attention kernels' own row maps: RowMap<Window> on a
// dense cache gives the logical position, RowMap<Ring> the ring slot.
__global__ __launch_bounds__(256) void select_kernel(const int32_t* lens, int W, int sink, int R_w,
                                                     int32_t* pos_out, int32_t* slot_out,
                                                     int32_t* n_sel_out, int32_t* err) {
  const int b = blockIdx.x;
  int S = lens[b];
  if (S < 0) {
    if (threadIdx.x == 0) raise_error(err, WMTP_DERR_LEN_RANGE);
    S = 0;
  }
  const int n = selected_count<KeyMap::Window>(S, W, sink);
  const RowMap<KeyMap::Window> wmap(S, W, sink, R_w);
  const int width = sink + W;
  const int64_t base = static_cast<int64_t>(b) * width;
  for (int j = threadIdx.x; j < width; j += blockDim.x) {
    pos_out[base + j] = j < n ? wmap.row(j) : -1;
  }
  if (slot_out != nullptr) {
    const RowMap<KeyMap::Ring> rmap(S, W, sink, R_w);
    for (int j = threadIdx.x; j < width; j += blockDim.x) slot_out[base + j] = j < n ? rmap.row(j) : -1;
  }
  if (threadIdx.x == 0) n_sel_out[b] = n;
}

}  // namespace

hipError_t launch_append(const AppendLaunch& L, hipStream_t st) {
  AppendArgs a;
  a.k = L.k; a.v = L.v; a.k_new = L.k_new; a.v_new = L.v_new;
  a.n_new = L.n_new; a.lens = L.lens; a.err = L.err;
  a.B = L.B; a.Hkv = L.Hkv; a.d = L.d; a.rows = L.rows;
  a.sink = L.sink; a.R_w = L.R_w; a.n_max = L.n_max;
  if (L.ring)
    hipLaunchKernelGGL(append_kernel<true>, dim3(L.B), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(append_kernel<false>, dim3(L.B), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_select(const int32_t* lens, int B, int W, int sink, int R_w, int32_t* pos_out,
                         int32_t* slot_out, int32_t* n_sel_out, int32_t* err, hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(256), 0, st, lens, W, sink, R_w, pos_out,
                     slot_out, n_sel_out, err);
  return hipGetLastError();
}

}  // namespace wmtp
