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
#include "fp8.h"
#include "index_map.h"
#include "launch.h"

#include <algorithm>
#include <climits>

namespace wmtp {
namespace {

struct AppendArgs {
  void* k;  // bf16 or E4M3 elements
  void* v;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const int32_t* n_new;
  int32_t* lens;
  int32_t* err;
  int B, Hkv, d;
  int64_t rows;
  int sink, R_w, n_max;
  float k_scale, v_scale;  // fp8: per-tensor scales the rows are divided by
  int32_t* lens_out;       // NULL: advance lens in place
};

template <bool RING, bool F8>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
  const int b = blockIdx.x;
  const int64_t cap = RING ? static_cast<int64_t>(INT_MAX) : a.rows;
  const bool report = threadIdx.x == 0;

  // Both counts are read before either is checked: a read placed after an
  // error report would wait for the first one.
  int L0 = a.lens[b];
  int n = a.n_new[b];
  if (L0 < 0 || L0 > cap) {
    if (report) raise_error(a.err, WMTP_DERR_LEN_RANGE);
    L0 = L0 < 0 ? 0 : static_cast<int>(cap);
  }
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
    const u32x4 kx = *reinterpret_cast<const u32x4*>(a.k_new + src);
    const u32x4 vx = *reinterpret_cast<const u32x4*>(a.v_new + src);
    if constexpr (F8) {
      *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(a.k) + dst) = bf16x8_to_fp8x8(kx, a.k_scale);
      *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(a.v) + dst) = bf16x8_to_fp8x8(vx, a.v_scale);
    } else {
      *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.k) + dst) = kx;
      *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.v) + dst) = vx;
    }
  }
  if (a.lens_out != nullptr) {
    if (threadIdx.x == 0) a.lens_out[b] = S_new;
    return;
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

// Speculation candidates (Windowed-MTP Section 7, tree speculation): one
// workgroup per request writes each candidate's draft row for position
// lens[b] + depth[b] -- candidate 0 at that position's ring slot (in place,
// as a chain writes), candidate c >= 1 at slot depth[b] of its private run
// -- then advances depth[b].  A request already at the largest depth is
// flagged and left unchanged.
__global__ __launch_bounds__(256) void tree_append_kernel(TreeAppendLaunch a) {
  const int b = blockIdx.x;
  const bool report = threadIdx.x == 0;
  int S = a.lens[b];
  if (S < 0 || S > INT_MAX - a.dd) {
    if (report) raise_error(a.err, WMTP_DERR_LEN_RANGE);
    S = S < 0 ? 0 : INT_MAX - a.dd;
  }
  const int i = a.depth[b];
  if (i < 0 || i >= a.dd) {  // uniform over the workgroup
    if (report) raise_error(a.err, WMTP_DERR_DEPTH);
    return;
  }
  const int p = S + i;
  const int ring_slot = p < a.sink ? p : a.sink + (p - a.sink) % a.R_w;
  const int units = a.Hkv * a.d / 8;  // 16-byte units per row
  const int64_t row_elems = static_cast<int64_t>(a.Hkv) * a.d;
  const int64_t ring_rows = static_cast<int64_t>(a.sink) + a.R_w;
  const int64_t run_rows = static_cast<int64_t>(a.width - 1) * a.dd;
  for (int u = threadIdx.x; u < a.width * units; u += blockDim.x) {
    const int c = u / units;
    const int off = (u % units) * 8;
    const int64_t src = (static_cast<int64_t>(b) * a.width + c) * row_elems + off;
    const u32x4 kx = *reinterpret_cast<const u32x4*>(a.k_new + src);
    const u32x4 vx = *reinterpret_cast<const u32x4*>(a.v_new + src);
    if (c == 0) {
      const int64_t dst = (static_cast<int64_t>(b) * ring_rows + ring_slot) * row_elems + off;
      *reinterpret_cast<u32x4*>(a.k + dst) = kx;
      *reinterpret_cast<u32x4*>(a.v + dst) = vx;
    } else {
      const int64_t dst = (static_cast<int64_t>(b) * run_rows + static_cast<int64_t>(c - 1) * a.dd + i) * row_elems + off;
      *reinterpret_cast<u32x4*>(a.k2 + dst) = kx;
      *reinterpret_cast<u32x4*>(a.v2 + dst) = vx;
    }
  }
  __syncthreads();  // every thread has read depth[b] before it changes
  if (threadIdx.x == 0) a.depth[b] = i + 1;
}

// counts[b] -= n_drop[b], or counts[b] = 0 without n_drop.
__global__ __launch_bounds__(256) void rollback_kernel(int32_t* counts, const int32_t* n_drop, int B,
                                                      int32_t* err) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  if (n_drop == nullptr) {
    counts[b] = 0;
    return;
  }
  const int c = counts[b];
  const int n = n_drop[b];
  if (n < 0 || c < 0 || n > c) {
    raise_error(err, WMTP_DERR_NNEW_RANGE);
    counts[b] = c < 0 ? 0 : (n < 0 ? c : 0);
    return;
  }
  counts[b] = c - n;
}

// The conversion exports run the appends' quantiser and the attention's
// widening on flat arrays, 8 elements per thread and step.
__global__ __launch_bounds__(256) void fp8_quantize_kernel(const uint16_t* x, int64_t units, float scale,
                                                          uint8_t* codes) {
  for (int64_t u = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; u < units;
       u += static_cast<int64_t>(gridDim.x) * blockDim.x)
    *reinterpret_cast<u32x2*>(codes + u * 8) =
        bf16x8_to_fp8x8(*reinterpret_cast<const u32x4*>(x + u * 8), scale);
}

__global__ __launch_bounds__(256) void fp8_dequantize_kernel(const uint8_t* codes, int64_t units,
                                                            uint16_t* out) {
  for (int64_t u = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; u < units;
       u += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const u32x2 c = *reinterpret_cast<const u32x2*>(codes + u * 8);
    *reinterpret_cast<u32x4*>(out + u * 8) = fp8x8_to_bf16x8(c[0], c[1]);
  }
}

}  // namespace

hipError_t launch_append(const AppendLaunch& L, hipStream_t st) {
  AppendArgs a;
  a.k = L.k; a.v = L.v; a.k_new = L.k_new; a.v_new = L.v_new;
  a.n_new = L.n_new; a.lens = L.lens; a.err = L.err;
  a.B = L.B; a.Hkv = L.Hkv; a.d = L.d; a.rows = L.rows;
  a.sink = L.sink; a.R_w = L.R_w; a.n_max = L.n_max;
  a.k_scale = L.k_scale; a.v_scale = L.v_scale;
  a.lens_out = L.lens_out;
  const dim3 grid(L.B), block(256);
  if (L.ring) {
    if (L.fp8)
      hipLaunchKernelGGL((append_kernel<true, true>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((append_kernel<true, false>), grid, block, 0, st, a);
  } else {
    if (L.fp8)
      hipLaunchKernelGGL((append_kernel<false, true>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((append_kernel<false, false>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_tree_append(const TreeAppendLaunch& L, hipStream_t st) {
  hipLaunchKernelGGL(tree_append_kernel, dim3(L.B), dim3(256), 0, st, L);
  return hipGetLastError();
}

hipError_t launch_rollback(int32_t* counts, const int32_t* n_drop, int B, int32_t* err, hipStream_t st) {
  hipLaunchKernelGGL(rollback_kernel, dim3((B + 255) / 256), dim3(256), 0, st, counts, n_drop, B, err);
  return hipGetLastError();
}

hipError_t launch_fp8_quantize(const uint16_t* x, int64_t n, float scale, uint8_t* codes,
                               hipStream_t st) {
  const int64_t units = n / 8;
  if (units == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((units + 255) / 256, 65536));
  hipLaunchKernelGGL(fp8_quantize_kernel, dim3(blocks), dim3(256), 0, st, x, units, scale, codes);
  return hipGetLastError();
}

hipError_t launch_fp8_dequantize(const uint8_t* codes, int64_t n, uint16_t* out, hipStream_t st) {
  const int64_t units = n / 8;
  if (units == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((units + 255) / 256, 65536));
  hipLaunchKernelGGL(fp8_dequantize_kernel, dim3(blocks), dim3(256), 0, st, codes, units, out);
  return hipGetLastError();
}

hipError_t launch_select(const int32_t* lens, int B, int W, int sink, int R_w, int32_t* pos_out,
                         int32_t* slot_out, int32_t* n_sel_out, int32_t* err, hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(256), 0, st, lens, W, sink, R_w, pos_out,
                     slot_out, n_sel_out, err);
  return hipGetLastError();
}

}  // namespace wmtp
