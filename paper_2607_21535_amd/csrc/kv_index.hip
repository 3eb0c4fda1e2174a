// The draft's KV-index builder over a paged token pool (page size 1).
//
// Windowed-MTP changes exactly this step (Section 4 "Mechanism"; Appendix A
// pseudocode): for request r of length S the draft's index list is
// req_to_token[r, keep] with keep = [0, S) natively, or the sink [0, sink)
// followed by the window [S - W, S) once S > sink + W.  The output is the
// packed list format of paged attention libraries: kv_indptr[B + 1] (prefix
// sums of the kept counts) and kv_indices (the kept keys' pool rows, request
// after request, ascending position).  The native list costs O(S) per request
// and step, the windowed one O(sink + W).
//
// Grid: (pieces of at most kPiece kept keys) x B.  Each workgroup finds its
// request's offset with a wave-level prefix sum over the device-resident
// lengths and copies its piece of the table with coalesced reads and writes.

#include "../../include/wmtp.h"
#include "common.h"
#include "index_map.h"
#include "launch.h"

namespace wmtp {
namespace {

constexpr int kPiece = 8192;  // kept keys per workgroup

struct IndexArgs {
  const int32_t* table;
  int64_t stride;
  const int32_t* lens;
  int32_t* indptr;
  int32_t* indices;
  int32_t* err;
  int B, W, sink;
};

__device__ __forceinline__ int read_len(const IndexArgs& a, int b, bool report) {
  int S = a.lens[b];
  if (S < 0 || static_cast<int64_t>(S) > a.stride) {
    if (report) raise_error(a.err, WMTP_DERR_LEN_RANGE);
    S = S < 0 ? 0 : static_cast<int>(a.stride);
  }
  return S;
}

template <KeyMap M>
__global__ __launch_bounds__(256) void kv_index_kernel(IndexArgs a) {
  const int b = blockIdx.y;
  const int piece = blockIdx.x;
  __shared__ int s_off, s_n, s_S;
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    long long before = 0;
    int mine = 0, myS = 0;
    for (int base = 0; base <= b; base += kWave) {
      const int bb = base + lane;
      if (bb <= b) {
        const int S = read_len(a, bb, bb == b && piece == 0);
        const int n = selected_count<M>(S, a.W, a.sink);
        if (bb < b) {
          before += n;
        } else {
          mine = n;
          myS = S;
        }
      }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      before += __shfl_xor(before, off);
      mine += __shfl_xor(mine, off);
      myS += __shfl_xor(myS, off);
    }
    if (lane == 0) {
      s_off = static_cast<int>(before);
      s_n = mine;
      s_S = myS;
    }
  }
  __syncthreads();
  const int off = s_off;
  const int n = s_n;
  if (piece == 0 && threadIdx.x == 0) {
    if (b == 0) a.indptr[0] = 0;
    a.indptr[b + 1] = off + n;
  }
  const int j0 = piece * kPiece;
  if (j0 >= n) return;
  const int j1 = min(j0 + kPiece, n);
  const RowMap<M> map(s_S, a.W, a.sink, 1);
  const int32_t* trow = a.table + static_cast<int64_t>(b) * a.stride;
  for (int j = j0 + static_cast<int>(threadIdx.x); j < j1; j += blockDim.x)
    a.indices[static_cast<int64_t>(off) + j] = trow[map.row(j)];
}

}  // namespace

hipError_t launch_kv_indices(const int32_t* table, int64_t table_stride, const int32_t* lens, int B,
                             bool windowed, int W, int sink, int64_t n_keys_max, int32_t* indptr,
                             int32_t* indices, int32_t* err, hipStream_t st) {
  IndexArgs a;
  a.table = table;
  a.stride = table_stride;
  a.lens = lens;
  a.indptr = indptr;
  a.indices = indices;
  a.err = err;
  a.B = B;
  a.W = W;
  a.sink = sink;
  const unsigned pieces = static_cast<unsigned>(n_keys_max > 0 ? (n_keys_max + kPiece - 1) / kPiece : 1);
  const dim3 grid(pieces, static_cast<unsigned>(B));
  if (windowed)
    hipLaunchKernelGGL(kv_index_kernel<KeyMap::PagedWindow>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(kv_index_kernel<KeyMap::PagedFull>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace wmtp
