// Key selection and ring slot arithmetic (Windowed-MTP, Section 4
// "Mechanism" and the Appendix A pseudocode of the windowing change).
//
// A sequence of length S exposes n_sel "virtual" keys j = 0 .. n_sel-1 in
// ascending logical position:
//   full      n_sel = S,                 position(j) = j
//   windowed  n_sel = min(S, sink + W);  when S > sink + W the positions are
//             0 .. sink-1 followed by S-W .. S-1, otherwise j itself
// The compact ring keeps position p in slot p (p < sink) or
// sink + (p - sink) mod R_w; the ring holds the whole window when R_w >= W.
// Everything here is O(1) integer arithmetic per key: no index table is
// built.  A paged pool adds one lookup of the request's token table
// (req_to_token[b][position]) per kept key -- for the windowed draft only at
// the sink + W kept positions (the Appendix A pseudocode's
// kv_index = req_to_token[r, keep]).
#pragma once

#include "common.h"

namespace wmtp {

// Key maps: where virtual key j of a query row is stored.
//   Full, Window       dense per-sequence cache, row = logical position
//   Ring               compact ring, row = ring slot of the position
//   PagedFull/Window   shared token pool, row = req_to_token[b][position]
//                      (the kernel resolves the table; RowMap gives positions)
//   Tree               speculation candidates over a ring (Section 7, tree
//                      speculation): candidate 0 and committed positions
//                      live at their ring slots; positions of candidate
//                      b >= 1 past the committed length live in its private
//                      run, rows numbered after the ring's
//   WindowStep, RingStep
//                      a windowed draft step fused with its append:
//                      positions before the old length live in the cache /
//                      ring, the step's new rows (at and past it) are read
//                      from the caller's new-row buffer, rows numbered after
//                      the cache's
enum class KeyMap : int {
  Full = 0, Window = 1, Ring = 2, PagedFull = 3, PagedWindow = 4, Tree = 5, WindowStep = 7, RingStep = 8
};

constexpr bool is_paged(KeyMap m) { return m == KeyMap::PagedFull || m == KeyMap::PagedWindow; }
constexpr bool is_windowed(KeyMap m) {
  return m == KeyMap::Window || m == KeyMap::Ring || m == KeyMap::PagedWindow || m == KeyMap::Tree ||
         m == KeyMap::WindowStep || m == KeyMap::RingStep;
}
constexpr bool is_ring(KeyMap m) { return m == KeyMap::Ring || m == KeyMap::Tree || m == KeyMap::RingStep; }
constexpr bool is_step(KeyMap m) { return m == KeyMap::WindowStep || m == KeyMap::RingStep; }
// Maps whose keys past a per-row boundary S_c come from a second buffer.
constexpr bool has_tail(KeyMap m) { return m == KeyMap::Tree || is_step(m); }

template <KeyMap M>
__device__ __forceinline__ int selected_count(int S, int W, int sink) {
  if constexpr (!is_windowed(M)) {
    return S;
  } else {
    return S > sink + W ? sink + W : S;
  }
}

// Storage row (dense, ring) or logical position (paged) of virtual key j,
// with the per-sequence part hoisted: one compare for the window, one
// compare-and-subtract for the ring wrap.
template <KeyMap M>
struct RowMap {
  int sink;
  int R_w;
  int shift;  // position(j) = j + shift for j >= sink
  int r0;     // shift mod R_w (ring maps only)
  int S_c = 0;     // tail maps: positions >= S_c come from the second buffer ...
  int bbase = -1;  // ... at rows bbase + (position - S_c); -1: no second buffer

  __device__ __forceinline__ RowMap(int S, int W, int sink_, int R_w_) : sink(sink_), R_w(R_w_) {
    shift = (is_windowed(M) && S > sink_ + W) ? S - W - sink_ : 0;
    r0 = is_ring(M) ? shift % R_w_ : 0;
  }

  __device__ __forceinline__ int row(int j) const {
    if constexpr (!is_windowed(M)) {
      if constexpr (has_tail(M)) {
        if (j >= S_c) return bbase + (j - S_c);
      }
      return j;
    } else if constexpr (!is_ring(M)) {
      const int pos = j < sink ? j : j + shift;
      if constexpr (has_tail(M)) {
        if (pos >= S_c) return bbase + (pos - S_c);
      }
      return pos;
    } else {
      if constexpr (has_tail(M)) {
        const int pos = j < sink ? j : j + shift;
        if (bbase >= 0 && pos >= S_c) return bbase + (pos - S_c);
      }
      // j - sink < W <= R_w and r0 < R_w, so one subtraction wraps.
      if (j < sink) return j;
      int t = (j - sink) + r0;
      if (t >= R_w) t -= R_w;
      return sink + t;
    }
  }
};

}  // namespace wmtp
