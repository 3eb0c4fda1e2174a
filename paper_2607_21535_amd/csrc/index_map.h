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
// Everything here is O(1) integer arithmetic per key: no index table exists.
#pragma once

#include "common.h"

namespace wmtp {

enum class KeyMap : int { Full = 0, Window = 1, Ring = 2 };

template <KeyMap M>
__device__ __forceinline__ int selected_count(int S, int W, int sink) {
  if constexpr (M == KeyMap::Full) {
    return S;
  } else {
    return S > sink + W ? sink + W : S;
  }
}

// Logical position of virtual key j (0 <= j < selected_count).
template <KeyMap M>
__device__ __forceinline__ int key_position(int j, int S, int W, int sink) {
  if constexpr (M == KeyMap::Full) {
    return j;
  } else {
    return (S > sink + W && j >= sink) ? S - W + (j - sink) : j;
  }
}

// Ring slot of logical position p.
__device__ __forceinline__ int ring_slot(int p, int sink, int R_w) {
  return p < sink ? p : sink + (p - sink) % R_w;
}

// Storage row of virtual key j, with the per-sequence part hoisted: one
// compare for the window, one compare-and-subtract for the ring wrap.
template <KeyMap M>
struct RowMap {
  int sink;
  int R_w;
  int shift;  // position(j) = j + shift for j >= sink
  int r0;     // shift mod R_w (ring only)

  __device__ __forceinline__ RowMap(int S, int W, int sink_, int R_w_) : sink(sink_), R_w(R_w_) {
    shift = (M != KeyMap::Full && S > sink_ + W) ? S - W - sink_ : 0;
    r0 = (M == KeyMap::Ring) ? shift % R_w_ : 0;
  }

  __device__ __forceinline__ int row(int j) const {
    if constexpr (M == KeyMap::Full) {
      return j;
    } else if constexpr (M == KeyMap::Window) {
      return j < sink ? j : j + shift;
    } else {
      // j - sink < W <= R_w and r0 < R_w, so one subtraction wraps.
      if (j < sink) return j;
      int t = (j - sink) + r0;
      if (t >= R_w) t -= R_w;
      return sink + t;
    }
  }
};

}  // namespace wmtp
