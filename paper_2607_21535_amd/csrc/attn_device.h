// Device pieces shared by the attention kernels: row lengths from the
// device-resident length arrays, streaming loads of the cache, the per-tile
// registers and the online softmax over 16-key MFMA tiles.
#pragma once

#include "../../include/wmtp.h"
#include "common.h"
#include "fp8.h"
#include "index_map.h"

#include <climits>

namespace wmtp {

// A length read from a device array, clamped to [0, cap] (flagged when out
// of range).
__device__ __forceinline__ int check_len(int S, int64_t cap, int32_t* err, bool report) {
  if (S < 0 || static_cast<int64_t>(S) > cap) {
    if (report) raise_error(err, WMTP_DERR_LEN_RANGE);
    S = S < 0 ? 0 : static_cast<int>(cap);
  }
  return S;
}

__device__ __forceinline__ int read_len(const int32_t* lens, int b, int64_t cap, int32_t* err,
                                        bool report) {
  return check_len(lens[b], cap, err, report);
}

// Tail maps.  Tree (speculation candidates): query row v = b * qps + t is
// candidate t of request b, whose committed length is lens[b] and
// speculative depth n_q[b] (0 .. dd); every candidate sees lens[b] + depth
// rows.  Fused windowed draft step: the row sees its old length lens[b] plus the
// n_q[b] (0 .. dd) rows appended by this call; a dense cache cannot grow
// past `cap` (flagged, the rows past it dropped).  Out-of-range values are
// clamped and flagged.  `s_commit` receives the old / committed length.
template <KeyMap M>
__device__ __forceinline__ int tail_len(const int32_t* lens, const int32_t* extra, int dd, int64_t cap,
                                        int b, int32_t* err, bool report, int& s_commit) {
  constexpr bool kDense = is_step(M) && !is_ring(M);
  const int64_t lim = kDense ? (cap < INT_MAX - dd ? cap : INT_MAX - dd) : INT_MAX - dd;
  // Both values are read before either is checked: a read placed after an
  // error report would wait for the first one (the report may write memory
  // the second read could alias).
  int S = lens[b];
  int i = extra[b];
  if (S < 0 || S > lim) {
    if (report) raise_error(err, WMTP_DERR_LEN_RANGE);
    S = S < 0 ? 0 : static_cast<int>(lim);
  }
  if (i < 0 || i > dd) {
    if (report) raise_error(err, WMTP_DERR_NNEW_RANGE);
    i = i < 0 ? 0 : dd;
  }
  if (kDense && static_cast<int64_t>(S) + i > cap) {
    if (report) raise_error(err, WMTP_DERR_CAPACITY);
    i = static_cast<int>(cap - S);
  }
  s_commit = S;
  return S + i;
}

// Query row v = b * qps + t is row t of sequence b.  lens[b] counts every
// cached row, including the n new rows of this call (n = n_q[b], or qps when
// n_q is NULL); row t attends causally: it sees the first lens[b] - n + t + 1
// rows (the draft decode step is the case qps = n = 1).  Rows t >= n, and
// every row of an empty sequence, have no keys; a non-empty sequence with
// fewer rows than n is flagged.  Tail maps use tail_len.  Returns that
// length; `b_out` receives the sequence.
template <KeyMap M>
__device__ __forceinline__ int visible_len(const int32_t* lens, const int32_t* n_q, int qps,
                                           int64_t cap, int32_t* err, int v, bool report,
                                           int& b_out, int dd) {
  if constexpr (has_tail(M)) {
    const int b = v / qps;
    b_out = b;
    int s_commit;
    return tail_len<M>(lens, n_q, dd, cap, b, err, report && v == b * qps, s_commit);
  }
  const int b = qps == 1 ? v : v / qps;
  const int t = v - b * qps;
  b_out = b;
  // Both values are read before either is checked (as in tail_len).
  const int S_read = lens[b];
  int n = n_q != nullptr ? n_q[b] : qps;
  const int S = check_len(S_read, cap, err, report);
  if (n_q != nullptr) {
    if (n < 0 || n > qps) {
      if (report) raise_error(err, WMTP_DERR_NNEW_RANGE);
      n = n < 0 ? 0 : qps;
    }
  }
  if (t >= n || S == 0) return 0;  // padding row, or an empty (padding) sequence
  const int L = S - n + t + 1;
  if (L < 1) {  // fewer cached rows than new query rows
    if (report) raise_error(err, WMTP_DERR_LEN_RANGE);
    return 0;
  }
  return L;
}

// Streaming loads of the KV cache: non-temporal (read once per call, kept out
// of the caches' way).
template <typename T, typename E>
__device__ __forceinline__ T stream_load(const E* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const T*>(p));
}

// Maximum and sum of x over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (one
// query head of an MFMA tile), as with shuffles by lane ^ 16 and then
// lane ^ 32, but without their LDS permutes and waits: v_permlane16_swap
// exchanges lanes 16..31 and 48..63 of its first register with lanes 0..15
// and 32..47 of its second, v_permlane32_swap lanes 32..63 of the first with
// lanes 0..31 of the second, so with x in both registers each lane then holds
// x of itself and of its partner, in one VALU op.  (The compiler's builtins
// for these swaps returned the first register twice in this toolchain, so
// they are written as inline assembly; the s_nop covers the wait a swap needs
// after a VALU write of its operands.)  The sum adds the same pairs in the
// same order as the shuffles, so its bits are theirs.
__device__ __forceinline__ void swap_rows16(float& a, float& b) {
  asm("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void swap_rows32(float& a, float& b) {
  asm("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ float max_across_rows(float x) {
  float a = x, b = x;
  swap_rows16(a, b);
  float c = fmaxf(a, b), e = c;
  swap_rows32(c, e);
  return fmaxf(c, e);
}
__device__ __forceinline__ float sum_across_rows(float x) {
  float a = x, b = x;
  swap_rows16(a, b);
  float c = a + b, e = c;
  swap_rows32(c, e);
  return c + e;
}

// Registers of one 16-key tile on one lane.  kx holds 16-byte units
// 64 i + lane of the tile's K rows, key-major (8 bf16 values or 16 fp8 codes
// each); vx holds the lane's VEC values (or codes) of keys 4*grp + i as words.
template <int D, bool F8>
struct TileRegs {
  u32x4 kx[D / 32];
  uint32_t vx[4][D / 32];
};
template <int D>
struct TileRegs<D, true> {
  u32x4 kx[D / 64];
  uint32_t vx[4][D / 64];
};

// Online softmax of one wave over 16-key tiles: 16 query heads (the lane's
// column col), the running maximum m (exp2 domain), the sums l of the
// bf16-rounded weights (normalises the output) and z of the fp32 weights
// (the log-sum-exp), and the output O^T[d, heads] in VEC MFMA accumulators:
// acc[e][jj] of lane (grp, col) holds head col at
// d = (e / SEG) * 16 * SEG + SEG * (4 grp + jj) + e % SEG, where SEG is the
// lane's run of contiguous value columns (min(VEC, 8) for bf16, VEC for fp8).
template <int D, bool F8>
struct OnlineHeads {
  static constexpr int VEC = D / 16;
  floatx4 acc[VEC];
  float m, l, z;

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = floatx4{0.f, 0.f, 0.f, 0.f};
    m = neg_inf();
    l = 0.f;
    z = 0.f;
  }

  // Takes the logits of NT consecutive 16-key tiles: s[u][i] is the raw
  // logit of key jt + 16 u + 4 grp + i for head col (keys at or past j_end
  // are masked out; kLateMask: only when the group reaches j_end, a branch
  // that pays off where the computation, not the memory, bounds the kernel).
  // Updates the running maximum, rescales the state when it grows and
  // returns the weights as the P^T operands of the tiles.
  template <int NT, bool kLateMask = false>
  __device__ __forceinline__ void weigh(const floatx4 (&s)[NT], int jt, int j_end, float sl2, int grp,
                                        bf16x4 (&pop)[NT]) {
    float sv[NT][4];
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i) sv[u][i] = s[u][i] * sl2;
    if (!kLateMask || jt + kTileKeys * NT > j_end) {  // wave-uniform
#pragma unroll
      for (int u = 0; u < NT; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (jt + kTileKeys * u + 4 * grp + i >= j_end) sv[u][i] = neg_inf();
    }
    float mt = neg_inf();
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i) mt = fmaxf(mt, sv[u][i]);
    const float m_new = fmaxf(m, max_across_rows(mt));
    if (__any(m_new > m)) {
      const float alpha = __builtin_amdgcn_exp2f(m - m_new);
      l *= alpha;
      z *= alpha;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] *= alpha;
    }
    m = m_new;
    // The weights of keys 4*grp + i for head col, rounded to bf16; the
    // denominator sums the same rounded weights.
#pragma unroll
    for (int u = 0; u < NT; ++u) {
      uint32_t pb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const float p0 = __builtin_amdgcn_exp2f(sv[u][2 * i] - m);
        const float p1 = __builtin_amdgcn_exp2f(sv[u][2 * i + 1] - m);
        pb[i] = pack_bf16x2(p0, p1);
        l += bf16_lo(pb[i]) + bf16_hi(pb[i]);
        z += p0 + p1;
      }
      pop[u] = __builtin_bit_cast(bf16x4, u32x2{pb[0], pb[1]});
    }
  }

  // weigh with fewer vector instructions, for the multi-row kernel (whose
  // time is set by its compute waves): the maximum is taken over the raw
  // logits (rounding is monotone, so it scales to the maximum of the scaled
  // ones), the scale is folded into the exponent, exp2(fma(s, sl2, -m)), and
  // the sum of the rounded weights is a bf16 dot product with (1, 1) per
  // weight pair.  Requires sl2 > 0: the kernel puts the sign of the scale
  // into its queries (exact) and stands in the smallest normal float for a
  // zero scale (every weight is then exp2 of a number within |s| 2^-126 of 0,
  // i.e. 1 to fp32 precision, as for the scale 0, and a masked key keeps
  // exp2(-inf) = 0 where -inf * 0 would be NaN).  The weights and sums may
  // differ from weigh's in the last bit.
  template <int NT>
  __device__ __forceinline__ void weigh_lean(const floatx4 (&s)[NT], int jt, int j_end, float sl2, int grp,
                                             bf16x4 (&pop)[NT]) {
    const bool tail = jt + kTileKeys * NT > j_end;  // wave-uniform: the group reaches the row's end
    float sv[NT][4];
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i) sv[u][i] = s[u][i];
    if (tail) {
#pragma unroll
      for (int u = 0; u < NT; ++u)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (jt + kTileKeys * u + 4 * grp + i >= j_end) sv[u][i] = neg_inf();
    }
    float mt = neg_inf();
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i) mt = fmaxf(mt, sv[u][i]);
    // Key jt is visible, so mt is finite after the exchange.
    const float m_new = fmaxf(m, max_across_rows(mt) * sl2);
    if (__any(m_new > m)) {
      const float alpha = __builtin_amdgcn_exp2f(m - m_new);
      l *= alpha;
      z *= alpha;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] *= alpha;
    }
    m = m_new;
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3f803f80u);
#pragma unroll
    for (int u = 0; u < NT; ++u) {
      uint32_t pb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[u][2 * i], sl2, -m));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[u][2 * i + 1], sl2, -m));
        pb[i] = pack_bf16x2(p0, p1);
        l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pb[i]), ones, l, false);
        z += p0 + p1;
      }
      pop[u] = __builtin_bit_cast(bf16x4, u32x2{pb[0], pb[1]});
    }
  }

  // O^T += V^T . P^T for one tile: vx holds the lane's value words of keys
  // 4 grp + i (bf16: VEC values, fp8: VEC codes, per key).
  template <int NW>
  __device__ __forceinline__ void accumulate(const bf16x4& pop, const uint32_t (&vx)[4][NW]) {
    if constexpr (F8) {
      // V^T operand for output tiles 4w .. 4w+3: interleave the codes of keys
      // (0, 1) and (2, 3) byte by byte, then widen pairs to bf16.
#pragma unroll
      for (int w = 0; w < VEC / 4; ++w) {
        const uint32_t p01 = __builtin_amdgcn_perm(vx[1][w], vx[0][w], 0x05010400u);
        const uint32_t q01 = __builtin_amdgcn_perm(vx[1][w], vx[0][w], 0x07030602u);
        const uint32_t p23 = __builtin_amdgcn_perm(vx[3][w], vx[2][w], 0x05010400u);
        const uint32_t q23 = __builtin_amdgcn_perm(vx[3][w], vx[2][w], 0x07030602u);
        const uint32_t lo01[4] = {fp8x2_to_bf16x2<false>(p01), fp8x2_to_bf16x2<true>(p01),
                                  fp8x2_to_bf16x2<false>(q01), fp8x2_to_bf16x2<true>(q01)};
        const uint32_t lo23[4] = {fp8x2_to_bf16x2<false>(p23), fp8x2_to_bf16x2<true>(p23),
                                  fp8x2_to_bf16x2<false>(q23), fp8x2_to_bf16x2<true>(q23)};
#pragma unroll
        for (int x = 0; x < 4; ++x)
          acc[4 * w + x] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
              __builtin_bit_cast(bf16x4, u32x2{lo01[x], lo23[x]}), pop, acc[4 * w + x], 0, 0, 0);
      }
    } else {
      // V^T operand for output tile e: this lane's four keys at its value
      // column e, packed from the loaded rows (low or high halves of a word).
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t a01 = __builtin_amdgcn_perm(vx[1][e >> 1], vx[0][e >> 1], sel);
        const uint32_t a23 = __builtin_amdgcn_perm(vx[3][e >> 1], vx[2][e >> 1], sel);
        acc[e] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, u32x2{a01, a23}),
                                                          pop, acc[e], 0, 0, 0);
      }
    }
  }

  // One tile: logits s (key jt + 4 grp + i), value words vx.
  template <int NW>
  __device__ __forceinline__ void add(const floatx4& s, const uint32_t (&vx)[4][NW], int jt, int j_end,
                                      float sl2, int grp) {
    const floatx4 s1[1] = {s};
    bf16x4 pop[1];
    weigh(s1, jt, j_end, sl2, grp, pop);
    accumulate(pop[0], vx);
  }
};

}  // namespace wmtp
