// Windowed draft decode attention in one launch: the attention sink plus the
// most recent W keys of each query row (Windowed-MTP Section 4 "Mechanism"
// and the Appendix A pseudocode), over a dense cache, the compact ring, the
// paged token pool, speculation candidates or the fused draft step; bf16 or
// fp8 (E4M3) cache.
//
// A windowed row attends at most sink + W keys whatever its length, so the
// work items of a row are fixed when the call is launched: item c of a row
// covers its selected keys [c * item_keys, (c + 1) * item_keys).  No length
// scan is needed to find an item, and the query and the row length are
// loaded together at the start.  The row's key set moves with its length,
// which is read on the device (a captured graph adapts to every replay).
//
// The value dimension is also cut into `NSL` slices of DS columns: the
// workgroup of (item, KV head, slice) computes the logits over whole key rows
// but accumulates only its slice of the value rows, so the partial result of
// an item is small and the merge of a (row, KV head, slice) reads little.
// The latency of one windowed call is set by a chain of dependent memory
// round trips, not by bandwidth: the row length, the key and value rows, the
// partials and the output.
//
// Merge in the same launch.  After writing its partial (maximum, two sums
// and the unnormalised output slice, as the split-K kernel writes them) a
// workgroup releases it at device scope and takes a ticket from the
// (row, KV head, slice) counter in the workspace.  The workgroup that takes
// the last ticket acquires every partial of its slice, combines them in item
// order -- the same order whichever workgroup finishes last, so the results
// are bitwise reproducible -- writes the output and resets the counter to
// zero for the next call.  No workgroup ever waits for another.
//
// Per 16-key tile and wave the arithmetic is that of the split-K kernel:
// S^T = K Q^T on v_mfma_f32_16x16x32_bf16 (K through LDS), the online
// softmax in the exp2 domain, O^T += V^T P^T on v_mfma_f32_16x16x16_bf16
// with P rounded to bf16 (OnlineHeads).

#include "../../include/wmtp.h"
#include "attn_device.h"
#include "launch.h"

#include <algorithm>
#include <climits>
#include <cstdlib>
#include <type_traits>

namespace wmtp {
namespace {

struct WinArgs {
  const uint16_t* q;
  const void* k;  // bf16 or fp8 elements
  const void* v;
  const int32_t* lens;
  const int32_t* n_q;    // new query rows per sequence (extend), depth (tree), n_new (step)
  const int32_t* table;  // paged: req_to_token [B, table_stride]
  int64_t table_stride;
  uint16_t* out;
  float* lse;
  int32_t* err;
  int32_t* lens_out;  // fused step: each row's new length
  int B, Hq, Hkv, G;
  int qps;        // query rows per sequence
  int64_t rows;   // dense: rows per sequence; ring: slots; paged: pool rows
  int64_t len_cap;
  int W, sink, R_w;
  float scale_log2;
  float out_scale;  // value scale of an fp8 cache (1 for bf16)
  const void* k2;   // tree: private runs; step: the new rows
  const void* v2;
  int64_t rows2;
  int dd;
  int item_keys;  // selected keys per work item (a multiple of 64)
  int n_items;    // work items per row
  int NI;         // work items in all: query rows x KV heads x n_items
  float* rec;         // partial records [query rows x KV heads x slices x n_items, kHdr + 16 DS]
  int32_t* tickets;   // [query rows x KV heads x slices], zero between calls
};

// Partials pass between workgroups on different XCDs, whose L2 caches are
// not coherent with each other.  They are written and read with device-scope
// accesses (buffer loads and stores with the sc1 policy), which the hardware
// performs at the device's point of coherence; an agent-scope release or
// acquire fence would instead write back or invalidate the whole L2 of the
// XCD (about a microsecond, serialised per workgroup).  Ordering: every
// thread waits for its stores to complete before the workgroup takes its
// ticket, and the merger reads only after it.
constexpr int kCohSc1 = 16;  // cache policy bit of the raw buffer builtins: sc1 (device scope)
constexpr int kHdr = 64;     // header floats of a partial record: m[16], l[16], z[16], 16 unused

// The base is uniform; it is passed through readfirstlane so that the
// descriptor is built in scalar registers (a descriptor the compiler
// believes divergent costs a loop around every load that uses it).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t record_rsrc(float* base) {
  // (the builtin returns int: each half goes back through uint32_t, or a
  // low half with bit 31 set would sign-extend into the high one)
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(p >> 32)));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(p & 0xffffffffu)));
  const uint64_t u = (static_cast<uint64_t>(hi) << 32) | lo;
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<float*>(u), 0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ void coherent_store16(__amdgpu_buffer_rsrc_t r, int byte_off, u32x4 x) {
  __builtin_amdgcn_raw_buffer_store_b128(x, r, byte_off, 0, kCohSc1);
}

// Waves per workgroup: four, one per SIMD.  (Eight, one 16-key tile each
// for a 128-key item, measured no faster: the item's tiles share the CU's
// four SIMDs either way.)
constexpr int win_waves(int) { return 4; }

template <int D, int DS, KeyMap M, bool F8>
__global__ __launch_bounds__(win_waves(DS) * kWave) void window_kernel(const int32_t* lens, const int32_t* n_q, const uint16_t* q, int NI, int n_items,
                                                                   int Hkv, int qps, int G, int Hq, int dd, WinArgs a) {
  constexpr int NW = win_waves(DS);
  constexpr int NT = NW * kWave;
  using KT = std::conditional_t<F8, uint8_t, uint16_t>;  // one cached K/V element
  constexpr int NSL = D / DS;  // value slices
  constexpr int VEC = DS / 16;  // slice values of one key per lane in the PV operand
  // A lane's VEC values come in pieces of SEG contiguous columns (16 bytes at
  // most), piece sg of lane col at slice column sg*16*SEG + SEG*col; fp8:
  // one piece of VEC codes.
  constexpr int SEG = F8 ? VEC : (VEC < 8 ? VEC : 8);
  constexpr int NSEG = VEC / SEG;
  constexpr int KCH = D / 32;  // 16x16x32 steps over d for the logits

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int grp = lane >> 4;
  const int col = lane & 15;

  // Workgroup -> (item it, slice s).  Consecutive workgroup ids land on
  // different XCDs; the NSL slices of one item get ids equal modulo 8, so
  // they read the same key rows through one L2.
  const int id = blockIdx.x;
  const int s = (id >> 3) % NSL;
  const int it = ((id >> 3) / NSL) * 8 + (id & 7);
  if (it >= NI) return;  // padding of the last group of eight: no item, no ticket
  const int c = it % n_items;
  const int vg = it / n_items;  // query row x KV heads + KV head
  const int g = vg % Hkv;
  const int v = vg / Hkv;
  const int b = qps == 1 ? v : v / qps;

  // Q^T operand (as in the split-K kernel): lane (grp, col) holds at step kk
  // the 8 d values of head col that the key operand holds.
  bf16x8 qf[KCH];
  {
    const bool live = col < G;
    const uint16_t* qp = q + (static_cast<int64_t>(v) * Hq + g * G + (live ? col : 0)) * D;
#pragma unroll
    for (int kk = 0; kk < KCH; ++kk) {
      const int d0 = F8 ? ((kk >> 1) * 4 + grp) * 16 + (kk & 1) * 8 : kk * 32 + grp * 8;
      u32x4 w = *reinterpret_cast<const u32x4*>(qp + d0);
      if (!live) w = u32x4{0u, 0u, 0u, 0u};
      qf[kk] = __builtin_bit_cast(bf16x8, w);
    }
  }
  const bool report = tid == 0 && c == 0 && s == 0 && g == 0;
  // The row's length; tail maps also give the committed / old length S_c
  // (one read of each length array: a second read would be ordered behind
  // the first one's error report).
  int S, S_c_len = 0;
  if constexpr (has_tail(M)) {
    S = tail_len<M>(lens, n_q, dd, a.len_cap, b, a.err, report && v == b * qps, S_c_len);
  } else {
    int b_unused;
    S = visible_len<M>(lens, n_q, qps, a.len_cap, a.err, v, report, b_unused, dd);
  }
  S = __builtin_amdgcn_readfirstlane(S);
  const int n_sel = selected_count<M>(S, a.W, a.sink);
  const int j0 = c * a.item_keys;
  const int j1 = min(j0 + a.item_keys, n_sel);

  // Rows of the cache (dense, ring or pool positions) come from the plain
  // map; a tail map reads the positions at and past S_c -- the fused step's
  // new rows, or a speculation candidate's own rows -- from the second
  // buffer, at virtual indices j >= j_c (one compare per load).
  constexpr KeyMap MB = M == KeyMap::WindowStep ? KeyMap::Window : (has_tail(M) ? KeyMap::Ring : M);
  RowMap<MB> map(S, a.W, a.sink, a.R_w);
  [[maybe_unused]] int S_c = S;
  [[maybe_unused]] int j_c = INT_MAX;
  [[maybe_unused]] int tbase = 0;  // first row of the candidate's run in the second buffer
  if constexpr (has_tail(M)) {
    S_c = __builtin_amdgcn_readfirstlane(S_c_len);
    bool tail = true;
    if constexpr (M == KeyMap::Tree) {
      const int cand = v - b * qps;
      tail = cand != 0;  // candidate 0 lives in the ring, as a chain writes it
      tbase = (cand - 1) * dd;
    }
    // The first virtual index whose position is >= S_c (positions grow with j).
    if (tail) j_c = S_c < a.sink ? S_c : max(a.sink, S_c - map.shift);
  }
  const int64_t rs = static_cast<int64_t>(Hkv) * D;  // elements between rows
  const int64_t seq_rows = is_paged(M) ? 0 : static_cast<int64_t>(b) * a.rows;
  const int64_t seq_off = (seq_rows * Hkv + g) * D;
  const KT* kbase = static_cast<const KT*>(a.k) + seq_off;
  const KT* vbase = static_cast<const KT*>(a.v) + seq_off;
  [[maybe_unused]] const int64_t off2 = (static_cast<int64_t>(b) * a.rows2 * Hkv + g) * D;
  [[maybe_unused]] const KT* kbase2 = has_tail(M) ? static_cast<const KT*>(a.k2) + off2 : nullptr;
  [[maybe_unused]] const KT* vbase2 = has_tail(M) ? static_cast<const KT*>(a.v2) + off2 : nullptr;
  // Second-buffer row of virtual index j >= j_c.
  [[maybe_unused]] auto tail_row = [&](int j) { return (j < a.sink ? j : j + map.shift) - S_c + tbase; };

  // Fused draft step: the first item of a row also writes its slice of its KV
  // head's new rows into the cache (ring: the resident ones).  No workgroup
  // of this launch reads those slots: the appended positions are read from
  // the new-row buffer, and on a ring (R_w >= W) a slot they overwrite held a
  // position outside every window of this call.  A thread's first unit is
  // loaded here, beside the tile loads, and stored once the workgroup has
  // its ticket (the merger: after the merge).
  [[maybe_unused]] constexpr int kCopyUnits = DS / 8;  // 16-byte units of the slice
  [[maybe_unused]] u32x4 cpy_k = {}, cpy_v = {};
  [[maybe_unused]] int64_t cpy_dst = -1;
  auto copy_unit = [&](int u, int64_t& dst) -> bool {  // false: nothing to write for unit u
    const int i = u / kCopyUnits;
    const int p = S_c + i;
    int slot = p;
    if constexpr (is_ring(M)) {
      if (p >= a.sink && p < S - a.R_w) return false;  // overwritten later in the same append
      slot = p < a.sink ? p : a.sink + (p - a.sink) % a.R_w;
    }
    dst = static_cast<int64_t>(slot) * rs + s * DS + (u % kCopyUnits) * 8;
    return true;
  };
  auto copy_src = [&](int u) { return off2 + static_cast<int64_t>(u / kCopyUnits) * rs + s * DS + (u % kCopyUnits) * 8; };
  if constexpr (is_step(M)) {
    if (c == 0 && tid < (S - S_c) * kCopyUnits) {
      int64_t dst;
      if (copy_unit(tid, dst)) {
        cpy_dst = dst;
        cpy_k = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.k2) + copy_src(tid));
        cpy_v = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v2) + copy_src(tid));
      }
    }
  }

  constexpr int kKUnits = F8 ? D / 16 : D / 8;  // 16-byte units per key row (one KV head)
  constexpr int kKPitch = kKUnits + 2;          // LDS row pitch in units (conflict-free operand reads)
  constexpr int kKLoads = kTileKeys * kKUnits / kWave;  // load instructions per tile
  constexpr int kStageBytes = NW * kTileKeys * kKPitch * 16;
  constexpr int kComboBytes = (NW / 2) * VEC * kWave * 16;  // the wave-combine regions
  constexpr int kRec = kHdr + kMaxGroup * DS;         // floats of one partial record
  constexpr int kLdsBytes = kStageBytes > kComboBytes ? kStageBytes : kComboBytes;
  static_assert(kRec * 4 <= kLdsBytes, "the partial record is staged in the K tiles' LDS");
  __shared__ __align__(16) unsigned char s_lds[kLdsBytes];
  __shared__ float s_m[NW][16];
  __shared__ float s_l[NW][16];
  __shared__ float s_z[NW][16];
  __shared__ int s_last;
  u32x4* s_k = reinterpret_cast<u32x4*>(s_lds) + wave * kTileKeys * kKPitch;

  // Paged: the pool rows of this item's keys, looked up once into LDS.
  [[maybe_unused]] int* slots = nullptr;
  if constexpr (is_paged(M)) {
    __shared__ int s_slot[kWinMaxItemKeys];
    slots = s_slot;
    const int32_t* trow = a.table + static_cast<int64_t>(b) * a.table_stride;
    bool bad = false;
    for (int j = j0 + tid; j < j1; j += NT) {
      int slot = trow[map.row(j)];
      if (slot < 0 || static_cast<int64_t>(slot) >= a.rows) {
        bad = true;
        slot = 0;
      }
      s_slot[j - j0] = slot;
    }
    if (bad) raise_error(a.err, WMTP_DERR_SLOT_RANGE);
    __syncthreads();
  }
  auto row_of = [&](int j) -> int {
    if constexpr (is_paged(M)) {
      return slots[j - j0];
    } else {
      return map.row(j);
    }
  };
  // `tail` (std::true_type / false_type): whether this item reaches the
  // tail keys; only the item holding a row's last keys does, so the others
  // load without the per-key choice.
  auto key_ptr = [&](int j, auto tail) -> const KT* {
    if constexpr (decltype(tail)::value) {
      if (j >= j_c) return kbase2 + static_cast<int64_t>(tail_row(j)) * rs;
    }
    return kbase + static_cast<int64_t>(row_of(j)) * rs;
  };
  auto value_ptr = [&](int j, auto tail) -> const KT* {
    if constexpr (decltype(tail)::value) {
      if (j >= j_c) return vbase2 + static_cast<int64_t>(tail_row(j)) * rs;
    }
    return vbase + static_cast<int64_t>(row_of(j)) * rs;
  };

  struct Tile {
    u32x4 kx[kKLoads];
    uint32_t vx[4][F8 ? VEC / 4 : VEC / 2];
  };
  const int n_tiles = j1 > j0 ? (j1 - j0 + kTileKeys - 1) / kTileKeys : 0;

  // Keys past j1 read a valid row (j0) and are masked out of the softmax; a
  // tile index past the end re-reads the last tile, so every path issues the
  // same loads and the waits cover exactly the tile being computed.
  auto load_tile = [&](Tile& T, int t, auto tail) {
    const int jt = j0 + min(t, n_tiles - 1) * kTileKeys;
#pragma unroll
    for (int i = 0; i < kKLoads; ++i) {
      const int f = i * kWave + lane;
      const int j = jt + f / kKUnits;
      T.kx[i] = stream_load<u32x4>(key_ptr(j < j1 ? j : j0, tail) + (f % kKUnits) * (16 / static_cast<int>(sizeof(KT))));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = jt + 4 * grp + i;
      const KT* p = value_ptr(j < j1 ? j : j0, tail) + s * DS + SEG * col;
      if constexpr (F8) {
        if constexpr (VEC == 16) {
          const u32x4 x = stream_load<u32x4>(p);
#pragma unroll
          for (int w = 0; w < 4; ++w) T.vx[i][w] = x[w];
        } else if constexpr (VEC == 8) {
          const u32x2 x = stream_load<u32x2>(p);
          T.vx[i][0] = x[0];
          T.vx[i][1] = x[1];
        } else {
          T.vx[i][0] = stream_load<uint32_t>(p);
        }
      } else {
#pragma unroll
        for (int sg = 0; sg < NSEG; ++sg) {
          if constexpr (SEG == 8) {
            const u32x4 x = stream_load<u32x4>(p + sg * 16 * SEG);
#pragma unroll
            for (int w = 0; w < 4; ++w) T.vx[i][sg * 4 + w] = x[w];
          } else {
            const u32x2 x = stream_load<u32x2>(p + sg * 16 * SEG);
            T.vx[i][sg * 2] = x[0];
            T.vx[i][sg * 2 + 1] = x[1];
          }
        }
      }
    }
  };

  OnlineHeads<DS, F8> st;
  st.init();
  const float sl2 = a.scale_log2;

  auto compute_tile = [&](const Tile& T, int t) {
    const int jt = j0 + t * kTileKeys;
    floatx4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < kKLoads; ++i) {
      const int f = i * kWave + lane;
      s_k[(f / kKUnits) * kKPitch + f % kKUnits] = T.kx[i];
    }
    if constexpr (F8) {
#pragma unroll
      for (int kk = 0; kk < D / 64; ++kk) {
        const u32x4 w = s_k[col * kKPitch + 4 * kk + grp];
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fp8x8_to_bf16x8(w[0], w[1])),
                                                     qf[2 * kk], sc, 0, 0, 0);
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fp8x8_to_bf16x8(w[2], w[3])),
                                                     qf[2 * kk + 1], sc, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < KCH; ++kk)
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, s_k[col * kKPitch + 4 * kk + grp]),
                                                     qf[kk], sc, 0, 0, 0);
    }
    st.add(sc, T.vx, jt, j1, sl2, grp);
  };

  // Two register buffers per wave (the next tile's loads in flight while the
  // current one is computed); the four waves take interleaved tiles.
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + NW - 1) / NW : 0;
  auto run_tiles = [&](auto tail) {
    Tile T0, T1;
    load_tile(T0, wave, tail);
    int i = 0;
    for (; i + 2 <= my_tiles; i += 2) {
      const int t = wave + i * NW;
      load_tile(T1, t + NW, tail);
      compute_tile(T0, t);
      load_tile(T0, t + 2 * NW, tail);
      compute_tile(T1, t + NW);
    }
    if (i < my_tiles) compute_tile(T0, wave + i * NW);
  };
  if (n_tiles > 0) {
    if constexpr (has_tail(M)) {
      if (j1 > j_c) {
        run_tiles(std::true_type{});
      } else {
        run_tiles(std::false_type{});
      }
    } else {
      run_tiles(std::false_type{});
    }

    // ---- combine the four waves: (m, l, z) per head, O pairwise ----
    float l_run = st.l, z_run = st.z;
    const float m_run = st.m;
    l_run = sum_across_rows(l_run);
    z_run = sum_across_rows(z_run);
    if (grp == 0) {
      s_m[wave][col] = m_run;
      s_l[wave][col] = l_run;
      s_z[wave][col] = z_run;
    }
    __syncthreads();
    float Mx = neg_inf();
#pragma unroll
    for (int w = 0; w < NW; ++w) Mx = fmaxf(Mx, s_m[w][col]);
    float Lx = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) Lx += s_l[w][col] * __builtin_amdgcn_exp2f(s_m[w][col] - Mx);
    float Zx = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) Zx += s_z[w][col] * __builtin_amdgcn_exp2f(s_m[w][col] - Mx);
    const float f = __builtin_amdgcn_exp2f(m_run - Mx);  // 0 for a wave with no tile
#pragma unroll
    for (int e = 0; e < VEC; ++e) st.acc[e] *= f;
    // O of the NW waves summed pairwise in a fixed tree ((w0 + w1) + (w2 +
    // w3)) + ..., through NW / 2 LDS regions; wave 0 ends with the total.
    floatx4* s_x = reinterpret_cast<floatx4*>(s_lds);
#pragma unroll
    for (int h = 1; h < NW; h <<= 1) {
      if (wave % (2 * h) == h) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) s_x[((wave / (2 * h)) * VEC + e) * kWave + lane] = st.acc[e];
      }
      __syncthreads();
      if (2 * h < NW) {
        if (wave % (2 * h) == 0) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) st.acc[e] += s_x[((wave / (2 * h)) * VEC + e) * kWave + lane];
        }
        __syncthreads();
      }
    }
    // The partial record of (row, KV head, slice, item): header m, l, z per
    // head, then o [16 heads, DS] (acc[e][jj] of lane (grp, col) is head col
    // at slice column (e / SEG) * 16 * SEG + SEG * (4 grp + jj) + e % SEG),
    // staged in LDS by wave 0 and stored by every thread, 16 bytes each.
    float* s_rec = reinterpret_cast<float*>(s_lds);
    if (wave == 0) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) st.acc[e] += s_x[e * kWave + lane];
      if (grp == 0) {
        s_rec[col] = Mx;
        s_rec[16 + col] = Lx;
        s_rec[32 + col] = Zx;
      }
#pragma unroll
      for (int sg = 0; sg < NSEG; ++sg)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
#pragma unroll
          for (int w = 0; w < SEG / 4; ++w) {
            const int e = sg * SEG + 4 * w;
            *reinterpret_cast<floatx4*>(s_rec + kHdr + col * DS + sg * 16 * SEG + SEG * (4 * grp + jj) + 4 * w) =
                floatx4{st.acc[e][jj], st.acc[e + 1][jj], st.acc[e + 2][jj], st.acc[e + 3][jj]};
          }
    }
    __syncthreads();
    const __amdgpu_buffer_rsrc_t rr = record_rsrc(a.rec + ((static_cast<int64_t>(vg) * NSL + s) * n_items + c) * kRec);
    for (int i = tid; i < kRec / 4; i += NT)
      coherent_store16(rr, i * 16, reinterpret_cast<const u32x4*>(s_rec)[i]);
    __builtin_amdgcn_s_waitcnt(0);  // the stores are complete at the point of coherence
  }

  // The fused step's copy of the new rows, stored after the ticket: a
  // store ahead of the merge's loads would hold them up (memory operations
  // of a wave complete in order).
  auto store_copy = [&]() {
    if constexpr (is_step(M)) {
      if (c == 0) {
        uint16_t* kw = const_cast<uint16_t*>(reinterpret_cast<const uint16_t*>(kbase));
        uint16_t* vw = const_cast<uint16_t*>(reinterpret_cast<const uint16_t*>(vbase));
        if (cpy_dst >= 0) {
          *reinterpret_cast<u32x4*>(kw + cpy_dst) = cpy_k;
          *reinterpret_cast<u32x4*>(vw + cpy_dst) = cpy_v;
        }
        for (int u = tid + NT; u < (S - S_c) * kCopyUnits; u += NT) {  // long appends
          int64_t dst;
          if (!copy_unit(u, dst)) continue;
          *reinterpret_cast<u32x4*>(kw + dst) =
              *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.k2) + copy_src(u));
          *reinterpret_cast<u32x4*>(vw + dst) =
              *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v2) + copy_src(u));
        }
      }
    }
  };

  // ---- ticket: the last workgroup of (row, KV head, slice) merges ----
  int32_t* ticket = a.tickets + (static_cast<int64_t>(vg) * NSL + s);
  __syncthreads();
  if (tid == 0) {
    const int old = __hip_atomic_fetch_add(ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = old == n_items - 1;
    if (last) __hip_atomic_store(ticket, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = last;
  }
  __syncthreads();
  if (!s_last) {
    store_copy();
    return;
  }

  // Combine the items that hold keys, in item order, in batches of NB:
  // M = running max of m, and O, L, Z the sums of o, l, z weighted by
  // 2^(m - M) (a batch rescales the sums of the earlier ones when M grows).
  // Thread t owns float4 columns t, t + NT, ... of [G heads x DS / 4] and
  // loads, for a batch's items, those columns and its heads' m, l, z into
  // registers, all loads in flight together; a slot past the batch's last
  // item holds m = -inf and zeros and gets weight 0, so the combine takes
  // runs of eight items with no branch inside a run.
  constexpr int Q4 = DS / 4;
  constexpr int CPT = (kMaxGroup * Q4 + NT - 1) / NT;  // columns per thread
  constexpr int NB = 32 / CPT;                                       // items per batch
  const int n_c = ceil_div_i(n_sel, a.item_keys);
  float* gbase = a.rec + (static_cast<int64_t>(vg) * NSL + s) * n_items * kRec;
  const __amdgpu_buffer_rsrc_t rg = record_rsrc(gbase);
  float Mrun[CPT], L[CPT], Z[CPT];
  floatx4 O[CPT];
#pragma unroll
  for (int x = 0; x < CPT; ++x) {
    Mrun[x] = neg_inf();
    L[x] = 0.f;
    Z[x] = 0.f;
    O[x] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  for (int c0 = 0; c0 < n_c; c0 += NB) {
    const int nb = min(NB, n_c - c0);
    floatx4 ov[NB][CPT];
    float hm[NB][CPT], hs[NB][CPT], hz[NB][CPT];
#pragma unroll
    for (int cc = 0; cc < NB; ++cc) {
      // The item's record offset is one uniform (scalar) operand of the
      // loads; a thread's offsets within a record are fixed (columns of
      // padding heads load those of head G - 1 and are not written).
      const int so = (c0 + cc) * kRec * 4;
#pragma unroll
      for (int x = 0; x < CPT; ++x) {
        const int colx = tid + x * NT;
        const int hl = min(colx / Q4, G - 1), q4 = colx % Q4;
        ov[cc][x] = floatx4{0.f, 0.f, 0.f, 0.f};
        hm[cc][x] = neg_inf();
        hs[cc][x] = 0.f;
        hz[cc][x] = 0.f;
        if (cc < nb) {
          ov[cc][x] = __builtin_bit_cast(
              floatx4, __builtin_amdgcn_raw_buffer_load_b128(rg, (kHdr + hl * DS + 4 * q4) * 4, so, kCohSc1));
          hm[cc][x] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, hl * 4, so, kCohSc1));
          hs[cc][x] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, (16 + hl) * 4, so, kCohSc1));
          hz[cc][x] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, (32 + hl) * 4, so, kCohSc1));
        }
      }
    }
#pragma unroll
    for (int x = 0; x < CPT; ++x) {
      float mb = Mrun[x];
#pragma unroll
      for (int cc = 0; cc < NB; ++cc) mb = fmaxf(mb, hm[cc][x]);
      const float f = mb == neg_inf() ? 0.f : __builtin_amdgcn_exp2f(Mrun[x] - mb);  // 0 before the first batch
      O[x] *= f;
      L[x] *= f;
      Z[x] *= f;
#pragma unroll
      for (int c8 = 0; c8 < NB; c8 += 8) {
        if (c8 < nb) {
#pragma unroll
          for (int i = 0; i < 8 && c8 + i < NB; ++i) {
            const int cc = c8 + i;
            const float w = cc < nb ? __builtin_amdgcn_exp2f(hm[cc][x] - mb) : 0.f;
            O[x] += w * ov[cc][x];
            L[x] += w * hs[cc][x];
            Z[x] += w * hz[cc][x];
          }
        }
      }
      Mrun[x] = mb;
    }
  }
#pragma unroll
  for (int x = 0; x < CPT; ++x) {
    const int colx = tid + x * NT;
    const int hl = colx / Q4, q4 = colx % Q4;
    if (hl >= G) continue;
    float r[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = n_c > 0 ? O[x][i] / L[x] * a.out_scale : 0.f;
    const int h = g * G + hl;
    *reinterpret_cast<u32x2*>(a.out + (static_cast<int64_t>(v) * Hq + h) * D + s * DS + 4 * q4) =
        u32x2{pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3])};
    if (a.lse != nullptr && s == 0 && q4 == 0)
      a.lse[static_cast<int64_t>(v) * Hq + h] = n_c > 0 ? (Mrun[x] + log2f(Z[x])) * kLn2 : neg_inf();
  }
  store_copy();
  if constexpr (is_step(M)) {
    if (g == 0 && s == 0 && tid == 0) a.lens_out[v] = S;  // this launch reads only the old lengths
  }
}

template <int D, int DS, KeyMap M, bool F8>
hipError_t launch_typed(const AttnLaunch& L, hipStream_t st) {
  WinArgs a;
  a.q = L.q; a.k = L.k; a.v = L.v; a.lens = L.lens; a.n_q = L.n_q;
  a.table = L.table; a.table_stride = L.table_stride;
  a.out = L.out; a.lse = L.lse; a.err = L.err; a.lens_out = L.lens_out;
  a.B = L.B; a.Hq = L.Hq; a.Hkv = L.Hkv; a.G = L.Hq / L.Hkv; a.qps = L.qps;
  a.rows = L.rows; a.len_cap = L.len_cap;
  a.W = L.W; a.sink = L.sink; a.R_w = L.R_w;
  a.scale_log2 = L.scale * L.k_scale * kLog2e;
  a.out_scale = L.v_scale;
  a.k2 = L.k2; a.v2 = L.v2; a.rows2 = L.rows2; a.dd = L.dd;
  a.item_keys = L.win_keys;
  a.n_items = L.win_items;
  const int64_t NI = static_cast<int64_t>(L.B) * L.qps * L.Hkv * L.win_items;
  a.NI = static_cast<int>(NI);
  a.rec = L.pm; a.tickets = L.tickets;
  const int64_t groups = (NI + 7) / 8;
  const dim3 grid(static_cast<unsigned>(groups * (D / DS) * 8));
  hipLaunchKernelGGL((window_kernel<D, DS, M, F8>), grid, dim3(win_waves(DS) * kWave), 0, st, a.lens, a.n_q, a.q,
                     a.NI, a.n_items, a.Hkv, a.qps, a.G, a.Hq, a.dd, a);
  return hipGetLastError();
}

template <int D, KeyMap M, bool F8>
hipError_t launch_slices(const AttnLaunch& L, hipStream_t st) {
  if constexpr (D > kWinSlice) {
    if (L.win_slices > 1) return launch_typed<D, kWinSlice, M, F8>(L, st);
  }
  return launch_typed<D, D, M, F8>(L, st);
}

template <int D>
hipError_t launch_d(const AttnLaunch& L, hipStream_t st) {
  if (L.kv_fp8) {
    switch (L.variant) {
      case WMTP_VARIANT_FULL: return launch_slices<D, KeyMap::Full, true>(L, st);
      case WMTP_VARIANT_WINDOWED: return launch_slices<D, KeyMap::Window, true>(L, st);
      case WMTP_VARIANT_RING: return launch_slices<D, KeyMap::Ring, true>(L, st);
      case WMTP_VARIANT_PAGED_FULL: return launch_slices<D, KeyMap::PagedFull, true>(L, st);
      case WMTP_VARIANT_PAGED_WINDOWED: return launch_slices<D, KeyMap::PagedWindow, true>(L, st);
      default: return hipErrorInvalidValue;  // no fp8 tree or fused-step kernels
    }
  }
  if (L.step) {
    switch (L.variant) {
      case WMTP_VARIANT_WINDOWED: return launch_slices<D, KeyMap::WindowStep, false>(L, st);
      case WMTP_VARIANT_RING: return launch_slices<D, KeyMap::RingStep, false>(L, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (L.variant) {
    case WMTP_VARIANT_FULL: return launch_slices<D, KeyMap::Full, false>(L, st);
    case WMTP_VARIANT_WINDOWED: return launch_slices<D, KeyMap::Window, false>(L, st);
    case WMTP_VARIANT_RING: return launch_slices<D, KeyMap::Ring, false>(L, st);
    case WMTP_VARIANT_PAGED_FULL: return launch_slices<D, KeyMap::PagedFull, false>(L, st);
    case WMTP_VARIANT_PAGED_WINDOWED: return launch_slices<D, KeyMap::PagedWindow, false>(L, st);
    case WMTP_VARIANT_TREE: return launch_slices<D, KeyMap::Tree, false>(L, st);
    default: return hipErrorInvalidValue;
  }
}

int env_int(const char* name, int dflt) {
  const char* e = std::getenv(name);
  if (e == nullptr || *e == '\0') return dflt;
  const int x = std::atoi(e);
  return x > 0 ? x : dflt;
}

// Estimated time (us) of one windowed call with the given layout: rounds of
// split workgroups (a round trip plus the item's bytes through one CU), then
// one merge (a round trip plus the slice's partials through one CU), and
// never less than the whole read at the device's bandwidth; ties (calls
// bound by that read) go to the layout with the shorter chain.  The unsliced
// kernel at d = 256 holds more than 256 registers per lane: one workgroup
// per CU.
double estimate_us(int64_t rows, int keys, int d, int elem, int item_keys, int slices, int cus) {
  const int64_t items = (keys + item_keys - 1) / item_keys;
  const int64_t wgs = rows * items * slices;
  const int64_t per_round = (d == 256 && slices == 1 ? 1LL : 2LL) * cus;
  const int64_t rounds = (wgs + per_round - 1) / per_round;
  const int ds = d / slices;
  const int64_t batches = (items + 32 / std::max(1, ds / 64) - 1) / (32 / std::max(1, ds / 64));
  const double per_cu = 1.0e5;  // bytes per us through one CU
  const double wg_bytes = static_cast<double>(item_keys) * (d + ds) * elem;
  const double merge_bytes = static_cast<double>(items) * kMaxGroup * ds * 4.0;
  const double chain = rounds * (1.5 + wg_bytes / per_cu) + 1.0 + batches * 1.5 + merge_bytes / per_cu;
  const double total = static_cast<double>(rows) * keys * (static_cast<double>(d) * slices + d) * elem;
  return std::max(chain, 3.0 + total / 6.0e6) + 1e-3 * chain;
}

}  // namespace

WinPlan plan_window(int NV, int Hq, int Hkv, int d, int keys) {
  WinPlan p{};
  if (NV <= 0 || keys <= 0) return p;
  static const int keys_env = env_int("WMTP_WIN_KEYS", 0);
  static const int slices_env = env_int("WMTP_WIN_SLICES", 0);
  (void)Hq;
  const int64_t rows = static_cast<int64_t>(NV) * Hkv;
  // Sliced layouts need one counter per (row, KV head, slice).
  const int sliced = d > kWinSlice && rows * (d / kWinSlice) <= kMaxTickets ? d / kWinSlice : 1;
  if (rows > kMaxTickets) return p;  // n_items = 0: not supported
  const int cap = std::min(kWinMaxItemKeys, (keys + kChunkQuantum - 1) / kChunkQuantum * kChunkQuantum);
  // The layout is chosen for a bf16 cache and kept for fp8 (one workspace
  // size serves both); the estimate is that of the bf16 read.
  double best = 0.0;
  for (int sl : {sliced, 1}) {
    if (slices_env > 0 && sl != (slices_env > 1 ? sliced : 1)) continue;
    for (int ik = kChunkQuantum; ik <= cap; ik *= 2) {
      if (keys_env > 0 && ik != std::min(cap, keys_env / kChunkQuantum * kChunkQuantum)) continue;
      const double e = estimate_us(rows, keys, d, 2, ik, sl, device_cus());
      if (p.item_keys == 0 || e < best) {
        best = e;
        p.item_keys = ik;
        p.slices = sl;
      }
    }
    if (sl == 1) break;
  }
  if (p.item_keys == 0) {  // an override outside the powers of two
    p.item_keys = std::min(cap, std::max(kChunkQuantum, keys_env / kChunkQuantum * kChunkQuantum));
    p.slices = slices_env > 1 ? sliced : 1;
  }
  p.n_items = (keys + p.item_keys - 1) / p.item_keys;
  // Partial records: per (row, KV head, slice, item) a header of kHdr floats
  // and o [16 heads, d / slices] in fp32.
  const size_t records = static_cast<size_t>(rows) * p.n_items * p.slices;
  const size_t rec_bytes = (kHdr + static_cast<size_t>(kMaxGroup) * (d / p.slices)) * sizeof(float);
  if (static_cast<int64_t>(p.n_items) * static_cast<int64_t>(rec_bytes) >= INT_MAX) {
    p.n_items = 0;  // record offsets within a (row, KV head, slice) are 32-bit
    return p;
  }
  p.off_pm = kTicketBytes;
  p.off_pl = p.off_pz = p.off_po = p.off_pm;  // (one array of records)
  p.bytes = p.off_pm + records * rec_bytes;
  return p;
}

bool use_window_kernel_full(int NV, int Hkv, int d, int64_t S_max) {
  // Short full contexts are launch-bound like windowed calls and take the
  // one-launch kernel under the same row limit, up to a capacity measured on
  // MI355X (graph-replayed calls, one sequence, Hkv = 2; split + merge / one
  // launch): d = 256, Hq = 32: 1K 11.1 / 8.1 us, 4K 12.5 / 10.3, 8K 14.4 /
  // 13.1, 16K 16.9 / 16.3, 32K 21.3 / 40.2; d = 128, Hq = 16: 1K 8.9 / 6.7,
  // 4K 9.6 / 8.7, 8K 10.3 / 10.6 (the best item size), 16K 11.1 / 15.1.
  // WMTP_WIN_FULL_MAX_KEYS overrides the capacity limit (0: never), read at
  // every call.
  int64_t max_keys = d >= 256 ? kWinFullMaxKeys : kWinFullMaxKeys / 4;
  if (const char* e = std::getenv("WMTP_WIN_FULL_MAX_KEYS"); e != nullptr && *e != '\0') {
    char* end = nullptr;
    const long long x = std::strtoll(e, &end, 10);
    if (end != e && x >= 0) max_keys = x;
  }
  return S_max > 0 && S_max <= max_keys && use_window_kernel(NV, Hkv);
}

bool use_window_kernel(int NV, int Hkv) {
  // Measured on MI355X at d = 256, Hq = 32, W = 2048: one sequence (2 rows of
  // KV heads) 13.1 us per draft step against 14.9 us with split + merge; 8
  // extend rows, 4 tree candidates or 8 sequences are faster with the
  // split + merge kernels, whose merge runs on a workgroup per row and head.
  // WMTP_WIN_ONE_LAUNCH_ROWS overrides the threshold (0: never), read at
  // every call so that tests can run both paths in one process.
  int64_t max_rows = kWinOneLaunchRows;
  if (const char* e = std::getenv("WMTP_WIN_ONE_LAUNCH_ROWS"); e != nullptr && *e != '\0') {
    char* end = nullptr;
    const long long x = std::strtoll(e, &end, 10);
    if (end != e && x >= 0) max_rows = x;
  }
  return static_cast<int64_t>(NV) * Hkv <= max_rows;
}

hipError_t launch_window(const AttnLaunch& L, hipStream_t st) {
  switch (L.d) {
    case 64: return launch_d<64>(L, st);
    case 128: return launch_d<128>(L, st);
    default: return launch_d<256>(L, st);
  }
}

}  // namespace wmtp
