// Split-K single-token GQA decode attention for gfx950 (full, windowed and
// ring key maps), followed by a log-sum-exp merge of the split partials.
//
// What is computed: for every sequence b and query head h, softmax attention
// of q[b,h] over the keys the variant selects (Windowed-MTP Section 4
// "Mechanism" and the Appendix A pseudocode; the native draft reads all S
// keys, Section 3).  The selection is the O(1) index arithmetic of
// index_map.h; no index table is built.
//
// Work decomposition.  Sequence b attends n_sel(b) keys, cut into work items
// of `chunk` keys; the items of all sequences are numbered consecutively (a
// prefix sum over the device-resident lengths, so variable-length batches
// pack without holes) and one 256-thread workgroup handles one (item, KV
// head).  The four waves of a workgroup take interleaved 16-key tiles, so the
// group streams one contiguous key range.
//
// Per 16-key tile, on one wave:
//   S^T[16 keys, 16 heads] = K_tile . Q^T   v_mfma_f32_16x16x32_bf16, d/32 steps
//   online softmax per head in the exp2 domain (scale * log2 e folded into the
//   fp32 logits); the head's running maximum is shared by the four lanes that
//   hold its 16 scores (two xor shuffles)
//   O^T[d, heads] += V^T . P^T              v_mfma_f32_16x16x4f32, P kept in fp32
// The orientation puts a query head on the same lane in the scores and in the
// output accumulator, so rescaling by exp2(m_old - m_new) is lane-local, and
// it lets every lane read its V operand as one contiguous run of d/16
// values of a single key (16 lanes cover one 2*d-byte row: coalesced).
// The four waves combine their (m, l, O) through LDS in a fixed order, and the
// merge kernel combines the items of a sequence in a fixed order: results are
// bitwise reproducible.
//
// Query heads beyond G in the 16-wide MFMA operand are zero and discarded.

#include "../../include/wmtp.h"
#include "common.h"
#include "index_map.h"
#include "launch.h"

#include <algorithm>
#include <cstdlib>

namespace wmtp {
namespace {

struct SplitArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* lens;
  float* pm;
  float* pl;
  float* po;
  int32_t* err;
  int B, Hq, Hkv, G;
  int64_t rows;
  int64_t len_cap;
  int W, sink, R_w;
  int chunk;
  float scale_log2;
};

struct MergeArgs {
  const int32_t* lens;
  const float* pm;
  const float* pl;
  const float* po;
  uint16_t* out;
  float* lse;
  int32_t* err;
  int B, Hq, Hkv, G;
  int64_t len_cap;
  int W, sink, chunk;
};

__device__ __forceinline__ int read_len(const int32_t* lens, int b, int64_t cap, int32_t* err,
                                        bool report) {
  int S = lens[b];
  if (S < 0 || static_cast<int64_t>(S) > cap) {
    if (report) raise_error(err, WMTP_DERR_LEN_RANGE);
    S = S < 0 ? 0 : static_cast<int>(cap);
  }
  return S;
}

// Sequence b owns ceil(n_sel(b) / chunk) consecutive work items.  Wave 0
// scans the lengths; the result is broadcast through LDS.  Returns false
// (for the whole workgroup) when `item` lies past the last sequence's items.
template <KeyMap M>
__device__ bool locate_item(const SplitArgs& a, int item, int& b_out, int& c_out, int& S_out) {
  __shared__ int s_b, s_c, s_S;
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    if (lane == 0) s_b = -1;
    int carry = 0;
    for (int base = 0; base < a.B; base += kWave) {
      const int b = base + lane;
      int S = 0, cnt = 0;
      if (b < a.B) {
        S = read_len(a.lens, b, a.len_cap, a.err, true);
        cnt = ceil_div_i(selected_count<M>(S, a.W, a.sink), a.chunk);
      }
      int incl = cnt;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int t = __shfl_up(incl, off);
        if (lane >= off) incl += t;
      }
      const int lo = carry + incl - cnt;
      if (cnt > 0 && item >= lo && item < lo + cnt) {
        s_b = b;
        s_c = item - lo;
        s_S = S;
      }
      carry += __shfl(incl, kWave - 1);
      if (carry > item) break;
    }
  }
  __syncthreads();
  b_out = s_b;
  c_out = s_c;
  S_out = s_S;
  return b_out >= 0;
}

template <int VW>
__device__ __forceinline__ void load_words(uint32_t (&dst)[VW], const uint16_t* p) {
  if constexpr (VW == 8) {
    const u32x4 x = reinterpret_cast<const u32x4*>(p)[0];
    const u32x4 y = reinterpret_cast<const u32x4*>(p)[1];
    dst[0] = x[0]; dst[1] = x[1]; dst[2] = x[2]; dst[3] = x[3];
    dst[4] = y[0]; dst[5] = y[1]; dst[6] = y[2]; dst[7] = y[3];
  } else if constexpr (VW == 4) {
    const u32x4 x = *reinterpret_cast<const u32x4*>(p);
    dst[0] = x[0]; dst[1] = x[1]; dst[2] = x[2]; dst[3] = x[3];
  } else {
    static_assert(VW == 2, "d must be 64, 128 or 256");
    const u32x2 x = *reinterpret_cast<const u32x2*>(p);
    dst[0] = x[0]; dst[1] = x[1];
  }
}

template <int D, KeyMap M>
__global__ __launch_bounds__(kThreads) void split_kernel(SplitArgs a) {
  constexpr int VEC = D / 16;  // d values of one key per lane in the PV operand
  constexpr int VW = VEC / 2;  // ... as 32-bit words
  constexpr int KCH = D / 32;  // 16x16x32 steps over d for the logits
  constexpr int OPAD = kWave + 1;

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int grp = lane >> 4;  // 0..3
  const int col = lane & 15;  // query head (within the group) owned by this lane
  const int g = blockIdx.x % a.Hkv;
  const int item = blockIdx.x / a.Hkv;

  int b, c, S;
  if (!locate_item<M>(a, item, b, c, S)) return;
  const int n_sel = selected_count<M>(S, a.W, a.sink);
  const int j0 = c * a.chunk;
  const int j1 = min(j0 + a.chunk, n_sel);
  const RowMap<M> map(S, a.W, a.sink, a.R_w);
  const int64_t rs = static_cast<int64_t>(a.Hkv) * D;  // elements between rows
  const int64_t seq_off = (static_cast<int64_t>(b) * a.rows * a.Hkv + g) * D;
  const uint16_t* kbase = a.k + seq_off;
  const uint16_t* vbase = a.v + seq_off;

  // Q^T operand: lane (grp, col) holds q[b, g*G + col, kk*32 + grp*8 .. +8].
  bf16x8 qf[KCH];
  {
    const bool live = col < a.G;
    const uint16_t* qp =
        a.q + (static_cast<int64_t>(b) * a.Hq + g * a.G + (live ? col : 0)) * D + grp * 8;
#pragma unroll
    for (int kk = 0; kk < KCH; ++kk) {
      u32x4 w = *reinterpret_cast<const u32x4*>(qp + kk * 32);
      if (!live) w = u32x4{0u, 0u, 0u, 0u};
      qf[kk] = __builtin_bit_cast(bf16x8, w);
    }
  }

  struct Tile {
    u32x4 kx[KCH];       // key (col) : d chunk kk*32 + grp*8
    uint32_t vx[4][VW];  // key 4*grp + i : d values col*VEC ..
  };

  // Keys past j1 read a valid row (j0) and are masked out of the softmax.
  auto load_tile = [&](Tile& T, int t) {
    const int jt = j0 + t * kTileKeys;
    {
      const int j = jt + col;
      const int r = map.row(j < j1 ? j : j0);
      const uint16_t* p = kbase + static_cast<int64_t>(r) * rs + grp * 8;
#pragma unroll
      for (int kk = 0; kk < KCH; ++kk) T.kx[kk] = *reinterpret_cast<const u32x4*>(p + kk * 32);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = jt + 4 * grp + i;
      const int r = map.row(j < j1 ? j : j0);
      load_words<VW>(T.vx[i], vbase + static_cast<int64_t>(r) * rs + col * VEC);
    }
  };

  floatx4 acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = neg_inf();
  float l_run = 0.f;
  const float sl2 = a.scale_log2;

  auto compute_tile = [&](const Tile& T, int t) {
    const int jt = j0 + t * kTileKeys;
    floatx4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KCH; ++kk)
      s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, T.kx[kk]), qf[kk], s,
                                                  0, 0, 0);
    // s[i] = logit of key jt + 4*grp + i for head col
    float sv[4];
    float mt = neg_inf();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = jt + 4 * grp + i;
      sv[i] = j < j1 ? s[i] * sl2 : neg_inf();
      mt = fmaxf(mt, sv[i]);
    }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    if (__any(m_new > m_run)) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] *= alpha;
    }
    m_run = m_new;
    float pv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      pv[i] = __builtin_amdgcn_exp2f(sv[i] - m_run);
      l_run += pv[i];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const uint32_t w = T.vx[i][e >> 1];
        const float vf = (e & 1) ? bf16_hi(w) : bf16_lo(w);
        acc[e] = __builtin_amdgcn_mfma_f32_16x16x4f32(vf, pv[i], acc[e], 0, 0, 0);
      }
    }
  };

  // Two register buffers: the next tile's loads are in flight while the
  // current tile is computed.
  const int n_tiles = (j1 - j0 + kTileKeys - 1) / kTileKeys;
  Tile T0, T1;
  int t = wave;
  if (t < n_tiles) load_tile(T0, t);
  while (t < n_tiles) {
    const int t1 = t + kWaves;
    if (t1 < n_tiles) load_tile(T1, t1);
    compute_tile(T0, t);
    if (t1 >= n_tiles) break;
    const int t2 = t1 + kWaves;
    if (t2 < n_tiles) load_tile(T0, t2);
    compute_tile(T1, t1);
    t = t2;
  }

  // ---- combine the four waves: (m, l) per head, then O in wave order ----
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  __shared__ float s_m[kWaves][16];
  __shared__ float s_l[kWaves][16];
  __shared__ float s_o[(D / 4) * OPAD];
  if (grp == 0) {
    s_m[wave][col] = m_run;
    s_l[wave][col] = l_run;
  }
  __syncthreads();
  float Mx = neg_inf();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) Mx = fmaxf(Mx, s_m[w][col]);
  float Lx = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) Lx += s_l[w][col] * __builtin_amdgcn_exp2f(s_m[w][col] - Mx);
  const float f = __builtin_amdgcn_exp2f(m_run - Mx);  // 0 for a wave with no tile
  for (int w = 0; w < kWaves; ++w) {
    if (wave == w) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int idx = (e * 4 + jj) * OPAD + lane;
          const float val = acc[e][jj] * f;
          s_o[idx] = (w == 0) ? val : s_o[idx] + val;
        }
      }
    }
    __syncthreads();
  }

  // Partial row of (item, g): pm/pl [G], po [G, D].  Lane l of any wave held
  // head l&15, d = VEC*(4*(l>>4) + jj) + e.
  const int64_t pidx = blockIdx.x;
  if (threadIdx.x < 16 && col < a.G) {
    a.pm[pidx * a.G + col] = Mx;
    a.pl[pidx * a.G + col] = Lx;
  }
  float* po = a.po + pidx * a.G * D;
  for (int idx = threadIdx.x; idx < a.G * D; idx += kThreads) {
    const int h = idx / D;
    const int d = idx % D;
    const int gq = d / (4 * VEC);
    const int rem = d % (4 * VEC);
    const int jj = rem / VEC;
    const int e = rem % VEC;
    po[idx] = s_o[(e * 4 + jj) * OPAD + gq * 16 + h];
  }
}

// One workgroup per (b, h, 64-wide slice of d).  Items of sequence b are
// combined in a fixed order: wave w takes items w, w+4, ...; then waves 0..3.
template <int D, KeyMap M>
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int b = blockIdx.x / a.Hq;
  const int h = blockIdx.x % a.Hq;
  const int g = h / a.G;
  const int hl = h % a.G;
  const int d = blockIdx.y * kWave + lane;

  __shared__ int s_base, s_cnt;
  __shared__ float s_red[4];
  __shared__ float s_o[4][kWave];
  __shared__ float s_L[4];
  if (threadIdx.x < kWave) {
    int before = 0, mine = 0;
    for (int base = 0; base <= b; base += kWave) {
      const int bb = base + lane;
      if (bb <= b) {
        const int S = read_len(a.lens, bb, a.len_cap, a.err, false);
        const int cnt = ceil_div_i(selected_count<M>(S, a.W, a.sink), a.chunk);
        if (bb < b) before += cnt; else mine = cnt;
      }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
      before += __shfl_xor(before, off);
      mine += __shfl_xor(mine, off);
    }
    if (lane == 0) {
      s_base = before;
      s_cnt = mine;
    }
  }
  __syncthreads();
  const int base = s_base;
  const int n = s_cnt;

  // Largest partial maximum.
  float mx = neg_inf();
  for (int c = threadIdx.x; c < n; c += 256)
    mx = fmaxf(mx, a.pm[(static_cast<int64_t>(base + c) * a.Hkv + g) * a.G + hl]);
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if (lane == 0) s_red[wave] = mx;
  __syncthreads();
  const float Mx = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));

  float o = 0.f, L = 0.f;
  for (int c = wave; c < n; c += 4) {
    const int64_t pr = (static_cast<int64_t>(base + c) * a.Hkv + g) * a.G + hl;
    const float w = __builtin_amdgcn_exp2f(a.pm[pr] - Mx);
    o += w * a.po[pr * D + d];
    L += w * a.pl[pr];
  }
  s_o[wave][lane] = o;
  if (lane == 0) s_L[wave] = L;
  __syncthreads();
  if (wave == 0) {
    const float ot = ((s_o[0][lane] + s_o[1][lane]) + s_o[2][lane]) + s_o[3][lane];
    const float Lt = ((s_L[0] + s_L[1]) + s_L[2]) + s_L[3];
    const float r = n > 0 ? ot / Lt : 0.f;
    a.out[(static_cast<int64_t>(b) * a.Hq + h) * D + d] = f32_to_bf16_rne(r);
    if (a.lse != nullptr && blockIdx.y == 0 && lane == 0)
      a.lse[static_cast<int64_t>(b) * a.Hq + h] = n > 0 ? (Mx + log2f(Lt)) * kLn2 : neg_inf();
  }
}

template <int D, KeyMap M>
hipError_t launch_typed(const AttnLaunch& L, hipStream_t st) {
  const int G = L.Hq / L.Hkv;
  if (L.max_items > 0) {
    SplitArgs a;
    a.q = L.q; a.k = L.k; a.v = L.v; a.lens = L.lens;
    a.pm = L.pm; a.pl = L.pl; a.po = L.po; a.err = L.err;
    a.B = L.B; a.Hq = L.Hq; a.Hkv = L.Hkv; a.G = G;
    a.rows = L.rows; a.len_cap = L.len_cap;
    a.W = L.W; a.sink = L.sink; a.R_w = L.R_w; a.chunk = L.chunk;
    a.scale_log2 = L.scale * kLog2e;
    const dim3 grid(static_cast<unsigned>(L.max_items) * static_cast<unsigned>(L.Hkv));
    hipLaunchKernelGGL((split_kernel<D, M>), grid, dim3(kThreads), 0, st, a);
  }
  MergeArgs m;
  m.lens = L.lens; m.pm = L.pm; m.pl = L.pl; m.po = L.po;
  m.out = L.out; m.lse = L.lse; m.err = L.err;
  m.B = L.B; m.Hq = L.Hq; m.Hkv = L.Hkv; m.G = G;
  m.len_cap = L.len_cap; m.W = L.W; m.sink = L.sink; m.chunk = L.chunk;
  const dim3 grid2(static_cast<unsigned>(L.B) * static_cast<unsigned>(L.Hq), D / kWave);
  hipLaunchKernelGGL((merge_kernel<D, M>), grid2, dim3(256), 0, st, m);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const AttnLaunch& L, hipStream_t st) {
  switch (L.variant) {
    case WMTP_VARIANT_FULL: return launch_typed<D, KeyMap::Full>(L, st);
    case WMTP_VARIANT_WINDOWED: return launch_typed<D, KeyMap::Window>(L, st);
    default: return launch_typed<D, KeyMap::Ring>(L, st);
  }
}

int env_int(const char* name, int dflt) {
  const char* s = std::getenv(name);
  if (s == nullptr || *s == '\0') return dflt;
  const int v = std::atoi(s);
  return v > 0 ? v : dflt;
}

}  // namespace

SplitPlan plan_split(int B, int Hq, int Hkv, int d, int64_t n_keys_max) {
  // Aim for about kTargetItems workgroups in total (several per CU on a
  // 256-CU part) with items of at most kChunkMax keys, so that long sequences
  // get many items and short ones still spread over the chip.
  static const int target = env_int("WMTP_TARGET_ITEMS", 1024);
  static const int chunk_max =
      std::max(kChunkQuantum, env_int("WMTP_CHUNK_MAX", 2048) / kChunkQuantum * kChunkQuantum);
  SplitPlan p{};
  const int64_t groups = std::max<int64_t>(1, static_cast<int64_t>(B) * Hkv);
  const int64_t per_seq = std::max<int64_t>(1, (target + groups - 1) / groups);
  int64_t chunk = (std::max<int64_t>(n_keys_max, 1) + per_seq - 1) / per_seq;
  chunk = (chunk + kChunkQuantum - 1) / kChunkQuantum * kChunkQuantum;
  chunk = std::min<int64_t>(std::max<int64_t>(chunk, kChunkQuantum), chunk_max);
  p.chunk = static_cast<int>(chunk);
  p.max_items = n_keys_max > 0 ? static_cast<int>(B * ((n_keys_max + chunk - 1) / chunk)) : 0;
  const size_t rows = static_cast<size_t>(p.max_items) * Hkv * (Hq / Hkv);
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  p.off_pl = up(rows * sizeof(float));
  p.off_po = p.off_pl + up(rows * sizeof(float));
  p.bytes = rows ? p.off_po + up(rows * static_cast<size_t>(d) * sizeof(float)) : 0;
  return p;
}

hipError_t launch_attention(const AttnLaunch& L, hipStream_t st) {
  switch (L.d) {
    case 64: return launch_d<64>(L, st);
    case 128: return launch_d<128>(L, st);
    default: return launch_d<256>(L, st);
  }
}

}  // namespace wmtp
