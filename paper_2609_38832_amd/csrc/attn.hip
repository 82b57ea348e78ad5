// Routed causal attention over the packed per-head subsequences, and the gated
// combine back to token order.
//
// Sec. 3.1 Eq. namoh-attention: the routed query (t, i) attends to the keys and
// values of tokens s <= t routed to the same head i.  Sec. 3.2
// Eq. namoh-head-rope: RoPE at the rank inside the head's subsequence.
// Sec. 3.2 "Efficient execution": every (batch, head) subsequence is an
// independent causal sequence; query tiles with large and small causal work
// are interleaved across compute units.
//
// Launch sequence for one call:
//   k_rope_table  cos/sin of p * base^(-2j/d), angles formed and reduced in
//                 double, stored f32 (skipped without RoPE).
//   bf16, d in {64, 128}:
//     k_pack_kv   workgroup 0 builds the work list of (segment, query block)
//                 items sorted by causal work, heaviest first (counting sort
//                 by key-tile count).  Every other workgroup gathers one
//                 64-row key tile of a segment by perm_token, applies RoPE at
//                 the key's rank while loading it, rounds to bf16 (packed
//                 row-major), and writes the values as a transposed d x 64
//                 tile (the operand layout of the P.V product).  The packed
//                 rotated keys / values are what a prefill hands to the
//                 per-head decode caches.
//     k_attn_mfma one workgroup per work item: the query block is gathered
//                 and rotated into registers once; key/value tiles stream
//                 through a ring of LDS stages; S^T = K Q^T and O^T += V^T P^T
//                 run on v_mfma_f32_32x32x16_bf16 with fp32 accumulation and
//                 an fp32 online softmax (exp2).
//   other dtype / width:
//     k_attn_schedule  the work list alone.
//     k_attn_generic  fp32 arithmetic, one lane per query, keys gathered and
//                 rotated while staging each tile.
//   k_combine     o_t = sum_k gate(t,k) * h[slot_pos(t,k)] in k order.
#include <cmath>

#include "common.h"
#include "internal.h"
#include "launch.h"
#include "sched.h"
#include "tile.h"

namespace namoh {

// MFMA kernel shape: NW waves per workgroup, NQT 32-query sub-tiles per wave,
// MINB workgroups per compute unit the register allocation must allow, NS
// key/value tile stages in LDS (NS - 1 tiles in flight while one is used),
// VPRE 16-key steps of value operands read from LDS while the softmax runs
// (the rest while the first P.V products execute; d = 128 reads half early
// to stay within 256 registers).
template <int D> struct MfmaShape;
template <> struct MfmaShape<64> {
  static constexpr int NW = 4, NQT = 1, MINB = 4, NS = 2, VPRE = 0;
};
template <> struct MfmaShape<128> {
  static constexpr int NW = 4, NQT = 1, MINB = 2, NS = 2, VPRE = 2;
};
// The running softmax maximum (log2 units) is only raised when a tile
// exceeds it by more than kLazyLog2 (probabilities then stay below
// 2^kLazyLog2 and the final normalisation is exact), so the output
// accumulator is rarely rescaled.
constexpr float kLazyLog2 = 8.f;
constexpr int kGenericBM = 64;

constexpr int kPackThreads = 256;

// ---------------------------------------------------------------------------
// RoPE table table[p * (d/2) + j] = (cos, sin)(p * base^(-2j/d)) for p < T,
// the angles formed and reduced in double.  Every position a rotation can
// use (a rank below the longest segment, or a token index) is below T, so
// the table does not wait for the routing; kTableEntries entries per thread.
constexpr int kTableThreads = 256, kTableEntries = 4;
__global__ __launch_bounds__(kTableThreads) void k_rope_table(int T, int d, double log_base,
                                                             float2* __restrict__ table) {
  __shared__ double s_theta[64];
  const int half = d / 2;
  const int tid = thread_x();
  if (tid < half) s_theta[tid] = exp(-(2.0 * tid / d) * log_base);
  __syncthreads();
  const size_t total = static_cast<size_t>(T) * half;
  const size_t i0 = static_cast<size_t>(block_x()) * kTableThreads * kTableEntries + tid;
#pragma unroll
  for (int e = 0; e < kTableEntries; ++e) {
    const size_t i = i0 + static_cast<size_t>(e) * kTableThreads;
    if (i < total) {
      const int p = static_cast<int>(i / half);
      const int j = static_cast<int>(i - static_cast<size_t>(p) * half);
      table[i] = rope_cos_sin(static_cast<double>(p) * s_theta[j]);
    }
  }
}

// The schedule on its own (paths without the packing kernel, which otherwise
// builds it in its workgroup 0).
__global__ __launch_bounds__(kPackThreads) void k_attn_schedule(
    const int32_t* __restrict__ seg_offsets, int BH, int T, int BM, int Nr, int max_items,
    int period, WorkItem* __restrict__ items, int32_t* __restrict__ meta) {
  __shared__ SchedLds L;
  attn_schedule<kPackThreads>(seg_offsets, BH, T, BM, Nr, max_items, period, 1, items, meta, L);
}

// ---------------------------------------------------------------------------

// Workgroup 0 builds the attention schedule (it only needs seg_offsets and
// runs alongside the packing); workgroup 1 + gt packs key tile gt.
template <int D>
struct PackLds {
  uint16_t sv[kBN][D + 8];
  int off[kSegLds + 1];
  float wnorm[kPackThreads / kWave];
  double freq[D / 2];
};

// theta_j / (2 pi) = base^(-2j/d) / (2 pi) for the rotation pairs j < d/2,
// in double.
NAMOH_DEV double rope_freq_rev(int j, int d, double log_base) {
  return exp(-(2.0 * j / d) * log_base) * 0.15915494309189535;
}

// Squared norm of 8 packed bf16 values.
NAMOH_DEV float sumsq8(const uint4 x) {
  float f[8];
  unpack8(x, f);
  float a = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) a = fmaf(f[e], f[e], a);
  return a;
}

template <int D>
__global__ __launch_bounds__(kPackThreads) void k_pack_kv(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, double log_base,
    double* __restrict__ freq_out, const int32_t* __restrict__ seg_offsets,
    const int32_t* __restrict__ perm_token, int BH, int T, int H, int Nr, int rope_mode,
    int BM, int max_items, int period, int G, WorkItem* __restrict__ items,
    int32_t* __restrict__ meta, uint16_t* __restrict__ Kp, uint16_t* __restrict__ Vt,
    float* __restrict__ knorm, int split_slots, SplitItem* __restrict__ splits,
    int resident_slots) {
  __shared__ __attribute__((aligned(16))) union {
    SchedLds sched;
    PackLds<D> pack;
  } L;
  if (block_x() == 0) {
    // the rotation frequencies for the attention kernel, then the schedule
    if (thread_x() < D / 2) freq_out[thread_x()] = rope_freq_rev(thread_x(), D, log_base);
    attn_schedule<kPackThreads>(seg_offsets, BH, T, BM, Nr, max_items, period, G, items, meta,
                                L.sched, split_slots, splits, resident_slots);
    return;
  }
  const int gt = block_x() - 1;
  const int tid = thread_x();
  if (rope_mode != 2 && tid < D / 2) L.pack.freq[tid] = rope_freq_rev(tid, D, log_base);
  // segment of tile gt: the last s with seg_tile0(off[s], s) <= gt
  const bool in_lds = BH <= kSegLds;
  if (in_lds)
    for (int i = tid; i <= BH; i += kPackThreads) L.pack.off[i] = seg_offsets[i];
  __syncthreads();
  const int32_t* off = in_lds ? L.pack.off : seg_offsets;
  int s;
  if (in_lds) {
    // seg_tile0(off[s], s) increases strictly with s, so the segment is the
    // number of segments whose first tile is at most gt, minus one: one
    // ballot per 64 segments (every wave computes it; no barrier)
    int cnt = 0;
    for (int s0 = 0; s0 < BH; s0 += kWave) {
      const int si = s0 + tid % kWave;
      cnt += __popcll(__ballot(si < BH && seg_tile0(off[si], si) <= gt));
    }
    s = cnt - 1;
  } else {
    int lo = 0, hi = BH;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (seg_tile0(off[mid], mid) <= gt) lo = mid; else hi = mid;
    }
    s = lo;
  }
  const int seg0 = off[s];
  const int n = off[s + 1] - seg0;
  const int r0 = (gt - seg_tile0(seg0, s)) * kBN;
  // a tile index in a gap between segments, or offsets that are not a
  // packing of [0, Nr) (the schedule is then empty): nothing to pack
  if (r0 < 0 || r0 >= n || seg0 < 0 || n > T || seg0 + n > Nr) return;
  auto& sv = L.pack.sv;
  const int b = s / H, h = s - (s / H) * H;
  const size_t head_base = (static_cast<size_t>(b) * H + h) * T;

  // Every load of the tile is issued before any of them is used: the
  // thread's rows' tokens, then its key granule pairs and value granules.
  // No load sits under a branch (a load under a branch is waited for where
  // the branch joins, which would serialise them): rows past the segment's
  // end load its last row and are zeroed after the load.
  constexpr int HP = D / 16;  // 8-element granule pairs (j, j + d/2) per key row
  constexpr int RG = D / 8;   // 16-byte granules per value row
  constexpr int KU = kBN * HP / kPackThreads, VU = kBN * RG / kPackThreads;
  static_assert(KU * kPackThreads == kBN * HP && VU * kPackThreads == kBN * RG, "units");
  static_assert(kWave % HP == 0, "a key row's units share one wave");
  auto token_of = [&](int row) {   // the segment's last row past its end
    const int r = min(r0 + row, n - 1);
    return static_cast<int>(min(static_cast<unsigned>(perm_token[seg0 + r]),
                                static_cast<unsigned>(T - 1)));
  };
  auto zero_unless = [](uint4 x, bool keep) {
    return keep ? x : make_uint4(0, 0, 0, 0);
  };
  int ktok[KU], vtok[VU];
#pragma unroll
  for (int i = 0; i < KU; ++i) ktok[i] = token_of((tid + i * kPackThreads) / HP);
#pragma unroll
  for (int i = 0; i < VU; ++i) vtok[i] = token_of((tid + i * kPackThreads) / RG);
  uint4 ka[KU], kb[KU], vx[VU];
#pragma unroll
  for (int i = 0; i < KU; ++i) {
    const int c = (tid + i * kPackThreads) % HP;
    const uint16_t* src = k + (head_base + ktok[i]) * D;
    ka[i] = *reinterpret_cast<const uint4*>(src + 8 * c);
    kb[i] = *reinterpret_cast<const uint4*>(src + D / 2 + 8 * c);
  }
#pragma unroll
  for (int i = 0; i < VU; ++i) {
    const int gr = (tid + i * kPackThreads) % RG;
    vx[i] = *reinterpret_cast<const uint4*>(v + (head_base + vtok[i]) * D + 8 * gr);
  }
#pragma unroll
  for (int i = 0; i < KU; ++i) {
    const bool in = r0 + (tid + i * kPackThreads) / HP < n;
    ka[i] = zero_unless(ka[i], in);
    kb[i] = zero_unless(kb[i], in);
  }
#pragma unroll
  for (int i = 0; i < VU; ++i) vx[i] = zero_unless(vx[i], r0 + (tid + i * kPackThreads) / RG < n);

  float rmax = 0.f;   // largest squared norm of a packed (rounded) key row seen
#pragma unroll
  for (int i = 0; i < KU; ++i) {
    const int u = tid + i * kPackThreads;
    const int row = u / HP, c = u % HP;
    uint4 o1 = ka[i], o2 = kb[i];
    if (rope_mode != 2) {   // rows past the end are zero and stay zero
      float x1[8], x2[8];
      unpack8(ka[i], x1);
      unpack8(kb[i], x2);
      const int pos = rope_mode == 0 ? r0 + row : ktok[i];
      float4 cs[4];
      rope8_rev(cs, static_cast<double>(pos), &L.pack.freq[8 * c]);
      rope8(x1, x2, cs);
      o1 = pack8(x1);
      o2 = pack8(x2);
    }
    uint16_t* dst = Kp + (static_cast<size_t>(gt) * kBN + row) * D;
    *reinterpret_cast<uint4*>(dst + 8 * c) = o1;
    *reinterpret_cast<uint4*>(dst + D / 2 + 8 * c) = o2;
    // the row's squared norm: its HP units are consecutive lanes
    float ss = sumsq8(o1) + sumsq8(o2);
    ss = group_sum<HP>(ss);
    rmax = fmaxf(rmax, ss);
  }
  // the tile's largest key norm (bounds every score of the tile, see
  // k_attn_mfma); written by the one workgroup that packs the tile
  rmax = group_max<kWave>(rmax);
  if (tid % kWave == 0) L.pack.wnorm[tid / kWave] = rmax;
#pragma unroll
  for (int i = 0; i < VU; ++i) {
    const int u = tid + i * kPackThreads;
    *reinterpret_cast<uint4*>(&sv[u / RG][8 * (u % RG)]) = vx[i];
  }
  __syncthreads();
  if (tid == 0) {
    float mx = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < kPackThreads / kWave; ++w2) mx = fmaxf(mx, L.pack.wnorm[w2]);
    knorm[gt] = sqrtf(mx);
  }
  for (int u = tid; u < D * (kBN / 8); u += kPackThreads) {
    const int m = u / (kBN / 8), pg = u - (u / (kBN / 8)) * (kBN / 8);
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = sv[vt_key_of_pos(8 * pg + 2 * e)][m];
      const uint32_t hi = sv[vt_key_of_pos(8 * pg + 2 * e + 1)][m];
      w[e] = lo | (hi << 16);
    }
    *reinterpret_cast<uint4*>(Vt + (static_cast<size_t>(gt) * D + m) * kBN + 8 * pg) =
        make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// S^T = K Q^T for one 64-key tile: 2 key sub-tiles x NQT query sub-tiles.
// All LDS operand reads of the tile are issued before the first MFMA (the
// scheduling barrier keeps them there), so LDS latency is paid once per tile
// instead of once per MFMA.
template <int D, int NQT>
NAMOH_DEV void qk_tile(f32x16 (&S)[2][NQT], const uint16_t* __restrict__ sKb,
                       const bf16x8 (&qB)[NQT][D / 16], const f32x16 (&minit)[NQT], int c,
                       int g) {
  constexpr int KS = D / 16;
  bf16x8 a[KS][2];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int row = 32 * kk + c;
      a[ks][kk] = *reinterpret_cast<const bf16x8*>(&sKb[row * D + swz<D / 8>(row, 2 * ks + g) * 8]);
    }
  // the accumulators start at -m (the query's running maximum), so the
  // scores leave the products already shifted
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
      S[kk][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0][kk], qB[qt][0], minit[qt], 0, 0, 0);
#pragma unroll
  for (int ks = 1; ks < KS; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt)
        S[kk][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks][kk], qB[qt][ks], S[kk][qt], 0, 0, 0);
}

// Mask, online softmax and O^T += V^T P^T for one 64-key tile.
//
// Scores arrive in log2 units (queries pre-scaled by scale * log2 e) and
// already shifted by the running maximum m (the accumulator start), so the
// common tile needs exp2 of the score and nothing else.  m is raised only
// when a tile's shifted maximum exceeds 2^kLazyLog2 in probability, and on
// a wave's first tile, which sets it to that tile's maximum; such a tile
// (rare) subtracts the raise from its scores, rescales O and l, and
// rebuilds the accumulator start.
// WIN: keys are visible only inside the window qr - window < key <= qr, and a
// lane's first tile with a visible key (fresh[qt]) sets its running maximum
// (without a window the item's first tile always holds key 0, visible to
// every query, and `first` plays that part for the whole wave).
template <int D, int NQT, int NW, bool WIN = false>
NAMOH_DEV void softmax_pv(f32x16 (&S)[2][NQT], f32x16 (&O)[D / 32][NQT],
                          float (&m_run)[NQT], float (&l_run)[NQT], f32x16 (&minit)[NQT],
                          bool first, bool fast, const uint16_t* __restrict__ sVb, int key0,
                          int q0, int wave, int n, int c, int g, int window = 0,
                          bool* fresh = nullptr) {
  // value operands: the first VPRE 16-key steps are read while the softmax
  // runs (all of them for d = 64; half for d = 128, to stay within 256
  // registers), the rest while the first P.V products execute
  constexpr int VPRE = MfmaShape<D>::VPRE;
  bf16x8 va[4][D / 32];
  auto vread = [&](int k2) {
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt) {
      const int row = 32 * mt + c;
      va[k2][mt] = *reinterpret_cast<const bf16x8*>(&sVb[row * kBN + swz<kBN / 8>(row, 2 * k2 + g) * 8]);
    }
  };
#pragma unroll
  for (int k2 = 0; k2 < VPRE; ++k2) vread(k2);
  // key 32kk + 8j + 4g + i of the tile is visible to query qr iff it is
  // <= min(qr, n - 1); with lim = min(qr, n - 1) - key0 - 4g the test is a
  // comparison of a constant with one per-lane value.
  if (key0 + kBN - 1 > q0 + 32 * wave || key0 + kBN > n) {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      const int qr = q0 + 32 * (qt * NW + wave) + c;
      const int lim = min(qr, n - 1) - key0 - 4 * g;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (32 * kk + 8 * j + i > lim) S[kk][qt][4 * j + i] = -INFINITY;
    }
  }
  if constexpr (WIN) {
    // the window's lower end: key >= qr - window + 1, i.e. index >= lo
    if (key0 < q0 + 32 * ((NQT - 1) * NW + wave) + 31 - window + 1) {
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt) {
        const int qr = q0 + 32 * (qt * NW + wave) + c;
        const int lo = qr - window + 1 - key0 - 4 * g;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (32 * kk + 8 * j + i < lo) S[kk][qt][4 * j + i] = -INFINITY;
      }
    }
  }
  bf16x8 pB[NQT][4];
  float alpha[NQT], delta[NQT];
  bool rescale = false;
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) alpha[qt] = 1.f;
  // fast: the tile's norm bound already keeps every score within kLazyLog2
  // of the running maximum, so the maximum is not needed
  if (!fast) {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      float mx = fmaxf(S[0][qt][0], S[0][qt][1]);
#pragma unroll
      for (int i = 2; i < 32; i += 2)
        mx = fmaxf(fmaxf(mx, S[i >> 4][qt][i & 15]), S[i >> 4][qt][(i & 15) + 1]);
      mx = pair_max32(mx);
      if constexpr (WIN) {
        // a lane with no visible key yet takes the first finite maximum (a
        // row fully masked in this tile keeps m = 0 and adds nothing)
        const bool fr = fresh[qt];
        const bool up = fr ? mx > -INFINITY : mx > kLazyLog2;
        delta[qt] = up ? mx : 0.f;
        alpha[qt] = (up && !fr) ? __builtin_amdgcn_exp2f(-mx) : 1.f;
        fresh[qt] = fr && !up;
        rescale |= up;
      } else {
        const bool up = first || mx > kLazyLog2;
        delta[qt] = up ? mx : 0.f;
        alpha[qt] = (up && !first) ? __builtin_amdgcn_exp2f(-mx) : 1.f;
        rescale |= up;
      }
    }
  } else if constexpr (WIN) {
    // the norm bound holds: m = 0 is the reference from here on
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) fresh[qt] = false;
  }
  if (!fast && __any(rescale)) {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int e = 0; e < 16; ++e) S[kk][qt][e] -= delta[qt];
      m_run[qt] += delta[qt];
#pragma unroll
      for (int e = 0; e < 16; ++e) minit[qt][e] = -m_run[qt];
    }
    if (WIN || !first) {   // (fresh lanes have alpha = 1 and O = 0)
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
          for (int e = 0; e < 16; ++e) O[mt][qt][e] *= alpha[qt];
    }
  }
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    float ls = 0.f;
#pragma unroll
    for (int k2 = 0; k2 < 4; ++k2) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pB[qt][k2][e] =
            static_cast<__bf16>(__builtin_amdgcn_exp2f(S[k2 >> 1][qt][8 * (k2 & 1) + e]));
      // row sum of the rounded probabilities: pairs times (1, 1)
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const bf16x2 pr = {pB[qt][k2][e], pB[qt][k2][e + 1]};
        ls = __builtin_amdgcn_fdot2_f32_bf16(pr, kOnes2, ls, false);
      }
    }
    l_run[qt] = l_run[qt] * alpha[qt] + ls;
  }
#pragma unroll
  for (int k2 = VPRE; k2 < 4; ++k2) vread(k2);
#pragma unroll
  for (int k2 = 0; k2 < 4; ++k2)
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt)
        O[mt][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[k2][mt], pB[qt][k2], O[mt][qt], 0, 0, 0);
}

// Part record: a 16-byte granule of a bf16 head-output row that the first
// key-range part of a split block writes in place of the row's values, in
// every granule of the row: element 0 is 0x7F81, a signalling NaN, which no
// value row holds (the attention's rows are rounded from arithmetic results,
// and arithmetic never yields a signalling NaN; the rounding of a quiet NaN
// gives a quiet NaN or a zero); elements 1-2 hold 1 + the index of the row's
// first partial row (the partial of part p is p * BM rows further on) and
// element 3 the part count P.
constexpr uint32_t kPartRecordTag = 0x7F81u;
NAMOH_DEV uint4 part_record(int first, int P) {
  const uint32_t code = static_cast<uint32_t>(first + 1);
  return make_uint4(kPartRecordTag | (code << 16), (code >> 16) | (static_cast<uint32_t>(P) << 16),
                    0u, 0u);
}
// The record's (first partial row, part count), or P = 0 for a value granule.
NAMOH_DEV void read_part_record(const uint4 u, int& first, int& P) {
  const bool rec = (u.x & 0xFFFFu) == kPartRecordTag;
  first = static_cast<int>((u.x >> 16) | ((u.y & 0xFFFFu) << 16)) - 1;
  P = rec ? static_cast<int>(u.y >> 16) : 0;
}

// ---------------------------------------------------------------------------
// bf16 MFMA flash attention over one (segment, query block) work item.
//
// (Operand order of v_mfma_f32_32x32x16_bf16: tile.h.)  The kernel computes
// the transposed scores S^T = K Q^T (keys are rows), so every lane owns one
// query and 16 of its keys per 32-key sub-tile: the softmax row reduction is
// in-lane plus one exchange with lane c ^ 32.  The probabilities leave the
// accumulators in B-operand order for O^T += V^T P^T, against the value
// tile stored transposed with the keys of each 16-key group permuted.
// WIN: sliding-window attention (keys qr - window < key <= qr); the item then
// starts at the first key tile that meets its first query's window.
template <int D, int NQT, int NW, bool HB, bool WIN = false>
__global__ __launch_bounds__(NW * 64, MfmaShape<D>::MINB) void k_attn_mfma(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ Kp,
    const uint16_t* __restrict__ Vt, const double* __restrict__ freq,
    const int32_t* __restrict__ perm_token, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ meta, const float* __restrict__ knorm, int T, int H, int G,
    int rope_mode, float scale_log2, void* __restrict__ hout, float* __restrict__ lse_out,
    int window, float* __restrict__ part_o, float* __restrict__ part_ml, int mark_parts) {
  constexpr int BM = 32 * NQT * NW;
  constexpr int KS = D / 16;  // reduction steps of S^T = K Q^T
  constexpr int MT = D / 32;  // 32-row tiles of O^T
  constexpr int NT = NW * 64;
  constexpr int KPT = kBN * D / 8 / NT;  // 16-byte granules per thread per tile
  static_assert(kBN * D / 8 % NT == 0, "tile/thread mismatch");

  constexpr int NS = MfmaShape<D>::NS;
  // two stages: each tile is published by a full vmcnt wait and a barrier
  // (partial waits are not relied on for LDS-DMA loads, see tile_dma)
  static_assert(NS == 2, "tile stages");
  __shared__ __attribute__((aligned(16))) uint16_t sK[NS][kBN * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV[NS][D * kBN];
  WorkItem it;
  if (!my_item(items, meta, it)) return;
  const int s = it.s;
  const int q0 = it.qb * BM;
  const int b = s / H, h = s - (s / H) * H;
  const int seg0 = it.seg0;
  const int n = it.n;
  const int tile0 = it.tile0;
  const int ntiles = (n + kBN - 1) / kBN;
  // key tiles of the item: the causal range, or a key-range part of it
  // (kt_lo, kt_hi) whose unnormalised partial k_attn_merge combines
  const int kt_end = WIN ? min(ntiles, (q0 + BM + kBN - 1) / kBN) : it.kt_hi;
  const int part = item_slot(it.qh);   // partial slot, -1 for a whole item
  const int tid = thread_x();
  const int wave = tid / 64, lane = tid % 64;
  const int c = lane & 31, g = lane >> 5;
  // key tiles this wave's queries see: up to its last valid row; none when
  // all its rows are padding past the segment's end
  const int wq_last = q0 + 32 * ((NQT - 1) * NW + wave) + 31;
  const int wave_tiles = q0 + 32 * wave < n ? min(wq_last, n - 1) / kBN + 1 : 0;
  // first key tile of the item and of this wave
  const int kb = WIN ? max(0, q0 - window + 1) / kBN : it.kt_lo;
  const int wave_first = WIN ? max(0, q0 + 32 * wave - window + 1) / kBN : kb;
  // query head of the item: head h of the key/value segment, or with key/value
  // groups of G query heads, head h * G + qh; its head outputs are row
  // (packed row) * G + qh
  const int qh = it.qh & ((1 << kQhBits) - 1);
  const size_t head_base = ((static_cast<size_t>(b) * H + h) * G + qh) * T;

  // token of each query row.  The tile loads below are invisible to the
  // compiler's wait counting: a count it places for the tokens would also
  // have to cover them, so the tokens are waited for before the first tile
  // load is issued.
  int qtok[NQT];
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    const int r = q0 + 32 * (qt * NW + wave) + c;
    qtok[qt] = perm_token[seg0 + (r < n ? r : n - 1)];
  }
  // largest key norm over the item's key tiles (lane-wise here, reduced
  // across the wave after the query gather); four independent loads per
  // lane per round, all issued before the wait below
  float kmax = 0.f;
  for (int i0 = kb; i0 < kt_end; i0 += 4 * kWave) {
    float kv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = i0 + j * kWave + lane;
      kv[j] = i < kt_end ? knorm[tile0 + i] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) kmax = fmaxf(kmax, kv[j]);
  }
  wait_vmcnt<0>();

  // ---- first NS - 1 key/value tiles: in flight during the query gather ---
  // (always NS - 1 loads, repeating the last tile when the item has fewer,
  // so the number of loads in flight is the same on every path; the
  // repeats land in stages the loop never reads and are complete before the
  // loop's last iteration)
  constexpr size_t TS = static_cast<size_t>(kBN) * D;   // elements per tile
  constexpr uint32_t TB = static_cast<uint32_t>(TS * 2);  // bytes per tile
  // (the buffer resource lives in scalar registers: the item's values are
  // uniform, and readfirstlane says so)
  const int tile0_s = __builtin_amdgcn_readfirstlane(tile0);
  const int kt_end_s = __builtin_amdgcn_readfirstlane(kt_end);
  const int kb_s = __builtin_amdgcn_readfirstlane(kb);
  const uint16_t* const bK = Kp + static_cast<size_t>(tile0_s) * TS;
  const uint16_t* const bV = Vt + static_cast<size_t>(tile0_s) * TS;
  const uint32_t nb = static_cast<uint32_t>(kt_end_s) * TB;   // below 2^32 (checked on the host)
  const uint32_t voffK = tile_voffset<D / 8, NT>(tid);
  const uint32_t voffV = tile_voffset<kBN / 8, NT>(tid);
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t lK = lds_address(&sK[0][0]) + wave_s * kWave * 16;
  const uint32_t lV = lds_address(&sV[0][0]) + wave_s * kWave * 16;
#pragma unroll
  for (int i = 0; i < NS - 1; ++i) {
    const uint32_t tb = static_cast<uint32_t>(min(kb_s + i, kt_end_s - 1)) * TB;
    tile_dma<KPT, NT>(bK, nb, tb, lK + i * TB, voffK);
    tile_dma<KPT, NT>(bV, nb, tb, lV + i * TB, voffV);
  }

  // ---- query block: gather, rotate, round to bf16 B operands -------------
  // (the query rows and the frequencies of the lane's rotation pairs are
  // loaded together; the frequencies are read in the no-RoPE mode too, where
  // the identity rotation replaces them)
  bf16x8 qB[NQT][KS];
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    const int r = q0 + 32 * (qt * NW + wave) + c;
    const int rr = r < n ? r : n - 1;
    const int t = min(static_cast<unsigned>(qtok[qt]), static_cast<unsigned>(T - 1));
    const uint16_t* qrow = q + (head_base + t) * D;
    const int pos = rope_mode == 0 ? rr : (rope_mode == 1 ? t : 0);
    const float qscale = r < n ? scale_log2 : 0.f;   // padding rows: zero queries
    u32x4 qa[KS / 2], qb2[KS / 2];
    double fr[KS / 2][8];
#pragma unroll
    for (int s2 = 0; s2 < KS / 2; ++s2) {
      qa[s2] = *reinterpret_cast<const u32x4*>(qrow + 16 * s2 + 8 * g);
      qb2[s2] = *reinterpret_cast<const u32x4*>(qrow + D / 2 + 16 * s2 + 8 * g);
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const double2 f2 = *reinterpret_cast<const double2*>(freq + 16 * s2 + 8 * g + e);
        fr[s2][e] = f2.x;
        fr[s2][e + 1] = f2.y;
      }
    }
#pragma unroll
    for (int s2 = 0; s2 < KS / 2; ++s2) {
      float x1[8], x2[8];
      unpack8(make_uint4(qa[s2][0], qa[s2][1], qa[s2][2], qa[s2][3]), x1);
      unpack8(make_uint4(qb2[s2][0], qb2[s2][1], qb2[s2][2], qb2[s2][3]), x2);
      float4 cs[4];
      if (rope_mode == 2) {   // identity rotation
#pragma unroll
        for (int e = 0; e < 4; ++e) cs[e] = make_float4(1.f, 0.f, 1.f, 0.f);
      } else {
        rope8_rev(cs, static_cast<double>(pos), fr[s2]);
      }
      rope8(x1, x2, cs);
#pragma unroll
      for (int e = 0; e < 8; ++e) {   // pre-scaled: scores come out in log2 units
        qB[qt][s2][e] = static_cast<__bf16>(x1[e] * qscale);
        qB[qt][s2 + KS / 2][e] = static_cast<__bf16>(x2[e] * qscale);
      }
    }
  }
  // query rows and first tiles in: no load the compiler tracks is left for
  // it to wait for inside the loop (where its wait would also cover the
  // tile loads issued since)
  wait_vmcnt<0>();
  // Norm bound of the scores.  Every (log2-unit) score of a query against
  // the item's keys is at most |q~| * max |k~| in magnitude (Cauchy-Schwarz
  // on the rounded operands; the small factor covers the fp32
  // accumulation), so while that product stays within kLazyLog2 of the
  // running maximum a tile's exact maximum is not needed.
  kmax = group_max<kWave>(kmax);
  float qn[NQT];
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    float ss = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = static_cast<float>(qB[qt][ks][e]);
        ss = fmaf(x, x, ss);
      }
    qn[qt] = sqrtf(pair_sum32(ss)) * kmax * 1.001f;
  }

  f32x16 O[MT][NQT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
      for (int e = 0; e < 16; ++e) O[mt][qt][e] = 0.f;
  float m_run[NQT], l_run[NQT];
  f32x16 minit[NQT];
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    m_run[qt] = 0.f;   // set from the first tile
    l_run[qt] = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) minit[qt][e] = 0.f;
  }

  // ---- tile loop: two-stage ring of K/V tiles, one barrier per tile -------
  // At the top of iteration kt the wave's loads of tile kt are the only ones
  // in flight: waiting for them and the barrier publish the tile.  After the
  // barrier every wave has finished tile kt - 1, so its stage receives tile
  // kt + 1.
  bool fresh[NQT];   // (WIN) no visible key seen yet by the lane's query
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) fresh[qt] = true;
  for (int kt = kb; kt < kt_end; ++kt) {
    const int st = (kt - kb) % NS;
    wait_vmcnt<0>();
    __syncthreads();
    if (kt + NS - 1 < kt_end) {
      const int nst = (kt - kb + NS - 1) % NS;
      const uint32_t tb = static_cast<uint32_t>(kt + NS - 1) * TB;
      tile_dma<KPT, NT>(bK, nb, tb, lK + nst * TB, voffK);
      tile_dma<KPT, NT>(bV, nb, tb, lV + nst * TB, voffV);
    }
    if (kt < wave_tiles && kt >= wave_first) {
      f32x16 S[2][NQT];
      qk_tile<D, NQT>(S, sK[st], qB, minit, c, g);
      bool within = true;
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt) within &= qn[qt] <= m_run[qt] + kLazyLog2;
      softmax_pv<D, NQT, NW, WIN>(S, O, m_run, l_run, minit, kt == kb, __all(within), sV[st],
                                  kt * kBN, q0, wave, n, c, g, window, fresh);
    }
  }

  // ---- epilogue: normalise and store the packed head outputs -----------
  if (!WIN && part >= 0) {
    // a key-range part: unnormalised rows O, the running maximum m (log2
    // units) and the row sum l, for k_attn_merge
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      const int ri = 32 * (qt * NW + wave) + c;   // row within the block
      const float lsum = pair_sum32(l_run[qt]);
      if (q0 + ri < n) {
        float* const orow = part_o + (static_cast<size_t>(part) * BM + ri) * D;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            *reinterpret_cast<float4*>(orow + 32 * mt + 8 * j + 4 * g) =
                make_float4(O[mt][qt][4 * j], O[mt][qt][4 * j + 1], O[mt][qt][4 * j + 2],
                            O[mt][qt][4 * j + 3]);
        if (g == 0)
          *reinterpret_cast<float2*>(part_ml + (static_cast<size_t>(part) * BM + ri) * 2) =
              make_float2(m_run[qt], lsum);
        // bf16 head outputs merged by the combine: the first part writes the
        // row as a record of where its P partials are (part_record)
        if (HB && mark_parts && kb == 0) {
          const uint4 rec = part_record(part * BM + ri, item_parts(it.qh));
          uint4* const hrow = reinterpret_cast<uint4*>(
              static_cast<uint16_t*>(hout) + (static_cast<size_t>(seg0 + q0 + ri) * G + qh) * D);
#pragma unroll
          for (int j = 0; j < D / 16; ++j) hrow[2 * j + g] = rec;
        }
      }
    }
    return;
  }
  if constexpr (HB) {
    // bf16 rows go out through LDS: the accumulator layout gives each lane 8
    // bytes of 32 different rows per store, the staged layout 16 bytes of
    // whole 128-byte lines.  The stage the loop's last barrier left unused
    // (no tile in it is read again, no DMA targets it) holds one 32-row
    // block per wave, 64 D bytes each; 16-byte granule G of row c is kept at
    // granule G ^ (c mod D/8), so the writes of a wave spread over the banks
    // and each row is still one run of D/8 granules.
    static_assert(NQT * NW <= 4, "epilogue staging: one 32-row block per wave in one stage");
    constexpr int NG = D / 8;          // 16-byte granules per output row
    constexpr int RPI = kWave / NG;    // rows per coalesced store
    const int fs = (kt_end_s - kb_s) % NS;
    uint16_t* const ho = static_cast<uint16_t*>(hout);
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      const int blk = qt * NW + wave_s;
      char* const stage =
          reinterpret_cast<char*>(blk < 2 ? &sK[fs][0] : &sV[fs][0]) + (blk & 1) * 64 * D;
      const float inv = 1.f / pair_sum32(l_run[qt]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int phys = (4 * mt + j) ^ (c % NG);
          *reinterpret_cast<uint2*>(stage + c * 2 * D + phys * 16 + 8 * g) =
              make_uint2(pack_bf16x2(O[mt][qt][4 * j] * inv, O[mt][qt][4 * j + 1] * inv),
                         pack_bf16x2(O[mt][qt][4 * j + 2] * inv, O[mt][qt][4 * j + 3] * inv));
        }
      // the wave reads back what its own lanes wrote: LDS work of one wave
      // completes in order, the fence keeps the compiler from moving the
      // reads above the writes
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      const int row0 = q0 + 32 * blk;
      const int gl = lane % NG;
#pragma unroll
      for (int i = 0; i < 32 / RPI; ++i) {
        const int rr = i * RPI + lane / NG;
        const uint4 v = *reinterpret_cast<const uint4*>(stage + rr * 2 * D + (gl ^ (rr % NG)) * 16);
        if (row0 + rr < n)
          *reinterpret_cast<uint4*>(
              ho + (static_cast<size_t>(seg0 + row0 + rr) * G + qh) * D + gl * 8) = v;
      }
    }
  } else {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt) {
      const float lsum = pair_sum32(l_run[qt]);
      const float inv = 1.f / lsum;
      const int r = q0 + 32 * (qt * NW + wave) + c;
      if (r < n) {
        // log-sum-exp of the row's scores in log2 units (the backward's
        // statistics): the probabilities were exp2(score - m_run)
        if (lse_out != nullptr && g == 0)
          lse_out[static_cast<size_t>(seg0 + r) * G + qh] = m_run[qt] + log2f(lsum);
        const size_t orow = (static_cast<size_t>(seg0 + r) * G + qh) * D;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            *reinterpret_cast<float4*>(static_cast<float*>(hout) + orow + 32 * mt + 8 * j + 4 * g) =
                make_float4(O[mt][qt][4 * j] * inv, O[mt][qt][4 * j + 1] * inv,
                            O[mt][qt][4 * j + 2] * inv, O[mt][qt][4 * j + 3] * inv);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Merge of key-range parts (see attn_schedule): every row of a split item's
// query block from its P partials (O_p unnormalised, m_p, l_p):
//   M = max over p of m_p,  h = sum_p 2^(m_p - M) O_p / sum_p 2^(m_p - M) l_p,
// written as the block's head-output row (bf16; or f32 with the row's
// log-sum-exp M + log2 of the denominator).  The work units are (split item,
// pass of RPP rows), strided over the workgroups; eight columns per thread.
// P is a template argument, so a row's 3P loads are issued together (a load
// under a branch would be waited for where the branch joins).
constexpr int kMergeThreads = 256;
template <int D, bool HB, int P>
NAMOH_DEV void merge_row(const SplitItem& si, int q0, int r, int sub,
                         const float* __restrict__ part_o, const float* __restrict__ part_ml,
                         int BM, int G, void* __restrict__ hout, float* __restrict__ lse_out) {
  float2 ml[P];
  float4 a[P][2];
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const size_t pr = static_cast<size_t>(si.base + p) * BM + r;
    ml[p] = *reinterpret_cast<const float2*>(part_ml + pr * 2);
    const float4* src = reinterpret_cast<const float4*>(part_o + pr * D + 8 * sub);
    a[p][0] = src[0];
    a[p][1] = src[1];
  }
  float M = -INFINITY;
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (ml[p].y > 0.f) M = fmaxf(M, ml[p].x);
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  float den = 0.f;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const float wgt = ml[p].y > 0.f ? __builtin_amdgcn_exp2f(ml[p].x - M) : 0.f;
    den = fmaf(wgt, ml[p].y, den);
    acc[0] = fmaf(wgt, a[p][0].x, acc[0]); acc[1] = fmaf(wgt, a[p][0].y, acc[1]);
    acc[2] = fmaf(wgt, a[p][0].z, acc[2]); acc[3] = fmaf(wgt, a[p][0].w, acc[3]);
    acc[4] = fmaf(wgt, a[p][1].x, acc[4]); acc[5] = fmaf(wgt, a[p][1].y, acc[5]);
    acc[6] = fmaf(wgt, a[p][1].z, acc[6]); acc[7] = fmaf(wgt, a[p][1].w, acc[7]);
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] *= inv;
  const size_t row = static_cast<size_t>(si.seg0 + q0 + r) * G + si.qh;
  if constexpr (HB) {
    reinterpret_cast<uint4*>(static_cast<uint16_t*>(hout) + row * D)[sub] = pack8(acc);
  } else {
    float4* dst = reinterpret_cast<float4*>(static_cast<float*>(hout) + row * D + 8 * sub);
    dst[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    dst[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    if (lse_out != nullptr && sub == 0) lse_out[row] = M + log2f(den);
  }
}

template <int D, bool HB>
__global__ __launch_bounds__(kMergeThreads) void k_attn_merge(
    const SplitItem* __restrict__ splits, const int32_t* __restrict__ meta,
    const float* __restrict__ part_o, const float* __restrict__ part_ml, int BM, int G,
    int nblocks, void* __restrict__ hout, float* __restrict__ lse_out) {
  constexpr int TPR = D / 8;                   // threads per row
  constexpr int RPP = kMergeThreads / TPR;     // rows per pass
  static_assert(kSplitMaxParts == 8, "merge_row instances");
  const int nsplit = meta[kMetaSplit];
  const int npass = (BM + RPP - 1) / RPP;
  const int tid = thread_x();
  const int sub = tid % TPR, rw = tid / TPR;
  for (int u = block_x(); u < nsplit * npass; u += nblocks) {
    const int j = u / npass;
    const int r = (u - j * npass) * RPP + rw;
    const SplitItem si = splits[j];
    const int q0 = si.qb * BM;
    if (r >= min(BM, si.n - q0)) continue;
#define NAMOH_MERGE(PP) \
  merge_row<D, HB, PP>(si, q0, r, sub, part_o, part_ml, BM, G, hout, lse_out)
    switch (si.P) {
      case 2: NAMOH_MERGE(2); break;
      case 3: NAMOH_MERGE(3); break;
      case 4: NAMOH_MERGE(4); break;
      case 5: NAMOH_MERGE(5); break;
      case 6: NAMOH_MERGE(6); break;
      case 7: NAMOH_MERGE(7); break;
      case 8: NAMOH_MERGE(8); break;
      default: break;   // (a split item has 2 .. kSplitMaxParts parts)
    }
#undef NAMOH_MERGE
  }
}

// ---------------------------------------------------------------------------
// fp32-arithmetic attention for every other dtype / head width: one lane per
// query, keys gathered by perm_token and rotated while each tile is staged.
template <int D, bool BF16>
NAMOH_DEV void load_row(const void* base, size_t row, float* out) {
  if constexpr (BF16) {
    const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + row * D);
#pragma unroll
    for (int i = 0; i < D / 8; ++i) unpack8(p[i], out + 8 * i);
  } else {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + row * D);
#pragma unroll
    for (int i = 0; i < D / 4; ++i) {
      const float4 x = p[i];
      out[4 * i] = x.x; out[4 * i + 1] = x.y; out[4 * i + 2] = x.z; out[4 * i + 3] = x.w;
    }
  }
}

template <int D>
NAMOH_DEV void rope_row(float* x, const float2* __restrict__ cs) {
#pragma unroll
  for (int j = 0; j < D / 2; ++j) {
    const float2 w = cs[j];
    const float a = x[j], bb = x[j + D / 2];
    x[j] = a * w.x - bb * w.y;
    x[j + D / 2] = bb * w.x + a * w.y;
  }
}

template <int D, bool BF16>
__global__ __launch_bounds__(64) void k_attn_generic(
    const void* __restrict__ q, const void* __restrict__ k,
    const void* __restrict__ v, const float2* __restrict__ table,
    const int32_t* __restrict__ perm_token, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ meta, int T, int H, int rope_mode, float scale,
    float* __restrict__ hout) {
  __shared__ float sK[kBN][D + 1];
  __shared__ float sV[kBN][D + 1];
  WorkItem it;
  if (!my_item(items, meta, it)) return;
  const int s = it.s;
  const int q0 = it.qb * kGenericBM;
  const int b = s / H, h = s - (s / H) * H;
  const int seg0 = it.seg0;
  const int n = it.n;
  const size_t head_base = (static_cast<size_t>(b) * H + h) * T;
  const int lane = thread_x();
  const int r = q0 + lane;

  float qv[D], acc[D], row[D];
  {
    const int rr = r < n ? r : n - 1;
    const int t = min(static_cast<unsigned>(perm_token[seg0 + rr]), static_cast<unsigned>(T - 1));
    load_row<D, BF16>(q, head_base + t, qv);
    if (rope_mode != 2)
      rope_row<D>(qv, table + static_cast<size_t>(rope_mode == 0 ? rr : t) * (D / 2));
#pragma unroll
    for (int d = 0; d < D; ++d) {
      qv[d] *= scale;
      acc[d] = 0.f;
    }
  }
  float m = -INFINITY, l = 0.f;
  const int ntiles = (n + kBN - 1) / kBN;
  const int kt_end = min(ntiles, (q0 + kGenericBM - 1) / kBN + 1);
  for (int kt = 0; kt < kt_end; ++kt) {
    const int key = kt * kBN + lane;
    if (key < n) {
      const int t = min(static_cast<unsigned>(perm_token[seg0 + key]), static_cast<unsigned>(T - 1));
      load_row<D, BF16>(k, head_base + t, row);
      if (rope_mode != 2)
        rope_row<D>(row, table + static_cast<size_t>(rope_mode == 0 ? key : t) * (D / 2));
#pragma unroll
      for (int d = 0; d < D; ++d) sK[lane][d] = row[d];
      load_row<D, BF16>(v, head_base + t, row);
#pragma unroll
      for (int d = 0; d < D; ++d) sV[lane][d] = row[d];
    }
    __syncthreads();
    const int jmax = min(min(kBN, n - kt * kBN), r - kt * kBN + 1);
    for (int j = 0; j < kBN; ++j) {
      float sc = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) sc = fmaf(qv[d], sK[j][d], sc);
      if (j < jmax) {
        const float mn = fmaxf(m, sc);
        const float corr = expf(m - mn);
        const float p = expf(sc - mn);
        l = l * corr + p;
#pragma unroll
        for (int d = 0; d < D; ++d) acc[d] = fmaf(p, sV[j][d], acc[d] * corr);
        m = mn;
      }
    }
    __syncthreads();
  }
  if (r < n) {
    const float inv = 1.f / l;
    float* orow = hout + static_cast<size_t>(seg0 + r) * D;
#pragma unroll
    for (int d = 0; d < D; d += 4)
      *reinterpret_cast<float4*>(orow + d) =
          make_float4(acc[d] * inv, acc[d + 1] * inv, acc[d + 2] * inv, acc[d + 3] * inv);
  }
}

// ---------------------------------------------------------------------------
// One thread per (token, 8 output elements).  The K slots are gathered eight
// at a time (all loads of a batch issued before their products) and summed
// in k order.  GC = 1 fixes G = 1 at compile time (no per-row division,
// whose branch would split the batch of loads).
//
// PartRows (bf16 head outputs of the forward only): the key-range parts' rows
// are merged here instead of by k_attn_merge.  The first part of a split
// block writes each of the block's head-output rows as a part record
// (part_record) instead of a value; such a row is formed from its P partials
// as k_attn_merge forms it (same operations in the same order, rounded to
// bf16) and added after the round's value rows.
struct PartRows {
  const float* part_o = nullptr;
  const float* part_ml = nullptr;
  int BM = 0;
  int rows = 0;   // partial rows in part_o / part_ml (indices are checked against it)
};

// Row of a split block from its partials (the arithmetic of merge_row with
// the part count at run time): x receives the 8 values of column group cc,
// rounded to bf16 as the merge kernel stores them.  An entry that does not
// name partial rows inside the buffers gives zeros.
NAMOH_DEV void merge_part_row(const PartRows& pr, int first, int P, int D, int cc, float* x) {
  if (P < 2 || P > kSplitMaxParts || first < 0 || first + (P - 1) * pr.BM >= pr.rows) {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = 0.f;
    return;
  }
  // the parts' (m, l) and the first two partial rows together (parts past P
  // repeat the last one and are left out), then two partial rows at a time:
  // few registers, so the combine keeps its occupancy
  auto row_of = [&](int p) { return static_cast<size_t>(first + min(p, P - 1) * pr.BM); };
  float2 ml[kSplitMaxParts];
  float4 a[2][2];
#pragma unroll
  for (int p = 0; p < kSplitMaxParts; ++p)
    ml[p] = *reinterpret_cast<const float2*>(pr.part_ml + row_of(p) * 2);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const float4* src = reinterpret_cast<const float4*>(pr.part_o + row_of(h) * D + 8 * cc);
    a[h][0] = src[0];
    a[h][1] = src[1];
  }
  float M = -INFINITY;
#pragma unroll
  for (int p = 0; p < kSplitMaxParts; ++p)
    if (p < P && ml[p].y > 0.f) M = fmaxf(M, ml[p].x);
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  float den = 0.f;
  auto add = [&](float2 m, const float4 (&v)[2]) {
    const float wgt = m.y > 0.f ? __builtin_amdgcn_exp2f(m.x - M) : 0.f;
    den = fmaf(wgt, m.y, den);
    acc[0] = fmaf(wgt, v[0].x, acc[0]); acc[1] = fmaf(wgt, v[0].y, acc[1]);
    acc[2] = fmaf(wgt, v[0].z, acc[2]); acc[3] = fmaf(wgt, v[0].w, acc[3]);
    acc[4] = fmaf(wgt, v[1].x, acc[4]); acc[5] = fmaf(wgt, v[1].y, acc[5]);
    acc[6] = fmaf(wgt, v[1].z, acc[6]); acc[7] = fmaf(wgt, v[1].w, acc[7]);
  };
  add(ml[0], a[0]);
  add(ml[1], a[1]);   // (P >= 2)
#pragma unroll 1
  for (int p0 = 2; p0 < P; p0 += 2) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float4* src = reinterpret_cast<const float4*>(pr.part_o + row_of(p0 + h) * D + 8 * cc);
      a[h][0] = src[0];
      a[h][1] = src[1];
    }
    const float2 m0 = *reinterpret_cast<const float2*>(pr.part_ml + row_of(p0) * 2);
    const float2 m1 = *reinterpret_cast<const float2*>(pr.part_ml + row_of(p0 + 1) * 2);
    add(m0, a[0]);
    if (p0 + 1 < P) add(m1, a[1]);
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] *= inv;
  unpack8(pack8(acc), x);
}

constexpr int kCombineThreads = 256;
template <bool IN_BF16, bool OUT_BF16, int GC = 0, bool MERGE = false>
__global__ __launch_bounds__(kCombineThreads) void k_combine(
    const void* __restrict__ hout, const float* __restrict__ gates,
    const int32_t* __restrict__ slot_pos, long BT, int K, int D, int Nr, int G,
    void* __restrict__ out, PartRows pr) {
  const int C = D / 8;
  const long idx = static_cast<long>(block_x()) * kCombineThreads + thread_x();
  const long tok = idx / C;
  const int cc = static_cast<int>(idx - tok * C);
  if (tok >= BT) return;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  const int32_t* sp = slot_pos + tok * K;
  const float* gp = gates + tok * K;
  // Rounds of KC rows: row v = k * G + u is head output u of selected slot k
  // (G = 1 without key/value groups), weighted by the slot's gate; first
  // their slots and gates, then all their rows in flight at once; the sum
  // runs over v in ascending order.  No load sits under a branch (a load
  // under a branch is waited for where the branch joins, which would
  // serialise the rows): indices are clamped, and rows past K * G or with a
  // slot outside the packed rows are replaced by zeros after the load.
  constexpr int KC = 8;
  if constexpr (GC == 1) G = 1;
  const int KV = K * G;
  for (int k0 = 0; k0 < KV; k0 += KC) {
    int p[KC];
    bool ok[KC];
    float gk[KC];
    float x[KC][8];
    bool rec[KC];
#pragma unroll
    for (int i = 0; i < KC; ++i) {
      const int vr = k0 + i;
      const int kk = min(GC == 1 ? vr : vr / G, K - 1);
      const int sl = sp[kk];
      const float gv = gp[kk];
      ok[i] = vr < KV && static_cast<unsigned>(sl) < static_cast<unsigned>(Nr);
      p[i] = ok[i] ? sl * G + (vr - kk * G) : 0;
      gk[i] = ok[i] ? gv : 0.f;
    }
#pragma unroll
    for (int i = 0; i < KC; ++i) {
      if constexpr (IN_BF16) {
        const uint4 u = reinterpret_cast<const uint4*>(hout)[static_cast<size_t>(p[i]) * C + cc];
        rec[i] = (u.x & 0xFFFFu) == kPartRecordTag;
        unpack8(u, x[i]);
      } else {
        rec[i] = false;
        const float4* src =
            reinterpret_cast<const float4*>(hout) + (static_cast<size_t>(p[i]) * C + cc) * 2;
        const float4 a = src[0], bb = src[1];
        x[i][0] = a.x; x[i][1] = a.y; x[i][2] = a.z; x[i][3] = a.w;
        x[i][4] = bb.x; x[i][5] = bb.y; x[i][6] = bb.z; x[i][7] = bb.w;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) x[i][e] = ok[i] ? x[i][e] : 0.f;
    }
    // value rows in order (a part record counts as zero here) ...
#pragma unroll
    for (int i = 0; i < KC; ++i)
      if (k0 + i < KV)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(gk[i], rec[i] ? 0.f : x[i][e], acc[e]);
    // ... then the rows of split blocks (rare), each formed from its
    // partials; their slot, gate and record are read again here (a loop
    // over a bit mask), so the common path keeps no registers for them
    if constexpr (MERGE) {
      unsigned mask = 0;
#pragma unroll
      for (int i = 0; i < KC; ++i) mask |= (ok[i] && rec[i] ? 1u : 0u) << i;
#pragma unroll 1
      for (; mask != 0; mask &= mask - 1) {
        const int vr = k0 + __builtin_ctz(mask);
        const int kk = min(GC == 1 ? vr : vr / G, K - 1);
        const int pv = sp[kk] * G + (vr - kk * G);   // (ok: a packed row)
        const float gv = gp[kk];
        const uint4 u = reinterpret_cast<const uint4*>(hout)[static_cast<size_t>(pv) * C + cc];
        int first, P;
        read_part_record(u, first, P);
        float xv[8];
        merge_part_row(pr, first, P, D, cc, xv);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(gv, xv[e], acc[e]);
      }
    }
  }
  if constexpr (OUT_BF16) {
    reinterpret_cast<uint4*>(out)[idx] = pack8(acc);
  } else {
    float4* dst = reinterpret_cast<float4*>(out) + idx * 2;
    dst[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    dst[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
}

// ---------------------------------------------------------------------------
static bool use_mfma(int d, int dtype) { return dtype == 1 && (d == 64 || d == 128); }

// Compute units of the current device (the period of the hardware's
// workgroup placement); 0 if the query fails, which turns the serpentine
// order off.
static int device_cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return n;
}

static int block_queries(int d, int dtype) {
  if (!use_mfma(d, dtype)) return kGenericBM;
  return d == 64 ? 32 * MfmaShape<64>::NQT * MfmaShape<64>::NW
                 : 32 * MfmaShape<128>::NQT * MfmaShape<128>::NW;
}

struct AttnWs {
  int32_t* meta;
  WorkItem* items;
  float2* table;
  uint16_t* Kp;
  uint16_t* Vt;
  float* knorm;
  double* freq;
  float* hpack;
  SplitItem* splits;   // split items, at most split_slots
  float* part_o;       // partial rows [2 split_slots][BM][d]
  float* part_ml;      // partial (m, l) [2 split_slots][BM]
  size_t bytes;
  size_t max_items, max_tiles;
  int split_slots;     // resident workgroups the fair share assumes (0: no parts)
};

// Resident workgroups of the MFMA attention on one MI355X (256 compute units
// times the workgroups each holds): the count the key-range parts' fair share
// and the workspace for them are sized with.
constexpr int kSplitCUs = 256;

// H, K: key/value heads (segments per sequence) and selected segments per
// token; G query heads per key/value head (1 without groups).
static AttnWs carve_attn(void* ws, int B, int T, int H, int K, int d, int dtype, int G = 1) {
  const size_t BH = static_cast<size_t>(B) * H;
  const size_t Nr = static_cast<size_t>(B) * T * K;
  const int BM = block_queries(d, dtype);
  AttnWs w;
  w.split_slots = !use_mfma(d, dtype)
                      ? 0
                      : kSplitCUs * (d == 64 ? MfmaShape<64>::MINB : MfmaShape<128>::MINB);
  w.max_items = (Nr / BM + BH + 1) * G + static_cast<size_t>(w.split_slots);
  w.max_tiles = Nr / kBN + BH + 1;
  Carver cv(ws);
  w.meta = cv.take<int32_t>(kMetaCount);
  w.items = cv.take<WorkItem>(w.max_items);
  w.table = cv.take<float2>(static_cast<size_t>(T) * (d / 2));
  if (use_mfma(d, dtype)) {
    w.Kp = cv.take<uint16_t>(w.max_tiles * kBN * d);
    w.Vt = cv.take<uint16_t>(w.max_tiles * kBN * d);
    w.knorm = cv.take<float>(w.max_tiles);
    w.freq = cv.take<double>(64);
  } else {
    w.Kp = w.Vt = nullptr;
    w.knorm = nullptr;
    w.freq = nullptr;
  }
  w.hpack = cv.take<float>(Nr * G * d);
  const size_t ps = 2 * static_cast<size_t>(w.split_slots);
  w.splits = cv.take<SplitItem>(static_cast<size_t>(w.split_slots));
  w.part_o = cv.take<float>(ps * BM * d);
  w.part_ml = cv.take<float>(ps * BM * 2);
  w.bytes = cv.off;
  return w;
}

size_t attn_workspace_bytes(int B, int T, int H, int K, int d, int dtype, int G) {
  return carve_attn(nullptr, B, T, H, K, d, dtype, G).bytes;
}

template <int D>
static void launch_mfma(const AttnWs& w, const void* q, const void* k, const void* v,
                        int B, int T, int H, int G, int Nr, int rope_mode, double log_base,
                        float scale_log2, const int32_t* seg_offsets, const int32_t* perm_token,
                        void* hout, bool hout_bf16, float* lse, hipStream_t st, int window = 0,
                        bool split = false, bool merge_in_combine = false) {
  constexpr int NW = MfmaShape<D>::NW, NQT = MfmaShape<D>::NQT;
  constexpr int BM = 32 * NQT * NW;
  // key-range parts only for the whole-prefix forward (the window variant and
  // the backward's work list keep whole items)
  const int slots = split && window == 0 ? w.split_slots : 0;
  launch_k("pack", k_pack_kv<D>, dim3(static_cast<unsigned>(1 + w.max_tiles)), dim3(kPackThreads),
           st, static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), log_base, w.freq,
           seg_offsets, perm_token, B * H, T, H, Nr, rope_mode, BM,
           static_cast<int>(w.max_items), device_cu_count(), G, w.items, w.meta, w.Kp, w.Vt,
           w.knorm, slots, w.splits, w.split_slots);
  const dim3 grid(static_cast<unsigned>(w.max_items)), block(NW * 64);
  const uint16_t* q16 = static_cast<const uint16_t*>(q);
  float* const nof = nullptr;
  // bf16 head outputs read only by the layer's combine: the combine merges
  // the parts' rows itself (one launch fewer)
  const int fused = slots > 0 && hout_bf16 && merge_in_combine ? 1 : 0;
  if (window > 0 && hout_bf16)
    launch_k("attn", k_attn_mfma<D, NQT, NW, true, true>, grid, block, st, q16, w.Kp, w.Vt,
             w.freq, perm_token, w.items, w.meta, w.knorm, T, H, G, rope_mode, scale_log2, hout,
             nof, window, nof, nof, 0);
  else if (window > 0)
    launch_k("attn", k_attn_mfma<D, NQT, NW, false, true>, grid, block, st, q16, w.Kp, w.Vt,
             w.freq, perm_token, w.items, w.meta, w.knorm, T, H, G, rope_mode, scale_log2, hout,
             nof, window, nof, nof, 0);
  else if (hout_bf16)
    launch_k("attn", k_attn_mfma<D, NQT, NW, true>, grid, block, st, q16, w.Kp, w.Vt, w.freq,
             perm_token, w.items, w.meta, w.knorm, T, H, G, rope_mode, scale_log2, hout, nof, 0,
             w.part_o, w.part_ml, fused);
  else
    launch_k("attn", k_attn_mfma<D, NQT, NW, false>, grid, block, st, q16, w.Kp, w.Vt, w.freq,
             perm_token, w.items, w.meta, w.knorm, T, H, G, rope_mode, scale_log2, hout, lse, 0,
             w.part_o, w.part_ml, 0);
  if (slots > 0 && !fused) {
    constexpr int kMergeBlocks = 512;   // about one (item, row pass) unit each
    if (hout_bf16)
      launch_k("merge", k_attn_merge<D, true>, dim3(kMergeBlocks), dim3(kMergeThreads), st,
               w.splits, w.meta, w.part_o, w.part_ml, BM, G, kMergeBlocks, hout, nof);
    else
      launch_k("merge", k_attn_merge<D, false>, dim3(kMergeBlocks), dim3(kMergeThreads), st,
               w.splits, w.meta, w.part_o, w.part_ml, BM, G, kMergeBlocks, hout, lse);
  }
}

template <int D, bool BF16>
static void launch_generic(const AttnWs& w, const void* q, const void* k, const void* v,
                           int T, int H, int rope_mode, float scale,
                           const int32_t* seg_offsets, const int32_t* perm_token,
                           float* hout, hipStream_t st) {
  launch_k("attn", k_attn_generic<D, BF16>, dim3(static_cast<unsigned>(w.max_items)), dim3(64),
           st, q, k, v, w.table, perm_token, w.items, w.meta, T, H, rope_mode, scale, hout);
}

hipError_t launch_attn(const void* q, const void* k, const void* v, int dtype,
                       int B, int T, int H, int K, int d, float rope_base,
                       int rope_mode, float scale, const float* gates,
                       const int32_t* seg_offsets, const int32_t* perm_token,
                       const int32_t* slot_pos, void* out, int out_dtype,
                       float* head_out, void* ws, hipStream_t st, int G) {
  const AttnWs w = carve_attn(ws, B, T, H, K, d, dtype, G);
  // Without a caller-supplied head_out, the MFMA path keeps the packed head
  // outputs in bf16 (half the traffic of the attention epilogue and of the
  // combine); the combine accumulates in fp32 either way.
  const bool hb = head_out == nullptr && use_mfma(d, dtype);
  void* hout = head_out ? static_cast<void*>(head_out) : static_cast<void*>(w.hpack);
  const int BM = block_queries(d, dtype);
  const int Nr = B * T * K;
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  // the MFMA path forms its rotation factors in the kernels; the fp32 path
  // reads them from the table
  if (rope_mode != 2 && !use_mfma(d, dtype)) {
    const size_t entries = static_cast<size_t>(T) * (d / 2);
    const size_t per_block = static_cast<size_t>(kTableThreads) * kTableEntries;
    k_rope_table<<<static_cast<unsigned>((entries + per_block - 1) / per_block), kTableThreads, 0,
                   st>>>(T, d, log_base, w.table);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (use_mfma(d, dtype)) {
    const float sl2 = scale * 1.4426950408889634f;
    const bool fuse = hb && out != nullptr;   // nobody but the combine reads the head outputs
    if (d == 64)
      launch_mfma<64>(w, q, k, v, B, T, H, G, Nr, rope_mode, log_base, sl2, seg_offsets,
                      perm_token, hout, hb, nullptr, st, 0, true, fuse);
    else
      launch_mfma<128>(w, q, k, v, B, T, H, G, Nr, rope_mode, log_base, sl2, seg_offsets,
                       perm_token, hout, hb, nullptr, st, 0, true, fuse);
  } else {
    if (G != 1) return hipErrorInvalidValue;   // key/value groups run on the MFMA path only
    k_attn_schedule<<<1, kPackThreads, 0, st>>>(seg_offsets, B * H, T, BM, Nr,
                                                static_cast<int>(w.max_items), device_cu_count(),
                                                w.items, w.meta);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const bool bf = dtype == 1;
#define NAMOH_GEN(DD)                                                                        \
  (bf ? launch_generic<DD, true>(w, q, k, v, T, H, rope_mode, scale, seg_offsets, perm_token, static_cast<float*>(hout), st) \
      : launch_generic<DD, false>(w, q, k, v, T, H, rope_mode, scale, seg_offsets, perm_token, static_cast<float*>(hout), st))
    if (d == 32) NAMOH_GEN(32);
    else if (d == 64) NAMOH_GEN(64);
    else NAMOH_GEN(128);
#undef NAMOH_GEN
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (out == nullptr) return hipSuccess;   // head outputs only
  const long BT = static_cast<long>(B) * T;
  const long threads = BT * (d / 8);
  const unsigned grid = static_cast<unsigned>((threads + kCombineThreads - 1) / kCombineThreads);
  const dim3 cg(grid), cb(kCombineThreads);
  PartRows pr;   // (hb: the forward's key-range parts, merged by the combine)
  if (hb) {
    pr.part_o = w.part_o;
    pr.part_ml = w.part_ml;
    pr.BM = BM;
    pr.rows = 2 * w.split_slots * BM;
  }
  if (hb && out_dtype == 1)
    launch_k("combine", G == 1 ? k_combine<true, true, 1, true> : k_combine<true, true, 0, true>,
             cg, cb, st, hout, gates, slot_pos, BT, K, d, Nr, G, out, pr);
  else if (hb)
    launch_k("combine", G == 1 ? k_combine<true, false, 1, true> : k_combine<true, false, 0, true>,
             cg, cb, st, hout, gates, slot_pos, BT, K, d, Nr, G, out, pr);
  else if (out_dtype == 1)
    launch_k("combine", G == 1 ? k_combine<false, true, 1> : k_combine<false, true>, cg, cb, st,
             hout, gates, slot_pos, BT, K, d, Nr, G, out, pr);
  else
    launch_k("combine", G == 1 ? k_combine<false, false, 1> : k_combine<false, false>, cg, cb,
             st, hout, gates, slot_pos, BT, K, d, Nr, G, out, pr);
  return hipGetLastError();
}

hipError_t launch_combine_f32(const float* rows, const float* gates, const int32_t* slot_pos,
                              long BT, int K, int D, int Nr, void* out, int out_dtype,
                              hipStream_t st) {
  const long threads = BT * (D / 8);
  const unsigned grid = static_cast<unsigned>((threads + kCombineThreads - 1) / kCombineThreads);
  if (out_dtype == 1)
    launch_k("combine", k_combine<false, true, 1>, dim3(grid), dim3(kCombineThreads), st, rows,
             gates, slot_pos, BT, K, D, Nr, 1, out, PartRows{});
  else
    launch_k("combine", k_combine<false, false, 1>, dim3(grid), dim3(kCombineThreads), st, rows,
             gates, slot_pos, BT, K, D, Nr, 1, out, PartRows{});
  return hipGetLastError();
}

hipError_t launch_combine_rows(const uint16_t* rows, const float* gates, const int32_t* slot_pos,
                               long BT, int K, int D, int Nr, void* out, int out_dtype,
                               hipStream_t st) {
  const long threads = BT * (D / 8);
  const unsigned grid = static_cast<unsigned>((threads + kCombineThreads - 1) / kCombineThreads);
  if (out_dtype == 1)
    k_combine<true, true, 1><<<grid, kCombineThreads, 0, st>>>(rows, gates, slot_pos, BT, K, D, Nr,
                                                              1, out, PartRows{});
  else
    k_combine<true, false, 1><<<grid, kCombineThreads, 0, st>>>(rows, gates, slot_pos, BT, K, D,
                                                               Nr, 1, out, PartRows{});
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Always-active shared heads (Sec. 4.4, shared heads for local context): every
// (sequence, shared head) is one segment holding all T tokens in order (so
// the rank is the global position), attended causally or inside a window of
// `window` tokens, and the heads' outputs are added to the layer output.
__global__ __launch_bounds__(256) void k_shared_setup(int BH, int T, int32_t* __restrict__ seg_offsets,
                                                      int32_t* __restrict__ perm_token) {
  const size_t i = static_cast<size_t>(block_x()) * 256 + thread_x();
  const size_t n = static_cast<size_t>(BH) * T;
  if (i <= static_cast<size_t>(BH)) seg_offsets[i] = static_cast<int32_t>(i * T);
  if (i < n) perm_token[i] = static_cast<int32_t>(i % T);
}

// out[b, t] = (ACC ? out[b, t] : 0) + sum over shared heads s (in order) of
// h[(b * Hs + s) * T + t]; one thread per 8 columns.
template <bool IN_BF16, bool OUT_BF16, bool ACC>
__global__ __launch_bounds__(256) void k_shared_add(const void* __restrict__ h, int B, int T,
                                                    int Hs, int D, void* __restrict__ out) {
  const int C = D / 8;
  const long idx = static_cast<long>(block_x()) * 256 + thread_x();
  const long bt = idx / C;
  const int cc = static_cast<int>(idx - bt * C);
  if (bt >= static_cast<long>(B) * T) return;
  const long b = bt / T, t = bt - b * T;
  float acc[8];
  if constexpr (ACC) {
    if constexpr (OUT_BF16) {
      unpack8(reinterpret_cast<const uint4*>(out)[idx], acc);
    } else {
      const float4* o = reinterpret_cast<const float4*>(out) + idx * 2;
      const float4 a = o[0], c = o[1];
      acc[0] = a.x; acc[1] = a.y; acc[2] = a.z; acc[3] = a.w;
      acc[4] = c.x; acc[5] = c.y; acc[6] = c.z; acc[7] = c.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  }
  for (int sh = 0; sh < Hs; ++sh) {
    const size_t row = (static_cast<size_t>(b) * Hs + sh) * T + t;
    float x[8];
    if constexpr (IN_BF16) {
      unpack8(reinterpret_cast<const uint4*>(h)[row * C + cc], x);
    } else {
      const float4* src = reinterpret_cast<const float4*>(h) + (row * C + cc) * 2;
      const float4 a = src[0], c = src[1];
      x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
      x[4] = c.x; x[5] = c.y; x[6] = c.z; x[7] = c.w;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += x[e];
  }
  if constexpr (OUT_BF16) {
    reinterpret_cast<uint4*>(out)[idx] = pack8(acc);
  } else {
    float4* dst = reinterpret_cast<float4*>(out) + idx * 2;
    dst[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    dst[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
}

struct SharedWs {
  AttnWs attn;
  int32_t* seg_offsets;
  int32_t* perm_token;
  size_t bytes;
};

static SharedWs carve_shared(void* ws, int B, int T, int Hs, int d) {
  SharedWs w;
  // every token is a row of every shared head: H = K = Hs
  w.attn = carve_attn(ws, B, T, Hs, Hs, d, 1);
  Carver cv(ws == nullptr ? nullptr : static_cast<char*>(ws) + w.attn.bytes);
  w.seg_offsets = cv.take<int32_t>(static_cast<size_t>(B) * Hs + 1);
  w.perm_token = cv.take<int32_t>(static_cast<size_t>(B) * Hs * T);
  w.bytes = w.attn.bytes + cv.off;
  return w;
}

size_t shared_workspace_bytes(int B, int T, int Hs, int d) {
  return carve_shared(nullptr, B, T, Hs, d).bytes;
}

hipError_t launch_shared(const void* q, const void* k, const void* v, int B, int T, int Hs, int d,
                         int window, float rope_base, int rope_mode, float scale, void* out,
                         int out_dtype, int accumulate, float* head_out, void* ws,
                         hipStream_t st) {
  const SharedWs w = carve_shared(ws, B, T, Hs, d);
  const int BH = B * Hs;
  const int Nr = B * T * Hs;
  const size_t n = static_cast<size_t>(BH) * T + 1;
  k_shared_setup<<<static_cast<unsigned>((n + 255) / 256), 256, 0, st>>>(BH, T, w.seg_offsets,
                                                                         w.perm_token);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const bool hb = head_out == nullptr;
  void* hout = hb ? static_cast<void*>(w.attn.hpack) : static_cast<void*>(head_out);
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  const float sl2 = scale * 1.4426950408889634f;
  // a window at least T long is the full causal prefix
  const int win = window >= T ? 0 : window;
  if (d == 64)
    launch_mfma<64>(w.attn, q, k, v, B, T, Hs, 1, Nr, rope_mode, log_base, sl2, w.seg_offsets,
                    w.perm_token, hout, hb, nullptr, st, win);
  else
    launch_mfma<128>(w.attn, q, k, v, B, T, Hs, 1, Nr, rope_mode, log_base, sl2, w.seg_offsets,
                     w.perm_token, hout, hb, nullptr, st, win);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (out == nullptr) return hipSuccess;
  const long threads = static_cast<long>(B) * T * (d / 8);
  const unsigned grid = static_cast<unsigned>((threads + 255) / 256);
#define NAMOH_SADD(IB, OB, AC) \
  k_shared_add<IB, OB, AC><<<grid, 256, 0, st>>>(hout, B, T, Hs, d, out)
  const bool ob = out_dtype == 1;
  if (hb) {
    if (ob) { if (accumulate) NAMOH_SADD(true, true, true); else NAMOH_SADD(true, true, false); }
    else { if (accumulate) NAMOH_SADD(true, false, true); else NAMOH_SADD(true, false, false); }
  } else {
    if (ob) { if (accumulate) NAMOH_SADD(false, true, true); else NAMOH_SADD(false, true, false); }
    else { if (accumulate) NAMOH_SADD(false, false, true); else NAMOH_SADD(false, false, false); }
  }
#undef NAMOH_SADD
  return hipGetLastError();
}

// The forward for the backward (bf16, d = 64 or 128): RoPE table, packed
// rotated key tiles and transposed value tiles, the work list, the f32
// packed head outputs and the per-row log-sum-exp in log2 units of the
// scores scaled by scale * log2 e.  The workspace is laid out as for
// launch_attn; `tiles` receives where each piece lives.
void attn_stats_tiles(void* ws, int B, int T, int H, int K, int d, AttnTiles& tiles) {
  const AttnWs w = carve_attn(ws, B, T, H, K, d, 1);
  tiles.Kp = w.Kp;
  tiles.Vt = w.Vt;
  tiles.freq = w.freq;
  tiles.items = w.items;
  tiles.meta = w.meta;
  tiles.splits = w.splits;
  tiles.part = w.part_o;
  tiles.h = w.hpack;
  tiles.max_items = static_cast<int>(w.max_items);
  tiles.max_tiles = static_cast<int>(w.max_tiles);
  tiles.BM = block_queries(d, 1);
  tiles.part_rows = 2 * w.split_slots * tiles.BM;
}

hipError_t launch_attn_stats(const void* q, const void* k, const void* v, int B, int T, int H,
                             int K, int d, float rope_base, int rope_mode, float scale,
                             const int32_t* seg_offsets, const int32_t* perm_token, float* lse,
                             void* ws, AttnTiles& tiles, hipStream_t st) {
  const AttnWs w = carve_attn(ws, B, T, H, K, d, 1);
  const int Nr = B * T * K;
  // (the backward rotates with the forward's frequencies, no table)
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  const float sl2 = scale * 1.4426950408889634f;
  // key-range parts as in the inference forward (the backward's query side
  // runs the same parts; the key side takes each split block once)
  if (d == 64)
    launch_mfma<64>(w, q, k, v, B, T, H, 1, Nr, rope_mode, log_base, sl2, seg_offsets,
                    perm_token, w.hpack, false, lse, st, 0, true);
  else
    launch_mfma<128>(w, q, k, v, B, T, H, 1, Nr, rope_mode, log_base, sl2, seg_offsets,
                     perm_token, w.hpack, false, lse, st, 0, true);
  attn_stats_tiles(ws, B, T, H, K, d, tiles);
  return hipGetLastError();
}

}  // namespace namoh
