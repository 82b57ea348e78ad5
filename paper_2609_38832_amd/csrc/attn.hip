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
//   k_attn_prep   workgroup 0: per segment key-tile counts and their running
//                 sum (tile_off), and the work list of (segment, query block)
//                 items: split over the 8 XCDs in segment order by causal
//                 work, heaviest first inside each XCD (counting sort by
//                 key-tile count).  Other workgroups: the RoPE table,
//                 cos/sin of p * base^(-2j/d) from double angles, stored f32.
//   bf16, d in {64, 128}:
//     k_pack_kv   gathers each 64-row key tile of a segment by perm_token,
//                 applies RoPE at the key's rank while loading it, rounds to
//                 bf16 (packed row-major), and writes the values as a
//                 transposed d x 64 tile (the operand layout of the P.V
//                 product).  The packed rotated keys / values are what a
//                 prefill hands to the per-head decode caches.
//     k_attn_mfma one workgroup per work item: the query block is gathered
//                 and rotated into registers once; key/value tiles are
//                 double-buffered through LDS; S^T = K Q^T and O^T += V^T P^T
//                 run on v_mfma_f32_32x32x16_bf16 with fp32 accumulation and
//                 an fp32 online softmax (exp2).
//   other dtype / width:
//     k_attn_generic  fp32 arithmetic, one lane per query, keys gathered and
//                 rotated while staging each tile.
//   k_combine     o_t = sum_k gate(t,k) * h[slot_pos(t,k)] in k order.
#include <cmath>

#include "common.h"
#include "internal.h"

namespace namoh {

constexpr int kBN = 64;            // keys per tile
constexpr int kPrepThreads = 1024;

// mfma kernel shape: waves per workgroup and 32-query sub-tiles per wave
#ifndef NAMOH_D64_NW
#define NAMOH_D64_NW 4
#endif
#ifndef NAMOH_D64_NQT
#define NAMOH_D64_NQT 1
#endif
#ifndef NAMOH_D128_NW
#define NAMOH_D128_NW 4
#endif
#ifndef NAMOH_D128_NQT
#define NAMOH_D128_NQT 1
#endif
#ifndef NAMOH_D64_MINB
#define NAMOH_D64_MINB 2
#endif
#ifndef NAMOH_D128_MINB
#define NAMOH_D128_MINB 2
#endif
// NW waves per workgroup, NQT 32-query sub-tiles per wave, MINB workgroups
// per compute unit the register allocation must allow.
template <int D> struct MfmaShape;
template <> struct MfmaShape<64> {
  static constexpr int NW = NAMOH_D64_NW, NQT = NAMOH_D64_NQT, MINB = NAMOH_D64_MINB;
};
template <> struct MfmaShape<128> {
  static constexpr int NW = NAMOH_D128_NW, NQT = NAMOH_D128_NQT, MINB = NAMOH_D128_MINB;
};
#ifndef NAMOH_ATTN_PIPE
#define NAMOH_ATTN_PIPE 0
#endif
// The running softmax maximum is only raised when a tile exceeds it by more
// than 2^kLazyLog2 (probabilities then stay below 2^kLazyLog2 and the final
// normalisation is exact), so the output accumulator is rarely rescaled.
constexpr float kLazyLog2 = 8.f;
constexpr int kGenericBM = 64;

// Work items are (segment, query block).  They are split over the 8 XCDs
// (each with its own L2): items are laid out in segment order, and an item
// goes to XCD floor(8 * work before it / total work), so every XCD gets an
// eighth of the causal work and a segment's key/value tiles stay in one L2
// (a segment spans two XCDs only at a split point).  Inside an XCD the items
// run heaviest first (longest-processing-time order).  Workgroup i runs item
// rank i / 8 of XCD i % 8, matching the round-robin order in which the
// hardware hands workgroups to XCDs.
constexpr int kXcd = 8;
constexpr int kXcdBins = 1024;     // work keys per XCD, clamped to this many
enum Meta {
  kMetaItems = 0, kMetaTiles = 1, kMetaTablePos = 2, kMetaBad = 3, kMetaStride = 4,
  kMetaXcd = 8, kMetaCount = 16
};

// ---------------------------------------------------------------------------
NAMOH_DEV void attn_schedule(
    const int32_t* __restrict__ seg_offsets, int BH, int T, int BM,
    int rope_mode, int Nr, int max_items, int32_t* __restrict__ tile_off,
    long long* __restrict__ work_off, int2* __restrict__ items,
    int32_t* __restrict__ meta) {
  __shared__ int s_hist[kXcd * kXcdBins];
  __shared__ int s_wave[kPrepThreads / kWave + 1];
  __shared__ int s_xbase[kXcd + 1];
  __shared__ int s_maxn;
  __shared__ int s_bad;
  __shared__ long long s_lwave[kPrepThreads / kWave + 1];
  const int tid = threadIdx.x;
  const int per_qb = BM / kBN;           // key tiles added per query block
  for (int i = tid; i < kXcd * kXcdBins; i += kPrepThreads) s_hist[i] = 0;
  if (tid == 0) {
    s_maxn = 0;
    s_bad = seg_offsets[0] != 0 || seg_offsets[BH] != Nr;
  }
  __syncthreads();
  // offsets that are not a valid packing of Nr rows disable the call: every
  // later kernel then sees zero items and zero tiles.
  for (int s = tid; s < BH; s += kPrepThreads)
    if (seg_offsets[s + 1] < seg_offsets[s] || seg_offsets[s + 1] - seg_offsets[s] > T) s_bad = 1;
  __syncthreads();
  if (s_bad) {
    if (tid == 0) {
      meta[kMetaItems] = 0;
      meta[kMetaTiles] = 0;
      meta[kMetaTablePos] = 0;
      meta[kMetaBad] = 1;
      meta[kMetaStride] = max_items;
      for (int x = 0; x < kXcd; ++x) meta[kMetaXcd + x] = 0;
    }
    return;
  }

  // pass 1: key-tile running sum (tile_off), longest segment, work running
  // sum over segments (work_off)
  int carry = 0;
  long long wcarry = 0;
  for (int start = 0; start < BH; start += kPrepThreads) {
    const int s = start + tid;
    const int n = s < BH ? seg_offsets[s + 1] - seg_offsets[s] : 0;
    const int tiles = (n + kBN - 1) / kBN;
    if (n > 0) atomicMax(&s_maxn, n);
    const int nqb = (n + BM - 1) / BM;
    long long wsum = 0;
    for (int qb = 0; qb < nqb; ++qb) wsum += min(tiles, (qb + 1) * per_qb);
    int total;
    const int ex = block_exclusive_scan<kPrepThreads>(tiles, s_wave, total);
    // 64-bit exclusive scan of the segment work (wave scans + one wave)
    long long incl = wsum;
    const int lane = tid % kWave, wave = tid / kWave;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const long long y = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += y;
    }
    if (lane == kWave - 1) s_lwave[wave] = incl;
    __syncthreads();
    if (tid == 0) {
      long long acc = 0;
      for (int w = 0; w < kPrepThreads / kWave; ++w) {
        const long long v = s_lwave[w];
        s_lwave[w] = acc;
        acc += v;
      }
      s_lwave[kPrepThreads / kWave] = acc;
    }
    __syncthreads();
    if (s < BH) {
      tile_off[s] = carry + ex;
      work_off[s] = wcarry + s_lwave[wave] + incl - wsum;
    }
    carry += total;
    wcarry += s_lwave[kPrepThreads / kWave];
    __syncthreads();
  }
  const long long wtotal = wcarry > 0 ? wcarry : 1;
  if (tid == 0) {
    tile_off[BH] = carry;
    meta[kMetaBad] = 0;
    meta[kMetaTiles] = carry;
    meta[kMetaTablePos] = rope_mode == 0 ? s_maxn : (rope_mode == 1 ? T : 0);
    meta[kMetaStride] = max_items;
  }
  __syncthreads();
  // pass 2: histogram of item work per XCD
  for (int s = tid; s < BH; s += kPrepThreads) {
    const int n = seg_offsets[s + 1] - seg_offsets[s];
    const int tiles = (n + kBN - 1) / kBN;
    const int nqb = (n + BM - 1) / BM;
    long long before = work_off[s];
    for (int qb = 0; qb < nqb; ++qb) {
      const int w = min(tiles, (qb + 1) * per_qb);
      const int x = static_cast<int>(min(static_cast<long long>(kXcd - 1), before * kXcd / wtotal));
      atomicAdd(&s_hist[x * kXcdBins + kXcdBins - 1 - min(w, kXcdBins - 1)], 1);
      before += w;
    }
  }
  __syncthreads();
  // per-XCD exclusive scans of the histograms (heaviest bin first)
  constexpr int PER = kXcd * kXcdBins / kPrepThreads;
  constexpr int TPX = kPrepThreads / kXcd;   // threads per XCD
  int h[PER];
  int sum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    h[i] = s_hist[tid * PER + i];
    sum += h[i];
  }
  int total;
  int run = block_exclusive_scan<kPrepThreads>(sum, s_wave, total);
  if (tid % TPX == 0) s_xbase[tid / TPX] = run;
  if (tid == 0) s_xbase[kXcd] = total;
  __syncthreads();
  run -= s_xbase[tid / TPX];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    s_hist[tid * PER + i] = run;
    run += h[i];
  }
  if (tid < kXcd) meta[kMetaXcd + tid] = min(s_xbase[tid + 1] - s_xbase[tid], max_items);
  if (tid == 0) meta[kMetaItems] = total;
  __syncthreads();
  // pass 3: place the items
  for (int s = tid; s < BH; s += kPrepThreads) {
    const int n = seg_offsets[s + 1] - seg_offsets[s];
    const int tiles = (n + kBN - 1) / kBN;
    const int nqb = (n + BM - 1) / BM;
    long long before = work_off[s];
    for (int qb = 0; qb < nqb; ++qb) {
      const int w = min(tiles, (qb + 1) * per_qb);
      const int x = static_cast<int>(min(static_cast<long long>(kXcd - 1), before * kXcd / wtotal));
      const int pos = atomicAdd(&s_hist[x * kXcdBins + kXcdBins - 1 - min(w, kXcdBins - 1)], 1);
      if (pos < max_items) items[static_cast<size_t>(x) * max_items + pos] = make_int2(s, qb);
      before += w;
    }
  }
}

// Work item of this workgroup, or false if it has none.
NAMOH_DEV bool my_item(const int2* __restrict__ items, const int32_t* __restrict__ meta,
                       int2& it) {
  const int x = blockIdx.x % kXcd;
  const int rank = blockIdx.x / kXcd;
  if (rank >= meta[kMetaXcd + x]) return false;
  it = items[static_cast<size_t>(x) * meta[kMetaStride] + rank];
  return true;
}

// ---------------------------------------------------------------------------
// Workgroup 0 builds the schedule (above); workgroups 1.. fill the RoPE table
// table[p * (d/2) + j] = (cos, sin)(p * base^(-2j/d)) for p < P, with angles
// in double.  P (longest segment for head-relative positions, T for global
// ones) is recomputed by each table workgroup from seg_offsets.
__global__ __launch_bounds__(kPrepThreads) void k_attn_prep(
    const int32_t* __restrict__ seg_offsets, int BH, int T, int BM,
    int rope_mode, int Nr, int max_items, int d, double log_base,
    int32_t* __restrict__ tile_off, long long* __restrict__ work_off,
    int2* __restrict__ items, int32_t* __restrict__ meta, float2* __restrict__ table) {
  if (blockIdx.x == 0) {
    attn_schedule(seg_offsets, BH, T, BM, rope_mode, Nr, max_items, tile_off, work_off, items,
                  meta);
    return;
  }
  if (rope_mode == 2) return;
  __shared__ int s_p;
  int P = T;
  if (rope_mode == 0) {
    if (threadIdx.x == 0) s_p = 0;
    __syncthreads();
    int mx = 0;
    for (int s = threadIdx.x; s < BH; s += kPrepThreads)
      mx = max(mx, min(seg_offsets[s + 1] - seg_offsets[s], T));
    atomicMax(&s_p, mx);
    __syncthreads();
    P = s_p;
  }
  const int half = d / 2;
  const size_t total = static_cast<size_t>(P) * half;
  const size_t stride = static_cast<size_t>(gridDim.x - 1) * kPrepThreads;
  for (size_t i = static_cast<size_t>(blockIdx.x - 1) * kPrepThreads + threadIdx.x; i < total;
       i += stride) {
    const int p = static_cast<int>(i / half);
    const int j = static_cast<int>(i - static_cast<size_t>(p) * half);
    const double theta = exp(-(2.0 * j / d) * log_base);
    double sn, cs;
    sincos(static_cast<double>(p) * theta, &sn, &cs);
    table[i] = make_float2(static_cast<float>(cs), static_cast<float>(sn));
  }
}

// ---------------------------------------------------------------------------
NAMOH_DEV int find_segment(const int32_t* __restrict__ tile_off, int BH, int gt) {
  int lo = 0, hi = BH;  // tile_off[lo] <= gt < tile_off[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tile_off[mid] <= gt) lo = mid; else hi = mid;
  }
  return lo;
}

NAMOH_DEV void unpack8(const uint4 x, float* f) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = lo_bf16(w[e]);
    f[2 * e + 1] = hi_bf16(w[e]);
  }
}

// Combine x of lanes l and l ^ 32 (v_permlane32_swap hands every lane both
// values; max and sum are symmetric, so the order of the pair is irrelevant).
NAMOH_DEV float pair_max32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
NAMOH_DEV float pair_sum32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

NAMOH_DEV uint4 pack8(const float* f) {
  return make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]),
                    pack_bf16x2(f[4], f[5]), pack_bf16x2(f[6], f[7]));
}

// Rotate the pair (x1[e], x2[e]) = (elements j, j + d/2) for 8 consecutive j
// starting at j0, with cs = table row of the position.
NAMOH_DEV void rope8(float* x1, float* x2, const float2* __restrict__ cs) {
  const float4* c4 = reinterpret_cast<const float4*>(cs);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float4 w = c4[e];  // (cos, sin) of j0+2e, then of j0+2e+1
    const float a0 = x1[2 * e], b0 = x2[2 * e];
    const float a1 = x1[2 * e + 1], b1 = x2[2 * e + 1];
    x1[2 * e] = a0 * w.x - b0 * w.y;
    x2[2 * e] = b0 * w.x + a0 * w.y;
    x1[2 * e + 1] = a1 * w.z - b1 * w.w;
    x2[2 * e + 1] = b1 * w.z + a1 * w.w;
  }
}

// Position of key `p16` within a 16-key group of the transposed value tile:
// bits 2 and 3 swapped (see k_attn_mfma, P.V operand order).
NAMOH_DEV int vt_key_of_pos(int p) {
  return (p & ~12) | ((p & 4) << 1) | ((p & 8) >> 1);
}

template <int D>
__global__ __launch_bounds__(256) void k_pack_kv(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const float2* __restrict__ table, const int32_t* __restrict__ seg_offsets,
    const int32_t* __restrict__ tile_off, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ meta, int BH, int T, int H, int rope_mode,
    uint16_t* __restrict__ Kp, uint16_t* __restrict__ Vt) {
  __shared__ __attribute__((aligned(16))) uint16_t sv[kBN][D + 8];
  const int gt = blockIdx.x;
  if (gt >= meta[kMetaTiles]) return;
  const int s = find_segment(tile_off, BH, gt);
  const int r0 = (gt - tile_off[s]) * kBN;
  const int b = s / H, h = s - (s / H) * H;
  const int seg0 = seg_offsets[s];
  const int n = seg_offsets[s + 1] - seg0;
  const size_t head_base = (static_cast<size_t>(b) * H + h) * T;
  const int tid = threadIdx.x;

  constexpr int HP = D / 16;  // 8-element granule pairs (j, j + d/2) per row
  for (int u = tid; u < kBN * HP; u += 256) {
    const int row = u / HP, c = u - (u / HP) * HP;
    const int r = r0 + row;
    float x1[8], x2[8];
    uint4 o1 = make_uint4(0, 0, 0, 0), o2 = o1;
    if (r < n) {
      const int t = min(static_cast<unsigned>(perm_token[seg0 + r]), static_cast<unsigned>(T - 1));
      const uint16_t* src = k + (head_base + t) * D;
      const uint4 a = *reinterpret_cast<const uint4*>(src + 8 * c);
      const uint4 bb = *reinterpret_cast<const uint4*>(src + D / 2 + 8 * c);
      if (rope_mode != 2) {
        unpack8(a, x1);
        unpack8(bb, x2);
        const int pos = rope_mode == 0 ? r : t;
        rope8(x1, x2, table + static_cast<size_t>(pos) * (D / 2) + 8 * c);
        o1 = pack8(x1);
        o2 = pack8(x2);
      } else {
        o1 = a;
        o2 = bb;
      }
    }
    uint16_t* dst = Kp + (static_cast<size_t>(gt) * kBN + row) * D;
    *reinterpret_cast<uint4*>(dst + 8 * c) = o1;
    *reinterpret_cast<uint4*>(dst + D / 2 + 8 * c) = o2;
  }
  constexpr int RG = D / 8;  // granules per value row
  for (int u = tid; u < kBN * RG; u += 256) {
    const int row = u / RG, gr = u - (u / RG) * RG;
    const int r = r0 + row;
    uint4 x = make_uint4(0, 0, 0, 0);
    if (r < n) {
      const int t = min(static_cast<unsigned>(perm_token[seg0 + r]), static_cast<unsigned>(T - 1));
      x = *reinterpret_cast<const uint4*>(v + (head_base + t) * D + 8 * gr);
    }
    *reinterpret_cast<uint4*>(&sv[row][8 * gr]) = x;
  }
  __syncthreads();
  for (int u = tid; u < D * (kBN / 8); u += 256) {
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

// LDS granule swizzle.  gfx950 LDS serves 256 bytes (64 banks) per clock,
// i.e. 16 lanes of a 16-byte read at once; the operand reads below have 16
// consecutive lanes read the same logical 16-byte granule of 16 consecutive
// rows.  XOR-ing the granule index with row bits makes those 16 reads cover
// all 64 banks: rows of 16 granules (256 B) use row & 15; rows of 8 granules
// (128 B, two rows per bank sweep) use (row >> 1) & 7.
template <int GPR>
NAMOH_DEV int swz(int row, int gr) {
  static_assert(GPR == 8 || GPR == 16, "granules per row");
  return GPR == 16 ? (gr ^ (row & 15)) : (gr ^ ((row >> 1) & 7));
}

// Tile staging: KPT 16-byte granules per thread of one packed key tile or
// one transposed value tile (contiguous in HBM) into registers, then into
// swizzled LDS.
template <int KPT, int NT>
NAMOH_DEV void tile_gload(const uint16_t* __restrict__ tile, int tid, u32x4 (&reg)[KPT]) {
  const u32x4* p = reinterpret_cast<const u32x4*>(tile);
#pragma unroll
  for (int i = 0; i < KPT; ++i) reg[i] = p[tid + i * NT];
}

// key tile: kBN rows of D elements
template <int D, int KPT, int NT>
NAMOH_DEV void tile_lstore_k(uint16_t* sKb, int tid, const u32x4 (&reg)[KPT]) {
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int u = tid + i * NT;
    const int row = u / (D / 8), gr = u % (D / 8);
    *reinterpret_cast<u32x4*>(&sKb[row * D + swz<D / 8>(row, gr) * 8]) = reg[i];
  }
}

// transposed value tile: D rows of kBN keys
template <int D, int KPT, int NT>
NAMOH_DEV void tile_lstore_v(uint16_t* sVb, int tid, const u32x4 (&reg)[KPT]) {
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int u = tid + i * NT;
    const int m = u / (kBN / 8), gv = u % (kBN / 8);
    *reinterpret_cast<u32x4*>(&sVb[m * kBN + swz<kBN / 8>(m, gv) * 8]) = reg[i];
  }
}

// Direct global -> LDS staging (global_load_lds_dwordx4): lane l of a wave
// instruction writes LDS granule base + l, so the swizzle is applied on the
// global side: the lane that fills physical granule P = row * GPR + phys
// fetches logical granule swz(row, phys) of that row (the XOR is its own
// inverse).  Completion is tracked by vmcnt: wait_tile_dma() before the
// barrier that publishes the tile.
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

template <int GPR, int KPT, int NT>
NAMOH_DEV void tile_dma(const uint16_t* __restrict__ tile, uint16_t* lds_tile, int tid) {
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const int P = tid + i * NT;                 // physical granule of this lane
    const int row = P / GPR, phys = P % GPR;
    const int gr = swz<GPR>(row, phys);
    const uint16_t* src = tile + (row * GPR + gr) * 8;
    uint16_t* dst = lds_tile + (P - (tid & 63)) * 8;   // wave-uniform base
    __builtin_amdgcn_global_load_lds((glb_void_t*)(src), (lds_void_t*)(dst), 16, 0, 0);
  }
}

NAMOH_DEV void wait_tile_dma() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// S^T = K Q^T for one 64-key tile: 2 key sub-tiles x NQT query sub-tiles.
// All LDS operand reads of the tile are issued before the first MFMA (the
// scheduling barrier keeps them there), so LDS latency is paid once per tile
// instead of once per MFMA.
template <int D, int NQT>
NAMOH_DEV void qk_tile(f32x16 (&S)[2][NQT], const uint16_t* __restrict__ sKb,
                       const bf16x8 (&qB)[NQT][D / 16], int c, int g) {
  constexpr int KS = D / 16;
  bf16x8 a[KS][2];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int row = 32 * kk + c;
      a[ks][kk] = *reinterpret_cast<const bf16x8*>(&sKb[row * D + swz<D / 8>(row, 2 * ks + g) * 8]);
    }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
      for (int e = 0; e < 16; ++e) S[kk][qt][e] = 0.f;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt)
        S[kk][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks][kk], qB[qt][ks], S[kk][qt], 0, 0, 0);
}

// Pieces of one tile's work for the software-pipelined loop.
template <int D>
NAMOH_DEV void qk_reads(bf16x8 (&a)[D / 16][2], const uint16_t* __restrict__ sKb, int c, int g) {
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int row = 32 * kk + c;
      a[ks][kk] = *reinterpret_cast<const bf16x8*>(&sKb[row * D + swz<D / 8>(row, 2 * ks + g) * 8]);
    }
}

template <int D, int NQT>
NAMOH_DEV void qk_mfma(f32x16 (&S)[2][NQT], const bf16x8 (&a)[D / 16][2],
                       const bf16x8 (&qB)[NQT][D / 16]) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
      for (int e = 0; e < 16; ++e) S[kk][qt][e] = 0.f;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt)
        S[kk][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks][kk], qB[qt][ks], S[kk][qt], 0, 0, 0);
}

template <int D>
NAMOH_DEV void v_reads(bf16x8 (&va)[4][D / 32], const uint16_t* __restrict__ sVb, int c, int g) {
#pragma unroll
  for (int k2 = 0; k2 < 4; ++k2)
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt) {
      const int row = 32 * mt + c;
      va[k2][mt] = *reinterpret_cast<const bf16x8*>(&sVb[row * kBN + swz<kBN / 8>(row, 2 * k2 + g) * 8]);
    }
}

// Probabilities of one unmasked tile (branch-free VALU work).
template <int NQT>
NAMOH_DEV void softmax_probs(f32x16 (&S)[2][NQT], bf16x8 (&pB)[NQT][4], float (&alpha)[NQT],
                             bool& rescale, float (&m_run)[NQT], float (&l_run)[NQT],
                             float scale_log2, float lazy_thr) {
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    float mx = -INFINITY;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int e = 0; e < 16; e += 2) mx = fmaxf(mx, fmaxf(S[kk][qt][e], S[kk][qt][e + 1]));
    mx = pair_max32(mx);
    const bool up = mx > m_run[qt] + lazy_thr;
    const float mnew = up ? mx : m_run[qt];
    alpha[qt] = up ? __builtin_amdgcn_exp2f((m_run[qt] - mnew) * scale_log2) : 1.f;
    rescale |= up;
    const float mc = mnew * scale_log2;
    float ls = 0.f;
#pragma unroll
    for (int k2 = 0; k2 < 4; ++k2) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pB[qt][k2][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(
            fmaf(S[k2 >> 1][qt][8 * (k2 & 1) + e], scale_log2, -mc)));
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const bf16x2 pr = {pB[qt][k2][e], pB[qt][k2][e + 1]};
        ls = __builtin_amdgcn_fdot2_f32_bf16(pr, kOnes2, ls, false);
      }
    }
    l_run[qt] = l_run[qt] * alpha[qt] + ls;
    m_run[qt] = mnew;
  }
}

template <int D, int NQT>
NAMOH_DEV void rescale_o(f32x16 (&O)[D / 32][NQT], const float (&alpha)[NQT]) {
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) O[mt][qt][e] *= alpha[qt];
}

template <int D, int NQT>
NAMOH_DEV void pv_mfma(f32x16 (&O)[D / 32][NQT], const bf16x8 (&va)[4][D / 32],
                       const bf16x8 (&pB)[NQT][4]) {
#pragma unroll
  for (int k2 = 0; k2 < 4; ++k2)
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
      for (int qt = 0; qt < NQT; ++qt)
        O[mt][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[k2][mt], pB[qt][k2], O[mt][qt], 0, 0, 0);
}

// Single 32-query sub-tile versions (the two-sub-tile ping-pong loop).
template <int D>
NAMOH_DEV void qk_mfma1(f32x16 (&S)[2], const bf16x8 (&a)[D / 16][2], const bf16x8 (&qB)[D / 16]) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int e = 0; e < 16; ++e) S[kk][e] = 0.f;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
      S[kk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks][kk], qB[ks], S[kk], 0, 0, 0);
}

NAMOH_DEV void softmax_probs1(f32x16 (&S)[2], bf16x8 (&pB)[4], float& alpha, bool& rescale,
                              float& m_run, float& l_run, float scale_log2, float lazy_thr) {
  float mx = -INFINITY;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int e = 0; e < 16; e += 2) mx = fmaxf(mx, fmaxf(S[kk][e], S[kk][e + 1]));
  mx = pair_max32(mx);
  const bool up = mx > m_run + lazy_thr;
  const float mnew = up ? mx : m_run;
  alpha = up ? __builtin_amdgcn_exp2f((m_run - mnew) * scale_log2) : 1.f;
  rescale = up;
  const float mc = mnew * scale_log2;
  float ls = 0.f;
#pragma unroll
  for (int k2 = 0; k2 < 4; ++k2) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      pB[k2][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(
          fmaf(S[k2 >> 1][8 * (k2 & 1) + e], scale_log2, -mc)));
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const bf16x2 pr = {pB[k2][e], pB[k2][e + 1]};
      ls = __builtin_amdgcn_fdot2_f32_bf16(pr, kOnes2, ls, false);
    }
  }
  l_run = l_run * alpha + ls;
  m_run = mnew;
}

template <int D, int NQT, int QT>
NAMOH_DEV void pv_mfma_q(f32x16 (&O)[D / 32][NQT], const bf16x8 (&va)[4][D / 32],
                         const bf16x8 (&pB)[4]) {
#pragma unroll
  for (int k2 = 0; k2 < 4; ++k2)
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
      O[mt][QT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[k2][mt], pB[k2], O[mt][QT], 0, 0, 0);
}

template <int D, int NQT, int QT>
NAMOH_DEV void rescale_q(f32x16 (&O)[D / 32][NQT], float alpha) {
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) O[mt][QT][e] *= alpha;
}

// Mask, online softmax and O^T += V^T P^T for one 64-key tile.
template <int D, int NQT, int NW>
NAMOH_DEV void softmax_pv(f32x16 (&S)[2][NQT], f32x16 (&O)[D / 32][NQT],
                          float (&m_run)[NQT], float (&l_run)[NQT],
                          const uint16_t* __restrict__ sVb, int key0, int q0,
                          int wave, int n, int c, int g, float scale_log2,
                          float lazy_thr) {
  // value operands: the first VPRE 16-key steps are read while the softmax
  // runs (all of them for d = 64; half for d = 128, to stay within 256
  // registers), the rest while the first P.V products execute
  constexpr int VPRE = D == 128 ? 2 : 4;
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
  bf16x8 pB[NQT][4];
  float alpha[NQT];
  bool rescale = false;
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    float mx = -INFINITY;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int e = 0; e < 16; e += 2) mx = fmaxf(mx, fmaxf(S[kk][qt][e], S[kk][qt][e + 1]));
    mx = pair_max32(mx);
    const bool up = mx > m_run[qt] + lazy_thr;
    const float mnew = up ? mx : m_run[qt];
    alpha[qt] = up ? __builtin_amdgcn_exp2f((m_run[qt] - mnew) * scale_log2) : 1.f;
    rescale |= up;
    const float mc = mnew * scale_log2;
    float ls = 0.f;
#pragma unroll
    for (int k2 = 0; k2 < 4; ++k2) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pB[qt][k2][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(
            fmaf(S[k2 >> 1][qt][8 * (k2 & 1) + e], scale_log2, -mc)));
      // row sum of the rounded probabilities: pairs times (1, 1)
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const bf16x2 pr = {pB[qt][k2][e], pB[qt][k2][e + 1]};
        ls = __builtin_amdgcn_fdot2_f32_bf16(pr, kOnes2, ls, false);
      }
    }
    l_run[qt] = l_run[qt] * alpha[qt] + ls;
    m_run[qt] = mnew;
  }
  if (__any(rescale)) {
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
      for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) O[mt][qt][e] *= alpha[qt];
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

// ---------------------------------------------------------------------------
// bf16 MFMA flash attention over one (segment, query block) work item.
//
// v_mfma_f32_32x32x16_bf16 operand order used here (wave64, lane = 32*g + c):
// A (32 x 16): lane holds row c, reduction slots 8g..8g+7; B (16 x 32): lane
// holds column c, the same reduction slots; C (32 x 32): lane holds column c,
// rows 8j + 4g + i in accumulator 4j + i.  The kernel computes the transposed
// scores S^T = K Q^T (keys are rows), so every lane owns one query and 16 of
// its keys per 32-key sub-tile: the softmax row reduction is in-lane plus one
// exchange with lane c ^ 32.  The probabilities of a 16-key reduction step
// are accumulators 8s..8s+7, i.e. keys 8a + 4g + i (a = 0, 1); the
// transposed value tile stores, inside each 16-key group, key 8a + 4g + i at
// position 8g + 4a + i, so one 16-byte LDS read gives the matching A operand.
template <int D, int NQT, int NW, bool HB>
__global__ __launch_bounds__(NW * 64, MfmaShape<D>::MINB) void k_attn_mfma(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ Kp,
    const uint16_t* __restrict__ Vt, const float2* __restrict__ table,
    const int32_t* __restrict__ seg_offsets, const int32_t* __restrict__ tile_off,
    const int32_t* __restrict__ perm_token, const int2* __restrict__ items,
    const int32_t* __restrict__ meta, int T, int H, int rope_mode,
    float scale_log2, void* __restrict__ hout) {
  constexpr int BM = 32 * NQT * NW;
  constexpr int KS = D / 16;  // reduction steps of S^T = K Q^T
  constexpr int MT = D / 32;  // 32-row tiles of O^T
  constexpr int NT = NW * 64;
  constexpr int KPT = kBN * D / 8 / NT;  // 16-byte granules per thread per tile
  static_assert(kBN * D / 8 % NT == 0, "tile/thread mismatch");

  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kBN * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][D * kBN];

  int2 it;
  if (!my_item(items, meta, it)) return;
  const int s = it.x;
  const int q0 = it.y * BM;
  const int b = s / H, h = s - (s / H) * H;
  const int seg0 = seg_offsets[s];
  const int n = seg_offsets[s + 1] - seg0;
  const int tile0 = tile_off[s];
  const int ntiles = (n + kBN - 1) / kBN;
  const int kt_end = min(ntiles, (q0 + BM + kBN - 1) / kBN);
  const int tid = threadIdx.x;
  const int wave = tid / 64, lane = tid % 64;
  const int c = lane & 31, g = lane >> 5;
  const int wq_last = q0 + 32 * ((NQT - 1) * NW + wave) + 31;
  const int wave_tiles = min(ntiles, wq_last / kBN + 1);
  const size_t head_base = (static_cast<size_t>(b) * H + h) * T;
  const float lazy_thr = kLazyLog2 / scale_log2;

  // ---- query block: gather, rotate, round to bf16 B operands -------------
  bf16x8 qB[NQT][KS];
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    const int r = q0 + 32 * (qt * NW + wave) + c;
    const int rr = r < n ? r : n - 1;
    const int t = min(static_cast<unsigned>(perm_token[seg0 + rr]), static_cast<unsigned>(T - 1));
    const uint16_t* qrow = q + (head_base + t) * D;
    const int pos = rope_mode == 0 ? rr : t;
#pragma unroll
    for (int s2 = 0; s2 < KS / 2; ++s2) {
      float x1[8], x2[8];
      unpack8(*reinterpret_cast<const uint4*>(qrow + 16 * s2 + 8 * g), x1);
      unpack8(*reinterpret_cast<const uint4*>(qrow + D / 2 + 16 * s2 + 8 * g), x2);
      if (rope_mode != 2)
        rope8(x1, x2, table + static_cast<size_t>(pos) * (D / 2) + 16 * s2 + 8 * g);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        qB[qt][s2][e] = static_cast<__bf16>(r < n ? x1[e] : 0.f);
        qB[qt][s2 + KS / 2][e] = static_cast<__bf16>(r < n ? x2[e] : 0.f);
      }
    }
  }

  f32x16 O[MT][NQT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int qt = 0; qt < NQT; ++qt)
#pragma unroll
      for (int e = 0; e < 16; ++e) O[mt][qt][e] = 0.f;
  float m_run[NQT], l_run[NQT];
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    m_run[qt] = -1e30f;
    l_run[qt] = 0.f;
  }

#if NAMOH_ATTN_PIPE == 2
  // ---- two-sub-tile ping-pong -------------------------------------------
  // Each wave owns two 32-query sub-tiles.  On tiles that need no mask, the
  // score MFMAs of sub-tile 1 are interleaved with the softmax of sub-tile 0,
  // and the P.V MFMAs of sub-tile 0 with the softmax of sub-tile 1, so the
  // wave keeps its matrix and vector pipes busy at the same time.
  static_assert(NQT == 2, "ping-pong loop needs two query sub-tiles per wave");
  constexpr size_t TS = static_cast<size_t>(kBN) * D;
  const uint16_t* Kbase = Kp + static_cast<size_t>(tile0) * TS;
  const uint16_t* Vbase = Vt + static_cast<size_t>(tile0) * TS;
  if (kt_end > 0) {
    tile_dma<D / 8, KPT, NT>(Kbase, sK[0], tid);
    tile_dma<kBN / 8, KPT, NT>(Vbase, sV[0], tid);
  }
  for (int kt = 0; kt < kt_end; ++kt) {
    const int buf = kt & 1;
    wait_tile_dma();
    __syncthreads();
    if (kt + 1 < kt_end) {
      tile_dma<D / 8, KPT, NT>(Kbase + (kt + 1) * TS, sK[buf ^ 1], tid);
      tile_dma<kBN / 8, KPT, NT>(Vbase + (kt + 1) * TS, sV[buf ^ 1], tid);
    }
    if (kt >= wave_tiles) continue;
    const int key0 = kt * kBN;
    if (key0 + kBN - 1 > q0 + 32 * wave || key0 + kBN > n) {
      f32x16 S[2][NQT];
      qk_tile<D, NQT>(S, sK[buf], qB, c, g);
      softmax_pv<D, NQT, NW>(S, O, m_run, l_run, sV[buf], key0, q0, wave, n, c, g,
                             scale_log2, lazy_thr);
      continue;
    }
    bf16x8 ka[KS][2];
    qk_reads<D>(ka, sK[buf], c, g);
    f32x16 S0[2], S1[2];
    qk_mfma1<D>(S0, ka, qB[0]);
    qk_mfma1<D>(S1, ka, qB[1]);
    bf16x8 p0[4], p1[4];
    float a0, a1;
    bool r0, r1;
    softmax_probs1(S0, p0, a0, r0, m_run[0], l_run[0], scale_log2, lazy_thr);
#pragma unroll
    for (int i = 0; i < 2 * KS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
      __builtin_amdgcn_sched_group_barrier(0x002, 5, 1);
    }
    bf16x8 va[4][MT];
    v_reads<D>(va, sV[buf], c, g);
    if (__any(r0)) rescale_q<D, NQT, 0>(O, a0);
    pv_mfma_q<D, NQT, 0>(O, va, p0);
    softmax_probs1(S1, p1, a1, r1, m_run[1], l_run[1], scale_log2, lazy_thr);
#pragma unroll
    for (int i = 0; i < 4 * MT; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
      __builtin_amdgcn_sched_group_barrier(0x002, 5, 2);
    }
    if (__any(r1)) rescale_q<D, NQT, 1>(O, a1);
    pv_mfma_q<D, NQT, 1>(O, va, p1);
  }

#elif NAMOH_ATTN_PIPE
  // ---- software-pipelined tile loop -------------------------------------
  // Iteration j issues the score MFMAs of tile j + 1 interleaved with the
  // softmax VALU work of tile j (only the wave's last, diagonal tile needs a
  // mask, so every other iteration is one branch-free block that the
  // scheduling barriers below interleave), then the P.V MFMAs of tile j.
  // LDS holds K_{j+1} and V_j during iteration j; after the barrier that
  // opens iteration j the wave stores K_{j+2} into the key buffer K_j used
  // and V_{j+1} into the value buffer V_{j-1} used (both idle: every wave has
  // left iteration j - 1), and starts the global loads of K_{j+3}, V_{j+2}.
  constexpr size_t TS = static_cast<size_t>(kBN) * D;
  const uint16_t* Kbase = Kp + static_cast<size_t>(tile0) * TS;
  const uint16_t* Vbase = Vt + static_cast<size_t>(tile0) * TS;
  u32x4 kreg[KPT], vreg[KPT];
  if (kt_end > 0) {
    tile_gload<KPT, NT>(Kbase, tid, kreg);
    tile_gload<KPT, NT>(Vbase, tid, vreg);
    tile_lstore_k<D, KPT, NT>(sK[0], tid, kreg);
    tile_lstore_v<D, KPT, NT>(sV[0], tid, vreg);
  }
  if (kt_end > 1) {
    tile_gload<KPT, NT>(Kbase + TS, tid, kreg);
    tile_lstore_k<D, KPT, NT>(sK[1], tid, kreg);
  }
  __syncthreads();
  if (kt_end > 2) tile_gload<KPT, NT>(Kbase + 2 * TS, tid, kreg);
  if (kt_end > 1) tile_gload<KPT, NT>(Vbase + TS, tid, vreg);
  f32x16 SA[2][NQT], SB[2][NQT];
  if (wave_tiles > 0) qk_tile<D, NQT>(SA, sK[0], qB, c, g);

  auto step = [&](int j, f32x16 (&Scur)[2][NQT], f32x16 (&Snext)[2][NQT]) {
    __syncthreads();
    if (j + 2 < kt_end) tile_lstore_k<D, KPT, NT>(sK[j & 1], tid, kreg);
    if (j + 1 < kt_end) tile_lstore_v<D, KPT, NT>(sV[(j + 1) & 1], tid, vreg);
    if (j + 3 < kt_end) tile_gload<KPT, NT>(Kbase + (j + 3) * TS, tid, kreg);
    if (j + 2 < kt_end) tile_gload<KPT, NT>(Vbase + (j + 2) * TS, tid, vreg);
    if (j + 1 < wave_tiles) {
      bf16x8 ka[D / 16][2];
      qk_reads<D>(ka, sK[(j + 1) & 1], c, g);
      bf16x8 pB[NQT][4];
      float alpha[NQT];
      bool rescale = false;
      softmax_probs<NQT>(Scur, pB, alpha, rescale, m_run, l_run, scale_log2, lazy_thr);
      qk_mfma<D, NQT>(Snext, ka, qB);
      // interleave: all LDS reads first, then one MFMA per VALU group
#pragma unroll
      for (int i = 0; i < 2 * (D / 16) * NQT; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
      }
      bf16x8 va[4][D / 32];
      v_reads<D>(va, sV[j & 1], c, g);
      if (__any(rescale)) rescale_o<D, NQT>(O, alpha);
      pv_mfma<D, NQT>(O, va, pB);
    } else if (j < wave_tiles) {
      softmax_pv<D, NQT, NW>(Scur, O, m_run, l_run, sV[j & 1], j * kBN, q0, wave, n, c, g,
                             scale_log2, lazy_thr);
    }
  };
  for (int j = 0; j < kt_end; j += 2) {
    step(j, SA, SB);
    if (j + 1 < kt_end) step(j + 1, SB, SA);
  }

#else
  // ---- tile loop: double-buffered K/V tiles, one barrier per tile --------
  // Tile kt + 1 is copied straight into the idle LDS buffer (global -> LDS)
  // while tile kt is computed; the barrier at the top of the next iteration
  // publishes it.
  constexpr size_t TS = static_cast<size_t>(kBN) * D;
  const uint16_t* Kbase = Kp + static_cast<size_t>(tile0) * TS;
  const uint16_t* Vbase = Vt + static_cast<size_t>(tile0) * TS;
  if (kt_end > 0) {
    tile_dma<D / 8, KPT, NT>(Kbase, sK[0], tid);
    tile_dma<kBN / 8, KPT, NT>(Vbase, sV[0], tid);
  }
  for (int kt = 0; kt < kt_end; ++kt) {
    const int buf = kt & 1;
    wait_tile_dma();
    __syncthreads();
    if (kt + 1 < kt_end) {
      tile_dma<D / 8, KPT, NT>(Kbase + (kt + 1) * TS, sK[buf ^ 1], tid);
      tile_dma<kBN / 8, KPT, NT>(Vbase + (kt + 1) * TS, sV[buf ^ 1], tid);
    }
    if (kt < wave_tiles) {
      f32x16 S[2][NQT];
      qk_tile<D, NQT>(S, sK[buf], qB, c, g);
      softmax_pv<D, NQT, NW>(S, O, m_run, l_run, sV[buf], kt * kBN, q0, wave, n, c, g,
                             scale_log2, lazy_thr);
    }
  }

#endif
  // ---- epilogue: normalise and store the packed head outputs -----------
#pragma unroll
  for (int qt = 0; qt < NQT; ++qt) {
    const float lt = pair_sum32(l_run[qt]);
    const float inv = 1.f / lt;
    const int r = q0 + 32 * (qt * NW + wave) + c;
    if (r < n) {
      const size_t orow = static_cast<size_t>(seg0 + r) * D;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int d0 = 32 * mt + 8 * j + 4 * g;
          const float4 o4 = make_float4(O[mt][qt][4 * j] * inv, O[mt][qt][4 * j + 1] * inv,
                                        O[mt][qt][4 * j + 2] * inv, O[mt][qt][4 * j + 3] * inv);
          if constexpr (HB)
            *reinterpret_cast<uint2*>(static_cast<uint16_t*>(hout) + orow + d0) =
                make_uint2(pack_bf16x2(o4.x, o4.y), pack_bf16x2(o4.z, o4.w));
          else
            *reinterpret_cast<float4*>(static_cast<float*>(hout) + orow + d0) = o4;
        }
    }
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
    const int32_t* __restrict__ seg_offsets, const int32_t* __restrict__ perm_token,
    const int2* __restrict__ items, const int32_t* __restrict__ meta, int T,
    int H, int rope_mode, float scale, float* __restrict__ hout) {
  __shared__ float sK[kBN][D + 1];
  __shared__ float sV[kBN][D + 1];
  int2 it;
  if (!my_item(items, meta, it)) return;
  const int s = it.x;
  const int q0 = it.y * kGenericBM;
  const int b = s / H, h = s - (s / H) * H;
  const int seg0 = seg_offsets[s];
  const int n = seg_offsets[s + 1] - seg0;
  const size_t head_base = (static_cast<size_t>(b) * H + h) * T;
  const int lane = threadIdx.x;
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
template <bool IN_BF16, bool OUT_BF16>
__global__ __launch_bounds__(256) void k_combine(
    const void* __restrict__ hout, const float* __restrict__ gates,
    const int32_t* __restrict__ slot_pos, long BT, int K, int D, int Nr,
    void* __restrict__ out) {
  const int C = D / 4;
  const long idx = static_cast<long>(blockIdx.x) * blockDim.x + threadIdx.x;
  const long tok = idx / C;
  const int cc = static_cast<int>(idx - tok * C);
  if (tok >= BT) return;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k = 0; k < K; ++k) {
    const int p = slot_pos[tok * K + k];
    if (static_cast<unsigned>(p) >= static_cast<unsigned>(Nr)) continue;
    const float gk = gates[tok * K + k];
    float4 x;
    if constexpr (IN_BF16) {
      const uint2 u = reinterpret_cast<const uint2*>(hout)[static_cast<size_t>(p) * C + cc];
      x = make_float4(lo_bf16(u.x), hi_bf16(u.x), lo_bf16(u.y), hi_bf16(u.y));
    } else {
      x = reinterpret_cast<const float4*>(hout)[static_cast<size_t>(p) * C + cc];
    }
    acc.x = fmaf(gk, x.x, acc.x);
    acc.y = fmaf(gk, x.y, acc.y);
    acc.z = fmaf(gk, x.z, acc.z);
    acc.w = fmaf(gk, x.w, acc.w);
  }
  if constexpr (OUT_BF16) {
    reinterpret_cast<uint2*>(out)[idx] =
        make_uint2(pack_bf16x2(acc.x, acc.y), pack_bf16x2(acc.z, acc.w));
  } else {
    reinterpret_cast<float4*>(out)[idx] = acc;
  }
}

// ---------------------------------------------------------------------------
static bool use_mfma(int d, int dtype) { return dtype == 1 && (d == 64 || d == 128); }

static int block_queries(int d, int dtype) {
  if (!use_mfma(d, dtype)) return kGenericBM;
  return d == 64 ? 32 * MfmaShape<64>::NQT * MfmaShape<64>::NW
                 : 32 * MfmaShape<128>::NQT * MfmaShape<128>::NW;
}

struct AttnWs {
  int32_t* meta;
  int32_t* tile_off;
  long long* work_off;
  int2* items;
  float2* table;
  uint16_t* Kp;
  uint16_t* Vt;
  float* hpack;
  size_t bytes;
  size_t max_items, max_tiles;
};

static AttnWs carve_attn(void* ws, int B, int T, int H, int K, int d, int dtype) {
  const size_t BH = static_cast<size_t>(B) * H;
  const size_t Nr = static_cast<size_t>(B) * T * K;
  const int BM = block_queries(d, dtype);
  AttnWs w;
  w.max_items = Nr / BM + BH + 1;
  w.max_tiles = Nr / kBN + BH + 1;
  Carver cv(ws);
  w.meta = cv.take<int32_t>(kMetaCount);
  w.tile_off = cv.take<int32_t>(BH + 1);
  w.work_off = cv.take<long long>(BH + 1);
  w.items = cv.take<int2>(kXcd * w.max_items);
  w.table = cv.take<float2>(static_cast<size_t>(T) * (d / 2));
  if (use_mfma(d, dtype)) {
    w.Kp = cv.take<uint16_t>(w.max_tiles * kBN * d);
    w.Vt = cv.take<uint16_t>(w.max_tiles * kBN * d);
  } else {
    w.Kp = w.Vt = nullptr;
  }
  w.hpack = cv.take<float>(Nr * d);
  w.bytes = cv.off;
  return w;
}

size_t attn_workspace_bytes(int B, int T, int H, int K, int d, int dtype) {
  return carve_attn(nullptr, B, T, H, K, d, dtype).bytes;
}

template <int D>
static void launch_mfma(const AttnWs& w, const void* q, const void* k, const void* v,
                        int B, int T, int H, int rope_mode, float scale_log2,
                        const int32_t* seg_offsets, const int32_t* perm_token,
                        void* hout, bool hout_bf16, hipStream_t st) {
  constexpr int NW = MfmaShape<D>::NW, NQT = MfmaShape<D>::NQT;
  prof_mark("pack", true, st);
  k_pack_kv<D><<<static_cast<unsigned>(w.max_tiles), 256, 0, st>>>(
      static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), w.table,
      seg_offsets, w.tile_off, perm_token, w.meta, B * H, T, H, rope_mode, w.Kp, w.Vt);
  prof_mark("pack", false, st);
  prof_mark("attn", true, st);
  if (hout_bf16)
    k_attn_mfma<D, NQT, NW, true><<<static_cast<unsigned>(kXcd * w.max_items), NW * 64, 0, st>>>(
        static_cast<const uint16_t*>(q), w.Kp, w.Vt, w.table, seg_offsets, w.tile_off,
        perm_token, w.items, w.meta, T, H, rope_mode, scale_log2, hout);
  else
    k_attn_mfma<D, NQT, NW, false><<<static_cast<unsigned>(kXcd * w.max_items), NW * 64, 0, st>>>(
        static_cast<const uint16_t*>(q), w.Kp, w.Vt, w.table, seg_offsets, w.tile_off,
        perm_token, w.items, w.meta, T, H, rope_mode, scale_log2, hout);
  prof_mark("attn", false, st);
}

template <int D, bool BF16>
static void launch_generic(const AttnWs& w, const void* q, const void* k, const void* v,
                           int T, int H, int rope_mode, float scale,
                           const int32_t* seg_offsets, const int32_t* perm_token,
                           float* hout, hipStream_t st) {
  prof_mark("attn", true, st);
  k_attn_generic<D, BF16><<<static_cast<unsigned>(kXcd * w.max_items), 64, 0, st>>>(
      q, k, v, w.table, seg_offsets, perm_token, w.items, w.meta, T, H, rope_mode,
      scale, hout);
  prof_mark("attn", false, st);
}

hipError_t launch_attn(const void* q, const void* k, const void* v, int dtype,
                       int B, int T, int H, int K, int d, float rope_base,
                       int rope_mode, float scale, const float* gates,
                       const int32_t* seg_offsets, const int32_t* perm_token,
                       const int32_t* slot_pos, void* out, int out_dtype,
                       float* head_out, void* ws, hipStream_t st) {
  const AttnWs w = carve_attn(ws, B, T, H, K, d, dtype);
  // Without a caller-supplied head_out, the MFMA path keeps the packed head
  // outputs in bf16 (half the traffic of the attention epilogue and of the
  // combine); the combine accumulates in fp32 either way.
  const bool hb = head_out == nullptr && use_mfma(d, dtype);
  void* hout = head_out ? static_cast<void*>(head_out) : static_cast<void*>(w.hpack);
  const int BM = block_queries(d, dtype);
  const int Nr = B * T * K;
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  k_attn_prep<<<1 + 64, kPrepThreads, 0, st>>>(seg_offsets, B * H, T, BM, rope_mode, Nr,
                                               static_cast<int>(w.max_items), d, log_base,
                                               w.tile_off, w.work_off, w.items, w.meta, w.table);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (use_mfma(d, dtype)) {
    const float sl2 = scale * 1.4426950408889634f;
    if (d == 64)
      launch_mfma<64>(w, q, k, v, B, T, H, rope_mode, sl2, seg_offsets, perm_token, hout, hb, st);
    else
      launch_mfma<128>(w, q, k, v, B, T, H, rope_mode, sl2, seg_offsets, perm_token, hout, hb, st);
  } else {
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
  const long BT = static_cast<long>(B) * T;
  const long threads = BT * (d / 4);
  const unsigned grid = static_cast<unsigned>((threads + 255) / 256);
  prof_mark("combine", true, st);
  if (hb && out_dtype == 1)
    k_combine<true, true><<<grid, 256, 0, st>>>(hout, gates, slot_pos, BT, K, d, Nr, out);
  else if (hb)
    k_combine<true, false><<<grid, 256, 0, st>>>(hout, gates, slot_pos, BT, K, d, Nr, out);
  else if (out_dtype == 1)
    k_combine<false, true><<<grid, 256, 0, st>>>(hout, gates, slot_pos, BT, K, d, Nr, out);
  else
    k_combine<false, false><<<grid, 256, 0, st>>>(hout, gates, slot_pos, BT, K, d, Nr, out);
  prof_mark("combine", false, st);
  return hipGetLastError();
}

}  // namespace namoh
