// Routed per-head projections (Sec. 3.1, Eq. namoh-qkv, and the output
// aggregation of Eq. namoh-attention with W_O^(i) kept).
//
// Tokens are dispatched to their heads before projection: for every
// (batch b, head i) segment the packed rows r < n_{b,i} are the tokens of the
// ordered index set I_i, and only those pairs are projected.
//
//   k_proj_big<QKV>   [q|k|v]_{t,i} = x_t W_QKV[i]^T for the segment's rows:
//                     a grouped GEMM (M = n_{b,i}, N = 3d, K = d_model) whose
//                     data rows are gathered by token; the 4-column runs of
//                     each result row go straight to the dense q, k, v rows
//                     of the pair (other rows are never written).
//   k_out_map +       dense output projection (H d <= 384 K): the tokens'
//   k_proj_big<OUT>   gated head rows against the stacked W_O over all heads.
//   k_proj_gemm +     per-pair output projection (otherwise): Y_r = h_r
//   k_combine         W_O[i]^T for every packed head-output row r (bf16 rows
//                     in packed order), then o_t = sum_k g_{t,k}
//                     Y[slot_pos(t,k)] in k order.
//
// The products are formed transposed, C^T = W X^T, on
// v_mfma_f32_32x32x16_bf16 (weights as the A operand, data rows as the B
// operand; operand order in tile.h), so each lane holds 16 output columns of
// one data row, as four runs of 4 consecutive columns.  K is walked in
// chunks of 64 staged through LDS (rows of 128 bytes with the 64-bank
// granule swizzle).  fp32 accumulation; operands bf16.
#include "common.h"
#include "internal.h"
#include "tile.h"

namespace namoh {

constexpr int kProjRows = 128;       // data rows per workgroup (4 waves x 32)
constexpr int kProjKC = 64;          // reduction chunk
constexpr int kProjThreads = 256;
constexpr int kProjSegLds = 1024;    // segment offsets staged in LDS up to this many

enum ProjMode { kProjQKV = 0, kProjOut = 1 };

// Packed 128-row tiles of segment s are numbered from seg0 / 128 + s (the
// same argument as seg_tile0 for 64-row tiles: disjoint, increasing, below
// Nr / 128 + BH + 1).
NAMOH_DEV int seg_ptile0(int seg0, int s) { return seg0 / kProjRows + s; }

template <int NT>
struct ProjLds {
  uint16_t w[NT * kProjKC];          // weight rows (output columns) x 64 k
  uint16_t x[kProjRows * kProjKC];   // data rows x 64 k
  int off[kProjSegLds + 1];
};

// Round 8 floats to bf16 (RNE) as one 16-byte granule.
NAMOH_DEV u32x4 f32x8_to_bf16(const float4 a, const float4 b) {
  return u32x4{pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w), pack_bf16x2(b.x, b.y),
               pack_bf16x2(b.z, b.w)};
}

// Chunk k0 of the thread's data granules (rows xrow[e], 16-byte granule
// (tid + 256 e) % 8; padding rows ~0 give zeros) and weight granules (row
// (tid + 256 e) / 8 of wbase) into registers.
template <int XG, int WG, bool SRC_F32>
NAMOH_DEV void proj_load(u32x4 (&xr)[XG], u32x4 (&wr)[WG], const void* __restrict__ src,
                         const size_t (&xrow)[XG], const uint16_t* __restrict__ wbase, int kdim,
                         int k0, int tid) {
#pragma unroll
  for (int e = 0; e < XG; ++e) {
    const int gr = (tid + e * kProjThreads) % 8;
    xr[e] = u32x4{0u, 0u, 0u, 0u};
    if (xrow[e] != ~static_cast<size_t>(0)) {
      if constexpr (SRC_F32) {
        const float4* p =
            reinterpret_cast<const float4*>(static_cast<const float*>(src) + xrow[e] + k0 + 8 * gr);
        xr[e] = f32x8_to_bf16(p[0], p[1]);
      } else {
        xr[e] = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(src) + xrow[e] + k0 +
                                                8 * gr);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < WG; ++e) {
    const int u = tid + e * kProjThreads;
    wr[e] = *reinterpret_cast<const u32x4*>(wbase + static_cast<size_t>(u / 8) * kdim + k0 +
                                            8 * (u % 8));
  }
}

// Per-pair output projection: one workgroup computes 128 packed rows x NT
// columns of one segment with four waves of 32 rows; the next chunk is loaded
// into registers while the current one is multiplied from LDS.  src = packed
// head outputs [Nr, d] (f32 if SRC_F32, else bf16; rounded to bf16 as they
// are staged), w = W_O [H, d_model, d] bf16, kdim = d, N = d_model; output Y
// [Nr, d_model] bf16 (dst0).
template <int MODE, int NT, bool SRC_F32>
__global__ __launch_bounds__(kProjThreads, 2) void k_proj_gemm(
    const void* __restrict__ src, const uint16_t* __restrict__ w,
    const int32_t* __restrict__ seg_offsets, const int32_t* __restrict__ perm_token, int BH,
    int H, int T, int Nr, int kdim, int N, int d, uint16_t* __restrict__ dst0,
    uint16_t* __restrict__ dst1, uint16_t* __restrict__ dst2) {
  static_assert(NT % 32 == 0 && (NT * kProjKC / 8) % kProjThreads == 0, "column tile");
  constexpr int CT = NT / 32;                                  // 32-column MFMA tiles
  constexpr int XG = kProjRows * kProjKC / 8 / kProjThreads;   // data granules per thread
  constexpr int WG = NT * kProjKC / 8 / kProjThreads;          // weight granules per thread
  __shared__ __attribute__((aligned(16))) ProjLds<NT> L;
  const int tid = thread_x();
  const int lane = tid % kWave, wave = tid / kWave;
  const int c = lane & 31, g = lane >> 5;
  const int gt = block_x();
  const int n0 = static_cast<int>(__builtin_amdgcn_workgroup_id_y()) * NT;

  // ---- segment of row tile gt (as in the packing kernel) ------------------
  const bool in_lds = BH <= kProjSegLds;
  if (in_lds)
    for (int i = tid; i <= BH; i += kProjThreads) L.off[i] = seg_offsets[i];
  __syncthreads();
  const int32_t* off = in_lds ? L.off : seg_offsets;
  int s;
  if (in_lds) {
    int cnt = 0;
    for (int s0 = 0; s0 < BH; s0 += kWave) {
      const int si = s0 + lane;
      cnt += __popcll(__ballot(si < BH && seg_ptile0(off[si], si) <= gt));
    }
    s = cnt - 1;
  } else {
    int lo = 0, hi = BH;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (seg_ptile0(off[mid], mid) <= gt) lo = mid; else hi = mid;
    }
    s = lo;
  }
  const int seg0 = off[s];
  const int n = off[s + 1] - seg0;
  const int r0 = (gt - seg_ptile0(seg0, s)) * kProjRows;
  // a tile in a gap between segments, or offsets that are not a packing
  if (r0 < 0 || r0 >= n || seg0 < 0 || n > T || seg0 + n > Nr) return;
  const int hh = s - (s / H) * H;

  // ---- the thread's data rows and weight rows -----------------------------
  // data granule u = tid + 256 e: row u / 8, 16-byte granule u % 8 of the
  // chunk; weight granule likewise over NT rows
  size_t xrow[XG];   // element offset of the row's start in src (or ~0: padding)
#pragma unroll
  for (int e = 0; e < XG; ++e) {
    const int r = r0 + (tid + e * kProjThreads) / 8;
    xrow[e] = ~static_cast<size_t>(0);
    if (r < n) xrow[e] = static_cast<size_t>(seg0 + r) * kdim;
  }
  const uint16_t* wbase = w + (static_cast<size_t>(hh) * N + n0) * kdim;

  u32x4 xr[XG], wr[WG];
  f32x16 C[CT];
#pragma unroll
  for (int t2 = 0; t2 < CT; ++t2)
#pragma unroll
    for (int e = 0; e < 16; ++e) C[t2][e] = 0.f;

  proj_load<XG, WG, SRC_F32>(xr, wr, src, xrow, wbase, kdim, 0, tid);
  const int drow = 32 * wave + c;   // this lane's data row in the tile (B operand column)
  for (int k0 = 0; k0 < kdim; k0 += kProjKC) {
    __syncthreads();            // the previous chunk's operand reads are done
#pragma unroll
    for (int e = 0; e < XG; ++e) {
      const int u = tid + e * kProjThreads, row = u / 8;
      *reinterpret_cast<u32x4*>(&L.x[row * kProjKC + swz<8>(row, u % 8) * 8]) = xr[e];
    }
#pragma unroll
    for (int e = 0; e < WG; ++e) {
      const int u = tid + e * kProjThreads, row = u / 8;
      *reinterpret_cast<u32x4*>(&L.w[row * kProjKC + swz<8>(row, u % 8) * 8]) = wr[e];
    }
    __syncthreads();
    if (k0 + kProjKC < kdim) proj_load<XG, WG, SRC_F32>(xr, wr, src, xrow, wbase, kdim, k0 + kProjKC, tid);
#pragma unroll
    for (int ks = 0; ks < kProjKC / 16; ++ks) {
      const bf16x8 bx =
          *reinterpret_cast<const bf16x8*>(&L.x[drow * kProjKC + swz<8>(drow, 2 * ks + g) * 8]);
#pragma unroll
      for (int t2 = 0; t2 < CT; ++t2) {
        const int wrow = 32 * t2 + c;
        const bf16x8 aw =
            *reinterpret_cast<const bf16x8*>(&L.w[wrow * kProjKC + swz<8>(wrow, 2 * ks + g) * 8]);
        C[t2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aw, bx, C[t2], 0, 0, 0);
      }
    }
  }

  // ---- epilogue: lane (c, g) holds data row drow, output columns
  // n0 + 32 t2 + 8 j + 4 g + i (i < 4) in accumulator 4 j + i ---------------
  const int r = r0 + drow;
  if (r >= n) return;
  {
    const size_t orow = static_cast<size_t>(seg0 + r) * N;
#pragma unroll
    for (int t2 = 0; t2 < CT; ++t2)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = n0 + 32 * t2 + 8 * j + 4 * g;
        *reinterpret_cast<uint2*>(dst0 + orow + col) =
            make_uint2(pack_bf16x2(C[t2][4 * j], C[t2][4 * j + 1]),
                       pack_bf16x2(C[t2][4 * j + 2], C[t2][4 * j + 3]));
      }
  }
}

// ---------------------------------------------------------------------------
// Output projection as one dense product over all heads of a token tile:
// o_t = sum_i [i selected for t] (g_{t,i} h_{t,i}) W_O[i]^T is the product of
// the gated head rows, laid out as a [B*T, H*d] operand whose blocks of
// unselected heads are zero, with the stacked weights [H*d, d_model].  That is
// H/K times the multiply-adds of the per-pair form, but no per-pair rows go
// through HBM: each token's gated rows are gathered straight into the operand
// tile, and the sum over the token's heads is the MFMA accumulation (head
// order, fp32).  Chosen when H*d is small against K (see out_proj_dense).
//
// k_out_map (32 tokens per workgroup): map[t * H + i] = packed row of head i
// for token t, or Nr when i is not selected (the head of a packed row is that
// of its segment: largest j with seg_offsets[j] <= row, head j % H); the
// gated rows G[r] = g h_r rounded to bf16 for every routed pair (r =
// slot_pos[t, k], g = gates[t, k]); and G[Nr] = 0, the row every unselected
// head reads.
constexpr int kMapTokens = 32;

template <bool SRC_F32>
__global__ __launch_bounds__(256) void k_out_map(
    const void* __restrict__ head_out, const float* __restrict__ gates,
    const int32_t* __restrict__ slot_pos, const int32_t* __restrict__ seg_offsets, long BT, int H,
    int K, int BH, int Nr, int d, int32_t* __restrict__ map, uint16_t* __restrict__ grows) {
  __shared__ int s_off[kProjSegLds + 1];
  __shared__ int s_tbl[kMapTokens * 64];
  __shared__ int s_row[kMapTokens * 64];
  __shared__ float s_gate[kMapTokens * 64];
  const int tid = thread_x();
  const long t0 = static_cast<long>(block_x()) * kMapTokens;
  const int nt = static_cast<int>(min(static_cast<long>(kMapTokens), BT - t0));
  const bool in_lds = BH <= kProjSegLds;
  if (in_lds)
    for (int i = tid; i <= BH; i += 256) s_off[i] = seg_offsets[i];
  for (int i = tid; i < nt * H; i += 256) s_tbl[i] = Nr;
  if (block_x() == 0)
    for (int i = tid; i < d / 8; i += 256)
      *reinterpret_cast<u32x4*>(grows + static_cast<size_t>(Nr) * d + 8 * i) = u32x4{0u, 0u, 0u, 0u};
  __syncthreads();
  const int32_t* off = in_lds ? s_off : seg_offsets;
  for (int i = tid; i < nt * K; i += 256) {
    const size_t gi = static_cast<size_t>(t0) * K + i;
    const int r = slot_pos[gi];
    const bool ok = r >= 0 && r < Nr;
    s_row[i] = ok ? r : -1;
    s_gate[i] = gates[gi];
    if (!ok) continue;
    int lo = 0, hi = BH;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (off[mid] <= r) lo = mid; else hi = mid;
    }
    s_tbl[(i / K) * H + lo % H] = r;
  }
  __syncthreads();
  for (int i = tid; i < nt * H; i += 256) map[static_cast<size_t>(t0) * H + i] = s_tbl[i];
  const int g8 = d / 8;
  for (int u = tid; u < nt * K * g8; u += 256) {
    const int i = u / g8, q = u - (u / g8) * g8;
    const int r = s_row[i];
    if (r < 0) continue;
    const float g = s_gate[i];
    const size_t o = static_cast<size_t>(r) * d + 8 * q;
    float f[8];
    if constexpr (SRC_F32) {
      const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(head_out) + o);
      const float4 a = p[0], b = p[1];
      f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
    } else {
      const u32x4 h = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(head_out) + o);
      const uint32_t hw[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        f[2 * e] = lo_bf16(hw[e]);
        f[2 * e + 1] = hi_bf16(hw[e]);
      }
    }
    *reinterpret_cast<u32x4*>(grows + o) =
        u32x4{pack_bf16x2(g * f[0], g * f[1]), pack_bf16x2(g * f[2], g * f[3]),
              pack_bf16x2(g * f[4], g * f[5]), pack_bf16x2(g * f[6], g * f[7])};
  }
}

// ---------------------------------------------------------------------------
// Big-tile GEMM of both projections: a workgroup computes 256 data rows x TN
// output columns with four waves of 128 rows x TN/2 columns (4 x TN/64 MFMA
// tiles per wave, accumulators in the AGPR half of the register file, one
// workgroup per CU).  The reduction runs in chunks of 64 through two LDS
// stages with one barrier per chunk.  Data rows are gathered, so their loads
// have the longer latency: they are issued three chunks ahead (two register
// sets), the weight rows two chunks ahead, each landing in LDS one chunk
// before use; the operand fragments of the next 16-wide step are read while
// the MFMAs of the current one run.
//   kProjQKV: data rows = the 256-row tiles of each (b, h) segment (tiles
//     numbered seg0 / 256 + s), gathered x rows; columns of W_QKV[h].
//   kProjOut: data rows = 256 consecutive tokens; the reduction runs over
//     H * d (chunk c is head c / (d / 64)); the rows are the tokens' gated
//     head rows G found through the head map (zero for unselected heads).
constexpr int kBigRows = 256;
constexpr int kQkvRows = 256;   // Q/K/V tiles (128: two workgroups per CU, measured no faster)
constexpr int kXcds = 8;        // XCDs of the device; workgroup i runs on XCD i % 8

template <int TM>
NAMOH_DEV int seg_btile0(int seg0, int s) { return seg0 / TM + s; }

template <int TM, int TN, int HM>
struct BigLds {
  uint16_t x[2][TM * kProjKC];
  uint16_t w[2][TN * kProjKC];
  int32_t map[TM * HM];   // OUT: the tile's head map (HM >= H); 160 KB in all at most
};
template <int TM, int TN>
struct BigLds<TM, TN, 0> {   // Q/K/V: no map (two 128-row workgroups fit one CU)
  uint16_t x[2][TM * kProjKC];
  uint16_t w[2][TN * kProjKC];
};

// Largest head count whose map tile fits beside the stages of a TN-wide tile.
constexpr int big_map_heads(int TN) { return TN == 256 ? 32 : 64; }

template <int MODE, int TM, int TN, bool OUT_BF16>
__global__ __launch_bounds__(kProjThreads, TM == 128 ? 2 : 1) void k_proj_big(
    const uint16_t* __restrict__ src, const uint16_t* __restrict__ w,
    const int32_t* __restrict__ seg_offsets, const int32_t* __restrict__ perm_token,
    const int32_t* __restrict__ map, int BH, int H, int T, long BT, int Nr, int kdim, int N, int d,
    int n_col_tiles, int classes, void* __restrict__ dst0, void* __restrict__ dst1,
    void* __restrict__ dst2) {
  constexpr int CT = TN / 64;                                  // 32-column tiles per wave
  constexpr int RT = TM / 64;                                   // 32-row tiles per wave
  constexpr int XG = TM * kProjKC / 8 / kProjThreads;          // data granules per thread
  constexpr int WG = TN * kProjKC / 8 / kProjThreads;          // weight granules per thread
  static_assert((TM == 128 || TM == 256) && TN % 64 == 0 && WG * kProjThreads * 8 == TN * kProjKC,
                "tile shape");
  constexpr int HM = MODE == kProjOut ? big_map_heads(TN) : 0;
  __shared__ __attribute__((aligned(16))) BigLds<TM, TN, HM> L;
  static_assert(sizeof(BigLds<TM, TN, HM>) <= 160 * 1024, "LDS");
  const int tid = thread_x();
  const int lane = tid % kWave, wave = tid / kWave;
  const int c = lane & 31, g = lane >> 5;
  const int wr = wave >> 1, wc = wave & 1;
  const int gr = tid % 8;   // the thread's 16-byte granule of a 64-wide chunk
  const int bid = block_x();
  const int rt0 = bid / n_col_tiles;
  int n0 = (bid - rt0 * n_col_tiles) * TN;

  // ---- the tile's data rows -------------------------------------------------
  int hh = 0, b = 0, seg0 = 0, nrow;
  long t0 = 0;
  size_t xrow[XG];   // QKV: element offset of the thread's x rows
  if constexpr (MODE == kProjQKV) {
    int* off = reinterpret_cast<int*>(&L.x[0][0]);   // staged before the ring is used
    const bool in_lds = BH <= kProjSegLds;
    if (in_lds)
      for (int i = tid; i <= BH; i += kProjThreads) off[i] = seg_offsets[i];
    __syncthreads();
    const int32_t* so = in_lds ? off : seg_offsets;
    int s, r0;
    if (classes > 1) {
      // XCD classes: workgroup bid runs on XCD bid % classes (dispatch is
      // round-robin over the XCDs) and takes the tiles of the heads h with
      // h % classes == bid % classes, so each XCD's L2 holds the weights of
      // its H / classes heads.  Class members (h, b) in order; tile j of the
      // class is found by a wave-wide scan of per-lane tile counts.
      const int x = bid % classes, i = bid / classes;
      n0 = (i % n_col_tiles) * TN;
      const int j = i / n_col_tiles;
      const int nb = BH / H;
      const int hc = x < H ? (H - x + classes - 1) / classes : 0;
      const int M = nb * hc;
      const int per = (M + kWave - 1) / kWave;
      const int m0 = min(M, lane * per), m1 = min(M, m0 + per);
      auto member = [&](int m) { return (m % nb) * H + x + classes * (m / nb); };
      int cnt = 0;
      for (int m = m0; m < m1; ++m) {
        const int sm = member(m);
        cnt += (max(0, so[sm + 1] - so[sm]) + TM - 1) / TM;
      }
      const int incl = wave_inclusive_scan(cnt);
      const uint64_t bal = __ballot(j >= incl - cnt && j < incl);
      int fs = -1, fr = 0;
      if (bal != 0 && lane == __ffsll(static_cast<unsigned long long>(bal)) - 1) {
        int acc = incl - cnt;
        for (int m = m0; m < m1; ++m) {
          const int sm = member(m);
          const int tcount = (max(0, so[sm + 1] - so[sm]) + TM - 1) / TM;
          if (j < acc + tcount) {
            fs = sm;
            fr = (j - acc) * TM;
            break;
          }
          acc += tcount;
        }
      }
      const int src_lane = bal != 0 ? __ffsll(static_cast<unsigned long long>(bal)) - 1 : 0;
      s = __shfl(fs, src_lane);
      r0 = __shfl(fr, src_lane);
    } else if (in_lds) {
      int cnt = 0;
      for (int s0 = 0; s0 < BH; s0 += kWave) {
        const int si = s0 + lane;
        cnt += __popcll(__ballot(si < BH && seg_btile0<TM>(so[si], si) <= rt0));
      }
      s = cnt - 1;
      r0 = (rt0 - seg_btile0<TM>(so[s], s)) * TM;
    } else {
      int lo = 0, hi = BH;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (seg_btile0<TM>(so[mid], mid) <= rt0) lo = mid; else hi = mid;
      }
      s = lo;
      r0 = (rt0 - seg_btile0<TM>(so[s], s)) * TM;
    }
    const int n = s >= 0 ? so[s + 1] - so[s] : 0;
    seg0 = s >= 0 ? so[s] : 0;
    __syncthreads();   // the staged offsets are read; the ring may be written
    if (s < 0 || r0 < 0 || r0 >= n || seg0 < 0 || n > T || seg0 + n > Nr) return;
    b = s / H;
    hh = s - (s / H) * H;
    seg0 += r0;
    nrow = min(TM, n - r0);
    // padding rows past the tile's end load the last row (their results are
    // never stored), so that no load needs a branch
#pragma unroll
    for (int e = 0; e < XG; ++e) {
      const int r = min(tid / 8 + 32 * e, nrow - 1);
      const int t = min(static_cast<unsigned>(perm_token[seg0 + r]), static_cast<unsigned>(T - 1));
      xrow[e] = (static_cast<size_t>(b) * T + t) * kdim;
    }
  } else {
    // the tile's head map into LDS (rows past the end repeat the last row;
    // their results are never stored)
    t0 = static_cast<long>(rt0) * TM;
    nrow = static_cast<int>(min(static_cast<long>(TM), BT - t0));
    // stored head-major ([h][row]): the 8 rows a wave reads for one head are
    // consecutive words, free of bank conflicts
    for (int i = tid; i < TM * H; i += kProjThreads) {
      const int row = i % TM, h = i / TM;
      const int32_t m = map[(static_cast<size_t>(t0) + min(row, nrow - 1)) * H + h];
      L.map[i] = static_cast<unsigned>(m) <= static_cast<unsigned>(Nr) ? m : Nr;
    }
    __syncthreads();
  }
  const int cph = d / kProjKC;                         // chunks per head (OUT)
  const int nchunk = MODE == kProjQKV ? kdim / kProjKC : H * cph;
  const int last = nchunk - 1;

  // two register sets for the weight rows too where the registers allow
  // (QKV; OUT with TN = 128): their loads are then also issued three chunks
  // ahead instead of two
  constexpr bool W2 = (MODE == kProjQKV && TM == 256) || (MODE == kProjOut && TN <= 128);
  u32x4 xs0[XG], xs1[XG], wv0[WG], wv1[W2 ? WG : 1];
  // one 16-byte granule e of the thread's data rows (rows tid / 8 + 32 e) or
  // weight rows of chunk ch
  auto load_x = [&](u32x4 (&xs)[XG], int ch, int e) {
    if constexpr (MODE == kProjQKV) {
      xs[e] = *reinterpret_cast<const u32x4*>(src + xrow[e] + ch * kProjKC + 8 * gr);
    } else {   // the gated row of the token's head (the zero row Nr if unselected)
      const int h = ch / cph, dd0 = (ch - h * cph) * kProjKC;
      const int m = L.map[h * TM + tid / 8 + 32 * e];
      xs[e] = *reinterpret_cast<const u32x4*>(src + static_cast<size_t>(m) * d + dd0 + 8 * gr);
    }
  };
  auto load_w = [&](u32x4 (&wv)[WG], int ch, int e) {
    const uint16_t* wb;
    size_t stride;
    if constexpr (MODE == kProjQKV) {
      wb = w + (static_cast<size_t>(hh) * N + n0) * kdim + ch * kProjKC;
      stride = kdim;
    } else {
      const int h = ch / cph, dd0 = (ch - h * cph) * kProjKC;
      wb = w + (static_cast<size_t>(h) * N + n0) * d + dd0;
      stride = d;
    }
    wv[e] = *reinterpret_cast<const u32x4*>(wb + static_cast<size_t>(tid / 8 + 32 * e) * stride + 8 * gr);
  };
  auto store_x = [&](const u32x4 (&xs)[XG], int stg, int e) {
    const int row = tid / 8 + 32 * e;
    *reinterpret_cast<u32x4*>(&L.x[stg][row * kProjKC + swz<8>(row, gr) * 8]) = xs[e];
  };
  auto store_w = [&](const u32x4 (&wv)[WG], int stg, int e) {
    const int row = tid / 8 + 32 * e;
    *reinterpret_cast<u32x4*>(&L.w[stg][row * kProjKC + swz<8>(row, gr) * 8]) = wv[e];
  };

  f32x16 C[CT][RT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int e = 0; e < 16; ++e) C[ct][rt][e] = 0.f;

  // One chunk step: chunk ch is multiplied from stage stg in four 16-wide
  // steps; behind the MFMAs of each step go a quarter of the LDS stores of
  // X(ch+1) (register set xn) and W(ch+1) into the free stage, each followed
  // by the load of the same granule of X(ch+3) and W(ch+2 or ch+3) into the
  // register it freed, so the staging runs in the shadow of the matrix work.
  // Operand fragments use two register sets: the reads of step ks + 1 are
  // issued before the MFMAs of step ks (scheduling barriers keep each step's
  // instructions together).  No branch surrounds a load or store (a load
  // under a branch is waited for where the branch joins, and the wait
  // counter is in order, so it would also wait for every load issued
  // before); indices past the end are clamped to the last chunk and land in
  // the stage that is no longer read.
  auto step = [&](int ch, u32x4 (&xn)[XG], u32x4 (&wn)[WG], int stg) {
    const int chx = min(ch + 3, last), chw = min(ch + (W2 ? 3 : 2), last);
    bf16x8 bx[2][RT], aw[2][CT];
    auto read_frags = [&](int ks, int set) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int drow = (TM / 2) * wr + 32 * rt + c;
        bx[set][rt] =
            *reinterpret_cast<const bf16x8*>(&L.x[stg][drow * kProjKC + swz<8>(drow, 2 * ks + g) * 8]);
      }
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) {
        const int wrow = (TN / 2) * wc + 32 * ct + c;
        aw[set][ct] =
            *reinterpret_cast<const bf16x8*>(&L.w[stg][wrow * kProjKC + swz<8>(wrow, 2 * ks + g) * 8]);
      }
    };
    read_frags(0, 0);
#pragma unroll
    for (int ks = 0; ks < kProjKC / 16; ++ks) {
      if (ks + 1 < kProjKC / 16) read_frags(ks + 1, (ks + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          C[ct][rt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aw[ks & 1][ct], bx[ks & 1][rt],
                                                              C[ct][rt], 0, 0, 0);
#pragma unroll
      for (int e = ks * XG / 4; e < (ks + 1) * XG / 4; ++e) {
        store_x(xn, stg ^ 1, e);
        load_x(xn, chx, e);
      }
#pragma unroll
      for (int e = ks * WG / 4; e < (ks + 1) * WG / 4; ++e) {
        store_w(wn, stg ^ 1, e);
        load_w(wn, chw, e);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
  };

  auto& wv1s = [&]() -> u32x4(&)[WG] {
    if constexpr (W2) return wv1; else return wv0;
  }();
#pragma unroll
  for (int e = 0; e < XG; ++e) load_x(xs0, 0, e);
#pragma unroll
  for (int e = 0; e < WG; ++e) load_w(wv0, 0, e);
#pragma unroll
  for (int e = 0; e < XG; ++e) store_x(xs0, 0, e);
#pragma unroll
  for (int e = 0; e < WG; ++e) store_w(wv0, 0, e);
#pragma unroll
  for (int e = 0; e < XG; ++e) load_x(xs1, min(1, last), e);
#pragma unroll
  for (int e = 0; e < WG; ++e) load_w(wv1s, min(1, last), e);
#pragma unroll
  for (int e = 0; e < XG; ++e) load_x(xs0, min(2, last), e);
  if constexpr (W2) {
#pragma unroll
    for (int e = 0; e < WG; ++e) load_w(wv0, min(2, last), e);
  }
  __syncthreads();
  int ch = 0;
  for (; ch + 1 < nchunk; ch += 2) {
    step(ch, xs1, wv1s, 0);
    step(ch + 1, xs0, wv0, 1);
  }
  if (ch < nchunk) step(ch, xs1, wv1s, 0);

  // ---- epilogue: lane (c, g) holds data row 128 wr + 32 rt + c, output
  // columns n0 + TN/2 wc + 32 ct + 8 j + 4 g + i in accumulator 4 j + i ----
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = (TM / 2) * wr + 32 * rt + c;
    if (r >= nrow) continue;
    size_t orow;
    if constexpr (MODE == kProjQKV) {
      const int t = min(static_cast<unsigned>(perm_token[seg0 + r]), static_cast<unsigned>(T - 1));
      orow = ((static_cast<size_t>(b) * H + hh) * T + t) * d;
    } else {
      orow = static_cast<size_t>(t0 + r) * N;
    }
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = n0 + (TN / 2) * wc + 32 * ct + 8 * j + 4 * g;
        const f32x16& A = C[ct][rt];
        if constexpr (MODE == kProjQKV) {
          const int which = col / d, cc = col - (col / d) * d;   // a 4-column run inside q, k or v
          uint16_t* dst = static_cast<uint16_t*>(which == 0 ? dst0 : (which == 1 ? dst1 : dst2));
          *reinterpret_cast<uint2*>(dst + orow + cc) =
              make_uint2(pack_bf16x2(A[4 * j], A[4 * j + 1]), pack_bf16x2(A[4 * j + 2], A[4 * j + 3]));
        } else if constexpr (OUT_BF16) {
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(dst0) + orow + col) =
              make_uint2(pack_bf16x2(A[4 * j], A[4 * j + 1]), pack_bf16x2(A[4 * j + 2], A[4 * j + 3]));
        } else {
          *reinterpret_cast<float4*>(static_cast<float*>(dst0) + orow + col) =
              make_float4(A[4 * j], A[4 * j + 1], A[4 * j + 2], A[4 * j + 3]);
        }
      }
  }
}

// The dense form costs 2 B T H d d_model multiply-add flops at MFMA rate; the
// per-pair form writes and re-reads B T K d_model bf16 rows.  With about
// 1 PFLOP/s sustained against about 4-5 TB/s for those rows the dense form is
// the faster one while H d < about 384 K (d 64: H/K <= 6; d 128: H/K <= 3).
bool out_proj_dense(int H, int K, int d) { return static_cast<long>(H) * d <= 384L * K && H <= 64; }

template <int TN>
static void launch_out_big(const uint16_t* grows, const uint16_t* w_o, const int32_t* map, long BT,
                           int Nr, int H, int d, int d_model, void* out, bool out_bf16,
                           hipStream_t st) {
  const int nct = d_model / TN;
  const unsigned grid = static_cast<unsigned>(((BT + kBigRows - 1) / kBigRows) * nct);
  if (out_bf16)
    k_proj_big<kProjOut, kBigRows, TN, true><<<grid, kProjThreads, 0, st>>>(
        grows, w_o, nullptr, nullptr, map, 0, H, 0, BT, Nr, d, d_model, d, nct, 1, out, nullptr, nullptr);
  else
    k_proj_big<kProjOut, kBigRows, TN, false><<<grid, kProjThreads, 0, st>>>(
        grows, w_o, nullptr, nullptr, map, 0, H, 0, BT, Nr, d, d_model, d, nct, 1, out, nullptr, nullptr);
}

// ---------------------------------------------------------------------------
static unsigned proj_row_tiles(int B, int T, int H, int K) {
  const size_t Nr = static_cast<size_t>(B) * T * K;
  return static_cast<unsigned>(Nr / kProjRows + static_cast<size_t>(B) * H + 1);
}

hipError_t launch_qkv_proj(const void* x, const void* w_qkv, int B, int T, int H, int K, int d,
                           int d_model, const int32_t* seg_offsets, const int32_t* perm_token,
                           void* q, void* k, void* v, hipStream_t st) {
  const int N = 3 * d;
  if (N % 192 != 0 || d_model % kProjKC != 0) return hipErrorInvalidValue;
  const size_t Nr = static_cast<size_t>(B) * T * K;
  const int nct = N / 192;
  constexpr int TM = kQkvRows;
  // XCD classes (heads h % 8 on XCD h % 8) when the offsets fit in LDS; the
  // grid then holds, per class, the most tiles a class can have (B T
  // min(K, H/8) / TM + B H/8 + 1); the rest of its workgroups find no tile
  const int classes = B * H <= kProjSegLds && H >= kXcds ? kXcds : 1;
  size_t tiles;
  if (classes > 1) {
    const size_t hc = (H + classes - 1) / classes;
    tiles = classes * (static_cast<size_t>(B) * T * std::min<size_t>(K, hc) / TM + B * hc + 1);
  } else {
    tiles = Nr / TM + static_cast<size_t>(B) * H + 1;
  }
  const unsigned grid = static_cast<unsigned>(tiles * nct);
  prof_mark("qkv_proj", true, st);
  k_proj_big<kProjQKV, TM, 192, false><<<grid, kProjThreads, 0, st>>>(
      static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w_qkv), seg_offsets,
      perm_token, nullptr, B * H, H, T,
      static_cast<long>(B) * T, B * T * K, d_model, N, d, nct, classes, q, k, v);
  prof_mark("qkv_proj", false, st);
  return hipGetLastError();
}

size_t out_proj_workspace_bytes(int B, int T, int H, int K, int d, int d_model) {
  if (out_proj_dense(H, K, d))   // head map + gated bf16 rows
    return align_up(static_cast<size_t>(B) * T * H * sizeof(int32_t)) +
           align_up((static_cast<size_t>(B) * T * K + 1) * d * 2);
  return align_up(static_cast<size_t>(B) * T * K * d_model * 2);
}

hipError_t launch_out_proj(const void* head_out, int head_out_dtype, const void* w_o,
                           const float* gates, const int32_t* slot_pos,
                           const int32_t* seg_offsets, int B, int T, int H, int K, int d,
                           int d_model, void* out, int out_dtype, void* ws, hipStream_t st) {
  if (d % kProjKC != 0 || d_model % 128 != 0) return hipErrorInvalidValue;
  if (out_proj_dense(H, K, d)) {
    const long BT = static_cast<long>(B) * T;
    int32_t* map = static_cast<int32_t*>(ws);
    uint16_t* grows = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) +
                                                  align_up(static_cast<size_t>(BT) * H * sizeof(int32_t)));
    const unsigned mgrid = static_cast<unsigned>((BT + kMapTokens - 1) / kMapTokens);
    prof_mark("out_proj", true, st);
    if (head_out_dtype == 0)
      k_out_map<true><<<mgrid, 256, 0, st>>>(head_out, gates, slot_pos, seg_offsets, BT, H, K, B * H,
                                             B * T * K, d, map, grows);
    else
      k_out_map<false><<<mgrid, 256, 0, st>>>(head_out, gates, slot_pos, seg_offsets, BT, H, K, B * H,
                                              B * T * K, d, map, grows);
    const uint16_t* w = static_cast<const uint16_t*>(w_o);
    if (d_model % 256 == 0 && H <= big_map_heads(256))
      launch_out_big<256>(grows, w, map, BT, B * T * K, H, d, d_model, out, out_dtype == 1, st);
    else
      launch_out_big<128>(grows, w, map, BT, B * T * K, H, d, d_model, out, out_dtype == 1, st);
    prof_mark("out_proj", false, st);
    return hipGetLastError();
  }
  uint16_t* Y = static_cast<uint16_t*>(ws);
  const dim3 grid(proj_row_tiles(B, T, H, K), static_cast<unsigned>(d_model / 128));
  prof_mark("out_proj", true, st);
  if (head_out_dtype == 0)
    k_proj_gemm<kProjOut, 128, true><<<grid, kProjThreads, 0, st>>>(
        head_out, static_cast<const uint16_t*>(w_o), seg_offsets, nullptr, B * H, H, T,
        B * T * K, d, d_model, d, Y, nullptr, nullptr);
  else
    k_proj_gemm<kProjOut, 128, false><<<grid, kProjThreads, 0, st>>>(
        head_out, static_cast<const uint16_t*>(w_o), seg_offsets, nullptr, B * H, H, T,
        B * T * K, d, d_model, d, Y, nullptr, nullptr);
  prof_mark("out_proj", false, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  prof_mark("out_combine", true, st);
  e = launch_combine_rows(Y, gates, slot_pos, static_cast<long>(B) * T, K, d_model, B * T * K,
                          out, out_dtype, st);
  prof_mark("out_combine", false, st);
  return e;
}

}  // namespace namoh
