// Routed per-head projections (Sec. 3.1, Eq. namoh-qkv, and the output
// aggregation of Eq. namoh-attention with W_O^(i) kept).
//
// Tokens are dispatched to their heads before projection: for every
// (batch b, head i) segment the packed rows r < n_{b,i} are the tokens of the
// ordered index set I_i, and only those pairs are projected.
//
//   k_proj_gemm<QKV>  [q|k|v]_{t,i} = x_t W_QKV[i]^T for the segment's rows:
//                     a grouped GEMM (M = n_{b,i}, N = 3d, K = d_model) whose
//                     data rows are gathered by token; the 4-column runs of
//                     each result row go straight to the dense q, k, v rows
//                     of the pair (other rows are never written).
//   k_proj_gemm<OUT>  Y_r = h_r W_O[i]^T for every packed head-output row r
//                     of the segment (M = n_{b,i}, N = d_model, K = d), bf16
//                     rows in packed order; k_combine then forms
//                     o_t = sum_k g_{t,k} Y[slot_pos(t,k)] in k order.
//
// One workgroup computes 128 rows x NT columns of one segment with four
// waves of 32 rows.  The product is formed transposed, C^T = W X^T, on
// v_mfma_f32_32x32x16_bf16 (weights as the A operand, data rows as the B
// operand; operand order in tile.h), so each lane holds 16 output columns of
// one data row, as four runs of 4 consecutive columns.  K is walked in
// chunks of 64: the next chunk is loaded into registers while the current
// one is multiplied from LDS (one LDS stage, rows of 128 bytes with the
// 64-bank granule swizzle).  fp32 accumulation; operands bf16 (fp32 head
// outputs are rounded to bf16 as they are staged).
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

// MODE kProjQKV: src = x [B, T, d_model] bf16, w = W_QKV [H, 3d, d_model] bf16,
//   kdim = d_model, N = 3d; outputs q, k, v [B, H, T, d] bf16 (dst0/1/2).
// MODE kProjOut: src = packed head outputs [Nr, d] (f32 if SRC_F32, else
//   bf16), w = W_O [H, d_model, d] bf16, kdim = d, N = d_model; output Y
//   [Nr, d_model] bf16 (dst0).
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
  const int b = s / H, hh = s - (s / H) * H;

  // ---- the thread's data rows and weight rows -----------------------------
  // data granule u = tid + 256 e: row u / 8, 16-byte granule u % 8 of the
  // chunk; weight granule likewise over NT rows
  size_t xrow[XG];   // element offset of the row's start in src (or ~0: padding)
#pragma unroll
  for (int e = 0; e < XG; ++e) {
    const int r = r0 + (tid + e * kProjThreads) / 8;
    xrow[e] = ~static_cast<size_t>(0);
    if (r < n) {
      if constexpr (MODE == kProjQKV) {
        const int t = min(static_cast<unsigned>(perm_token[seg0 + r]), static_cast<unsigned>(T - 1));
        xrow[e] = (static_cast<size_t>(b) * T + t) * kdim;
      } else {
        xrow[e] = static_cast<size_t>(seg0 + r) * kdim;
      }
    }
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
  if constexpr (MODE == kProjQKV) {
    const int t = min(static_cast<unsigned>(perm_token[seg0 + r]), static_cast<unsigned>(T - 1));
    const size_t orow = ((static_cast<size_t>(b) * H + hh) * T + t) * d;
#pragma unroll
    for (int t2 = 0; t2 < CT; ++t2)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = n0 + 32 * t2 + 8 * j + 4 * g;   // 4-column run inside one of q, k, v
        const int which = col / d, cc = col - (col / d) * d;
        uint16_t* dst = which == 0 ? dst0 : (which == 1 ? dst1 : dst2);
        *reinterpret_cast<uint2*>(dst + orow + cc) =
            make_uint2(pack_bf16x2(C[t2][4 * j], C[t2][4 * j + 1]),
                       pack_bf16x2(C[t2][4 * j + 2], C[t2][4 * j + 3]));
      }
  } else {
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
static unsigned proj_row_tiles(int B, int T, int H, int K) {
  const size_t Nr = static_cast<size_t>(B) * T * K;
  return static_cast<unsigned>(Nr / kProjRows + static_cast<size_t>(B) * H + 1);
}

hipError_t launch_qkv_proj(const void* x, const void* w_qkv, int B, int T, int H, int K, int d,
                           int d_model, const int32_t* seg_offsets, const int32_t* perm_token,
                           void* q, void* k, void* v, hipStream_t st) {
  const int N = 3 * d;
  if (N % 192 != 0 || d_model % kProjKC != 0) return hipErrorInvalidValue;
  const dim3 grid(proj_row_tiles(B, T, H, K), static_cast<unsigned>(N / 192));
  prof_mark("qkv_proj", true, st);
  k_proj_gemm<kProjQKV, 192, false><<<grid, kProjThreads, 0, st>>>(
      x, static_cast<const uint16_t*>(w_qkv), seg_offsets, perm_token, B * H, H, T, B * T * K,
      d_model, N, d, static_cast<uint16_t*>(q), static_cast<uint16_t*>(k),
      static_cast<uint16_t*>(v));
  prof_mark("qkv_proj", false, st);
  return hipGetLastError();
}

size_t out_proj_workspace_bytes(int B, int T, int K, int d_model) {
  return align_up(static_cast<size_t>(B) * T * K * d_model * 2);
}

hipError_t launch_out_proj(const void* head_out, int head_out_dtype, const void* w_o,
                           const float* gates, const int32_t* slot_pos,
                           const int32_t* seg_offsets, int B, int T, int H, int K, int d,
                           int d_model, void* out, int out_dtype, void* ws, hipStream_t st) {
  if (d % kProjKC != 0 || d_model % 128 != 0) return hipErrorInvalidValue;
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
