// Backward of the routed mixture-of-head attention layer (training path).
//
// The exact gradient of Sec. 3.1, Eqs. namoh-gates (gates as inputs),
// namoh-head-rope and namoh-attention, for the packed varlen attention of
// Sec. 3.2 "Efficient execution" that training uses too, with the selection
// S_K held fixed (it is piecewise constant).  Per (b, h) segment, with the
// rotated rows Q~, K~, S = Q~ K~^T scale (causal), P = softmax(S), O = P V
// and dO_r = g_r dout_t:  dV = P^T dO,  dS = P (dO V^T - rowsum(dO O)),
// dQ~ = dS K~ scale,  dK~ = dS^T Q~ scale,  then dq = dQ~ R^T (rotation by
// minus the angle) at the token's row, and dgates[t,k] = <h(t, k), dout_t>.
//
// fp32 arithmetic throughout; the forward statistics (log-sum-exp, O) are
// recomputed here, so the gradients do not depend on how the forward ran.
//   k_bwd_zero     clears the dense gradients (rows of tokens a head does
//                  not see get none).
//   k_bwd_gather   one thread per (packed row, 8-pair group): rotated q, k,
//                  the value row and dO = g dout, packed fp32; the row's
//                  segment (binary search over the offsets, staged in LDS)
//                  and its k slot.
//   k_bwd_q        one lane per query of a 64-query block of a segment:
//                  pass 1 over the block's keys (64-key tiles in LDS) for the
//                  log-sum-exp and O, then D = <dO, O> and the gate gradient;
//                  pass 2 for dQ~.
//   k_bwd_kv       one lane per key of a 64-key block: pass 1 over the later
//                  queries (tiles of Q~, dO, lse, D in LDS) for dV, pass 2
//                  for dK~.
//   k_bwd_scatter  un-rotates dQ~, dK~ and writes dq, dk, dv at the token
//                  rows; dgates at the (t, k) slots.
#include <algorithm>
#include <cmath>

#include "common.h"
#include "internal.h"
#include "sched.h"
#include "tile.h"

namespace namoh {

constexpr int kBwdBlock = 64;       // rows per LDS tile
constexpr int kBwdSegLds = 2048;    // segment offsets staged in LDS up to this many

template <bool BF16>
NAMOH_DEV float ldx(const void* p, size_t i) {
  if constexpr (BF16) return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
  else return static_cast<const float*>(p)[i];
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_bwd_zero(float4* __restrict__ a, float4* __restrict__ b,
                                                  float4* __restrict__ c, size_t n4) {
  const size_t i = static_cast<size_t>(block_x()) * 256 + thread_x();
  if (i < n4) {
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    a[i] = z;
    b[i] = z;
    c[i] = z;
  }
}

// ---------------------------------------------------------------------------
template <int D, bool BF16>
__global__ __launch_bounds__(256) void k_bwd_gather(
    const void* __restrict__ q, const void* __restrict__ k, const void* __restrict__ v,
    const int32_t* __restrict__ topk_idx, const float* __restrict__ gates,
    const float* __restrict__ dout, const int32_t* __restrict__ seg_offsets,
    const int32_t* __restrict__ perm_token, int BH, int H, int T, int K, int Nr, int rope_mode,
    double log_base, float* __restrict__ Qr, float* __restrict__ Kr, float* __restrict__ Vp,
    float* __restrict__ dOp, int32_t* __restrict__ seg_of, int32_t* __restrict__ kslot) {
  constexpr int G = D / 16;               // 8-pair groups per row
  constexpr int RW = 256 / G;             // rows per workgroup
  __shared__ double s_theta[D / 2];
  __shared__ int s_off[kBwdSegLds + 1];
  const int tid = thread_x();
  if (tid < D / 2) s_theta[tid] = exp(-(2.0 * tid / D) * log_base);
  const bool in_lds = BH <= kBwdSegLds;
  if (in_lds)
    for (int i = tid; i <= BH; i += 256) s_off[i] = seg_offsets[i];
  __syncthreads();
  const int32_t* off = in_lds ? s_off : seg_offsets;
  const int r = block_x() * RW + tid / G;
  const int j0 = (tid % G) * 8;
  if (r >= Nr) return;
  int lo = 0, hi = BH;   // the last segment starting at or before r
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (off[mid] <= r) lo = mid; else hi = mid;
  }
  const int s = lo, rank = r - off[lo];
  const int t = perm_token[r];
  if (t < 0 || t >= T || r >= off[lo + 1] || rank < 0) {   // not a packing: mark the row
    if (j0 == 0) {
      seg_of[r] = -1;
      kslot[r] = -1;
    }
    return;
  }
  const int b = s / H, h = s - (s / H) * H;
  int ks = -1;   // which of the token's K selections this segment is
  const int32_t* sel = topk_idx + (static_cast<size_t>(b) * T + t) * K;
  for (int k0 = 0; k0 < K; k0 += 8) {   // eight independent loads per round
    int sv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) sv[u] = sel[min(k0 + u, K - 1)];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (k0 + u < K && sv[u] == h) ks = k0 + u;
  }
  const float gv = gates[(static_cast<size_t>(b) * T + t) * K + max(ks, 0)];
  const float g = ks >= 0 ? gv : 0.f;
  if (j0 == 0) {
    seg_of[r] = s;
    kslot[r] = ks;
  }
  const size_t src = (static_cast<size_t>(s) * T + t) * D;
  const size_t dst = static_cast<size_t>(r) * D;
  const double pos = rope_mode == 0 ? rank : t;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int j = j0 + e;
    float cs = 1.f, sn = 0.f;
    if (rope_mode != 2) {
      const float2 w = rope_cos_sin(pos * s_theta[j]);
      cs = w.x;
      sn = w.y;
    }
    const float q1 = ldx<BF16>(q, src + j), q2 = ldx<BF16>(q, src + j + D / 2);
    const float k1 = ldx<BF16>(k, src + j), k2 = ldx<BF16>(k, src + j + D / 2);
    Qr[dst + j] = q1 * cs - q2 * sn;
    Qr[dst + j + D / 2] = q2 * cs + q1 * sn;
    Kr[dst + j] = k1 * cs - k2 * sn;
    Kr[dst + j + D / 2] = k2 * cs + k1 * sn;
    Vp[dst + j] = ldx<BF16>(v, src + j);
    Vp[dst + j + D / 2] = ldx<BF16>(v, src + j + D / 2);
    const size_t drow = (static_cast<size_t>(b) * T + t) * D;
    dOp[dst + j] = g * dout[drow + j];
    dOp[dst + j + D / 2] = g * dout[drow + j + D / 2];
  }
}

// ---------------------------------------------------------------------------
// Row split: a row of D values is held by LPR = D / 64 lanes (one for d <= 64,
// two at d = 128), each with DH = D / LPR of its values; dot products add the
// lanes' partial sums with one exchange.  A wave holds 64 / LPR rows and a
// workgroup of kBwdWaves waves shares every 64-row tile staged in LDS (rows
// padded to D + 4 floats, so 16-byte reads stay aligned).
constexpr int kBwdWaves = 4;
constexpr int kBwdWgThreads = kBwdWaves * kWave;
template <int D> struct BwdShape {
  static constexpr int LPR = D > 64 ? D / 64 : 1;
  static constexpr int DH = D / LPR;
  static constexpr int RW = kWave / LPR;          // rows per wave
  static constexpr int RB = kBwdWaves * RW;       // rows per workgroup
  static constexpr int LD = D + 4;                // LDS row stride (floats)
};

template <int LPR>
NAMOH_DEV float row_sum(float x) {
  if constexpr (LPR == 2) x = group_sum<2>(x);
  return x;
}

// rows [r0, r0 + 64) of a packed fp32 array (rows past n as zeros) into an
// LDS tile, 16-byte loads all issued before the stores
template <int D>
NAMOH_DEV void stage_tile(float* tile, const float* __restrict__ src, size_t a, int r0, int n,
                          int tid) {
  constexpr int LD = BwdShape<D>::LD;
  constexpr int C4 = D / 4;                               // float4 per row
  constexpr int PER = kBwdBlock * C4 / kBwdWgThreads;     // float4 per thread
  float4 x[PER];
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int u = tid + m * kBwdWgThreads;
    const int rr = u / C4, c4 = u - rr * C4;
    x[m] = r0 + rr < n ? *reinterpret_cast<const float4*>(src + (a + r0 + rr) * D + 4 * c4)
                       : make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int u = tid + m * kBwdWgThreads;
    const int rr = u / C4, c4 = u - rr * C4;
    *reinterpret_cast<float4*>(tile + rr * LD + 4 * c4) = x[m];
  }
}

template <int DH>
NAMOH_DEV float dot_lds(const float* v, const float* row) {
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < DH; e += 4) {
    const float4 r = *reinterpret_cast<const float4*>(row + e);
    s = fmaf(v[e], r.x, s);
    s = fmaf(v[e + 1], r.y, s);
    s = fmaf(v[e + 2], r.z, s);
    s = fmaf(v[e + 3], r.w, s);
  }
  return s;
}

template <int DH>
NAMOH_DEV void axpy_lds(float* acc, float a, const float* row) {
#pragma unroll
  for (int e = 0; e < DH; e += 4) {
    const float4 r = *reinterpret_cast<const float4*>(row + e);
    acc[e] = fmaf(a, r.x, acc[e]);
    acc[e + 1] = fmaf(a, r.y, acc[e + 1]);
    acc[e + 2] = fmaf(a, r.z, acc[e + 2]);
    acc[e + 3] = fmaf(a, r.w, acc[e + 3]);
  }
}

constexpr float kLog2e = 1.4426950408889634f;

// Query side.  Workgroup qb of segment s (grid y = segment, x = block;
// blocks past the segment's end exit); lanes (row i, part).  Scores are kept
// in log2 units (q scaled by scale log2 e), so exp2 applies directly.
template <int D>
__global__ __launch_bounds__(kBwdWgThreads, 1) void k_bwd_q(
    const float* __restrict__ Qr, const float* __restrict__ Kr, const float* __restrict__ Vp,
    const float* __restrict__ dOp, const float* __restrict__ dout,
    const int32_t* __restrict__ seg_offsets, const int32_t* __restrict__ perm_token, int H, int T,
    int Nr, float scale, float* __restrict__ lse, float* __restrict__ Dr, float* __restrict__ dgp,
    float* __restrict__ dQr) {
  using S = BwdShape<D>;
  constexpr int DH = S::DH, RB = S::RB, LD = S::LD;
  __shared__ __attribute__((aligned(16))) float sk[kBwdBlock * LD];
  __shared__ __attribute__((aligned(16))) float sv[kBwdBlock * LD];
  const int s = static_cast<int>(__builtin_amdgcn_workgroup_id_y());
  const int qb = block_x();
  const int a = seg_offsets[s], n = seg_offsets[s + 1] - a;
  const int i0 = qb * RB;
  if (i0 >= n || a < 0 || n > T || a + n > Nr) return;   // past the end, or not a packing
  const int tid = thread_x();
  const int wave = tid / kWave, lane = tid % kWave;
  const int i = i0 + wave * S::RW + lane / S::LPR, c0 = (lane % S::LPR) * DH;
  const bool valid = i < n;
  const size_t row = static_cast<size_t>(a) + (valid ? i : n - 1);
  const float sl2 = scale * kLog2e;
  float qv[DH], acc[DH];
#pragma unroll
  for (int e = 0; e < DH; ++e) {
    qv[e] = Qr[row * D + c0 + e] * sl2;
    acc[e] = 0.f;
  }
  const int ntile = (min(n, i0 + RB) + kBwdBlock - 1) / kBwdBlock;
  auto stage = [&](int kt) {
    __syncthreads();
    stage_tile<D>(sk, Kr, a, kt * kBwdBlock, n, tid);
    stage_tile<D>(sv, Vp, a, kt * kBwdBlock, n, tid);
    __syncthreads();
  };
  float m = -INFINITY, l = 0.f;
  // pass 1: log-sum-exp and O (the accumulator is rescaled only when the
  // running maximum rises)
  for (int kt = 0; kt < ntile; ++kt) {
    stage(kt);
    const int j0 = kt * kBwdBlock;
    const int jn = min(kBwdBlock, i + 1 - j0);   // keys j0 .. i (the same for a row's lanes)
    for (int jj = 0; jj < jn; ++jj) {
      const float sc = row_sum<S::LPR>(dot_lds<DH>(qv, sk + jj * LD + c0));
      if (sc > m) {
        const float corr = exp2f(m - sc);
        l *= corr;
#pragma unroll
        for (int e = 0; e < DH; ++e) acc[e] *= corr;
        m = sc;
      }
      const float p = exp2f(sc - m);
      l += p;
      axpy_lds<DH>(acc, p, sv + jj * LD + c0);
    }
  }
  // D = <dO, O>, gate gradient <O, dout_t>
  const float inv = 1.f / l;
  const int t = min(static_cast<unsigned>(perm_token[row]), static_cast<unsigned>(T - 1));
  const int b = s / H;
  float dsum = 0.f, gsum = 0.f;
  float dov[DH];
#pragma unroll
  for (int e = 0; e < DH; ++e) {
    const float o = acc[e] * inv;
    dov[e] = dOp[row * D + c0 + e];
    dsum = fmaf(dov[e], o, dsum);
    gsum = fmaf(dout[(static_cast<size_t>(b) * T + t) * D + c0 + e], o, gsum);
    acc[e] = 0.f;
  }
  dsum = row_sum<S::LPR>(dsum);
  gsum = row_sum<S::LPR>(gsum);
  const float lse2 = m + log2f(l);   // log2 units
  if (valid && c0 == 0) {
    lse[row] = lse2;
    Dr[row] = dsum;
    dgp[row] = gsum;
  }
  // pass 2: dQ~ = scale * sum_j P_ij (dO_i . v_j - D_i) k~_j
  for (int kt = 0; kt < ntile; ++kt) {
    stage(kt);
    const int j0 = kt * kBwdBlock;
    const int jn = min(kBwdBlock, i + 1 - j0);
    for (int jj = 0; jj < jn; ++jj) {
      const float sc = row_sum<S::LPR>(dot_lds<DH>(qv, sk + jj * LD + c0));
      const float dp = row_sum<S::LPR>(dot_lds<DH>(dov, sv + jj * LD + c0));
      const float ds = exp2f(sc - lse2) * (dp - dsum) * scale;
      axpy_lds<DH>(acc, ds, sk + jj * LD + c0);
    }
  }
  if (valid) {
#pragma unroll
    for (int e = 0; e < DH; ++e) dQr[row * D + c0 + e] = acc[e];
  }
}

// ---------------------------------------------------------------------------
// Key side.  Workgroup kb of segment s; lanes (key row j, part); queries
// i >= j, their tiles (Q~, dO, log-sum-exp in log2 units, D) staged in LDS.
template <int D>
__global__ __launch_bounds__(kBwdWgThreads, 1) void k_bwd_kv(
    const float* __restrict__ Qr, const float* __restrict__ Kr, const float* __restrict__ Vp,
    const float* __restrict__ dOp, const float* __restrict__ lse, const float* __restrict__ Dr,
    const int32_t* __restrict__ seg_offsets, int T, int Nr, float scale, float* __restrict__ dKr,
    float* __restrict__ dVp) {
  using S = BwdShape<D>;
  constexpr int DH = S::DH, RB = S::RB, LD = S::LD;
  __shared__ __attribute__((aligned(16))) float sq[kBwdBlock * LD];
  __shared__ __attribute__((aligned(16))) float sdo[kBwdBlock * LD];
  __shared__ float sl[kBwdBlock], sd[kBwdBlock];
  const int s = static_cast<int>(__builtin_amdgcn_workgroup_id_y());
  const int kb = block_x();
  const int a = seg_offsets[s], n = seg_offsets[s + 1] - a;
  const int j0 = kb * RB;
  if (j0 >= n || a < 0 || n > T || a + n > Nr) return;   // past the end, or not a packing
  const int tid = thread_x();
  const int wave = tid / kWave, lane = tid % kWave;
  const int j = j0 + wave * S::RW + lane / S::LPR, c0 = (lane % S::LPR) * DH;
  const bool valid = j < n;
  const size_t row = static_cast<size_t>(a) + (valid ? j : n - 1);
  const float sl2 = scale * kLog2e;
  float kv[DH], acc[DH];
#pragma unroll
  for (int e = 0; e < DH; ++e) {
    kv[e] = Kr[row * D + c0 + e] * sl2;
    acc[e] = 0.f;
  }
  const int nqt = (n + kBwdBlock - 1) / kBwdBlock;
  const int qt0 = j0 / kBwdBlock;
  auto stage = [&](int qt) {
    const int i0 = qt * kBwdBlock;
    __syncthreads();
    stage_tile<D>(sq, Qr, a, i0, n, tid);
    stage_tile<D>(sdo, dOp, a, i0, n, tid);
    if (tid < kBwdBlock) {
      const bool in = i0 + tid < n;
      sl[tid] = in ? lse[static_cast<size_t>(a) + i0 + tid] : 0.f;
      sd[tid] = in ? Dr[static_cast<size_t>(a) + i0 + tid] : 0.f;
    }
    __syncthreads();
  };
  // pass 1: dV_j = sum_{i >= j} P_ij dO_i
  for (int qt = qt0; qt < nqt; ++qt) {
    stage(qt);
    const int i0 = qt * kBwdBlock;
    const int ib = max(0, j - i0), ie = min(kBwdBlock, n - i0);
    for (int ii = ib; ii < ie; ++ii) {
      const float sc = row_sum<S::LPR>(dot_lds<DH>(kv, sq + ii * LD + c0));
      axpy_lds<DH>(acc, exp2f(sc - sl[ii]), sdo + ii * LD + c0);
    }
  }
  if (valid) {
#pragma unroll
    for (int e = 0; e < DH; ++e) dVp[row * D + c0 + e] = acc[e];
  }
  // pass 2: dK~_j = scale * sum_{i >= j} P_ij (dO_i . v_j - D_i) q~_i
  float vv[DH];
#pragma unroll
  for (int e = 0; e < DH; ++e) {
    vv[e] = Vp[row * D + c0 + e];
    acc[e] = 0.f;
  }
  for (int qt = qt0; qt < nqt; ++qt) {
    stage(qt);
    const int i0 = qt * kBwdBlock;
    const int ib = max(0, j - i0), ie = min(kBwdBlock, n - i0);
    for (int ii = ib; ii < ie; ++ii) {
      const float sc = row_sum<S::LPR>(dot_lds<DH>(kv, sq + ii * LD + c0));
      const float dp = row_sum<S::LPR>(dot_lds<DH>(vv, sdo + ii * LD + c0));
      const float ds = exp2f(sc - sl[ii]) * (dp - sd[ii]) * scale;
      axpy_lds<DH>(acc, ds, sq + ii * LD + c0);
    }
  }
  if (valid) {
#pragma unroll
    for (int e = 0; e < DH; ++e) dKr[row * D + c0 + e] = acc[e];
  }
}

// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void k_bwd_scatter(
    const float* __restrict__ dQr, const float* __restrict__ dKr, const float* __restrict__ dVp,
    const float* __restrict__ dgp, const int32_t* __restrict__ seg_of,
    const int32_t* __restrict__ kslot, const int32_t* __restrict__ seg_offsets,
    const int32_t* __restrict__ perm_token, int BH, int H, int T, int K, int Nr, int rope_mode,
    double log_base, float* __restrict__ dq, float* __restrict__ dk, float* __restrict__ dv,
    float* __restrict__ dgates, int packed) {
  constexpr int G = D / 16;
  constexpr int RW = 256 / G;
  __shared__ double s_theta[D / 2];
  const int tid = thread_x();
  if (tid < D / 2) s_theta[tid] = exp(-(2.0 * tid / D) * log_base);
  __syncthreads();
  const int r = block_x() * RW + tid / G;
  const int j0 = (tid % G) * 8;
  if (r >= Nr) return;
  const int t = perm_token[r];
  const int s = seg_of[r];
  if (t < 0 || t >= T || s < 0 || s >= BH) return;
  const int rank = r - seg_offsets[s];
  const int b = s / H;
  const int ks = kslot[r];
  if (j0 == 0 && ks >= 0 && ks < K) dgates[(static_cast<size_t>(b) * T + t) * K + ks] = dgp[r];
  const size_t src = static_cast<size_t>(r) * D;
  // dense [B, H, T, d] rows, or (packed) the routed row's own packed row
  const size_t dst = packed ? static_cast<size_t>(r) * D : (static_cast<size_t>(s) * T + t) * D;
  const double pos = rope_mode == 0 ? rank : t;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int j = j0 + e;
    float cs = 1.f, sn = 0.f;
    if (rope_mode != 2) {
      const float2 w = rope_cos_sin(pos * s_theta[j]);
      cs = w.x;
      sn = w.y;
    }
    // gradient through x' = (x1 c - x2 s, x2 c + x1 s): (d1 c + d2 s, d2 c - d1 s)
    const float q1 = dQr[src + j], q2 = dQr[src + j + D / 2];
    const float k1 = dKr[src + j], k2 = dKr[src + j + D / 2];
    dq[dst + j] = q1 * cs + q2 * sn;
    dq[dst + j + D / 2] = q2 * cs - q1 * sn;
    dk[dst + j] = k1 * cs + k2 * sn;
    dk[dst + j + D / 2] = k2 * cs - k1 * sn;
    dv[dst + j] = dVp[src + j];
    dv[dst + j + D / 2] = dVp[src + j + D / 2];
  }
}

// ===========================================================================
// bf16 MFMA path (d = 64 or 128).
//
// The forward (launch_attn_stats) leaves the rotated key tiles Kp, the
// transposed value tiles Vt, the work list, h and the log-sum-exp of every
// row.  k_bwd_pack adds, in the same numbering of 64-row tiles (row r of
// segment s at packed row 64 * seg_tile0 + r, rows past n zero):
//   Qs  = bf16(q~ * scale * log2 e), exactly the forward's query operand;
//   dO  = bf16(g * dout);  Vp = v;  (row-major, like Kp)
//   LD  = (lse, D) per row, D = <dO, h>; (+inf, 0) past n, so padding rows
//   get zero probabilities.
// k_bwd_dq (one wave per 32 queries, key tiles streamed): S^T - lse and
// dP^T - D start from the accumulators, dS^T = exp2(S^T - lse) (dP^T - D),
// dQ^T += K^T dS^T.  k_bwd_dkdv (one wave per 32 keys, query tiles
// streamed from the key block on): S - lse, dP - D, dV^T += dO^T P,
// dK^T += Q^T dS.  The transposed operands (K^T, dO^T, Q^T) are read from the
// same row-major LDS tiles with gfx950's transposing LDS reads.  Both take the forward's work list (heaviest first); the
// key side reads item (s, qb) as key block ceil(n / 128) - 1 - qb, whose work
// (the later queries) is what the query block's was (the earlier keys).
constexpr int kBwdPackThreads = 256;
constexpr int kBwdMfmaThreads = 256;   // 4 waves of 32 rows: 128-row blocks
constexpr int kBwdMfmaBlock = 128;
constexpr float kLn2 = 0.6931471805599453f;

// The key side's own work list (built by the packing kernel's workgroup 0):
// where it goes, its capacity, and the placement (period: compute units;
// resident: the key-side kernel's resident workgroups).
struct KeyList {
  WorkItem* items;
  int32_t* meta;
  int max_items, period, resident;
};

template <int D>
struct BwdPackLds {
  int off[kBwdSegLds + 1];
  int tok[kBN], ks[kBN];       // per tile row: token, k slot (-1: none)
  float g[kBN];                // per tile row: gate
  double freq[D / 2];          // RoPE theta_j / (2 pi)
};

template <int D>
__global__ __launch_bounds__(kBwdPackThreads) void k_bwd_pack(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ v,
    const float* __restrict__ dout, const int32_t* __restrict__ topk_idx,
    const float* __restrict__ gates, const int32_t* __restrict__ seg_offsets,
    const int32_t* __restrict__ perm_token, const double* __restrict__ freq,
    const float* __restrict__ hpack, const float* __restrict__ lse, int BH, int H, int T, int K,
    int Nr, int rope_mode, float scale_log2, uint16_t* __restrict__ Qs, uint16_t* __restrict__ dO,
    uint16_t* __restrict__ Vp, float2* __restrict__ LD, float* __restrict__ dgates, KeyList kl) {
  __shared__ __attribute__((aligned(16))) union {
    BwdPackLds<D> pack;
    SchedLds sched;
  } U;
  BwdPackLds<D>& L = U.pack;
  if (block_x() == 0) {
    // the key side's work list: whole blocks, heaviest first, placed for the
    // key-side kernel's resident workgroups (it runs alongside the packing)
    attn_schedule<kBwdPackThreads>(seg_offsets, BH, T, kBwdMfmaBlock, Nr, kl.max_items, kl.period,
                                   1, kl.items, kl.meta, U.sched, 0, nullptr, kl.resident);
    return;
  }
  const int gt = block_x() - 1;   // the tile this workgroup packs
  const int tid = thread_x();
  const bool in_lds = BH <= kBwdSegLds;
  // (published by the barrier before the rows are packed)
  if (rope_mode != 2 && tid < D / 2) L.freq[tid] = freq[tid];
  if (in_lds) {
    for (int i = tid; i <= BH; i += kBwdPackThreads) L.off[i] = seg_offsets[i];
    __syncthreads();
  }
  const int32_t* off = in_lds ? L.off : seg_offsets;
  int lo = 0, hi = BH;   // the segment of tile gt: last s with seg_tile0(off[s], s) <= gt
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (seg_tile0(off[mid], mid) <= gt) lo = mid; else hi = mid;
  }
  const int s = lo;
  const int seg0 = off[s];
  const int n = off[s + 1] - seg0;
  const int r0 = (gt - seg_tile0(seg0, s)) * kBN;
  // a tile in a gap between segments, or offsets that are not a packing
  if (r0 < 0 || r0 >= n || seg0 < 0 || n > T || seg0 + n > Nr) return;
  const int b = s / H, hh = s - (s / H) * H;
  const size_t head_base = (static_cast<size_t>(b) * H + hh) * T;
  const size_t prow0 = static_cast<size_t>(gt) * kBN;
  // token, k slot and gate of each tile row, once per row (r < n)
  if (tid < kBN && r0 + tid < n) {
    const int t = min(static_cast<unsigned>(perm_token[seg0 + r0 + tid]),
                      static_cast<unsigned>(T - 1));
    const int32_t* sel = topk_idx + (static_cast<size_t>(b) * T + t) * K;
    // the token's slot of head hh: eight independent loads per round (no
    // load under a branch, so they are in flight together)
    int ks = -1;
    for (int k0 = 0; k0 < K; k0 += 8) {
      int sv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) sv[u] = sel[min(k0 + u, K - 1)];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (k0 + u < K && sv[u] == hh) ks = k0 + u;
    }
    const float gv = gates[(static_cast<size_t>(b) * T + t) * K + max(ks, 0)];
    L.tok[tid] = t;
    L.ks[tid] = ks;
    L.g[tid] = ks >= 0 ? gv : 0.f;
  }
  __syncthreads();

  // rows: rotated, scaled queries (as the forward rounds them), gated output
  // gradients, values; one 8-pair group (j, j + d/2) per unit
  constexpr int HP = D / 16;
  for (int u = tid; u < kBN * HP; u += kBwdPackThreads) {
    const int row = u / HP, c = u - (u / HP) * HP;
    const int r = r0 + row;
    uint4 q1 = make_uint4(0, 0, 0, 0), q2 = q1, o1 = q1, o2 = q1, v1 = q1, v2 = q1;
    if (r < n) {
      const int t = L.tok[row];
      const float g = L.g[row];
      const uint16_t* qrow = q + (head_base + t) * D;
      float x1[8], x2[8];
      unpack8(*reinterpret_cast<const uint4*>(qrow + 8 * c), x1);
      unpack8(*reinterpret_cast<const uint4*>(qrow + D / 2 + 8 * c), x2);
      if (rope_mode != 2) {
        float4 cs[4];
        // the factors the forward rotated its queries with
        rope8_rev(cs, static_cast<double>(rope_mode == 0 ? r : t), &L.freq[8 * c]);
        rope8(x1, x2, cs);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x1[e] *= scale_log2;
        x2[e] *= scale_log2;
      }
      q1 = pack8(x1);
      q2 = pack8(x2);
      const float4* drow = reinterpret_cast<const float4*>(dout + (static_cast<size_t>(b) * T + t) * D);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const float4 a = drow[2 * c + e], a2 = drow[D / 8 + 2 * c + e];
        x1[4 * e] = g * a.x; x1[4 * e + 1] = g * a.y; x1[4 * e + 2] = g * a.z; x1[4 * e + 3] = g * a.w;
        x2[4 * e] = g * a2.x; x2[4 * e + 1] = g * a2.y; x2[4 * e + 2] = g * a2.z; x2[4 * e + 3] = g * a2.w;
      }
      o1 = pack8(x1);
      o2 = pack8(x2);
      const uint16_t* vrow = v + (head_base + t) * D;
      v1 = *reinterpret_cast<const uint4*>(vrow + 8 * c);
      v2 = *reinterpret_cast<const uint4*>(vrow + D / 2 + 8 * c);
    }
    const size_t o = (prow0 + row) * D;
    *reinterpret_cast<uint4*>(Qs + o + 8 * c) = q1;
    *reinterpret_cast<uint4*>(Qs + o + D / 2 + 8 * c) = q2;
    *reinterpret_cast<uint4*>(dO + o + 8 * c) = o1;
    *reinterpret_cast<uint4*>(dO + o + D / 2 + 8 * c) = o2;
    *reinterpret_cast<uint4*>(Vp + o + 8 * c) = v1;
    *reinterpret_cast<uint4*>(Vp + o + D / 2 + 8 * c) = v2;
  }
  // per row: D = <dO, h> (dO as rounded for the products), the gate
  // gradient <dout, h>, the log-sum-exp; four lanes per row
  {
    static_assert(kBwdPackThreads == 4 * kBN, "four lanes per row");
    const int row = tid >> 2, part = tid & 3;
    const int r = r0 + row;
    float dd = 0.f, dg = 0.f;
    int ks = -1, t = 0;
    if (r < n) {
      t = L.tok[row];
      ks = L.ks[row];
      const float g = L.g[row];
      const float4* hrow = reinterpret_cast<const float4*>(hpack + static_cast<size_t>(seg0 + r) * D);
      const float4* drow = reinterpret_cast<const float4*>(dout + (static_cast<size_t>(b) * T + t) * D);
#pragma unroll
      for (int e4 = part * (D / 16); e4 < (part + 1) * (D / 16); ++e4) {
        const float4 h4 = hrow[e4], d4 = drow[e4];
        const float hv[4] = {h4.x, h4.y, h4.z, h4.w}, dv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          dg = fmaf(dv[i], hv[i], dg);
          dd = fmaf(bf16_to_f32(f32_to_bf16(g * dv[i])), hv[i], dd);
        }
      }
    }
    dd = group_sum<4>(dd);
    dg = group_sum<4>(dg);
    if (part == 0) {
      LD[prow0 + row] = r < n ? make_float2(lse[seg0 + r], dd) : make_float2(INFINITY, 0.f);
      if (r < n && ks >= 0) dgates[(static_cast<size_t>(b) * T + t) * K + ks] = dg;
    }
  }
}

// C[kk] = A[kk] B for the two 32-row halves kk of a 64-row row-major LDS
// tile (swizzled as the tile loads store it) against D/16 register B
// operands, the accumulators starting at init[kk].  All LDS reads are issued
// before the first product.
template <int D>
NAMOH_DEV void tile_rows_x_regs(f32x16 (&C)[2], const uint16_t* __restrict__ tile,
                                const bf16x8 (&bop)[D / 16], const f32x16& init0,
                                const f32x16& init1, int c, int g) {
  constexpr int KS = D / 16;
  bf16x8 a[KS][2];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int row = 32 * kk + c;
      a[ks][kk] = *reinterpret_cast<const bf16x8*>(&tile[row * D + swz<D / 8>(row, 2 * ks + g) * 8]);
    }
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
    C[kk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0][kk], bop[0], kk == 0 ? init0 : init1, 0, 0, 0);
#pragma unroll
  for (int ks = 1; ks < KS; ++ks)
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
      C[kk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks][kk], bop[ks], C[kk], 0, 0, 0);
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
// The lane's byte offsets inside a tile for slot step 0 (read hh, column
// block mt); step ks adds 16 ks rows, a constant the read's offset field
// carries (row & 15 and so the swizzle do not change with ks).
template <int D>
struct TrOff {
  uint32_t o[2][D / 32];
};
template <int D>
NAMOH_DEV TrOff<D> tr_offsets(int lane) {
  const int grp = lane >> 4, i = lane & 15;
  TrOff<D> t;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt) {
      const int col = 32 * mt + 16 * (grp & 1) + 4 * (i & 3);
      const int row = vt_key_of_pos(8 * (grp >> 1) + 4 * hh + (i >> 2));
      t.o[hh][mt] = static_cast<uint32_t>((row * D + swz<D / 8>(row, col >> 3) * 8 + (col & 7)) * 2);
    }
  return t;
}
// A operand of the transposed view of a row-major 64-row LDS tile X [64][D]
// (granules swizzled by swz<D/8>, as the tile loads store it): lane (c, g)
// gets X[row(16 ks + 8 g + e)][32 mt + c], e = 0..7, with row(p) =
// vt_key_of_pos(p), the slot order of the C-layout B operands below.  Two
// transposing LDS reads (ds_read_b64_tr_b16): within each 16-lane group,
// source lane a + 4k names 4 consecutive columns 4a .. 4a + 3 of the row of
// slot k, and destination lane 4a + b receives column 4a + b of the four
// rows k = 0..3, so lanes 0-15 / 16-31 cover columns 0-15 / 16-31 of the
// 32-column block and lanes 32-63 the slots 8 .. 15.
template <int D>
NAMOH_DEV bf16x8 tr_operand(uint32_t tile_lds, const TrOff<D>& t, int mt, int ks) {
  union {
    i16x4 h[2];
    bf16x8 v;
  } u;
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const uint32_t a = tile_lds + t.o[hh][mt] + static_cast<uint32_t>(16 * ks * D * 2);
    u.h[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(static_cast<size_t>(a)));
  }
  return u.v;
}

// acc[mt] += X^T(rows 32 mt + c) Y over the tile's 64 reduction slots: X the
// row-major tile [64][D] in LDS read transposed, Y given as four 16-slot B
// operands taken from C-layout accumulators (slot order as tile.h describes).
template <int D>
NAMOH_DEV void rows_tposed_x_c(f32x16 (&acc)[D / 32], uint32_t tile_lds, const TrOff<D>& t,
                               const bf16x8 (&x)[4]) {
#pragma unroll
  for (int k2 = 0; k2 < 4; ++k2) {
    bf16x8 a[D / 32];
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt) a[mt] = tr_operand<D>(tile_lds, t, mt, k2);
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
      acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mt], x[k2], acc[mt], 0, 0, 0);
  }
}

// One 32-row half of tile_rows_x_regs: rows 32 kk .. 32 kk + 31 (kk wave
// uniform) of the tile against the register B operands.
template <int D>
NAMOH_DEV void tile_half_x_regs(f32x16& C, const uint16_t* __restrict__ tile,
                                const bf16x8 (&bop)[D / 16], const f32x16& init, int kk, int c,
                                int g) {
  constexpr int KS = D / 16;
  const int row = 32 * kk + c;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const bf16x8 a =
        *reinterpret_cast<const bf16x8*>(&tile[row * D + swz<D / 8>(row, 2 * ks + g) * 8]);
    C = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bop[ks], ks == 0 ? init : C, 0, 0, 0);
  }
}

// rows_tposed_x_c over the 32 reduction slots 32 kk .. 32 kk + 31 (kk wave
// uniform), Y given as their two 16-slot B operands.
template <int D>
NAMOH_DEV void rows_tposed_half_x_c(f32x16 (&acc)[D / 32], uint32_t tile_lds,
                                    const TrOff<D>& t, const bf16x8 (&x)[2], int kk) {
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt) {
      const bf16x8 a = tr_operand<D>(tile_lds, t, mt, 2 * kk + kh);
      acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, x[kh], acc[mt], 0, 0, 0);
    }
}

// (lse, D) pairs of one 64-row tile: 512 bytes, 32 lanes of wave 0 (the
// other waves issue nothing, and every wait below is for all loads).
NAMOH_DEV void ld_tile_dma(const float2* base, uint32_t nbytes, uint32_t tile_bytes,
                           uint32_t lds, int wave, int lane) {
  if (wave == 0) {
    const i32x4 rsrc = buffer_rsrc(reinterpret_cast<const uint16_t*>(base), nbytes);
    const int tb = __builtin_amdgcn_readfirstlane(static_cast<int>(tile_bytes));
    if (lane < 32) lds_dma16(rsrc, __builtin_amdgcn_readfirstlane(lds), lane * 16, tb);
  }
}

// A lane's pieces of one gradient row into the dense [B, H, T, d] output:
// acc[mt][4j + i] holds element 32 mt + 8 j + 4 g + i, times f.  The RoPE
// pair partner of element x < d/2 is x + d/2, in tile mt + d/64 of the same
// lane, so the gradient goes back through the rotation in registers:
// x' = (x1 c - x2 s, x2 c + x1 s) gives (d1 c + d2 s, d2 c - d1 s).  The
// factors of position pos are formed as the forward's (freq: theta_j /
// (2 pi) of the pairs, or NULL for no rotation).
template <int D>
NAMOH_DEV void store_row_unrotated(float* __restrict__ dst, const f32x16 (&acc)[D / 32], float f,
                                   const double* __restrict__ freq, double pos, int g) {
  constexpr int MH = D / 64;
#pragma unroll
  for (int mt = 0; mt < MH; ++mt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int x = 32 * mt + 8 * j + 4 * g;
      float a[4], b2[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = acc[mt][4 * j + i] * f;
        b2[i] = acc[mt + MH][4 * j + i] * f;
      }
      if (freq != nullptr) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float2 w = rope_cs_rev(pos, freq[x + i]);
          const float d1 = a[i], d2 = b2[i];
          a[i] = d1 * w.x + d2 * w.y;
          b2[i] = d2 * w.x - d1 * w.y;
        }
      }
      *reinterpret_cast<float4*>(dst + x) = make_float4(a[0], a[1], a[2], a[3]);
      *reinterpret_cast<float4*>(dst + x + D / 2) = make_float4(b2[0], b2[1], b2[2], b2[3]);
    }
}

// Zero rows of the dense gradients for the (token, head) pairs the routing
// did not select (the others are written by the MFMA kernels): one float4
// of a row per thread, rows of D / 4 threads.
constexpr int kZeroThreads = 256;
template <int D>
__global__ __launch_bounds__(kZeroThreads) void k_bwd_zero_unrouted(
    const int32_t* __restrict__ topk_idx, int H, int T, int K, size_t rows,
    float* __restrict__ dq, float* __restrict__ dk, float* __restrict__ dv) {
  constexpr int C4 = D / 4, RPB = kZeroThreads / C4;
  const size_t row = static_cast<size_t>(block_x()) * RPB + thread_x() / C4;
  const int c4 = thread_x() % C4;
  if (row >= rows) return;
  const size_t bh = row / T;
  const int t = static_cast<int>(row - bh * T);
  const int b = static_cast<int>(bh / H), h = static_cast<int>(bh - (bh / H) * H);
  const int32_t* tk = topk_idx + (static_cast<size_t>(b) * T + t) * K;
  bool routed = false;
  for (int k0 = 0; k0 < K; k0 += 8) {   // eight independent loads per round
    int sv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) sv[u] = tk[min(k0 + u, K - 1)];
#pragma unroll
    for (int u = 0; u < 8; ++u) routed |= sv[u] == h;   // clamped repeats change nothing
  }
  if (routed) return;
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  const size_t o = row * D + 4 * c4;
  *reinterpret_cast<float4*>(dq + o) = z;
  *reinterpret_cast<float4*>(dk + o) = z;
  *reinterpret_cast<float4*>(dv + o) = z;
}

template <int D> struct BwdMfmaShape {
  static constexpr int MINB = D == 64 ? 2 : 1;   // workgroups per CU (key side)
  static constexpr int MINB_Q = 2;               // (query side; 3 at d = 64 spills)
};

// A work record checked before it addresses anything (the saved backward
// takes the list from the caller's workspace): its segment, rows and tiles
// inside the packed arrays, a whole item (the backward's list holds no
// key-range parts) and a block inside its segment.  A record that fails is
// skipped.
NAMOH_DEV bool bwd_item_ok(const WorkItem& it, int BH, int T, int Nr, int max_tiles) {
  if (it.s < 0 || it.s >= BH || it.n <= 0 || it.n > T || it.seg0 < 0 || it.seg0 > Nr - it.n)
    return false;
  const int nt = (it.n + kBN - 1) / kBN;
  return it.qb >= 0 && it.qb < (it.n + kBwdMfmaBlock - 1) / kBwdMfmaBlock && it.tile0 >= 0 &&
         it.tile0 <= max_tiles - nt && it.kt_lo >= 0 && it.kt_lo < it.kt_hi && it.kt_hi <= nt;
}

// The key side runs its own list of whole blocks, where every item passes
// this test.  It guards that list: were the key side given a list with
// key-range parts, it would take a split block once, whole, at its part 1
// and skip the other parts, so no block's dK, dV would be written twice.
NAMOH_DEV bool bwd_key_side_item(const WorkItem& it) {
  return item_parts(it.qh) <= 1 || item_part(it.qh) == 1;
}

// Query side: dQ~ of one (segment, 128-query block) item.
template <int D>
__global__ __launch_bounds__(kBwdMfmaThreads, BwdMfmaShape<D>::MINB_Q) void k_bwd_dq(
    const uint16_t* __restrict__ Qs, const uint16_t* __restrict__ dO,
    const float2* __restrict__ LD, const uint16_t* __restrict__ Kp,
    const uint16_t* __restrict__ Vp, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ meta,
    const int32_t* __restrict__ perm_token, const double* __restrict__ freq, int T,
    int rope_mode, float scale, float* __restrict__ dq, int packed, int BH, int Nr,
    int max_tiles, float* __restrict__ part, int part_rows) {
  constexpr int NT = kBwdMfmaThreads, BM = kBwdMfmaBlock;
  constexpr int KS = D / 16, MT = D / 32;
  constexpr int KPT = kBN * D / 8 / NT;
  constexpr size_t TS = static_cast<size_t>(kBN) * D;
  constexpr uint32_t TB = static_cast<uint32_t>(TS * 2);
  // K and V tiles double-buffered; the dQ products read the key tile
  // transposed (64 KB per workgroup at d = 128)
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kBN * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][kBN * D];
  WorkItem it;
  if (!my_item(items, meta, it) || !bwd_item_ok(it, BH, T, Nr, max_tiles)) return;
  // a key-range part of a split block adds its keys' share of dQ~ to the
  // block's partial rows (summed by the key-side kernel's merge workgroups)
  const int slot = item_slot(it.qh);
  if (slot >= 0 && (part == nullptr || (slot + 1) * BM > part_rows)) return;
  const int q0 = it.qb * BM;
  const int seg0 = it.seg0, n = it.n, tile0 = it.tile0;
  const int kt_lo = it.kt_lo, kt_end = it.kt_hi;
  const int tid = thread_x();
  const int wave = tid / 64, lane = tid % 64;
  const int c = lane & 31, g = lane >> 5;
  const int r = q0 + 32 * wave + c;
  const bool valid = r < n;
  const int wave_tiles = q0 + 32 * wave < n ? min(q0 + 32 * wave + 31, n - 1) / kBN + 1 : 0;
  const size_t prow = static_cast<size_t>(tile0) * kBN + (valid ? r : n - 1);

  // the first key and value tiles go in first, so their latency overlaps
  // the query operands' (one full wait covers both)
  const int tile0_s = __builtin_amdgcn_readfirstlane(tile0);
  const int kt_end_s = __builtin_amdgcn_readfirstlane(kt_end);
  const uint16_t* const bK = Kp + static_cast<size_t>(tile0_s) * TS;
  const uint16_t* const bV = Vp + static_cast<size_t>(tile0_s) * TS;
  const uint32_t nb = static_cast<uint32_t>(kt_end_s) * TB;
  const uint32_t voffR = tile_voffset<D / 8, NT>(tid);
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t lK0 = lds_address(&sK[0][0]);
  const uint32_t lK = lK0 + wave_s * kWave * 16;
  const uint32_t lV = lds_address(&sV[0][0]) + wave_s * kWave * 16;
  const TrOff<D> tro = tr_offsets<D>(lane);
  tile_dma<KPT, NT>(bK, nb, static_cast<uint32_t>(kt_lo) * TB, lK, voffR);
  tile_dma<KPT, NT>(bV, nb, static_cast<uint32_t>(kt_lo) * TB, lV, voffR);

  // the query's operands and statistics (padding rows: zero operands,
  // lse = +inf, so their probabilities are 0)
  bf16x8 qB[KS], doB[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qB[ks] = *reinterpret_cast<const bf16x8*>(Qs + prow * D + 16 * ks + 8 * g);
    doB[ks] = *reinterpret_cast<const bf16x8*>(dO + prow * D + 16 * ks + 8 * g);
  }
  const float2 ld = LD[prow];
  wait_vmcnt<0>();
  // every accumulator of the lane's query starts at -lse (scores) and -D
  // (probability gradients): one tuple each serves both key halves
  f32x16 init_l, init_d;
  {
    const float nl = valid ? -ld.x : -INFINITY, nd = valid ? -ld.y : 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      init_l[e] = nl;
      init_d[e] = nd;
    }
  }

  f32x16 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[mt][e] = 0.f;
  // Per tile: wait for K, V of tile kt; the barrier also ends every wave's
  // reads of the other stage (tile kt - 1), so K, V of tile kt + 1 go there
  // now, behind the tile's products.
  for (int kt = kt_lo; kt < kt_end; ++kt) {
    const int st = (kt - kt_lo) & 1;
    wait_vmcnt<0>();
    __syncthreads();
    const bool more = kt + 1 < kt_end;
    if (more) {
      const uint32_t tb = static_cast<uint32_t>(kt + 1) * TB;
      const int ns = st ^ 1;
      tile_dma<KPT, NT>(bK, nb, tb, lK + ns * TB, voffR);
      tile_dma<KPT, NT>(bV, nb, tb, lV + ns * TB, voffR);
    }
    if (kt < wave_tiles) {
      f32x16 S[2], dP[2];
      tile_rows_x_regs<D>(S, sK[st], qB, init_l, init_l, c, g);    // S^T - lse (log2 units)
      tile_rows_x_regs<D>(dP, sV[st], doB, init_d, init_d, c, g);  // dP^T - D
      const int key0 = kt * kBN;
      if (key0 + kBN - 1 > q0 + 32 * wave || key0 + kBN > n) {
        const int lim = min(r, n - 1) - key0 - 4 * g;   // key 32kk + 8j + 4g + i visible iff <= lim + 4g
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (32 * kk + 8 * j + i > lim) S[kk][4 * j + i] = -INFINITY;
      }
      bf16x8 dsB[4];
#pragma unroll
      for (int k2 = 0; k2 < 4; ++k2)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int a = 8 * (k2 & 1) + e;
          dsB[k2][e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(S[k2 >> 1][a]) * dP[k2 >> 1][a]);
        }
      rows_tposed_x_c<D>(acc, lK0 + st * TB, tro, dsB);   // dQ^T += K^T dS^T
    }
  }
  if (valid && slot >= 0) {   // the part's sum, unscaled and in the rotated frame
    store_row_unrotated<D>(part + (static_cast<size_t>(slot) * BM + (r - q0)) * D, acc, 1.f,
                           nullptr, 0.0, g);
  } else if (valid) {   // dq~ = scale sum_j dS k~_j, back through the query's rotation
    const int t = min(static_cast<unsigned>(perm_token[seg0 + r]), static_cast<unsigned>(T - 1));
    const double* fq = rope_mode == 2 ? nullptr : freq;
    const double pos = rope_mode == 0 ? r : t;
    const size_t o = packed ? static_cast<size_t>(seg0 + r) * D : (static_cast<size_t>(it.s) * T + t) * D;
    store_row_unrotated<D>(dq + o, acc, scale, fq, pos, g);
  }
}

// dQ rows of the split blocks: the sum of their parts' partial rows in part
// order, scaled and back through the query's rotation as k_bwd_dq stores a
// whole block's rows.  Run by the workgroups past the key-side kernel's work
// items (k_bwd_dq has finished by then); units are (split block, pass of
// NT / (D / 8) rows), each thread four rotation pairs (x, x + d/2) of a row.
constexpr int kDqMergeGroups = 64;
struct DqMerge {
  const SplitItem* splits;
  const int32_t* meta;
  const float* part;
  float* dq;
  int part_rows, packed, rope_mode;
  float scale;
  int BH, Nr;
};
template <int D, int NT>
NAMOH_DEV void dq_merge_units(const DqMerge& m, int unit0, int nunits_wg,
                              const int32_t* __restrict__ perm_token,
                              const double* __restrict__ freq, int T) {
  constexpr int BM = kBwdMfmaBlock;
  constexpr int TPR = D / 8;          // threads per row
  constexpr int RPP = NT / TPR;       // rows per pass
  constexpr int NPASS = (BM + RPP - 1) / RPP;
  // (the records come from the caller's workspace: the count and every
  // record are range-checked before use; at most part_rows / (2 BM) blocks)
  const int nsplit = min(max(m.meta[kMetaSplit], 0), m.part_rows / (2 * BM));
  const int tid = thread_x();
  const int sub = tid % TPR, rw = tid / TPR;
  const int x = 4 * sub;              // pairs x .. x + 3 with x + d/2 .. x + d/2 + 3
  for (int u = unit0; u < nsplit * NPASS; u += nunits_wg) {
    const int j = u / NPASS;
    const int ri = (u - j * NPASS) * RPP + rw;
    const SplitItem si = m.splits[j];
    const int q0 = si.qb * BM;
    const int r = q0 + ri;
    if (ri >= BM || si.qb < 0 || r >= si.n || si.n > T || si.s < 0 || si.s >= m.BH ||
        si.seg0 < 0 || si.seg0 > m.Nr - si.n || si.P < 2 || si.P > 8 || si.base < 0 ||
        (si.base + si.P) * BM > m.part_rows)
      continue;
    float a[4] = {0.f, 0.f, 0.f, 0.f}, b[4] = {0.f, 0.f, 0.f, 0.f};
    for (int p = 0; p < si.P; ++p) {
      const float* row = m.part + (static_cast<size_t>(si.base + p) * BM + ri) * D;
      const float4 u1 = *reinterpret_cast<const float4*>(row + x);
      const float4 u2 = *reinterpret_cast<const float4*>(row + x + D / 2);
      a[0] += u1.x; a[1] += u1.y; a[2] += u1.z; a[3] += u1.w;
      b[0] += u2.x; b[1] += u2.y; b[2] += u2.z; b[3] += u2.w;
    }
    const int t = min(static_cast<unsigned>(perm_token[si.seg0 + r]), static_cast<unsigned>(T - 1));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[i] *= m.scale;
      b[i] *= m.scale;
    }
    if (m.rope_mode != 2) {
      const double pos = m.rope_mode == 0 ? r : t;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float2 w = rope_cs_rev(pos, freq[x + i]);
        const float d1 = a[i], d2 = b[i];
        a[i] = d1 * w.x + d2 * w.y;
        b[i] = d2 * w.x - d1 * w.y;
      }
    }
    const size_t o = m.packed ? static_cast<size_t>(si.seg0 + r) * D
                              : (static_cast<size_t>(si.s) * T + t) * D;
    *reinterpret_cast<float4*>(m.dq + o + x) = make_float4(a[0], a[1], a[2], a[3]);
    *reinterpret_cast<float4*>(m.dq + o + x + D / 2) = make_float4(b[0], b[1], b[2], b[3]);
  }
}

// Key side: dK~ and dV of one (segment, 128-key block) item.
template <int D>
__global__ __launch_bounds__(kBwdMfmaThreads, BwdMfmaShape<D>::MINB) void k_bwd_dkdv(
    const uint16_t* __restrict__ Qs, const uint16_t* __restrict__ dO,
    const float2* __restrict__ LD, const uint16_t* __restrict__ Kp,
    const uint16_t* __restrict__ Vp, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ meta, const int32_t* __restrict__ perm_token,
    const double* __restrict__ freq, int T, int rope_mode, float* __restrict__ dk,
    float* __restrict__ dv, int packed, int BH, int Nr, int max_tiles, int n_list, DqMerge dqm) {
  constexpr int NT = kBwdMfmaThreads, BM = kBwdMfmaBlock;
  constexpr int KS = D / 16, MT = D / 32;
  constexpr int KPT = kBN * D / 8 / NT;
  constexpr size_t TS = static_cast<size_t>(kBN) * D;
  constexpr uint32_t TB = static_cast<uint32_t>(TS * 2);
  constexpr uint32_t LB = kBN * sizeof(float2);
  // query and output-gradient tiles, read row-major for S and dP and
  // transposed for dV and dK
  __shared__ __attribute__((aligned(16))) uint16_t sQ[2][kBN * D];
  __shared__ __attribute__((aligned(16))) uint16_t sdO[2][kBN * D];
  __shared__ __attribute__((aligned(16))) float2 sLD[2][kBN];
  WorkItem it;
  if (block_x() >= n_list) {   // past the work list: the split blocks' dQ rows
    dq_merge_units<D, NT>(dqm, block_x() - n_list, static_cast<int>(gridDim.x) - n_list,
                          perm_token, freq, T);
    return;
  }
  if (!my_item(items, meta, it) || !bwd_item_ok(it, BH, T, Nr, max_tiles) ||
      !bwd_key_side_item(it))
    return;
  const int seg0 = it.seg0, n = it.n, tile0 = it.tile0;
  const int nkb = (n + BM - 1) / BM;
  const int j0 = (nkb - 1 - it.qb) * BM;
  const int ntiles = (n + kBN - 1) / kBN;
  const int qt0 = j0 / kBN;
  const int tid = thread_x();
  const int wave = tid / 64, lane = tid % 64;
  const int c = lane & 31, g = lane >> 5;
  const int jw0 = j0 + 32 * wave;   // the wave's first key
  const int j = jw0 + c;
  const bool valid = j < n;
  const bool wave_on = jw0 < n;
  const size_t prow = static_cast<size_t>(tile0) * kBN + (valid ? j : n - 1);

  // the first query tile goes in first, so its latency overlaps the key
  // operands' (one full wait covers both)
  const int tile0_s = __builtin_amdgcn_readfirstlane(tile0);
  const int nt_s = __builtin_amdgcn_readfirstlane(ntiles);
  const int qt0_s = __builtin_amdgcn_readfirstlane(qt0);
  const uint16_t* const bQ = Qs + static_cast<size_t>(tile0_s) * TS;
  const uint16_t* const bdO = dO + static_cast<size_t>(tile0_s) * TS;
  const float2* const bLD = LD + static_cast<size_t>(tile0_s) * kBN;
  const uint32_t nb = static_cast<uint32_t>(nt_s) * TB;
  const uint32_t nbl = static_cast<uint32_t>(nt_s) * LB;
  const uint32_t voffR = tile_voffset<D / 8, NT>(tid);
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t lQ0 = lds_address(&sQ[0][0]), ldO0 = lds_address(&sdO[0][0]);
  const uint32_t lQ = lQ0 + wave_s * kWave * 16;
  const uint32_t ldO = ldO0 + wave_s * kWave * 16;
  const uint32_t lLD = lds_address(&sLD[0][0]);
  const TrOff<D> tro = tr_offsets<D>(lane);
  auto issue = [&](int qt, int stage) {
    const uint32_t tb = static_cast<uint32_t>(qt) * TB;
    tile_dma<KPT, NT>(bQ, nb, tb, lQ + stage * TB, voffR);
    tile_dma<KPT, NT>(bdO, nb, tb, ldO + stage * TB, voffR);
    ld_tile_dma(bLD, nbl, static_cast<uint32_t>(qt) * LB, lLD + stage * LB, wave_s, lane);
  };
  issue(qt0_s, 0);

  bf16x8 kB[KS], vB[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kB[ks] = *reinterpret_cast<const bf16x8*>(Kp + prow * D + 16 * ks + 8 * g);
    vB[ks] = *reinterpret_cast<const bf16x8*>(Vp + prow * D + 16 * ks + 8 * g);
  }
  wait_vmcnt<0>();
  if (!valid) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) kB[ks][e] = vB[ks][e] = static_cast<__bf16>(0.f);
  }

  f32x16 aK[MT], aV[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) aK[mt][e] = aV[mt][e] = 0.f;
  for (int qt = qt0; qt < ntiles; ++qt) {
    const int st = (qt - qt0) & 1;
    wait_vmcnt<0>();
    __syncthreads();
    if (qt + 1 < ntiles) issue(qt + 1, st ^ 1);
    const int i0 = qt * kBN;
    // queries i0 .. i0 + 63 against the wave's keys: none visible when the
    // tile ends before the first key
    if (wave_on && i0 + kBN - 1 >= jw0) {
      // accumulator starts: -lse and -D of query rows 32kk + 8jj + 4g + i
      f32x16 S[2], dP[2];
      {
        f32x16 il[2], id[2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const float4* p = reinterpret_cast<const float4*>(&sLD[st][32 * kk + 8 * jj + 4 * g]);
            const float4 a = p[0], bq = p[1];
            il[kk][4 * jj] = -a.x;     id[kk][4 * jj] = -a.y;
            il[kk][4 * jj + 1] = -a.z; id[kk][4 * jj + 1] = -a.w;
            il[kk][4 * jj + 2] = -bq.x; id[kk][4 * jj + 2] = -bq.y;
            il[kk][4 * jj + 3] = -bq.z; id[kk][4 * jj + 3] = -bq.w;
          }
        tile_rows_x_regs<D>(S, sQ[st], kB, il[0], il[1], c, g);    // S - lse (log2 units)
        tile_rows_x_regs<D>(dP, sdO[st], vB, id[0], id[1], c, g);  // dP - D
      }
      if (i0 < jw0 + 32) {   // the diagonal: key j visible to query i iff j <= i
        const int lim = j - i0 - 4 * g;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (32 * kk + 8 * jj + i < lim) S[kk][4 * jj + i] = -INFINITY;
      }
      bf16x8 pB[4], dsB[4];
#pragma unroll
      for (int k2 = 0; k2 < 4; ++k2)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int a = 8 * (k2 & 1) + e;
          const float p = __builtin_amdgcn_exp2f(S[k2 >> 1][a]);
          pB[k2][e] = static_cast<__bf16>(p);
          dsB[k2][e] = static_cast<__bf16>(p * dP[k2 >> 1][a]);
        }
      rows_tposed_x_c<D>(aV, ldO0 + st * TB, tro, pB);   // dV^T += dO^T P
      rows_tposed_x_c<D>(aK, lQ0 + st * TB, tro, dsB);   // dK^T += Q^T dS
    }
  }
  if (valid) {
    // the queries were scaled by scale * log2 e: dk~ = ln 2 * sum dS Qs,
    // back through the key's rotation; dv as it is
    const int t = min(static_cast<unsigned>(perm_token[seg0 + j]), static_cast<unsigned>(T - 1));
    const size_t o = packed ? static_cast<size_t>(seg0 + j) * D : (static_cast<size_t>(it.s) * T + t) * D;
    const double* fq = rope_mode == 2 ? nullptr : freq;
    const double pos = rope_mode == 0 ? j : t;
    store_row_unrotated<D>(dk + o, aK, kLn2, fq, pos, g);
    store_row_unrotated<D>(dv + o, aV, 1.f, nullptr, 0.0, g);
  }
}

// Key side at d = 128 with two waves per SIMD: eight waves, wave w takes the
// keys of group w mod 4 (32 keys, as in k_bwd_dkdv) against query half
// w / 4 (rows 32 qh .. 32 qh + 31) of every query tile, so S, dP, P and dS
// are half as large per wave and a SIMD interleaves two waves of one
// workgroup (k_bwd_dkdv's 430 registers allow one).  The two halves' dK and
// dV partials of a key are summed through LDS at the end.
template <int D>
__global__ __launch_bounds__(2 * kBwdMfmaThreads, 1) void k_bwd_dkdv8(
    const uint16_t* __restrict__ Qs, const uint16_t* __restrict__ dO,
    const float2* __restrict__ LD, const uint16_t* __restrict__ Kp,
    const uint16_t* __restrict__ Vp, const WorkItem* __restrict__ items,
    const int32_t* __restrict__ meta, const int32_t* __restrict__ perm_token,
    const double* __restrict__ freq, int T, int rope_mode, float* __restrict__ dk,
    float* __restrict__ dv, int packed, int BH, int Nr, int max_tiles, int n_list, DqMerge dqm) {
  constexpr int NT = 2 * kBwdMfmaThreads, BM = kBwdMfmaBlock;
  constexpr int KS = D / 16, MT = D / 32;
  constexpr int KPT = kBN * D / 8 / NT;
  constexpr size_t TS = static_cast<size_t>(kBN) * D;
  constexpr uint32_t TB = static_cast<uint32_t>(TS * 2);
  constexpr uint32_t LB = kBN * sizeof(float2);
  static_assert(KPT >= 1 && KPT * NT * 8 == kBN * D, "tile/thread mismatch");
  // query and output-gradient tiles, read row-major for S and dP and
  // transposed for dV and dK
  __shared__ __attribute__((aligned(16))) uint16_t sQ[2][kBN * D];
  __shared__ __attribute__((aligned(16))) uint16_t sdO[2][kBN * D];
  __shared__ __attribute__((aligned(16))) float2 sLD[2][kBN];
  // the partials of query half 1, one 2 * MT * 16 * 64-float block per key
  // group: groups 0 and 1 in the tile stages once the loop is done, groups
  // 2 and 3 here (one workgroup per compute unit: 129 KB at d = 128)
  __shared__ __attribute__((aligned(16))) float sPart[2][2 * MT * 16 * 64];
  static_assert(sizeof(sQ) >= 2 * MT * 16 * 64 * sizeof(float), "partial staging");
  WorkItem it;
  if (block_x() >= n_list) {   // past the work list: the split blocks' dQ rows
    dq_merge_units<D, NT>(dqm, block_x() - n_list, static_cast<int>(gridDim.x) - n_list,
                          perm_token, freq, T);
    return;
  }
  if (!my_item(items, meta, it) || !bwd_item_ok(it, BH, T, Nr, max_tiles) ||
      !bwd_key_side_item(it))
    return;
  const int seg0 = it.seg0, n = it.n, tile0 = it.tile0;
  const int nkb = (n + BM - 1) / BM;
  const int j0 = (nkb - 1 - it.qb) * BM;
  const int ntiles = (n + kBN - 1) / kBN;
  const int qt0 = j0 / kBN;
  const int tid = thread_x();
  const int wave = tid / 64, lane = tid % 64;
  const int kgw = wave % 4, qh = wave / 4;   // key group, query half
  const int c = lane & 31, g = lane >> 5;
  const int jw0 = j0 + 32 * kgw;   // the wave's first key
  const int j = jw0 + c;
  const bool valid = j < n;
  const bool wave_on = jw0 < n;
  const size_t prow = static_cast<size_t>(tile0) * kBN + (valid ? j : n - 1);

  // the first query tile goes in first, so its latency overlaps the key
  // operands' (one full wait covers both)
  const int tile0_s = __builtin_amdgcn_readfirstlane(tile0);
  const int nt_s = __builtin_amdgcn_readfirstlane(ntiles);
  const int qt0_s = __builtin_amdgcn_readfirstlane(qt0);
  const int qh_s = __builtin_amdgcn_readfirstlane(qh);
  const uint16_t* const bQ = Qs + static_cast<size_t>(tile0_s) * TS;
  const uint16_t* const bdO = dO + static_cast<size_t>(tile0_s) * TS;
  const float2* const bLD = LD + static_cast<size_t>(tile0_s) * kBN;
  const uint32_t nb = static_cast<uint32_t>(nt_s) * TB;
  const uint32_t nbl = static_cast<uint32_t>(nt_s) * LB;
  const uint32_t voffR = tile_voffset<D / 8, NT>(tid);
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t lQ0 = lds_address(&sQ[0][0]), ldO0 = lds_address(&sdO[0][0]);
  const uint32_t lQ = lQ0 + wave_s * kWave * 16;
  const uint32_t ldO = ldO0 + wave_s * kWave * 16;
  const uint32_t lLD = lds_address(&sLD[0][0]);
  const TrOff<D> tro = tr_offsets<D>(lane);
  auto issue = [&](int qt, int stage) {
    const uint32_t tb = static_cast<uint32_t>(qt) * TB;
    tile_dma<KPT, NT>(bQ, nb, tb, lQ + stage * TB, voffR);
    tile_dma<KPT, NT>(bdO, nb, tb, ldO + stage * TB, voffR);
    ld_tile_dma(bLD, nbl, static_cast<uint32_t>(qt) * LB, lLD + stage * LB, wave_s, lane);
  };
  issue(qt0_s, 0);

  bf16x8 kB[KS], vB[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kB[ks] = *reinterpret_cast<const bf16x8*>(Kp + prow * D + 16 * ks + 8 * g);
    vB[ks] = *reinterpret_cast<const bf16x8*>(Vp + prow * D + 16 * ks + 8 * g);
  }
  wait_vmcnt<0>();
  if (!valid) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) kB[ks][e] = vB[ks][e] = static_cast<__bf16>(0.f);
  }

  f32x16 aK[MT], aV[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) aK[mt][e] = aV[mt][e] = 0.f;
  for (int qt = qt0; qt < ntiles; ++qt) {
    const int st = (qt - qt0) & 1;
    wait_vmcnt<0>();
    __syncthreads();
    if (qt + 1 < ntiles) issue(qt + 1, st ^ 1);
    const int i0 = qt * kBN + 32 * qh_s;   // the wave's first query of the tile
    // its 32 queries against its keys: none visible when they end before
    // the first key
    if (wave_on && i0 + 31 >= jw0) {
      // accumulator starts: -lse and -D of query rows 8jj + 4g + i
      f32x16 S, dP;
      {
        f32x16 il, id;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const float4* p = reinterpret_cast<const float4*>(&sLD[st][32 * qh_s + 8 * jj + 4 * g]);
          const float4 a = p[0], bq = p[1];
          il[4 * jj] = -a.x;     id[4 * jj] = -a.y;
          il[4 * jj + 1] = -a.z; id[4 * jj + 1] = -a.w;
          il[4 * jj + 2] = -bq.x; id[4 * jj + 2] = -bq.y;
          il[4 * jj + 3] = -bq.z; id[4 * jj + 3] = -bq.w;
        }
        tile_half_x_regs<D>(S, sQ[st], kB, il, qh_s, c, g);    // S - lse (log2 units)
        tile_half_x_regs<D>(dP, sdO[st], vB, id, qh_s, c, g);  // dP - D
      }
      if (i0 < jw0 + 32) {   // the diagonal: key j visible to query i iff j <= i
        const int lim = j - i0 - 4 * g;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (8 * jj + i < lim) S[4 * jj + i] = -INFINITY;
      }
      bf16x8 pB[2], dsB[2];
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int a = 8 * kh + e;
          const float p = __builtin_amdgcn_exp2f(S[a]);
          pB[kh][e] = static_cast<__bf16>(p);
          dsB[kh][e] = static_cast<__bf16>(p * dP[a]);
        }
      rows_tposed_half_x_c<D>(aV, ldO0 + st * TB, tro, pB, qh_s);   // dV^T += dO^T P
      rows_tposed_half_x_c<D>(aK, lQ0 + st * TB, tro, dsB, qh_s);   // dK^T += Q^T dS
    }
  }
  // the two query halves' partials of each key: half 1 hands its dK partial
  // to half 0 and half 0 its dV partial to half 1 through LDS (the tile
  // stages of the key group, idle by now, or sPart); half 0 then stores dK,
  // half 1 dV, so all eight waves share the epilogue
  __syncthreads();   // every wave is done with the tiles
  float* const stage = kgw == 0 ? reinterpret_cast<float*>(&sQ[0][0])
                     : kgw == 1 ? reinterpret_cast<float*>(&sdO[0][0])
                                : &sPart[kgw - 2][0];
  float* const give = stage + (qh == 1 ? 0 : MT * 16 * 64);   // dK from half 1, dV from half 0
  float* const take = stage + (qh == 1 ? MT * 16 * 64 : 0);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) give[(mt * 16 + e) * 64 + lane] = qh == 1 ? aK[mt][e] : aV[mt][e];
  __syncthreads();
  f32x16 (&mine)[MT] = qh == 1 ? aV : aK;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) mine[mt][e] += take[(mt * 16 + e) * 64 + lane];
  if (valid) {
    const int t = min(static_cast<unsigned>(perm_token[seg0 + j]), static_cast<unsigned>(T - 1));
    const size_t o = packed ? static_cast<size_t>(seg0 + j) * D : (static_cast<size_t>(it.s) * T + t) * D;
    if (qh == 0) {
      // the queries were scaled by scale * log2 e: dk~ = ln 2 * sum dS Qs,
      // back through the key's rotation
      const double* fq = rope_mode == 2 ? nullptr : freq;
      const double pos = rope_mode == 0 ? j : t;
      store_row_unrotated<D>(dk + o, aK, kLn2, fq, pos, g);
    } else {
      store_row_unrotated<D>(dv + o, aV, 1.f, nullptr, 0.0, g);   // dv as it is
    }
  }
}

// ---------------------------------------------------------------------------
struct BwdWs {
  float *Qr, *Kr, *Vp, *dOp, *dQr, *dKr, *dVp, *lse, *Dr, *dgp;
  int32_t *seg_of, *kslot;
  size_t bytes;
};

static BwdWs carve_bwd(void* ws, int B, int T, int K, int d) {
  const size_t Nr = static_cast<size_t>(B) * T * K;
  Carver cv(ws);
  BwdWs w;
  w.Qr = cv.take<float>(Nr * d);
  w.Kr = cv.take<float>(Nr * d);
  w.Vp = cv.take<float>(Nr * d);
  w.dOp = cv.take<float>(Nr * d);
  w.dQr = cv.take<float>(Nr * d);
  w.dKr = cv.take<float>(Nr * d);
  w.dVp = cv.take<float>(Nr * d);
  w.lse = cv.take<float>(Nr);
  w.Dr = cv.take<float>(Nr);
  w.dgp = cv.take<float>(Nr);
  w.seg_of = cv.take<int32_t>(Nr);
  w.kslot = cv.take<int32_t>(Nr);
  w.bytes = cv.off;
  return w;
}

struct BwdMfmaWs {
  void* attn;
  float* lse;
  uint16_t *Qs, *dO, *Vp;
  float2* LD;
  WorkItem* kitems;   // the key side's work list (whole blocks)
  int32_t* kmeta;
  size_t rows, bytes;
};

static BwdMfmaWs carve_bwd_mfma(void* ws, int B, int T, int H, int K, int d) {
  const size_t Nr = static_cast<size_t>(B) * T * K;
  const size_t BH = static_cast<size_t>(B) * H;
  Carver cv(ws);
  BwdMfmaWs w;
  w.rows = (Nr / kBN + BH + 1) * kBN;   // every 64-row tile a segment can use
  w.attn = cv.take<char>(attn_workspace_bytes(B, T, H, K, d, 1));
  w.lse = cv.take<float>(Nr);
  w.Qs = cv.take<uint16_t>(w.rows * d);
  w.dO = cv.take<uint16_t>(w.rows * d);
  w.Vp = cv.take<uint16_t>(w.rows * d);
  w.LD = cv.take<float2>(w.rows);
  AttnTiles tl;
  attn_stats_tiles(nullptr, B, T, H, K, d, tl);
  w.kitems = cv.take<WorkItem>(static_cast<size_t>(tl.max_items));
  w.kmeta = cv.take<int32_t>(kMetaCount);
  w.bytes = cv.off;
  return w;
}

static bool bwd_uses_mfma(int dtype, int d) { return dtype == 1 && (d == 64 || d == 128); }

// Compute units of the current device (the period of the hardware's
// workgroup placement; 0 turns the alternating placement off).
static int bwd_cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return n;
}

// Large enough for either path (the size query takes no dtype).
size_t attn_bwd_workspace_bytes(int B, int T, int H, int K, int d) {
  size_t bytes = carve_bwd(nullptr, B, T, K, d).bytes;
  if (d == 64 || d == 128) bytes = std::max(bytes, carve_bwd_mfma(nullptr, B, T, H, K, d).bytes);
  return bytes;
}

template <int D>
static hipError_t run_bwd_mfma(const void* q, const void* k, const void* v, int B, int T, int H,
                               int K, float rope_base, int rope_mode, float scale,
                               const int32_t* topk_idx, const float* gates,
                               const int32_t* seg_offsets, const int32_t* perm_token,
                               const float* dout, float* dq, float* dk, float* dv,
                               float* dgates, void* ws, hipStream_t st, bool packed,
                               bool saved) {
  const BwdMfmaWs w = carve_bwd_mfma(ws, B, T, H, K, D);
  const int BH = B * H;
  const int Nr = B * T * K;
  AttnTiles tl;
  hipError_t e = hipSuccess;
  if (saved)   // launch_train_fwd left the statistics and tiles in this workspace
    attn_stats_tiles(w.attn, B, T, H, K, D, tl);
  else
    e = launch_attn_stats(q, k, v, B, T, H, K, D, rope_base, rope_mode, scale, seg_offsets,
                          perm_token, w.lse, w.attn, tl, st);
  if (e != hipSuccess) return e;
  if (tl.BM != kBwdMfmaBlock || static_cast<size_t>(tl.max_tiles) * kBN > w.rows)
    return hipErrorInvalidValue;   // the forward's blocks and tiles must match these kernels
  if (!packed) {   // dense gradients: rows of tokens not routed to the head are zero
    const size_t rows = static_cast<size_t>(BH) * T;
    constexpr int RPB = kZeroThreads / (D / 4);
    k_bwd_zero_unrouted<D><<<static_cast<unsigned>((rows + RPB - 1) / RPB), kZeroThreads, 0,
                             st>>>(topk_idx, H, T, K, rows, dq, dk, dv);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const double* freq = tl.freq;
  prof_mark("bwd_pack", true, st);
  // the key side takes whole blocks: its own list, heaviest first, placed for
  // its own resident workgroups (the query side runs the forward's list with
  // its key-range parts)
  const int cus = bwd_cu_count();
  const KeyList kl{w.kitems, w.kmeta, tl.max_items, cus, cus * BwdMfmaShape<D>::MINB};
  k_bwd_pack<D><<<static_cast<unsigned>(tl.max_tiles) + 1, kBwdPackThreads, 0, st>>>(
      static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(v), dout, topk_idx, gates,
      seg_offsets, perm_token, freq, tl.h, w.lse, BH, H, T, K, Nr, rope_mode, scale * kLog2e,
      w.Qs, w.dO, w.Vp, w.LD, dgates, kl);
  prof_mark("bwd_pack", false, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  prof_mark("bwd_dq", true, st);
  k_bwd_dq<D><<<static_cast<unsigned>(tl.max_items), kBwdMfmaThreads, 0, st>>>(
      w.Qs, w.dO, w.LD, tl.Kp, w.Vp, tl.items, tl.meta, perm_token, freq, T, rope_mode,
      scale, dq, packed ? 1 : 0, BH, Nr, tl.max_tiles, tl.part, tl.part_rows);
  prof_mark("bwd_dq", false, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  prof_mark("bwd_dkdv", true, st);
  // the key-side grid carries kDqMergeGroups more workgroups, which sum the
  // split blocks' dQ partials (the query-side kernel has finished)
  const DqMerge dqm{tl.splits, tl.meta, tl.part, dq, tl.part_rows, packed ? 1 : 0, rope_mode,
                    scale, BH, Nr};
  const unsigned kgrid = static_cast<unsigned>(tl.max_items) + kDqMergeGroups;
  if constexpr (D == 128)
    k_bwd_dkdv8<D><<<kgrid, 2 * kBwdMfmaThreads, 0, st>>>(
        w.Qs, w.dO, w.LD, tl.Kp, w.Vp, w.kitems, w.kmeta, perm_token, freq, T,
        rope_mode, dk, dv, packed ? 1 : 0, BH, Nr, tl.max_tiles, tl.max_items, dqm);
  else
    k_bwd_dkdv<D><<<kgrid, kBwdMfmaThreads, 0, st>>>(
        w.Qs, w.dO, w.LD, tl.Kp, w.Vp, w.kitems, w.kmeta, perm_token, freq, T,
        rope_mode, dk, dv, packed ? 1 : 0, BH, Nr, tl.max_tiles, tl.max_items, dqm);
  prof_mark("bwd_dkdv", false, st);
  return hipGetLastError();
}

template <int D, bool BF16>
static hipError_t run_bwd(const void* q, const void* k, const void* v, int B, int T, int H, int K,
                          float rope_base, int rope_mode, float scale, const int32_t* topk_idx,
                          const float* gates, const int32_t* seg_offsets,
                          const int32_t* perm_token, const float* dout, float* dq, float* dk,
                          float* dv, float* dgates, void* ws, hipStream_t st, bool packed) {
  const BwdWs w = carve_bwd(ws, B, T, K, D);
  const int BH = B * H;
  const int Nr = B * T * K;
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  hipError_t e = hipSuccess;
  if (!packed) {   // dense gradients: rows of tokens not routed to the head are zero
    const size_t n4 = static_cast<size_t>(BH) * T * D / 4;
    k_bwd_zero<<<static_cast<unsigned>((n4 + 255) / 256), 256, 0, st>>>(
        reinterpret_cast<float4*>(dq), reinterpret_cast<float4*>(dk),
        reinterpret_cast<float4*>(dv), n4);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  constexpr int RW = 256 / (D / 16);
  const unsigned rgrid = static_cast<unsigned>((Nr + RW - 1) / RW);
  k_bwd_gather<D, BF16><<<rgrid, 256, 0, st>>>(q, k, v, topk_idx, gates, dout, seg_offsets,
                                               perm_token, BH, H, T, K, Nr, rope_mode, log_base,
                                               w.Qr, w.Kr, w.Vp, w.dOp, w.seg_of, w.kslot);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  constexpr int RB = BwdShape<D>::RB;
  const dim3 sgrid(static_cast<unsigned>((T + RB - 1) / RB), static_cast<unsigned>(BH));
  k_bwd_q<D><<<sgrid, kBwdWgThreads, 0, st>>>(w.Qr, w.Kr, w.Vp, w.dOp, dout, seg_offsets,
                                            perm_token, H, T, Nr, scale, w.lse, w.Dr, w.dgp,
                                            w.dQr);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_bwd_kv<D><<<sgrid, kBwdWgThreads, 0, st>>>(w.Qr, w.Kr, w.Vp, w.dOp, w.lse, w.Dr, seg_offsets,
                                             T, Nr, scale, w.dKr, w.dVp);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_bwd_scatter<D><<<rgrid, 256, 0, st>>>(w.dQr, w.dKr, w.dVp, w.dgp, w.seg_of, w.kslot,
                                          seg_offsets, perm_token, BH, H, T, K, Nr, rope_mode,
                                          log_base, dq, dk, dv, dgates, packed ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const void* q, const void* k, const void* v, int dtype, int B, int T,
                           int H, int K, int d, float rope_base, int rope_mode, float scale,
                           const int32_t* topk_idx, const float* gates,
                           const int32_t* seg_offsets, const int32_t* perm_token,
                           const float* dout, float* dq, float* dk, float* dv, float* dgates,
                           void* ws, hipStream_t st, bool packed, bool saved) {
#define NAMOH_BWD(DD, BF)                                                                      \
  return run_bwd<DD, BF>(q, k, v, B, T, H, K, rope_base, rope_mode, scale, topk_idx, gates,   \
                         seg_offsets, perm_token, dout, dq, dk, dv, dgates, ws, st, packed)
  if (bwd_uses_mfma(dtype, d)) {
    if (d == 64)
      return run_bwd_mfma<64>(q, k, v, B, T, H, K, rope_base, rope_mode, scale, topk_idx, gates,
                              seg_offsets, perm_token, dout, dq, dk, dv, dgates, ws, st, packed,
                              saved);
    return run_bwd_mfma<128>(q, k, v, B, T, H, K, rope_base, rope_mode, scale, topk_idx, gates,
                             seg_offsets, perm_token, dout, dq, dk, dv, dgates, ws, st, packed,
                             saved);
  }
  if (saved) return hipErrorInvalidValue;   // (the host checks: matrix-core path only)
  if (dtype == 1) NAMOH_BWD(32, true);
  if (d == 32) NAMOH_BWD(32, false);
  if (d == 64) NAMOH_BWD(64, false);
  NAMOH_BWD(128, false);
#undef NAMOH_BWD
}

bool attn_train_supported(int dtype, int d) { return bwd_uses_mfma(dtype, d); }

// Training forward: the forward with the row statistics into the backward's
// workspace (what launch_attn_bwd with saved = true reads back), and the
// layer output combined from its f32 head outputs.
hipError_t launch_train_fwd(const void* q, const void* k, const void* v, int dtype, int B,
                            int T, int H, int K, int d, float rope_base, int rope_mode,
                            float scale, const float* gates, const int32_t* seg_offsets,
                            const int32_t* perm_token, const int32_t* slot_pos, void* out,
                            int out_dtype, void* ws, hipStream_t st) {
  if (!bwd_uses_mfma(dtype, d)) return hipErrorInvalidValue;
  const BwdMfmaWs w = carve_bwd_mfma(ws, B, T, H, K, d);
  AttnTiles tl;
  hipError_t e = launch_attn_stats(q, k, v, B, T, H, K, d, rope_base, rope_mode, scale,
                                   seg_offsets, perm_token, w.lse, w.attn, tl, st);
  if (e != hipSuccess) return e;
  return launch_combine_f32(tl.h, gates, slot_pos, static_cast<long>(B) * T, K, d, B * T * K,
                            out, out_dtype, st);
}

// ---------------------------------------------------------------------------
// Router gradient through the gates (selection fixed): one thread per token.
// SOFTMAX_SELECTED: dl_j = g_j (dg_j - sum_k g_k dg_k) on the selected heads;
// SOFTMAX_ALL (and the loss-free balancing gates): dl = a (da - <a, da>).
// One workgroup per kRouteBwdTokens tokens: one thread per token forms the
// token's gradient row in LDS (dense, H entries), then the block of rows is
// written out with consecutive threads on consecutive floats.
constexpr int kRouteBwdTokens = 128;
__global__ __launch_bounds__(256) void k_route_bwd(const float* __restrict__ logits,
                                                   const int32_t* __restrict__ topk_idx,
                                                   const float* __restrict__ gates,
                                                   const float* __restrict__ dgates, long BT,
                                                   int H, int K, int gate_mode,
                                                   float* __restrict__ dlogits) {
  __shared__ float s_dl[kRouteBwdTokens * 64];
  const int tid = thread_x();
  const long tok0 = static_cast<long>(block_x()) * kRouteBwdTokens;
  const int ntok = static_cast<int>(min(static_cast<long>(kRouteBwdTokens), BT - tok0));
  for (int i = tid; i < ntok * H; i += 256) s_dl[i] = 0.f;
  __syncthreads();
  if (tid < ntok) {
    const long tok = tok0 + tid;
    const float* l = logits + tok * H;
    const int32_t* tk = topk_idx + tok * K;
    const float* g = gates + tok * K;
    const float* dg = dgates + tok * K;
    float* dl = s_dl + tid * H;
    bool valid = true;
    for (int kk = 0; kk < K; ++kk) valid &= tk[kk] >= 0 && tk[kk] < H;
    if (valid) {   // not a selection: no gradient
      if (gate_mode == 0) {
        float sum = 0.f;
        for (int kk = 0; kk < K; ++kk) sum = fmaf(g[kk], dg[kk], sum);
        for (int kk = 0; kk < K; ++kk) dl[tk[kk]] = g[kk] * (dg[kk] - sum);
      } else {
        float mx = l[0];
        for (int h = 1; h < H; ++h) mx = fmaxf(mx, l[h]);
        float z = 0.f;
        for (int h = 0; h < H; ++h) z += expf(l[h] - mx);
        const float iz = 1.f / z;
        float sum = 0.f;   // <a, da>
        for (int kk = 0; kk < K; ++kk) sum = fmaf(expf(l[tk[kk]] - mx) * iz, dg[kk], sum);
        for (int h = 0; h < H; ++h) dl[h] = -expf(l[h] - mx) * iz * sum;
        for (int kk = 0; kk < K; ++kk) dl[tk[kk]] += expf(l[tk[kk]] - mx) * iz * dg[kk];
      }
    }
  }
  __syncthreads();
  float* out = dlogits + tok0 * H;
  for (int i = tid; i < ntok * H; i += 256) out[i] = s_dl[i];
}

hipError_t launch_route_bwd(const float* logits, const int32_t* topk_idx, const float* gates,
                            const float* dgates, int B, int T, int H, int K, int gate_mode,
                            float* dlogits, hipStream_t st) {
  const long BT = static_cast<long>(B) * T;
  if (H > 64) return hipErrorInvalidValue;   // the API allows H <= 64
  k_route_bwd<<<static_cast<unsigned>((BT + kRouteBwdTokens - 1) / kRouteBwdTokens), 256, 0, st>>>(
      logits, topk_idx, gates, dgates, BT, H, K, gate_mode, dlogits);
  return hipGetLastError();
}

}  // namespace namoh
