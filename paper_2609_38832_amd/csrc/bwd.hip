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
  for (int kk = 0; kk < K; ++kk)
    if (topk_idx[(static_cast<size_t>(b) * T + t) * K + kk] == h) ks = kk;
  const float g = ks >= 0 ? gates[(static_cast<size_t>(b) * T + t) * K + ks] : 0.f;
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
  if constexpr (LPR == 2) x += __shfl_xor(x, 1);
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
    float* __restrict__ dgates) {
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
  if (j0 == 0 && kslot[r] >= 0) dgates[(static_cast<size_t>(b) * T + t) * K + kslot[r]] = dgp[r];
  const size_t src = static_cast<size_t>(r) * D;
  const size_t dst = (static_cast<size_t>(s) * T + t) * D;
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

size_t attn_bwd_workspace_bytes(int B, int T, int /*H*/, int K, int d) {
  return carve_bwd(nullptr, B, T, K, d).bytes;
}

template <int D, bool BF16>
static hipError_t run_bwd(const void* q, const void* k, const void* v, int B, int T, int H, int K,
                          float rope_base, int rope_mode, float scale, const int32_t* topk_idx,
                          const float* gates, const int32_t* seg_offsets,
                          const int32_t* perm_token, const float* dout, float* dq, float* dk,
                          float* dv, float* dgates, void* ws, hipStream_t st) {
  const BwdWs w = carve_bwd(ws, B, T, K, D);
  const int BH = B * H;
  const int Nr = B * T * K;
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  const size_t n4 = static_cast<size_t>(BH) * T * D / 4;
  k_bwd_zero<<<static_cast<unsigned>((n4 + 255) / 256), 256, 0, st>>>(
      reinterpret_cast<float4*>(dq), reinterpret_cast<float4*>(dk), reinterpret_cast<float4*>(dv),
      n4);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
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
                                          log_base, dq, dk, dv, dgates);
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const void* q, const void* k, const void* v, int dtype, int B, int T,
                           int H, int K, int d, float rope_base, int rope_mode, float scale,
                           const int32_t* topk_idx, const float* gates,
                           const int32_t* seg_offsets, const int32_t* perm_token,
                           const float* dout, float* dq, float* dk, float* dv, float* dgates,
                           void* ws, hipStream_t st) {
#define NAMOH_BWD(DD, BF)                                                                      \
  return run_bwd<DD, BF>(q, k, v, B, T, H, K, rope_base, rope_mode, scale, topk_idx, gates,   \
                         seg_offsets, perm_token, dout, dq, dk, dv, dgates, ws, st)
  if (dtype == 1) {
    if (d == 32) NAMOH_BWD(32, true);
    if (d == 64) NAMOH_BWD(64, true);
    NAMOH_BWD(128, true);
  }
  if (d == 32) NAMOH_BWD(32, false);
  if (d == 64) NAMOH_BWD(64, false);
  NAMOH_BWD(128, false);
#undef NAMOH_BWD
}

// ---------------------------------------------------------------------------
// Router gradient through the gates (selection fixed): one thread per token.
// SOFTMAX_SELECTED: dl_j = g_j (dg_j - sum_k g_k dg_k) on the selected heads;
// SOFTMAX_ALL (and the loss-free balancing gates): dl = a (da - <a, da>).
__global__ __launch_bounds__(256) void k_route_bwd(const float* __restrict__ logits,
                                                   const int32_t* __restrict__ topk_idx,
                                                   const float* __restrict__ gates,
                                                   const float* __restrict__ dgates, long BT,
                                                   int H, int K, int gate_mode,
                                                   float* __restrict__ dlogits) {
  const long tok = static_cast<long>(block_x()) * 256 + thread_x();
  if (tok >= BT) return;
  const float* l = logits + tok * H;
  const int32_t* tk = topk_idx + tok * K;
  const float* g = gates + tok * K;
  const float* dg = dgates + tok * K;
  float* dl = dlogits + tok * H;
  for (int h = 0; h < H; ++h) dl[h] = 0.f;
  for (int kk = 0; kk < K; ++kk)
    if (tk[kk] < 0 || tk[kk] >= H) return;   // not a selection: no gradient
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

hipError_t launch_route_bwd(const float* logits, const int32_t* topk_idx, const float* gates,
                            const float* dgates, int B, int T, int H, int K, int gate_mode,
                            float* dlogits, hipStream_t st) {
  const long BT = static_cast<long>(B) * T;
  k_route_bwd<<<static_cast<unsigned>((BT + 255) / 256), 256, 0, st>>>(
      logits, topk_idx, gates, dgates, BT, H, K, gate_mode, dlogits);
  return hipGetLastError();
}

}  // namespace namoh
