// One decoding step: route the new token, append it to its selected heads'
// caches, attend over each selected head's history, gate and combine.
//
// Sec. 3.1: routing uses only the current token, so incremental decoding is
// the same causal computation as prefill; the new token's rank in head h is
// that head's current length n (Eq. namoh-head-rope) and it attends to itself.
// Sec. 3.2: only the active heads' queries run, and only their caches are read
// or written.  Eq. namoh-kv-cost: the step reads sum over the selected heads
// of (n + 1) cached rows, which makes it HBM-bound.
//
//   k_decode_route_append  one workgroup per sequence: in every wave lane =
//                          head, the rank of each head under (logit desc,
//                          index asc) by H comparisons, gates; then wave w
//                          handles the selected heads w, w + 4, ...: rotation
//                          of q and k at rank n (angles in double), the cache
//                          append and the length update.
//   k_decode_attn          split over 512-row chunks of every selected head's
//                          history: 16-byte coalesced loads of K and V rows
//                          (a row spans d*esize/16 lanes), several rows in
//                          flight per lane, online softmax in exp2 domain,
//                          one (max, sum, acc[d]) partial per chunk.
//   k_decode_combine       merges the chunk partials of each head by
//                          log-sum-exp and sums the gated head outputs.
//   k_prefill_cache        the prefill -> decode hand-off: every packed
//                          prompt row (segment b*H + h, rank r, token t)
//                          writes its rotated key and its value to row r of
//                          head h's caches; cache_len = the segment lengths.
#include <algorithm>
#include <cmath>
#include <mutex>

#include "common.h"
#include "internal.h"
#include "launch.h"

namespace namoh {

constexpr int kDecChunk = 512;   // cached rows per attention workgroup
constexpr int kDecUnroll = 8;    // rows per lane in flight

template <bool BF16>
NAMOH_DEV float ld_elem(const void* p, size_t i) {
  if constexpr (BF16) return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
  else return static_cast<const float*>(p)[i];
}

template <bool BF16>
NAMOH_DEV void st_elem(void* p, size_t i, float x) {
  if constexpr (BF16) static_cast<uint16_t*>(p)[i] = f32_to_bf16(x);
  else static_cast<float*>(p)[i] = x;
}

constexpr int kAppendWaves = 4;

template <int D, bool BF16>
__global__ __launch_bounds__(64 * kAppendWaves) void k_decode_route_append(
    const float* __restrict__ logits, const void* __restrict__ q,
    const void* __restrict__ k, const void* __restrict__ v,
    void* __restrict__ k_cache, void* __restrict__ v_cache,
    int32_t* __restrict__ cache_len, const int32_t* __restrict__ seq_pos,
    int H, int K, long cap, double log_base, int rope_mode, int gate_mode,
    const float* __restrict__ bias, float qscale, int32_t* __restrict__ topk_idx,
    float* __restrict__ gates, int32_t* __restrict__ dev_status, float* __restrict__ qrot,
    int32_t* __restrict__ rows, int G) {
  const int b = block_x();
  const int lane = thread_x() % 64;
  const int wave = thread_x() / 64;
  const bool real = lane < H;
  const float l = real ? logits[static_cast<size_t>(b) * H + lane] : 0.f;
  // selection key: the logit, or with loss-free balancing biases the score
  // float(a + b) with the affinity a = softmax of the logits in double
  // (App. "Auxiliary-Loss-Free Balancing", Eq. namoh-biased-routing)
  float key = l, aff = 0.f;
  if (bias != nullptr) {
    float mx = real ? l : -INFINITY;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    double ex = real ? exp(static_cast<double>(l) - static_cast<double>(mx)) : 0.0;
    double z = ex;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) z += __shfl_xor(z, o);
    const double a = ex / z;
    aff = static_cast<float>(a);
    key = real ? static_cast<float>(a + static_cast<double>(bias[lane])) : 0.f;
  }
  int rank = 0;
  for (int j = 0; j < H; ++j) {
    const float kj = __shfl(key, j);
    rank += (kj > key) || (kj == key && j < lane);
  }
  const bool sel = real && rank < K;
  const uint64_t first = __ballot(real && rank == 0);
  const float lmax = __shfl(l, __ffsll(static_cast<long long>(first)) - 1);
  const float e_sel = sel ? expf(l - lmax) : 0.f;
  float e_den = gate_mode == 1 ? (real ? expf(l - lmax) : 0.f) : e_sel;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) e_den += __shfl_xor(e_den, o);
  if (sel && wave == 0) {
    topk_idx[static_cast<size_t>(b) * K + rank] = lane;
    gates[static_cast<size_t>(b) * K + rank] = bias != nullptr ? aff : e_sel / e_den;
  }

  // every wave routed the token; wave w appends heads w, w + 4, ...
  for (int kk = wave; kk < K; kk += kAppendWaves) {
    const uint64_t mk = __ballot(sel && rank == kk);
    const size_t bk = static_cast<size_t>(b) * K + kk;
    if (mk == 0) {  // only reachable with NaN logits (outside the contract)
      if (lane == 0) {
        rows[bk] = 0;
        topk_idx[bk] = -1;
        if (dev_status) dev_status[0] = 2;
      }
      continue;
    }
    const int h = __ffsll(static_cast<long long>(mk)) - 1;
    const size_t bh = static_cast<size_t>(b) * H + h;
    const int n = cache_len[bh];
    if (n < 0 || n >= cap) {
      if (lane == 0) {
        rows[bk] = 0;
        if (dev_status) dev_status[0] = 1;
      }
      continue;
    }
    const long pos = rope_mode == 0 ? n : (rope_mode == 1 ? seq_pos[b] : 0);
    const size_t src = bh * D;
    const size_t dst = (bh * cap + n) * D;
    for (int j = lane; j < D / 2; j += 64) {
      float cs = 1.f, sn = 0.f;
      if (rope_mode != 2) {
        const float2 w = rope_cos_sin(static_cast<double>(pos) * exp(-(2.0 * j / D) * log_base));
        cs = w.x;
        sn = w.y;
      }
      const float k1 = ld_elem<BF16>(k, src + j), k2 = ld_elem<BF16>(k, src + j + D / 2);
      st_elem<BF16>(k_cache, dst + j, k1 * cs - k2 * sn);
      st_elem<BF16>(k_cache, dst + j + D / 2, k2 * cs + k1 * sn);
      st_elem<BF16>(v_cache, dst + j, ld_elem<BF16>(v, src + j));
      st_elem<BF16>(v_cache, dst + j + D / 2, ld_elem<BF16>(v, src + j + D / 2));
      // the head's G query heads (G = 1 without key/value groups), rotated at
      // the same rank
      for (int u = 0; u < G; ++u) {
        const size_t qs = (bh * G + u) * D;
        const float q1 = ld_elem<BF16>(q, qs + j), q2 = ld_elem<BF16>(q, qs + j + D / 2);
        qrot[(bk * G + u) * D + j] = (q1 * cs - q2 * sn) * qscale;
        qrot[(bk * G + u) * D + j + D / 2] = (q2 * cs + q1 * sn) * qscale;
      }
    }
    if (lane == 0) {
      cache_len[bh] = n + 1;
      rows[bk] = n + 1;
    }
  }
}

// GQ queries per history row (the query heads of a key/value group; 1
// without groups): each row is read once and scored against all of them, with
// one online softmax per query; the partial of query u of selected head bk is
// (bk * GQ + u) * nchunk + chunk.
// RING (shared heads with a window): the caches are rings of cap rows and
// history row r of bk is physical row (row0[bk] + r) mod cap.
template <int D, bool BF16, int GQ = 1, bool RING = false>
__global__ __launch_bounds__(256) void k_decode_attn(
    const void* __restrict__ k_cache, const void* __restrict__ v_cache,
    const int32_t* __restrict__ topk_idx, const int32_t* __restrict__ rows,
    const float* __restrict__ qrot, int H, int K, long cap, int nchunk,
    float* __restrict__ part_acc, float* __restrict__ part_ml,
    const int32_t* __restrict__ row0 = nullptr) {
  constexpr int EPG = BF16 ? 8 : 4;   // elements per 16-byte granule
  constexpr int G = D / EPG;          // lanes per row
  constexpr int RPW = 64 / G;         // rows per wave per step
  constexpr int RPB = 4 * RPW;        // rows per workgroup per step
  // rows per lane in flight, fewer with more queries per row (registers)
  constexpr int U = GQ <= 2 ? kDecUnroll : (GQ == 4 ? kDecUnroll / 2 : kDecUnroll / 4);
  __shared__ float s_ml[GQ][RPB][2];
  __shared__ float s_acc[GQ][RPB][D];

  const int bk = block_x() / nchunk;
  const int chunk = block_x() - bk * nchunk;
  const int L = rows[bk];
  const int r0 = chunk * kDecChunk;
  if (r0 >= L) return;
  const int r1 = min(L, r0 + kDecChunk);
  const int b = bk / K;
  const int h = topk_idx[bk];
  const size_t rowbase = (static_cast<size_t>(b) * H + h) * cap;
  const int ring0 = RING ? row0[bk] : 0;
  const int tid = thread_x();
  const int lane = tid % 64, wave = tid / 64;
  const int sub = lane % G;
  const int grp = wave * RPW + lane / G;

  float qv[GQ][EPG];
#pragma unroll
  for (int u = 0; u < GQ; ++u)
#pragma unroll
    for (int e = 0; e < EPG; ++e)
      qv[u][e] = qrot[(static_cast<size_t>(bk) * GQ + u) * D + sub * EPG + e];
  float m[GQ], lsum[GQ], acc[GQ][EPG];
#pragma unroll
  for (int u = 0; u < GQ; ++u) {
    m[u] = -1e30f;
    lsum[u] = 0.f;
#pragma unroll
    for (int e = 0; e < EPG; ++e) acc[u][e] = 0.f;
  }

  const u32x4* kc = reinterpret_cast<const u32x4*>(k_cache);
  const u32x4* vc = reinterpret_cast<const u32x4*>(v_cache);
  for (int rb = r0; rb < r1; rb += RPB * U) {
    u32x4 kx[U], vx[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = rb + u * RPB + grp;
      if (r < r1) {
        long pr = r;
        if constexpr (RING) {
          pr += ring0;
          if (pr >= cap) pr -= cap;
        }
        const size_t gi = (rowbase + pr) * G + sub;
        kx[u] = kc[gi];
        vx[u] = vc[gi];
      } else {
        kx[u] = u32x4{0u, 0u, 0u, 0u};
        vx[u] = kx[u];
      }
    }
    float sc[GQ][U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float f[EPG];
      if constexpr (BF16) {
        const uint32_t w[4] = {kx[u].x, kx[u].y, kx[u].z, kx[u].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          f[2 * e] = lo_bf16(w[e]);
          f[2 * e + 1] = hi_bf16(w[e]);
        }
      } else {
        f[0] = __uint_as_float(kx[u].x); f[1] = __uint_as_float(kx[u].y);
        f[2] = __uint_as_float(kx[u].z); f[3] = __uint_as_float(kx[u].w);
      }
#pragma unroll
      for (int qq = 0; qq < GQ; ++qq) {
        float dsum = 0.f;
#pragma unroll
        for (int e = 0; e < EPG; ++e) dsum = fmaf(qv[qq][e], f[e], dsum);
        dsum = group_sum<G>(dsum);
        sc[qq][u] = (rb + u * RPB + grp < r1) ? dsum : -INFINITY;
      }
    }
    float p[GQ][U];
#pragma unroll
    for (int qq = 0; qq < GQ; ++qq) {
      float mx = sc[qq][0];
#pragma unroll
      for (int u = 1; u < U; ++u) mx = fmaxf(mx, sc[qq][u]);
      const float mnew = fmaxf(m[qq], mx);
      const float corr = __builtin_amdgcn_exp2f(m[qq] - mnew);
      lsum[qq] *= corr;
#pragma unroll
      for (int e = 0; e < EPG; ++e) acc[qq][e] *= corr;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        p[qq][u] = __builtin_amdgcn_exp2f(sc[qq][u] - mnew);
        lsum[qq] += p[qq][u];
      }
      m[qq] = mnew;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float f[EPG];
      if constexpr (BF16) {
        const uint32_t w[4] = {vx[u].x, vx[u].y, vx[u].z, vx[u].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          f[2 * e] = lo_bf16(w[e]);
          f[2 * e + 1] = hi_bf16(w[e]);
        }
      } else {
        f[0] = __uint_as_float(vx[u].x); f[1] = __uint_as_float(vx[u].y);
        f[2] = __uint_as_float(vx[u].z); f[3] = __uint_as_float(vx[u].w);
      }
#pragma unroll
      for (int qq = 0; qq < GQ; ++qq)
#pragma unroll
        for (int e = 0; e < EPG; ++e) acc[qq][e] = fmaf(p[qq][u], f[e], acc[qq][e]);
    }
  }
#pragma unroll
  for (int qq = 0; qq < GQ; ++qq) {
    if (sub == 0) {
      s_ml[qq][grp][0] = m[qq];
      s_ml[qq][grp][1] = lsum[qq];
    }
#pragma unroll
    for (int e = 0; e < EPG; ++e) s_acc[qq][grp][sub * EPG + e] = acc[qq][e];
  }
  __syncthreads();
  for (int t2 = tid; t2 < GQ * D; t2 += 256) {
    const int qq = t2 / D, dd = t2 - (t2 / D) * D;
    float M = -1e30f;
    for (int gi = 0; gi < RPB; ++gi) M = fmaxf(M, s_ml[qq][gi][0]);
    float Ls = 0.f, A = 0.f;
    for (int gi = 0; gi < RPB; ++gi) {
      const float w = __builtin_amdgcn_exp2f(s_ml[qq][gi][0] - M);
      Ls = fmaf(s_ml[qq][gi][1], w, Ls);
      A = fmaf(s_acc[qq][gi][dd], w, A);
    }
    const size_t pi = (static_cast<size_t>(bk) * GQ + qq) * nchunk + chunk;
    part_acc[pi * D + dd] = A;
    if (dd == 0) {
      part_ml[2 * pi] = M;
      part_ml[2 * pi + 1] = Ls;
    }
  }
}

// Grouped decode on the matrix cores (GQ = 4 or 8 query heads share each
// cached row).  A wave takes 128 rows of the chunk in blocks of 32 and uses
// v_mfma_f32_16x16x32_bf16 (lane l: A row / B column / C column l % 16,
// reduction slots 8 (l / 16) .. + 7; C rows 4 (l / 16) + i in accumulator
// i):
//   the block's key and value rows are loaded whole (each lane a 16-byte
//     granule of D / 16 consecutive rows: coalesced 16-byte loads) and
//     rearranged through wave-private LDS: key rows row-major with padded
//     rows (s_k), and each lane's run of rows of one column written as one
//     run of a V^T row (s_vt); the next block's loads are issued before the
//     current block is processed;
//   S[q][r] = Q K^T for two 16-row tiles: A = the GQ rotated queries (rows
//     >= GQ zero), B = the key rows read back from s_k;
//   online softmax per query in exp2 units: the 16 lanes of one reduction
//     group hold a query's 16 scores of a tile;
//   O[q][d] += P V over the 32 rows: A = P and B = V^T read from the
//     wave-private LDS tiles (P as [query][row], V^T as [d][row], both
//     16-byte reads).
// LDS: about 81 KB per workgroup at D = 128, so the two workgroups per
// compute unit that the launch bounds ask for fill its 160 KB.
// The reduction group kg = l / 16 of every layout holds queries 4 kg .. 4 kg
// + 3, so a lane's rescale factors apply to its own output accumulators.
// Partials as in k_decode_attn: (bk * GQ + q) * nchunk + chunk.
template <int D, int GQ>
__global__ __launch_bounds__(256, 2) void k_decode_attn_mfma(
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ topk_idx, const int32_t* __restrict__ rows,
    const float* __restrict__ qrot, int H, int K, long cap, int nchunk,
    float* __restrict__ part_acc, float* __restrict__ part_ml) {
  static_assert(GQ == 4 || GQ == 8, "queries per cached row");
  static_assert(D == 64 || D == 128, "head width");
  constexpr int KS = D / 32;           // reduction steps of the score product
  constexpr int NT = D / 16;           // 16-column output tiles
  constexpr int VP = 40;               // padded row length (elements) of the LDS tiles
  constexpr int RPW = kDecChunk / 4;   // rows per wave
  // the V^T tiles are dead after the loop; the per-wave output rows reuse them
  static_assert(4 * GQ * D * 4 <= 4 * D * VP * 2, "output rows fit the V^T tiles");
  constexpr int KP = D + 8;             // padded key row (elements) of the LDS key tile
  constexpr int GR = D / 8;             // 16-byte granules per cached row
  constexpr int RPL = GR / 2;           // rows per lane per 32-row block (coalesced loads)
  __shared__ __attribute__((aligned(16))) uint16_t s_vt[4][D * VP];
  __shared__ __attribute__((aligned(16))) uint16_t s_k[4][32 * KP];
  __shared__ __attribute__((aligned(16))) uint16_t s_p[4][16 * VP];
  __shared__ float s_ml[4][GQ][2];
  float (*s_o)[GQ][D] = reinterpret_cast<float (*)[GQ][D]>(&s_vt[0][0]);

  const int bk = block_x() / nchunk;
  const int chunk = block_x() - bk * nchunk;
  const int L = rows[bk];
  const int r0 = chunk * kDecChunk;
  if (r0 >= L) return;
  const int r1 = min(L, r0 + kDecChunk);
  const int b = bk / K;
  const int h = topk_idx[bk];
  const size_t rowbase = (static_cast<size_t>(b) * H + h) * cap;
  const int tid = thread_x();
  const int lane = tid % 64, wave = tid / 64;
  const int j16 = lane & 15, kg = lane >> 4;
  const int w0 = r0 + wave * RPW;
  const int w1 = min(r1, w0 + RPW);

  // A operand rows >= GQ are zero: they read query GQ - 1 and are cleared
  // after the loads (a load under a branch would be waited for at the join,
  // one round trip per load)
  bf16x8 qa[KS];
  {
    const float4* qrow = reinterpret_cast<const float4*>(
        qrot + (static_cast<size_t>(bk) * GQ + min(j16, GQ - 1)) * D + 8 * kg);
    float4 f[KS][2];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      f[s][0] = qrow[8 * s];
      f[s][1] = qrow[8 * s + 1];
    }
    const bool keep = j16 < GQ;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const float x[8] = {f[s][0].x, f[s][0].y, f[s][0].z, f[s][0].w,
                          f[s][1].x, f[s][1].y, f[s][1].z, f[s][1].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) qa[s][e] = static_cast<__bf16>(keep ? x[e] : 0.f);
    }
  }
  float m[4], l[4];
  f32x4 O[NT];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m[i] = -1e30f;
    l[i] = 0.f;
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) O[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  const u32x4* kc = reinterpret_cast<const u32x4*>(k_cache);
  const u32x4* vc = reinterpret_cast<const u32x4*>(v_cache);
  uint16_t* vt = s_vt[wave];
  uint16_t* pt = s_p[wave];
  // Coalesced loads: lane (granule lane % GR, row group lane / GR) reads rows
  // RPL * group + i, i < RPL, of the block, so each load instruction covers
  // whole rows.  Rows past the wave's end read its last row (finite values;
  // masked).  The next block is loaded while the current one is processed
  // (its loads are issued unconditionally, clamped like the tail).
  const int lg = lane % GR, lq = lane / GR;
  u32x4 kx[RPL], vx[RPL], kn[RPL], vn[RPL];
  auto load_block = [&](int rb, u32x4 (&kd)[RPL], u32x4 (&vd)[RPL]) {
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
      const size_t row = rowbase + min(rb + RPL * lq + i, w1 - 1);
      kd[i] = kc[row * GR + lg];
      vd[i] = vc[row * GR + lg];
    }
  };
  if (w0 < w1) load_block(w0, kx, vx);
  for (int rb = w0; rb < w1; rb += 32) {
    load_block(min(rb + 32, w1 - 1), kn, vn);
    // key rows into the wave's LDS tile (row-major, padded rows), values
    // transposed into V^T: lane's RPL consecutive rows of one granule become,
    // per column, one RPL-element run of a V^T row
    uint16_t* kt = s_k[wave];
#pragma unroll
    for (int i = 0; i < RPL; ++i)
      *reinterpret_cast<u32x4*>(&kt[(RPL * lq + i) * KP + 8 * lg]) = kx[i];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t run[RPL / 2];
#pragma unroll
      for (int m = 0; m < RPL / 2; ++m) {
        const uint32_t a = vx[2 * m][e / 2], c2 = vx[2 * m + 1][e / 2];
        run[m] = (e & 1) ? ((a >> 16) | (c2 & 0xFFFF0000u)) : ((a & 0xFFFFu) | (c2 << 16));
      }
      uint16_t* dst = &s_vt[wave][(8 * lg + e) * VP + RPL * lq];
      if constexpr (RPL == 8)
        *reinterpret_cast<u32x4*>(dst) = u32x4{run[0], run[1], run[2], run[3]};
      else
        *reinterpret_cast<uint2*>(dst) = make_uint2(run[0], run[1]);
    }
    f32x4 S[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      S[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bf16x8 kb =
            *reinterpret_cast<const bf16x8*>(&kt[(16 * tt + j16) * KP + 32 * s + 8 * kg]);
        S[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[s], kb, S[tt], 0, 0, 0);
      }
    }
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
      if (rb + 16 * tt + j16 >= w1) S[tt] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = fmaxf(S[0][i], S[1][i]);
      mx = group_max<16>(mx);
      const float mnew = fmaxf(m[i], mx);
      const float corr = __builtin_amdgcn_exp2f(m[i] - mnew);
      m[i] = mnew;
      const float p0 = __builtin_amdgcn_exp2f(S[0][i] - mnew);
      const float p1 = __builtin_amdgcn_exp2f(S[1][i] - mnew);
      float ps = p0 + p1;
      ps = group_sum<16>(ps);
      l[i] = l[i] * corr + ps;
#pragma unroll
      for (int t = 0; t < NT; ++t) O[t][i] *= corr;
      pt[(4 * kg + i) * VP + j16] = f32_to_bf16(p0);
      pt[(4 * kg + i) * VP + 16 + j16] = f32_to_bf16(p1);
    }
    // the tiles are wave-private: LDS operations of one wave complete in order
    const bf16x8 pa = *reinterpret_cast<const bf16x8*>(&pt[j16 * VP + 8 * kg]);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const bf16x8 vb = *reinterpret_cast<const bf16x8*>(&vt[(16 * t + j16) * VP + 8 * kg]);
      O[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vb, O[t], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
      kx[i] = kn[i];
      vx[i] = vn[i];
    }
  }

  // ---- merge the four waves' partials of every query -----------------------
  __syncthreads();   // every wave is done with its V^T tile (reused for s_o)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int q = 4 * kg + i;
    if (q < GQ) {
      if (j16 == 0) {
        s_ml[wave][q][0] = m[i];
        s_ml[wave][q][1] = l[i];
      }
#pragma unroll
      for (int t = 0; t < NT; ++t) s_o[wave][q][16 * t + j16] = O[t][i];
    }
  }
  __syncthreads();
  for (int t2 = tid; t2 < GQ * D; t2 += 256) {
    const int q = t2 / D, dd = t2 - (t2 / D) * D;
    float M = -1e30f;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_ml[w][q][0]);
    float Ls = 0.f, A = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float sc = __builtin_amdgcn_exp2f(s_ml[w][q][0] - M);
      Ls = fmaf(s_ml[w][q][1], sc, Ls);
      A = fmaf(s_o[w][q][dd], sc, A);
    }
    const size_t pi = (static_cast<size_t>(bk) * GQ + q) * nchunk + chunk;
    part_acc[pi * D + dd] = A;
    if (dd == 0) {
      part_ml[2 * pi] = M;
      part_ml[2 * pi + 1] = Ls;
    }
  }
}

// One workgroup per sequence; wave w merges the chunk partials of heads
// w, w + 4, ... (lane c holds chunk c's max and sum; the accumulators are
// read column-wise, d = lane + 64 i), then the gated head outputs are summed
// in head order.
// With key/value groups (G query heads per selected head) the G heads of a
// slot share its gate and are summed in head order.
template <int D, bool OUT_BF16>
__global__ __launch_bounds__(256) void k_decode_combine(
    const float* __restrict__ gates, const int32_t* __restrict__ rows,
    const float* __restrict__ part_acc, const float* __restrict__ part_ml,
    int K, int nchunk, void* __restrict__ out, int G, int accumulate = 0) {
  constexpr int NWV = 4;
  constexpr int DPL = (D + 63) / 64;  // output columns per lane
  __shared__ float s_o[NWV][D];
  const int b = block_x();
  const int lane = thread_x() % 64, wave = thread_x() / 64;
  float o[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) o[i] = 0.f;
  for (int vk = wave; vk < K * G; vk += NWV) {
    const int kk = vk / G;
    const size_t bk = static_cast<size_t>(b) * K + kk;
    const size_t bq = bk * G + (vk - kk * G);   // the head's partials
    const int L = rows[bk];
    if (L == 0) continue;
    const int nc = (L + kDecChunk - 1) / kDecChunk;
    const float* ml = part_ml + bq * nchunk * 2;
    float M = -1e30f;
    for (int c = lane; c < nc; c += 64) M = fmaxf(M, ml[2 * c]);
    M = group_max<64>(M);
    float Ls = 0.f;
    for (int c = lane; c < nc; c += 64) Ls += ml[2 * c + 1] * __builtin_amdgcn_exp2f(ml[2 * c] - M);
    Ls = group_sum<64>(Ls);
    const float scale = gates[bk] / Ls;
    float a[DPL];
#pragma unroll
    for (int i = 0; i < DPL; ++i) a[i] = 0.f;
    const float* pa = part_acc + bq * nchunk * D;
#pragma unroll 4
    for (int c = 0; c < nc; ++c) {
      const float w = __builtin_amdgcn_exp2f(ml[2 * c] - M);
#pragma unroll
      for (int i = 0; i < DPL; ++i) {
        const int d = lane + 64 * i;
        if (d < D) a[i] = fmaf(pa[static_cast<size_t>(c) * D + d], w, a[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < DPL; ++i) o[i] = fmaf(a[i], scale, o[i]);
  }
#pragma unroll
  for (int i = 0; i < DPL; ++i) {
    const int d = lane + 64 * i;
    if (d < D) s_o[wave][d] = o[i];
  }
  __syncthreads();
  if (thread_x() < D) {
    const size_t oi = static_cast<size_t>(b) * D + thread_x();
    float r = 0.f;
    if (accumulate) {   // added to what out holds (shared heads after the routed step)
      if constexpr (OUT_BF16) r = bf16_to_f32(static_cast<const uint16_t*>(out)[oi]);
      else r = static_cast<const float*>(out)[oi];
    }
#pragma unroll
    for (int w = 0; w < NWV; ++w) r += s_o[w][thread_x()];
    if constexpr (OUT_BF16) static_cast<uint16_t*>(out)[oi] = f32_to_bf16(r);
    else static_cast<float*>(out)[oi] = r;
  }
}

static int dec_nchunk(int cap) { return (cap + kDecChunk - 1) / kDecChunk; }

struct DecWs {
  float* qrot;
  int32_t* rows;
  float* part_acc;
  float* part_ml;
  size_t bytes;
};

static DecWs carve_dec(void* ws, int B, int K, int d, int cap, int G = 1) {
  const size_t BK = static_cast<size_t>(B) * K;
  const size_t nc = dec_nchunk(cap);
  Carver cv(ws);
  DecWs w;
  w.qrot = cv.take<float>(BK * G * d);
  w.rows = cv.take<int32_t>(BK);
  w.part_acc = cv.take<float>(BK * G * nc * d);
  w.part_ml = cv.take<float>(BK * G * nc * 2);
  w.bytes = cv.off;
  return w;
}

size_t decode_workspace_bytes(int B, int /*H*/, int K, int d, int cap, int G) {
  return carve_dec(nullptr, B, K, d, cap, G).bytes;
}

// ---------------------------------------------------------------------------
// Scratch of the decode step that allocates nothing (namoh_decode_step_noalloc):
// the step's workspace (rotated queries, history lengths, per-chunk partials)
// in a file-scope device array.  Every GPU the library runs on holds its own
// copy for the life of the process; every call on one GPU uses that GPU's
// copy, so calls that overlap on one GPU race.  Nothing in it needs to start
// at zero: the append kernel writes every row length and rotated query the
// attention reads, and each chunk writes the partial the combine reads.
constexpr size_t kDecodeScratchBytes = static_cast<size_t>(32) << 20;
static __device__ __attribute__((aligned(256))) unsigned char scratch[kDecodeScratchBytes];

size_t decode_scratch_bytes() { return kDecodeScratchBytes; }

// Device address of the array on the current device.  In host code the
// array's name only stands in for the symbol; its device address comes from
// hipGetSymbolAddress, taken once per device (with that device current) and
// kept.
hipError_t decode_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// Prefill -> decode hand-off (Sec. 3.2, efficient execution: a decoding step
// reads and extends only its active heads' caches, so those must hold the
// prompt's rotated keys and values of each head in rank order, Eq.
// namoh-head-rope).  A workgroup takes 4096 / D consecutive packed rows: the
// segment of each row by binary search over seg_offsets (staged in LDS), then one 8-pair
// group (elements j..j+7 and j+d/2..j+d/2+7) per thread, 16-byte loads and
// stores, angles formed and reduced in double as in the decode append.  Rows
// whose offsets are not a packing of [0, Nr) with ranks below cap and tokens
// below T are skipped.
constexpr int kCacheThreads = 256;
constexpr int kCacheSegLds = 2048;   // segment offsets staged in LDS up to this many segments
template <int D>
constexpr int cache_rows() { return kCacheThreads * 16 / D; }

template <bool BF16>
NAMOH_DEV void ld8(const void* p, size_t i, float* x) {
  if constexpr (BF16) {
    const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + i);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = lo_bf16(w[e]);
      x[2 * e + 1] = hi_bf16(w[e]);
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
    const float4 c = *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = c.x; x[5] = c.y; x[6] = c.z; x[7] = c.w;
  }
}

template <bool BF16>
NAMOH_DEV void st8(void* p, size_t i, const float* x) {
  if constexpr (BF16) {
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p) + i) =
        make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                   pack_bf16x2(x[6], x[7]));
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(p) + i) = make_float4(x[0], x[1], x[2], x[3]);
    *reinterpret_cast<float4*>(static_cast<float*>(p) + i + 4) = make_float4(x[4], x[5], x[6], x[7]);
  }
}

template <int D, bool BF16>
__global__ __launch_bounds__(kCacheThreads) void k_prefill_cache(
    const void* __restrict__ k, const void* __restrict__ v,
    const int32_t* __restrict__ seg_offsets, const int32_t* __restrict__ perm_token, int BH,
    int H, int T, int Nr, long cap, double log_base, int rope_mode, int nblocks,
    void* __restrict__ k_cache, void* __restrict__ v_cache, int32_t* __restrict__ cache_len) {
  constexpr int RW = cache_rows<D>();
  constexpr int G = D / 16;   // 8-pair groups per row
  static_assert(RW * G == kCacheThreads, "one group per thread");
  __shared__ double s_theta[D / 2];
  __shared__ int s_seg[RW], s_rank[RW], s_tok[RW];
  __shared__ int s_off[kCacheSegLds + 1];
  const int tid = thread_x();
  const int row0 = block_x() * RW;
  for (int s = block_x() * kCacheThreads + tid; s < BH; s += nblocks * kCacheThreads)
    cache_len[s] = seg_offsets[s + 1] - seg_offsets[s];
  if (tid < D / 2) s_theta[tid] = exp(-(2.0 * tid / D) * log_base);
  const bool in_lds = BH <= kCacheSegLds;
  if (in_lds)
    for (int i = tid; i <= BH; i += kCacheThreads) s_off[i] = seg_offsets[i];
  __syncthreads();
  const int32_t* off = in_lds ? s_off : seg_offsets;
  if (tid < RW) {
    const int pr = row0 + tid;
    int seg = -1, rank = -1, tok = -1;
    if (pr < Nr) {
      tok = perm_token[pr];
      int lo = 0, hi = BH;   // the last segment starting at or before pr
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (off[mid] <= pr) lo = mid; else hi = mid;
      }
      seg = lo;
      rank = pr - off[lo];
      if (rank < 0 || rank >= cap || pr >= off[lo + 1] || tok < 0 || tok >= T) seg = -1;
    }
    s_seg[tid] = seg;
    s_rank[tid] = rank;
    s_tok[tid] = tok;
  }
  __syncthreads();
  const int row = tid / G, j0 = (tid - row * G) * 8;
  const int seg = s_seg[row];
  if (seg < 0) return;
  const int r = s_rank[row], t = s_tok[row];
  const size_t src = (static_cast<size_t>(seg) * T + t) * D;
  const size_t dst = (static_cast<size_t>(seg) * cap + r) * D;
  float k1[8], k2[8], v1[8], v2[8];
  ld8<BF16>(k, src + j0, k1);
  ld8<BF16>(k, src + j0 + D / 2, k2);
  ld8<BF16>(v, src + j0, v1);
  ld8<BF16>(v, src + j0 + D / 2, v2);
  if (rope_mode != 2) {
    const double pos = rope_mode == 0 ? r : t;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float2 w = rope_cos_sin(pos * s_theta[j0 + e]);
      const float a = k1[e], c = k2[e];
      k1[e] = a * w.x - c * w.y;
      k2[e] = c * w.x + a * w.y;
    }
  }
  st8<BF16>(k_cache, dst + j0, k1);
  st8<BF16>(k_cache, dst + j0 + D / 2, k2);
  st8<BF16>(v_cache, dst + j0, v1);
  st8<BF16>(v_cache, dst + j0 + D / 2, v2);
}

template <int D, bool BF16>
static hipError_t run_prefill_cache(const void* k, const void* v, int B, int T, int H, int K,
                                    float rope_base, int rope_mode, const int32_t* seg_offsets,
                                    const int32_t* perm_token, void* k_cache, void* v_cache,
                                    int32_t* cache_len, int cap, hipStream_t st) {
  const int BH = B * H;
  const long Nr = static_cast<long>(B) * T * K;
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  constexpr int RW = cache_rows<D>();
  const long blocks = std::max((Nr + RW - 1) / RW,
                               static_cast<long>((BH + kCacheThreads - 1) / kCacheThreads));
  k_prefill_cache<D, BF16><<<static_cast<unsigned>(blocks), kCacheThreads, 0, st>>>(
      k, v, seg_offsets, perm_token, BH, H, T, static_cast<int>(Nr), cap, log_base, rope_mode,
      static_cast<int>(blocks), k_cache, v_cache, cache_len);
  return hipGetLastError();
}

hipError_t launch_prefill_cache(const void* k, const void* v, int dtype, int B, int T, int H,
                                int K, int d, float rope_base, int rope_mode,
                                const int32_t* seg_offsets, const int32_t* perm_token,
                                void* k_cache, void* v_cache, int32_t* cache_len, int cap,
                                hipStream_t st) {
#define NAMOH_PC(DD, BF)                                                                       \
  return run_prefill_cache<DD, BF>(k, v, B, T, H, K, rope_base, rope_mode, seg_offsets,       \
                                   perm_token, k_cache, v_cache, cache_len, cap, st)
  if (dtype == 1) {
    if (d == 32) NAMOH_PC(32, true);
    if (d == 64) NAMOH_PC(64, true);
    NAMOH_PC(128, true);
  }
  if (d == 32) NAMOH_PC(32, false);
  if (d == 64) NAMOH_PC(64, false);
  NAMOH_PC(128, false);
#undef NAMOH_PC
}

template <int D, bool BF16, int GQ = 1>
static hipError_t run_decode(const float* logits, const float* bias, const void* q, const void* k,
                             const void* v, void* k_cache, void* v_cache,
                             int32_t* cache_len, const int32_t* seq_pos, int B,
                             int H, int K, int cap, float rope_base,
                             int rope_mode, int gate_mode, float scale,
                             int32_t* topk_idx, float* gates, void* out,
                             int out_dtype, int32_t* dev_status, void* ws,
                             hipStream_t st) {
  const DecWs w = carve_dec(ws, B, K, D, cap, GQ);
  const int nc = dec_nchunk(cap);
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  k_decode_route_append<D, BF16><<<B, 64 * kAppendWaves, 0, st>>>(
      logits, q, k, v, k_cache, v_cache, cache_len, seq_pos, H, K, cap, log_base,
      rope_mode, gate_mode, bias, scale * 1.4426950408889634f, topk_idx, gates,
      dev_status, w.qrot, w.rows, GQ);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t grid = static_cast<size_t>(B) * K * nc;
  if constexpr (BF16 && (GQ == 4 || GQ == 8))
    launch_k("decode_attn", k_decode_attn_mfma<D, GQ>, dim3(static_cast<unsigned>(grid)),
             dim3(256), st, static_cast<const uint16_t*>(k_cache),
             static_cast<const uint16_t*>(v_cache), topk_idx, w.rows, w.qrot, H, K, cap, nc,
             w.part_acc, w.part_ml);
  else
    launch_k("decode_attn", k_decode_attn<D, BF16, GQ>, dim3(static_cast<unsigned>(grid)),
             dim3(256), st, k_cache, v_cache, topk_idx, w.rows, w.qrot, H, K, cap, nc,
             w.part_acc, w.part_ml, static_cast<const int32_t*>(nullptr));
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (out_dtype == 1)
    k_decode_combine<D, true><<<B, 256, 0, st>>>(gates, w.rows, w.part_acc, w.part_ml, K, nc, out,
                                                GQ);
  else
    k_decode_combine<D, false><<<B, 256, 0, st>>>(gates, w.rows, w.part_acc, w.part_ml, K, nc,
                                                 out, GQ);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Shared heads in the decode step (Sec. 4.4, shared heads for local context):
// the new token of sequence b, at global position p = cache_len[b], enters
// every one of the Hs always-active heads.  Its key (rotated at p, or not at
// all) and value go to row p mod cap of the head's caches, and its query
// attends over the keys at positions max(0, p + 1 - window) .. p (window 0:
// 0 .. p), itself included; the head outputs are summed without a gate.
// With a window the caches are rings that keep the most recent cap >= window
// tokens; without one row p must exist (p < cap), else the step skips the
// sequence and reports it.
//
//   k_shared_decode_append  one workgroup per sequence: wave w takes heads
//                           w, w + 4, ...: rotation (angles in double), the
//                           cache rows, the scaled rotated query, and the
//                           history each head reads (length, first ring row).
//   k_decode_attn<…, RING>  the routed step's split-K attention over those
//                           histories.
//   k_decode_combine        the routed step's merge, gates 1, added to out.
template <int D, bool BF16>
__global__ __launch_bounds__(64 * kAppendWaves) void k_shared_decode_append(
    const void* __restrict__ q, const void* __restrict__ k, const void* __restrict__ v,
    void* __restrict__ k_cache, void* __restrict__ v_cache, int32_t* __restrict__ cache_len,
    int Hs, long cap, int window, double log_base, int rope_mode, float qscale,
    int32_t* __restrict__ dev_status, float* __restrict__ qrot, int32_t* __restrict__ rows,
    int32_t* __restrict__ row0, int32_t* __restrict__ heads, float* __restrict__ gates) {
  const int b = block_x();
  const int lane = thread_x() % 64, wave = thread_x() / 64;
  const int p = cache_len[b];
  const bool over = p < 0 || (window == 0 && p >= cap);
  const int m = over ? 0 : (window > 0 ? min(p + 1, window) : p + 1);
  const long slot = over ? 0 : p % cap;
  for (int s = wave; s < Hs; s += kAppendWaves) {
    const size_t bs = static_cast<size_t>(b) * Hs + s;
    if (lane == 0) {
      rows[bs] = m;
      row0[bs] = over ? 0 : static_cast<int>((static_cast<long>(p) + 1 - m) % cap);
      heads[bs] = s;
      gates[bs] = 1.f;
    }
    if (over) continue;
    const size_t src = bs * D;
    const size_t dst = (bs * cap + slot) * D;
    for (int j = lane; j < D / 2; j += 64) {
      float cs = 1.f, sn = 0.f;
      if (rope_mode != 2) {
        const float2 w = rope_cos_sin(static_cast<double>(p) * exp(-(2.0 * j / D) * log_base));
        cs = w.x;
        sn = w.y;
      }
      const float k1 = ld_elem<BF16>(k, src + j), k2 = ld_elem<BF16>(k, src + j + D / 2);
      st_elem<BF16>(k_cache, dst + j, k1 * cs - k2 * sn);
      st_elem<BF16>(k_cache, dst + j + D / 2, k2 * cs + k1 * sn);
      st_elem<BF16>(v_cache, dst + j, ld_elem<BF16>(v, src + j));
      st_elem<BF16>(v_cache, dst + j + D / 2, ld_elem<BF16>(v, src + j + D / 2));
      const float q1 = ld_elem<BF16>(q, src + j), q2 = ld_elem<BF16>(q, src + j + D / 2);
      qrot[src + j] = (q1 * cs - q2 * sn) * qscale;
      qrot[src + j + D / 2] = (q2 * cs + q1 * sn) * qscale;
    }
  }
  __syncthreads();   // every wave has read cache_len[b]
  if (thread_x() == 0) {
    if (over) {
      if (dev_status) dev_status[0] = 1;
    } else {
      cache_len[b] = p + 1;
    }
  }
}

// Prefill -> decode hand-off of the shared heads: token t of the prompt
// (rotated at t, or not at all) goes to row t mod cap of every shared head's
// caches, for the last min(T, cap) tokens (with a window the earlier ones are
// never read again); cache_len[b] = T.  One thread per (row, rotation pair).
template <int D, bool BF16>
__global__ __launch_bounds__(256) void k_shared_prefill_cache(
    const void* __restrict__ k, const void* __restrict__ v, int T, int Hs, long cap,
    long first, double log_base, int rope_mode, void* __restrict__ k_cache,
    void* __restrict__ v_cache, int32_t* __restrict__ cache_len, long nrows) {
  const long idx = static_cast<long>(block_x()) * 256 + thread_x();
  const long row = idx / (D / 2);
  const int j = static_cast<int>(idx - row * (D / 2));
  if (row >= nrows) return;
  const long keep = T - first;              // tokens first .. T - 1
  const long bs = row / keep;               // b * Hs + s
  const long t = first + (row - bs * keep);
  if (j == 0 && t == T - 1 && bs % Hs == 0) cache_len[bs / Hs] = T;
  float cs = 1.f, sn = 0.f;
  if (rope_mode != 2) {
    const float2 w = rope_cos_sin(static_cast<double>(t) * exp(-(2.0 * j / D) * log_base));
    cs = w.x;
    sn = w.y;
  }
  const size_t src = (static_cast<size_t>(bs) * T + t) * D;
  const size_t dst = (static_cast<size_t>(bs) * cap + t % cap) * D;
  const float k1 = ld_elem<BF16>(k, src + j), k2 = ld_elem<BF16>(k, src + j + D / 2);
  st_elem<BF16>(k_cache, dst + j, k1 * cs - k2 * sn);
  st_elem<BF16>(k_cache, dst + j + D / 2, k2 * cs + k1 * sn);
  st_elem<BF16>(v_cache, dst + j, ld_elem<BF16>(v, src + j));
  st_elem<BF16>(v_cache, dst + j + D / 2, ld_elem<BF16>(v, src + j + D / 2));
}

struct SharedDecWs {
  float* qrot;
  int32_t* rows;
  int32_t* row0;
  int32_t* heads;
  float* gates;
  float* part_acc;
  float* part_ml;
  size_t bytes;
};

static SharedDecWs carve_shared_dec(void* ws, int B, int Hs, int d, int cap) {
  const size_t BS = static_cast<size_t>(B) * Hs;
  const size_t nc = dec_nchunk(cap);
  Carver cv(ws);
  SharedDecWs w;
  w.qrot = cv.take<float>(BS * d);
  w.rows = cv.take<int32_t>(BS);
  w.row0 = cv.take<int32_t>(BS);
  w.heads = cv.take<int32_t>(BS);
  w.gates = cv.take<float>(BS);
  w.part_acc = cv.take<float>(BS * nc * d);
  w.part_ml = cv.take<float>(BS * nc * 2);
  w.bytes = cv.off;
  return w;
}

size_t shared_decode_workspace_bytes(int B, int Hs, int d, int cap) {
  return carve_shared_dec(nullptr, B, Hs, d, cap).bytes;
}

template <int D, bool BF16>
static hipError_t run_shared_decode(const void* q, const void* k, const void* v, void* k_cache,
                                    void* v_cache, int32_t* cache_len, int B, int Hs, int cap,
                                    int window, float rope_base, int rope_mode, float scale,
                                    void* out, int out_dtype, int accumulate,
                                    int32_t* dev_status, void* ws, hipStream_t st) {
  const SharedDecWs w = carve_shared_dec(ws, B, Hs, D, cap);
  const int nc = dec_nchunk(cap);
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
  k_shared_decode_append<D, BF16><<<B, 64 * kAppendWaves, 0, st>>>(
      q, k, v, k_cache, v_cache, cache_len, Hs, cap, window, log_base, rope_mode,
      scale * 1.4426950408889634f, dev_status, w.qrot, w.rows, w.row0, w.heads, w.gates);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t grid = static_cast<size_t>(B) * Hs * nc;
  launch_k("decode_attn", k_decode_attn<D, BF16, 1, true>, dim3(static_cast<unsigned>(grid)),
           dim3(256), st, k_cache, v_cache, w.heads, w.rows, w.qrot, Hs, Hs, cap, nc, w.part_acc,
           w.part_ml, w.row0);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (out_dtype == 1)
    k_decode_combine<D, true><<<B, 256, 0, st>>>(w.gates, w.rows, w.part_acc, w.part_ml, Hs, nc,
                                                out, 1, accumulate);
  else
    k_decode_combine<D, false><<<B, 256, 0, st>>>(w.gates, w.rows, w.part_acc, w.part_ml, Hs, nc,
                                                 out, 1, accumulate);
  return hipGetLastError();
}

hipError_t launch_shared_decode(const void* q, const void* k, const void* v, int dtype,
                                void* k_cache, void* v_cache, int32_t* cache_len, int B, int Hs,
                                int d, int cap, int window, float rope_base, int rope_mode,
                                float scale, void* out, int out_dtype, int accumulate,
                                int32_t* dev_status, void* ws, hipStream_t st) {
#define NAMOH_SDEC(DD, BF)                                                                    \
  return run_shared_decode<DD, BF>(q, k, v, k_cache, v_cache, cache_len, B, Hs, cap, window, \
                                   rope_base, rope_mode, scale, out, out_dtype, accumulate,  \
                                   dev_status, ws, st)
  if (dtype == 1) {
    if (d == 32) NAMOH_SDEC(32, true);
    if (d == 64) NAMOH_SDEC(64, true);
    NAMOH_SDEC(128, true);
  }
  if (d == 32) NAMOH_SDEC(32, false);
  if (d == 64) NAMOH_SDEC(64, false);
  NAMOH_SDEC(128, false);
#undef NAMOH_SDEC
}

hipError_t launch_shared_prefill_cache(const void* k, const void* v, int dtype, int B, int T,
                                       int Hs, int d, int cap, float rope_base, int rope_mode,
                                       void* k_cache, void* v_cache, int32_t* cache_len,
                                       hipStream_t st) {
  const long first = T > cap ? static_cast<long>(T) - cap : 0;
  const long nrows = static_cast<long>(B) * Hs * (T - first);
  const long threads = nrows * (d / 2);
  const unsigned grid = static_cast<unsigned>((threads + 255) / 256);
  const double log_base = rope_mode == 2 ? 0.0 : std::log(static_cast<double>(rope_base));
#define NAMOH_SPC(DD, BF)                                                                       \
  k_shared_prefill_cache<DD, BF><<<grid, 256, 0, st>>>(k, v, T, Hs, cap, first, log_base,       \
                                                        rope_mode, k_cache, v_cache, cache_len, \
                                                        nrows)
  if (dtype == 1) {
    if (d == 32) NAMOH_SPC(32, true);
    else if (d == 64) NAMOH_SPC(64, true);
    else NAMOH_SPC(128, true);
  } else {
    if (d == 32) NAMOH_SPC(32, false);
    else if (d == 64) NAMOH_SPC(64, false);
    else NAMOH_SPC(128, false);
  }
#undef NAMOH_SPC
  return hipGetLastError();
}

hipError_t launch_decode(const float* logits, const float* bias, const void* q, const void* k,
                         const void* v, int dtype, void* k_cache,
                         void* v_cache, int32_t* cache_len,
                         const int32_t* seq_pos, int B, int H, int K, int d,
                         int cap, float rope_base, int rope_mode,
                         int gate_mode, float scale, int32_t* topk_idx,
                         float* gates, void* out, int out_dtype,
                         int32_t* dev_status, void* ws, hipStream_t st) {
#define NAMOH_DEC(DD, BF)                                                               \
  return run_decode<DD, BF>(logits, bias, q, k, v, k_cache, v_cache, cache_len, seq_pos, B, H, \
                            K, cap, rope_base, rope_mode, gate_mode, scale, topk_idx,    \
                            gates, out, out_dtype, dev_status, ws, st)
  if (dtype == 1) {
    if (d == 32) NAMOH_DEC(32, true);
    if (d == 64) NAMOH_DEC(64, true);
    NAMOH_DEC(128, true);
  }
  if (d == 32) NAMOH_DEC(32, false);
  if (d == 64) NAMOH_DEC(64, false);
  NAMOH_DEC(128, false);
#undef NAMOH_DEC
}

hipError_t launch_decode_grouped(const float* logits, const void* q, const void* k, const void* v,
                                 void* k_cache, void* v_cache, int32_t* cache_len,
                                 const int32_t* seq_pos, int B, int H, int K, int G, int d, int cap,
                                 float rope_base, int rope_mode, int gate_mode, float scale,
                                 int32_t* topk_idx, float* gates, void* out, int out_dtype,
                                 int32_t* dev_status, void* ws, hipStream_t st) {
#define NAMOH_DECG(DD, GG)                                                                    \
  return run_decode<DD, true, GG>(logits, nullptr, q, k, v, k_cache, v_cache, cache_len, seq_pos, \
                                  B, H, K, cap, rope_base, rope_mode, gate_mode, scale, topk_idx, \
                                  gates, out, out_dtype, dev_status, ws, st)
  if (d == 64) {
    if (G == 1) NAMOH_DECG(64, 1);
    if (G == 2) NAMOH_DECG(64, 2);
    if (G == 4) NAMOH_DECG(64, 4);
    if (G == 8) NAMOH_DECG(64, 8);
  } else if (d == 128) {
    if (G == 1) NAMOH_DECG(128, 1);
    if (G == 2) NAMOH_DECG(128, 2);
    if (G == 4) NAMOH_DECG(128, 4);
    if (G == 8) NAMOH_DECG(128, 8);
  }
#undef NAMOH_DECG
  return hipErrorInvalidValue;
}

}  // namespace namoh
