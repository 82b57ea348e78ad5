// Router top-K, gates, and the packed per-head token permutation.
//
// Sec. 3.1, Eq. namoh-gates: S_K(t) = TopK of the token's head scores,
// m_{t,i}, gates.  Sec. 3.1 (ordered index sets I_i) and Sec. 3.2 (packing of
// every (batch, head) subsequence): the permutation is a stable counting sort
// of the (token, head) pairs by segment b*H + h.
//
// Three launches; the only atomics are integer adds of counts, so every
// output is deterministic:
//   1. k_route_count   eight lanes per token, 64 tokens per workgroup: K
//                      rounds of a cooperative argmax under the total order
//                      (logit desc, head asc) on order-preserving integer
//                      keys, the gates, and per 64-token chunk the number of
//                      tokens routed to each head (LDS integer adds, exact).
//   2. k_route_scan    one wave per (b, h) segment: exclusive scan of the
//                      segment's chunk counts and the head length n.
//   3. k_route_scatter one wave per chunk: the segment offsets of sequence b
//                      are b*T*K plus a scan of its H head lengths (every
//                      sequence contributes exactly T*K pairs); a pair's
//                      packed position = segment offset + earlier chunks of the
//                      segment + lower lanes of this chunk routed to the same
//                      head (popcount of ballot & lanes-below).
#include <climits>

#include "common.h"
#include "internal.h"

namespace namoh {

constexpr int kRC = kRouteChunk;   // tokens per chunk
constexpr int kLPT = 8;            // lanes per token in k_route_count
constexpr int kCountThreads = kRC * kLPT;

// Order-preserving integer key of a float logit (-0.0 first made +0.0); the
// map is its own inverse.
NAMOH_DEV int logit_key(float f) {
  const int bits = __float_as_int(f == 0.f ? 0.f : f);
  return bits ^ ((bits >> 31) & 0x7FFFFFFF);
}
NAMOH_DEV float key_logit(int k) { return __int_as_float(k ^ ((k >> 31) & 0x7FFFFFFF)); }

// 8 lanes per token, each holding HMAX/8 heads.  Round k picks the largest
// (key, -head) pair below the previous round's winner: every lane scans its
// heads, then three xor-shuffles inside the 8-lane group reduce to the
// winner (larger key, then lower head index).  Real logits have keys above
// INT_MIN, so the INT_MIN padding of heads >= H never wins while K <= H.
template <int HMAX, int KMAX>
__global__ __launch_bounds__(kCountThreads) void k_route_count(
    const float* __restrict__ logits, int T, int H, int K, int gate_mode,
    int nchunk, int32_t* __restrict__ topk_idx, float* __restrict__ gates,
    int32_t* __restrict__ chunk_counts) {
  constexpr int HL = HMAX / kLPT;
  __shared__ int s_cnt[64];
  const int b = blockIdx.x / nchunk;
  const int c = blockIdx.x - b * nchunk;
  const int tid = threadIdx.x;
  const int sub = tid % kLPT;
  const int t = c * kRC + tid / kLPT;
  const bool valid = t < T;
  const size_t row = static_cast<size_t>(b) * T + (valid ? t : 0);
  if (tid < 64) s_cnt[tid] = 0;

  int key[HL];
  float val[HL];
  const float* lp = logits + row * H;
#pragma unroll
  for (int e = 0; e < HL; ++e) {
    const int j = sub * HL + e;
    val[e] = (valid && j < H) ? lp[j] : -INFINITY;
    key[e] = (valid && j < H) ? logit_key(val[e]) : INT_MIN;
  }
  int32_t* tk = topk_idx + row * K;
  float* gk = gates + row * K;
  int pk = INT_MAX, pj = -1;     // previous winner
  unsigned own = 0;              // selected heads owned by this lane
  float lmax = 0.f, denom = 0.f;
  // with K <= KMAX (<= 8) the winners stay in registers and lane k of the
  // group stores round k; otherwise lane 0 stores and rescales in place
  int wj[KMAX];
  float we[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    wj[k] = 0;
    we[k] = 0.f;
  }
#pragma unroll (KMAX <= 8 ? KMAX : 1)
  for (int k = 0; k < (KMAX <= 8 ? KMAX : K); ++k) {
    if (KMAX <= 8 && k >= K) break;
    int bk = INT_MIN, bj = INT_MAX;
#pragma unroll
    for (int e = 0; e < HL; ++e) {
      const int j = sub * HL + e;
      const bool cand = key[e] < pk || (key[e] == pk && j > pj);
      const bool better = cand && (key[e] > bk || (key[e] == bk && j < bj));
      bk = better ? key[e] : bk;
      bj = better ? j : bj;
    }
#pragma unroll
    for (int o = 1; o < kLPT; o <<= 1) {
      const int ok = __shfl_xor(bk, o, kLPT);
      const int oj = __shfl_xor(bj, o, kLPT);
      const bool better = ok > bk || (ok == bk && oj < bj);
      bk = better ? ok : bk;
      bj = better ? oj : bj;
    }
    pk = bk;
    pj = bj;
    if (bj / HL == sub) own |= 1u << (bj - sub * HL);
    const float v = key_logit(bk);
    if (k == 0) lmax = v;
    const float e = expf(v - lmax);
    denom += e;
    if constexpr (KMAX <= 8) {
      wj[k] = bj;
      we[k] = e;
    } else if (valid && sub == 0) {
      tk[k] = bj;
      gk[k] = e;  // unnormalised; scaled below
    }
  }
  if (gate_mode == 1) {  // softmax over all H logits, no renormalisation
    float part = 0.f;
#pragma unroll
    for (int e = 0; e < HL; ++e)
      if (sub * HL + e < H) part += expf(val[e] - lmax);
#pragma unroll
    for (int o = 1; o < kLPT; o <<= 1) part += __shfl_xor(part, o, kLPT);
    denom = part;
  }
  const float inv = 1.f / denom;
  if constexpr (KMAX <= 8) {
    int mj = 0;
    float me = 0.f;
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
      if (sub == k) {
        mj = wj[k];
        me = we[k];
      }
    if (valid && sub < K) {
      tk[sub] = mj;
      gk[sub] = me * inv;
    }
  } else if (valid && sub == 0) {
    for (int k = 0; k < K; ++k) gk[k] *= inv;
  }
  __syncthreads();
  if (valid)
#pragma unroll
    for (int e = 0; e < HL; ++e)
      if ((own >> e) & 1u) atomicAdd(&s_cnt[sub * HL + e], 1);
  __syncthreads();
  if (tid < H) chunk_counts[(static_cast<size_t>(b) * H + tid) * nchunk + c] = s_cnt[tid];
}

__global__ __launch_bounds__(kWave) void k_route_scan(
    const int32_t* __restrict__ counts, int nchunk, int32_t* __restrict__ within,
    int32_t* __restrict__ head_len) {
  const int s = blockIdx.x;
  const int lane = threadIdx.x;
  const size_t base = static_cast<size_t>(s) * nchunk;
  int carry = 0;
  for (int i0 = 0; i0 < nchunk; i0 += kWave) {
    const int i = i0 + lane;
    const int x = i < nchunk ? counts[base + i] : 0;
    const int incl = wave_inclusive_scan(x);
    if (i < nchunk) within[base + i] = carry + incl - x;
    carry += __shfl(incl, kWave - 1);
  }
  if (lane == 0) head_len[s] = carry;
}

__global__ __launch_bounds__(kRC) void k_route_scatter(
    const int32_t* __restrict__ topk_idx, int B, int T, int H, int K, int nchunk,
    const int32_t* __restrict__ within, const int32_t* __restrict__ head_len,
    int32_t* __restrict__ seg_offsets, int32_t* __restrict__ perm_token,
    int32_t* __restrict__ slot_pos) {
  __shared__ uint64_t s_bal[64];
  __shared__ int s_base[64];
  const int b = blockIdx.x / nchunk;
  const int c = blockIdx.x - b * nchunk;
  const int lane = threadIdx.x;
  const int t = c * kRC + lane;
  const bool valid = t < T;
  const size_t row = static_cast<size_t>(b) * T + (valid ? t : 0);
  const int32_t* tk = topk_idx + row * K;

  // segment offsets of sequence b
  const int hl = lane < H ? head_len[static_cast<size_t>(b) * H + lane] : 0;
  const int seg_off = b * T * K + wave_inclusive_scan(hl) - hl;
  if (lane < H) {
    if (c == 0) seg_offsets[static_cast<size_t>(b) * H + lane] = seg_off;
    s_base[lane] = seg_off + within[(static_cast<size_t>(b) * H + lane) * nchunk + c];
  }
  if (c == 0 && b == B - 1 && lane == 0) seg_offsets[static_cast<size_t>(B) * H] = B * T * K;

  uint64_t mask = 0;
  if (valid)
    for (int k = 0; k < K; ++k) mask |= 1ull << tk[k];
  uint64_t mine = 0;
  for (int h = 0; h < H; ++h) {
    const uint64_t bal = __ballot((mask >> h) & 1ull);
    if (lane == h) mine = bal;
  }
  s_bal[lane] = mine;
  __syncthreads();
  if (valid) {
    const uint64_t below = lanemask_lt();
    int32_t* sp = slot_pos + row * K;
    for (int k = 0; k < K; ++k) {
      const int h = tk[k];
      const int pos = s_base[h] + __popcll(s_bal[h] & below);
      perm_token[pos] = t;
      sp[k] = pos;
    }
  }
}

size_t route_workspace_bytes(int B, int T, int H, int /*K*/) {
  const size_t nchunk = (static_cast<size_t>(T) + kRouteChunk - 1) / kRouteChunk;
  const size_t L = static_cast<size_t>(B) * H * nchunk;
  return 2 * align_up(L * sizeof(int32_t));
}

hipError_t launch_route(const float* logits, int B, int T, int H, int K,
                        int gate_mode, int32_t* topk_idx, float* gates,
                        int32_t* head_len, int32_t* seg_offsets,
                        int32_t* perm_token, int32_t* slot_pos, void* ws,
                        hipStream_t st) {
  const int nchunk = (T + kRouteChunk - 1) / kRouteChunk;
  const size_t L = static_cast<size_t>(B) * H * nchunk;
  Carver cv(ws);
  int32_t* counts = cv.take<int32_t>(L);
  int32_t* within = cv.take<int32_t>(L);
  const dim3 grid(static_cast<unsigned>(static_cast<size_t>(B) * nchunk));
#define NAMOH_RC(HM, KM) \
  k_route_count<HM, KM><<<grid, kCountThreads, 0, st>>>(logits, T, H, K, gate_mode, nchunk, topk_idx, gates, counts)
  const bool small_k = K <= 8;
  if (H <= 8) NAMOH_RC(8, 8);
  else if (H <= 16) { if (small_k) NAMOH_RC(16, 8); else NAMOH_RC(16, 64); }
  else if (H <= 32) { if (small_k) NAMOH_RC(32, 8); else NAMOH_RC(32, 64); }
  else { if (small_k) NAMOH_RC(64, 8); else NAMOH_RC(64, 64); }
#undef NAMOH_RC
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_route_scan<<<B * H, kWave, 0, st>>>(counts, nchunk, within, head_len);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_route_scatter<<<grid, kRC, 0, st>>>(topk_idx, B, T, H, K, nchunk, within, head_len,
                                        seg_offsets, perm_token, slot_pos);
  return hipGetLastError();
}

}  // namespace namoh
