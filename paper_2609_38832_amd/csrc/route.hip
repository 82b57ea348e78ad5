// Router top-K, gates, and the packed per-head token permutation.
//
// Sec. 3.1, Eq. namoh-gates: S_K(t) = TopK of the token's head scores,
// m_{t,i}, gates.  Sec. 3.1 (ordered index sets I_i) and Sec. 3.2 (packing of
// every (batch, head) subsequence): the permutation is a stable counting sort
// of the (token, head) pairs by segment b*H + h.
//
// Two or three launches; no global atomics, so every output is deterministic
// (the loss-free-balancing variant orders by biased affinities, see
// k_route_count; k_route_bias_update applies the per-batch bias step):
//   1. k_route_count   eight lanes per token, 64 tokens per workgroup: K
//                      rounds of a cooperative argmax under the total order
//                      (logit desc, head asc), the gates, and for every
//                      selected (token, head) its rank among the chunk's
//                      tokens routed to that head (stored in slot_pos for
//                      now), plus the chunk's per-head counts.
//   2. k_route_scan    one wave per (b, h) segment: exclusive scan of the
//                      segment's chunk counts and the head length n (only
//                      for long sequences; otherwise the scatter sums its
//                      own prefixes from the counts, one launch fewer).
//   3. k_route_scatter one workgroup per chunk: the segment offsets of
//                      sequence b are b*T*K plus a scan of its H head
//                      lengths (every sequence contributes exactly T*K
//                      pairs); a pair's packed position = segment offset +
//                      earlier chunks of the segment + its rank in the chunk.
#include <climits>

#include "common.h"
#include "internal.h"
#include "launch.h"

namespace namoh {

constexpr int kRC = kRouteChunk;   // tokens per chunk
constexpr int kLPT = 8;            // lanes per token in k_route_count
constexpr int kCountThreads = kRC * kLPT;
constexpr int kCountWaves = kCountThreads / kWave;
constexpr int kScatterThreads = 512;
constexpr long kFusedScan = 8192;   // chunks x heads per sequence summed inside the scatter

// Order-preserving integer key of a float logit (-0.0 first made +0.0); the
// map is its own inverse.
NAMOH_DEV int logit_key(float f) {
  const int bits = __float_as_int(f == 0.f ? 0.f : f);
  return bits ^ ((bits >> 31) & 0x7FFFFFFF);
}
NAMOH_DEV float key_logit(int k) { return __int_as_float(k ^ ((k >> 31) & 0x7FFFFFFF)); }

// Candidate (logit, head) as one unsigned 64-bit value whose order is the
// selection order: the logit key (sign flipped to unsigned order) above,
// 255 - head below (equal logits: the lower head index is larger).  0 is
// below every real candidate and marks padding and removed heads.
NAMOH_DEV uint64_t cand(int key, int j) {
  return (static_cast<uint64_t>(static_cast<uint32_t>(key) ^ 0x80000000u) << 32) |
         static_cast<uint32_t>(255 - j);
}
NAMOH_DEV int cand_head(uint64_t c) { return 255 - static_cast<int>(c & 0xFFu); }
NAMOH_DEV int cand_key(uint64_t c) {
  return static_cast<int>(static_cast<uint32_t>(c >> 32) ^ 0x80000000u);
}

// 64-bit max with the value of another lane of the 8-lane group, moved by a
// DPP lane pattern (quad_perm [1,0,3,2] = xor 1, [2,3,0,1] = xor 2,
// row_half_mirror = lane 7 - i inside each 8-lane group).
template <int CTRL>
NAMOH_DEV uint64_t max_dpp(uint64_t x) {
  const int lo = __builtin_amdgcn_mov_dpp(static_cast<int>(static_cast<uint32_t>(x)), CTRL, 0xF,
                                          0xF, true);
  const int hi = __builtin_amdgcn_mov_dpp(static_cast<int>(static_cast<uint32_t>(x >> 32)), CTRL,
                                          0xF, 0xF, true);
  const uint64_t y = (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) |
                     static_cast<uint32_t>(lo);
  return y > x ? y : x;
}

// 8 lanes per token, lane `sub` holding heads sub*HL .. sub*HL + HL - 1.
// Round k: every lane takes the largest of its remaining candidates, three
// DPP steps reduce the group to the winner (after the first two the four
// lanes of each quad agree, so the mirror exchange pairs the two quads), and
// the owning lane removes it.  K <= KMAX <= 8 keeps the winners in
// registers and lane k of the group stores round k; otherwise lane 0 stores
// and rescales in place.
//
// BIASED (loss-free balancing, App. "Auxiliary-Loss-Free Balancing", Eq.
// namoh-biased-routing): the order is (score desc, head asc) with score =
// float(a + b), a = softmax over the H logits formed in double (exp of
// l - max, sum over the token's eight lanes), b the head's bias, and the
// gates are the selected affinities a (rounded to float, not renormalised);
// each lane writes the gates of the heads it owns.
template <int HMAX, int KMAX, bool BIASED>
__global__ __launch_bounds__(kCountThreads) void k_route_count(
    const float* __restrict__ logits, const float* __restrict__ bias, int T, int H, int K,
    int gate_mode, int nchunk, int32_t* __restrict__ topk_idx, float* __restrict__ gates,
    int32_t* __restrict__ slot_rank, int32_t* __restrict__ chunk_counts) {
  constexpr int HL = HMAX / kLPT;
  __shared__ int s_wcnt[kCountWaves][HMAX];
  const int b = block_x() / nchunk;
  const int c = block_x() - b * nchunk;
  const int tid = thread_x();
  const int sub = tid % kLPT;
  const int wave = tid / kWave, lane = tid % kWave;
  const int t = c * kRC + tid / kLPT;
  const bool valid = t < T;
  const size_t row = static_cast<size_t>(b) * T + (valid ? t : 0);

  float val[HL];
  const float* lp = logits + row * H + sub * HL;
  const bool vec = H == HMAX && (reinterpret_cast<uintptr_t>(logits) & 31) == 0;
  if (vec && valid) {   // whole rows of a 32-byte aligned array: vector loads
    if constexpr (HL == 8) {
      const float4 x0 = reinterpret_cast<const float4*>(lp)[0];
      const float4 x1 = reinterpret_cast<const float4*>(lp)[1];
      val[0] = x0.x; val[1] = x0.y; val[2] = x0.z; val[3] = x0.w;
      val[4] = x1.x; val[5] = x1.y; val[6] = x1.z; val[7] = x1.w;
    } else if constexpr (HL == 4) {
      const float4 x0 = *reinterpret_cast<const float4*>(lp);
      val[0] = x0.x; val[1] = x0.y; val[2] = x0.z; val[3] = x0.w;
    } else if constexpr (HL == 2) {
      const float2 x0 = *reinterpret_cast<const float2*>(lp);
      val[0] = x0.x; val[1] = x0.y;
    } else {
      val[0] = lp[0];
    }
  } else {
#pragma unroll
    for (int e = 0; e < HL; ++e) val[e] = (valid && sub * HL + e < H) ? lp[e] : -INFINITY;
  }
  uint64_t ck[HL];
  float aff[BIASED ? HL : 1];   // BIASED: the affinities of this lane's heads
  if constexpr (BIASED) {
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < HL; ++e)
      if (sub * HL + e < H) mx = fmaxf(mx, val[e]);
#pragma unroll
    for (int o = 1; o < kLPT; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kLPT));
    double ex[HL], z = 0.0;
#pragma unroll
    for (int e = 0; e < HL; ++e) {
      ex[e] = sub * HL + e < H ? exp(static_cast<double>(val[e]) - static_cast<double>(mx)) : 0.0;
      z += ex[e];
    }
#pragma unroll
    for (int o = 1; o < kLPT; o <<= 1) z += __shfl_xor(z, o, kLPT);
#pragma unroll
    for (int e = 0; e < HL; ++e) {
      const int j = sub * HL + e;
      const double a = ex[e] / z;
      aff[e] = static_cast<float>(a);
      const float score = j < H ? static_cast<float>(a + static_cast<double>(bias[j])) : 0.f;
      ck[e] = (valid && j < H) ? cand(logit_key(score), j) : 0ull;
    }
  } else {
#pragma unroll
    for (int e = 0; e < HL; ++e) {
      const int j = sub * HL + e;
      ck[e] = (valid && j < H) ? cand(logit_key(val[e]), j) : 0ull;
    }
  }

  int32_t* tk = topk_idx + row * K;
  float* gk = gates + row * K;
  unsigned own = 0;              // selected heads held by this lane (bit e)
  int own_k[HL];                 // ... and the round that selected each
  float lmax = 0.f, denom = 0.f;
  int wj[KMAX <= 8 ? KMAX : 1];
  float we[KMAX <= 8 ? KMAX : 1];
#pragma unroll
  for (int e = 0; e < HL; ++e) own_k[e] = 0;
#pragma unroll
  for (int k = 0; k < (KMAX <= 8 ? KMAX : 1); ++k) {
    wj[k] = 0;
    we[k] = 0.f;
  }
#pragma unroll(KMAX <= 8 ? KMAX : 1)
  for (int k = 0; k < (KMAX <= 8 ? KMAX : K); ++k) {
    if (KMAX <= 8 && k >= K) break;
    uint64_t best = ck[0];
#pragma unroll
    for (int e = 1; e < HL; ++e) best = ck[e] > best ? ck[e] : best;
    best = max_dpp<kDppXor1>(best);
    best = max_dpp<kDppXor2>(best);
    best = max_dpp<kDppRowHalfMirror>(best);
#pragma unroll
    for (int e = 0; e < HL; ++e)
      if (valid && ck[e] == best) {
        ck[e] = 0ull;
        own |= 1u << e;
        own_k[e] = k;
      }
    const int bj = cand_head(best);
    float e = 0.f;
    if constexpr (!BIASED) {
      const float v = key_logit(cand_key(best));
      if (k == 0) lmax = v;
      e = expf(v - lmax);
      denom += e;
    }
    if constexpr (KMAX <= 8) {
#pragma unroll
      for (int kk = 0; kk < KMAX; ++kk)
        if (kk == k) {
          wj[kk] = bj;
          we[kk] = e;
        }
    } else if (valid && sub == 0) {
      tk[k] = bj;
      if constexpr (!BIASED) gk[k] = e;  // unnormalised; scaled below
    }
  }
  if (!BIASED && gate_mode == 1) {  // softmax over all H logits, no renormalisation
    float part = 0.f;
#pragma unroll
    for (int e = 0; e < HL; ++e)
      if (sub * HL + e < H) part += expf(val[e] - lmax);
#pragma unroll
    for (int o = 1; o < kLPT; o <<= 1) part += __shfl_xor(part, o, kLPT);
    denom = part;
  }
  const float inv = BIASED ? 0.f : 1.f / denom;
  int mj = 0;
  float me = 0.f;
  if constexpr (KMAX <= 8) {
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
      if (sub == k) {
        mj = wj[k];
        me = we[k];
      }
  }

  // Ranks inside the chunk.  Ballot e marks the lanes holding their bit e;
  // head h = s*HL + e lives in lane s of every token group, so the wave's
  // tokens routed to h are ballot_e & (lanes s, s+8, ...).
  uint64_t bal[HL];
#pragma unroll
  for (int e = 0; e < HL; ++e) bal[e] = __ballot((own >> e) & 1u);
  const uint64_t same_sub = 0x0101010101010101ull << sub;
  if (lane < HMAX) {   // wave count of head `lane`
    const int hs = lane / HL, he = lane % HL;
    uint64_t be = bal[0];
#pragma unroll
    for (int e = 1; e < HL; ++e) be = he == e ? bal[e] : be;
    s_wcnt[wave][lane] = __popcll(be & (0x0101010101010101ull << hs));
  }
  __syncthreads();
  if (valid) {
    const uint64_t below = lanemask_lt() & same_sub;
    int32_t* rk = slot_rank + row * K;
#pragma unroll
    for (int e = 0; e < HL; ++e)
      if ((own >> e) & 1u) {
        const int h = sub * HL + e;
        int r = __popcll(bal[e] & below);
        for (int w = 0; w < wave; ++w) r += s_wcnt[w][h];
        rk[own_k[e]] = r;
      }
  }
  if (tid < H) {
    int n = 0;
#pragma unroll
    for (int w = 0; w < kCountWaves; ++w) n += s_wcnt[w][tid];
    chunk_counts[(static_cast<size_t>(b) * H + tid) * nchunk + c] = n;
  }
  // the selections and gates are stored last: a barrier after a global
  // store would wait for the store to complete
  if constexpr (BIASED) {
    if constexpr (KMAX <= 8)
      if (valid && sub < K) tk[sub] = mj;
    if (valid) {
#pragma unroll
      for (int e = 0; e < HL; ++e)
        if ((own >> e) & 1u) gk[own_k[e]] = aff[e];
    }
  } else if constexpr (KMAX <= 8) {
    if (valid && sub < K) {
      tk[sub] = mj;
      gk[sub] = me * inv;
    }
  } else if (valid && sub == 0) {
    for (int k = 0; k < K; ++k) gk[k] *= inv;
  }
}

// Loss-free balancing update (App. "Auxiliary-Loss-Free Balancing", Eq.
// namoh-loss-free): c_i = sum over the batch of head_len[b][i], c_bar =
// B T K / H, b_i += eta sign(c_bar - c_i); the sign is taken exactly as
// sign(B T K - H c_i) in 64-bit integers, the update is one float add.
__global__ __launch_bounds__(kWave) void k_route_bias_update(const int32_t* __restrict__ head_len,
                                                             int B, long long total, int H,
                                                             float eta, float* __restrict__ bias) {
  const int h = thread_x();
  if (h >= H) return;
  long long c = 0;
  for (int b = 0; b < B; ++b) c += head_len[static_cast<size_t>(b) * H + h];
  const long long diff = total - static_cast<long long>(H) * c;
  const float step = diff > 0 ? eta : (diff < 0 ? -eta : 0.f);
  bias[h] = bias[h] + step;
}

__global__ __launch_bounds__(kWave) void k_route_scan(
    const int32_t* __restrict__ counts, int nchunk, int32_t* __restrict__ within,
    int32_t* __restrict__ head_len) {
  const int s = block_x();
  const int lane = thread_x();
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

// FUSED: the chunk prefixes and head lengths of sequence b are summed here
// from the chunk counts (8 lanes per head, used when the sequence has few
// chunks x heads), instead of being read from k_route_scan's output.
template <bool FUSED>
__global__ __launch_bounds__(kScatterThreads) void k_route_scatter(
    const int32_t* __restrict__ topk_idx, int B, int T, int H, int K, int nchunk,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ within,
    int32_t* __restrict__ head_len, int32_t* __restrict__ seg_offsets,
    int32_t* __restrict__ perm_token, int32_t* __restrict__ slot_pos) {
  __shared__ int s_base[64];
  __shared__ int s_before[64];
  __shared__ int s_len[64];
  const int b = block_x() / nchunk;
  const int c = block_x() - b * nchunk;
  const int tid = thread_x();
  if constexpr (FUSED) {
    static_assert(kScatterThreads == 8 * 64, "8 lanes per head");
    const int h = tid / 8, j = tid % 8;
    int before = 0, total = 0;
    // eight independent loads per round (indices clamped, no load under a
    // branch, so they are in flight together); lanes of heads >= H add 0
    const int32_t* cp = counts + (static_cast<size_t>(b) * H + min(h, H - 1)) * nchunk;
    for (int c0 = j; c0 < nchunk; c0 += 64) {
      int x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = cp[min(c0 + 8 * u, nchunk - 1)];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int cc = c0 + 8 * u;
        const int v = cc < nchunk && h < H ? x[u] : 0;
        total += v;
        before += cc < c ? v : 0;
      }
    }
    before = group_sum_i<8>(before);
    total = group_sum_i<8>(total);
    if (j == 0) {
      s_before[h] = before;
      s_len[h] = total;
    }
    __syncthreads();
  }
  if (tid < kWave) {
    // segment offsets of sequence b and this chunk's start in each segment
    const int hl = tid < H ? (FUSED ? s_len[tid] : head_len[static_cast<size_t>(b) * H + tid]) : 0;
    const int seg_off = b * T * K + wave_inclusive_scan(hl) - hl;
    if (tid < H) {
      if (c == 0) {
        seg_offsets[static_cast<size_t>(b) * H + tid] = seg_off;
        if (FUSED) head_len[static_cast<size_t>(b) * H + tid] = hl;
      }
      s_base[tid] = seg_off + (FUSED ? s_before[tid]
                                     : within[(static_cast<size_t>(b) * H + tid) * nchunk + c]);
    }
    if (c == 0 && b == B - 1 && tid == 0) seg_offsets[static_cast<size_t>(B) * H] = B * T * K;
  }
  __syncthreads();
  const int t0 = c * kRC;
  const int nt = min(kRC, T - t0);
  const size_t e0 = (static_cast<size_t>(b) * T + t0) * K;
  const unsigned nr = static_cast<unsigned>(B) * T * K;
  for (int e = tid; e < nt * K; e += kScatterThreads) {
    const int h = topk_idx[e0 + e];
    const int rank = slot_pos[e0 + e];
    // the head and the in-chunk rank come from k_route_count; a position
    // outside [0, B*T*K) can only come from a corrupted workspace and is
    // not stored
    const int pos = static_cast<unsigned>(h) < static_cast<unsigned>(H)
                        ? s_base[min(max(h, 0), H - 1)] + rank : -1;
    if (static_cast<unsigned>(pos) < nr) perm_token[pos] = t0 + e / K;
    slot_pos[e0 + e] = pos;
  }
}

size_t route_workspace_bytes(int B, int T, int H, int /*K*/) {
  const size_t nchunk = (static_cast<size_t>(T) + kRouteChunk - 1) / kRouteChunk;
  const size_t L = static_cast<size_t>(B) * H * nchunk;
  return 2 * align_up(L * sizeof(int32_t));
}

hipError_t launch_route_bias_update(const int32_t* head_len, int B, int T, int H, int K,
                                   float eta, float* bias, hipStream_t st) {
  k_route_bias_update<<<1, kWave, 0, st>>>(head_len, B, static_cast<long long>(B) * T * K, H,
                                            eta, bias);
  return hipGetLastError();
}

hipError_t launch_route(const float* logits, const float* bias, int B, int T, int H, int K,
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
#define NAMOH_RC(HM, KM)                                                                   \
  do {                                                                                     \
    if (bias)                                                                              \
      launch_k("route_count", k_route_count<HM, KM, true>, grid, dim3(kCountThreads), st,  \
               logits, bias, T, H, K, gate_mode, nchunk, topk_idx, gates, slot_pos,        \
               counts);                                                                    \
    else                                                                                   \
      launch_k("route_count", k_route_count<HM, KM, false>, grid, dim3(kCountThreads), st, \
               logits, nullptr, T, H, K, gate_mode, nchunk, topk_idx, gates, slot_pos,     \
               counts);                                                                    \
  } while (0)
  const bool small_k = K <= 8;
  if (H <= 8) NAMOH_RC(8, 8);
  else if (H <= 16) { if (small_k) NAMOH_RC(16, 8); else NAMOH_RC(16, 64); }
  else if (H <= 32) { if (small_k) NAMOH_RC(32, 8); else NAMOH_RC(32, 64); }
  else { if (small_k) NAMOH_RC(64, 8); else NAMOH_RC(64, 64); }
#undef NAMOH_RC
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (static_cast<long>(nchunk) * H <= kFusedScan) {
    launch_k("route_scatter", k_route_scatter<true>, grid, dim3(kScatterThreads), st, topk_idx,
             B, T, H, K, nchunk, counts, within, head_len, seg_offsets, perm_token, slot_pos);
  } else {
    launch_k("route_scan", k_route_scan, dim3(B * H), dim3(kWave), st, counts, nchunk, within,
             head_len);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    launch_k("route_scatter", k_route_scatter<false>, grid, dim3(kScatterThreads), st, topk_idx,
             B, T, H, K, nchunk, counts, within, head_len, seg_offsets, perm_token, slot_pos);
  }
  return hipGetLastError();
}

}  // namespace namoh
