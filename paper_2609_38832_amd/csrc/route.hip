// Router top-K, gates, and the packed per-head token permutation.
//
// Sec. 3.1, Eq. namoh-gates: S_K(t) = TopK of the token's head scores,
// m_{t,i}, gates.  Sec. 3.1 (ordered index sets I_i) and Sec. 3.2 (packing of
// every (batch, head) subsequence): the permutation is a stable counting sort
// of the (token, head) pairs by segment b*H + h.
//
// Three launches, no atomics, so every output is deterministic:
//   1. k_route_count   one lane per token: K passes of a register argmax over
//                      the H logits (strict '>' scanning heads upward, so equal
//                      logits resolve to the lower head index), gates, and per
//                      256-token chunk the number of tokens routed to each head
//                      (wave ballot + popcount).
//   2. k_route_scan    one workgroup: exclusive scan of the chunk counts laid
//                      out [b][h][chunk], which is exactly segment order, then
//                      tokens-in-chunk order.  Gives seg_offsets and head_len.
//   3. k_route_scatter recomputes the chunk's ballots; a pair's packed
//                      position = chunk base + earlier waves' counts + the
//                      number of lower lanes in its wave routed to the same
//                      head (popcount of ballot & lanes-below).
#include "common.h"
#include "internal.h"

namespace namoh {

template <int HMAX>
__global__ __launch_bounds__(kRouteChunk) void k_route_count(
    const float* __restrict__ logits, int T, int H, int K, int gate_mode,
    int nchunk, int32_t* __restrict__ topk_idx, float* __restrict__ gates,
    int32_t* __restrict__ chunk_counts) {
  const int b = blockIdx.x / nchunk;
  const int c = blockIdx.x - b * nchunk;
  const int t = c * kRouteChunk + threadIdx.x;
  const bool valid = t < T;
  const size_t row = static_cast<size_t>(b) * T + (valid ? t : 0);

  float l[HMAX];
  const float* lp = logits + row * H;
#pragma unroll
  for (int j = 0; j < HMAX; ++j) l[j] = (valid && j < H) ? lp[j] : 0.f;

  int32_t* tk = topk_idx + row * K;
  float* gk = gates + row * K;
  uint64_t taken = 0;
  float lmax = 0.f, denom = 0.f;
  for (int k = 0; k < K; ++k) {
    int best = -1;
    float bv = 0.f;
#pragma unroll
    for (int j = 0; j < HMAX; ++j) {
      const bool avail = (j < H) && !((taken >> j) & 1ull);
      const bool better = avail && (best < 0 || l[j] > bv);
      best = better ? j : best;
      bv = better ? l[j] : bv;
    }
    taken |= 1ull << best;
    if (k == 0) lmax = bv;
    const float e = expf(bv - lmax);
    denom += e;
    if (valid) {
      tk[k] = best;
      gk[k] = e;  // unnormalised; scaled below
    }
  }
  if (gate_mode == 1) {  // softmax over all H logits, no renormalisation
    denom = 0.f;
#pragma unroll
    for (int j = 0; j < HMAX; ++j)
      if (j < H) denom += expf(l[j] - lmax);
  }
  if (valid) {
    const float inv = 1.f / denom;
    for (int k = 0; k < K; ++k) gk[k] *= inv;
  }

  // per-chunk head counts
  __shared__ int s_cnt[kRouteChunk / kWave][64];
  const int lane = __lane_id();
  const int wave = threadIdx.x / kWave;
  int mine = 0;
  for (int h = 0; h < H; ++h) {
    const uint64_t bal = __ballot(valid && ((taken >> h) & 1ull));
    if (lane == h) mine = __popcll(bal);
  }
  s_cnt[wave][lane] = mine;
  __syncthreads();
  if (threadIdx.x < H) {
    int s = 0;
#pragma unroll
    for (int w = 0; w < kRouteChunk / kWave; ++w) s += s_cnt[w][threadIdx.x];
    chunk_counts[(static_cast<size_t>(b) * H + threadIdx.x) * nchunk + c] = s;
  }
}

constexpr int kScanThreads = 1024;
constexpr int kScanItems = 4;

__global__ __launch_bounds__(kScanThreads) void k_route_scan(
    const int32_t* __restrict__ counts, int L, int nchunk, int BH,
    int32_t* __restrict__ base, int32_t* __restrict__ seg_offsets,
    int32_t* __restrict__ head_len) {
  __shared__ int s_wave[kScanThreads / kWave];
  __shared__ int s_carry;
  const int tid = threadIdx.x;
  const int lane = __lane_id();
  const int wave = tid / kWave;
  if (tid == 0) s_carry = 0;
  __syncthreads();
  for (int start = 0; start < L; start += kScanThreads * kScanItems) {
    int v[kScanItems];
    int sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
      const int idx = start + tid * kScanItems + i;
      v[i] = idx < L ? counts[idx] : 0;
      sum += v[i];
    }
    const int incl = wave_inclusive_scan(sum);
    if (lane == kWave - 1) s_wave[wave] = incl;
    __syncthreads();
    if (wave == 0) {
      const int wv = lane < kScanThreads / kWave ? s_wave[lane] : 0;
      const int wi = wave_inclusive_scan(wv);
      if (lane < kScanThreads / kWave) s_wave[lane] = wi - wv;  // exclusive
    }
    __syncthreads();
    int run = s_carry + s_wave[wave] + incl - sum;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
      const int idx = start + tid * kScanItems + i;
      if (idx < L) {
        base[idx] = run;
        if (idx % nchunk == 0) seg_offsets[idx / nchunk] = run;
      }
      run += v[i];
    }
    __syncthreads();
    if (tid == kScanThreads - 1) s_carry = run;
    __syncthreads();
  }
  if (tid == 0) seg_offsets[BH] = s_carry;
  for (int s = tid; s < BH; s += kScanThreads) {
    int n = 0;
    for (int c = 0; c < nchunk; ++c) n += counts[static_cast<size_t>(s) * nchunk + c];
    head_len[s] = n;
  }
}

__global__ __launch_bounds__(kRouteChunk) void k_route_scatter(
    const int32_t* __restrict__ topk_idx, int T, int H, int K, int nchunk,
    const int32_t* __restrict__ base, int32_t* __restrict__ perm_token,
    int32_t* __restrict__ slot_pos) {
  __shared__ uint64_t s_bal[kRouteChunk / kWave][64];
  __shared__ int s_base[kRouteChunk / kWave][64];
  const int b = blockIdx.x / nchunk;
  const int c = blockIdx.x - b * nchunk;
  const int t = c * kRouteChunk + threadIdx.x;
  const bool valid = t < T;
  const int lane = __lane_id();
  const int wave = threadIdx.x / kWave;
  const size_t row = static_cast<size_t>(b) * T + (valid ? t : 0);
  const int32_t* tk = topk_idx + row * K;

  uint64_t mask = 0;
  if (valid)
    for (int k = 0; k < K; ++k) mask |= 1ull << tk[k];
  uint64_t mine = 0;
  for (int h = 0; h < H; ++h) {
    const uint64_t bal = __ballot((mask >> h) & 1ull);
    if (lane == h) mine = bal;
  }
  s_bal[wave][lane] = mine;
  __syncthreads();
  if (threadIdx.x < H) {
    const int h = threadIdx.x;
    int acc = base[(static_cast<size_t>(b) * H + h) * nchunk + c];
#pragma unroll
    for (int w = 0; w < kRouteChunk / kWave; ++w) {
      s_base[w][h] = acc;
      acc += __popcll(s_bal[w][h]);
    }
  }
  __syncthreads();
  if (valid) {
    const uint64_t below = lanemask_lt();
    int32_t* sp = slot_pos + row * K;
    for (int k = 0; k < K; ++k) {
      const int h = tk[k];
      const int pos = s_base[wave][h] + __popcll(s_bal[wave][h] & below);
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
  int32_t* base = cv.take<int32_t>(L);
  const dim3 grid(static_cast<unsigned>(static_cast<size_t>(B) * nchunk));
  if (H <= 8)
    k_route_count<8><<<grid, kRouteChunk, 0, st>>>(logits, T, H, K, gate_mode, nchunk, topk_idx, gates, counts);
  else if (H <= 16)
    k_route_count<16><<<grid, kRouteChunk, 0, st>>>(logits, T, H, K, gate_mode, nchunk, topk_idx, gates, counts);
  else if (H <= 32)
    k_route_count<32><<<grid, kRouteChunk, 0, st>>>(logits, T, H, K, gate_mode, nchunk, topk_idx, gates, counts);
  else
    k_route_count<64><<<grid, kRouteChunk, 0, st>>>(logits, T, H, K, gate_mode, nchunk, topk_idx, gates, counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_route_scan<<<1, kScanThreads, 0, st>>>(counts, static_cast<int>(L), nchunk, B * H, base, seg_offsets, head_len);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_route_scatter<<<grid, kRouteChunk, 0, st>>>(topk_idx, T, H, K, nchunk, base, perm_token, slot_pos);
  return hipGetLastError();
}

}  // namespace namoh
