// The attention work list: (segment, query block) items ordered heaviest
// first for the hardware's in-order dispatch, with key-range parts for
// blocks heavier than a workgroup's fair share (Sec. 3.2, length-aware
// scheduling).  Built on the device by one workgroup (attn_schedule); used by
// the forward kernels (attn.hip) and the backward (bwd.hip).
#pragma once

#include "common.h"
#include "tile.h"

namespace namoh {

constexpr int kSortBins = 2048;    // work keys (key tiles) are clamped to this many bins
constexpr int kSegLds = 1024;      // segment offsets staged in LDS up to this many segments

// ---------------------------------------------------------------------------
// The work list: items sorted by causal work (key tiles), heaviest first,
// by a counting sort; workgroup i runs item i, and the hardware dispatches
// workgroups in index order, which makes the assignment to compute units
// longest-processing-time first.  (Placing items by XCD so that a segment's
// key/value tiles stay in one L2 measured no faster: the tiles are re-read
// from the shared last-level cache at a rate the kernel does not saturate.)
// The sort visits one (segment, query block) cell per thread per round and
// reserves its ranks with LDS atomics (two per cell at most).
// Offsets that are not a valid packing of Nr rows (out of order, a segment
// longer than T, or not ending at Nr) produce an empty list.  The global
// stores come last: a barrier after a store would wait for it.
//
// Key-range parts (split_slots > 0).  With `split_slots` resident workgroups,
// a slot's fair share of the work is F = ceil(total key tiles / split_slots).
// An item with more than F key tiles (and at least kSplitMinTiles) would
// outlast the rest of the kernel on its compute unit, so it is cut into P
// parts of at most L = ceil(w / P0) tiles (P0 = min(kSplitMaxParts,
// ceil(w / F))), taken from the end of its key range (the last part holds
// the diagonal tiles, every other part only keys before the block's first
// query); each part writes an unnormalised partial (O, m, l) that
// k_attn_merge combines.  Below kSplitMinTiles a part's fixed cost (query
// gather, first tiles, partial rows) outweighs the balance it buys.  The
// parts add at most split_slots items, at most 2 split_slots partial slots
// and at most split_slots split items (sum of w over the split items is at
// least (number of split items) F, and each adds at most w / F parts).
constexpr int kSplitMinTiles = 32;
constexpr int kSplitMaxParts = 8;

// Dispatch positions: `resident_slots` workgroups of the attention kernel are
// resident at once (256 units times the kernel's workgroups per unit); only
// the first round of ranks is placed in alternating block order
// (resident_pos), with or without key-range parts.
//
// Late pairs (split_slots > 0, S = split_slots resident slots, E = items - S
// with 0 < E <= S / kPairMaxFrac).  The E items past the slots would start
// only when a slot frees, late in the kernel, and end it.  The hardware puts
// workgroup i on XCD i mod 8, and on compute unit i mod (units) while every
// unit has room; a unit issues for its oldest wave first, so the workgroups
// of the first block of positions run ahead and the youngest lag.  Pair j
// (j < E) joins the lightest extra item (rank S + j) with the lightest
// placed one (rank S - 1 - j, whose serpentine position is in the last,
// reversed block, on unit j): the light item takes position j, the oldest
// on unit j, and finishes first; the other items of unit j each move one
// block later, keeping their order; and rank S - 1 - j is dispatched after
// all slots are taken, at S + k with k = j (mod 8), so it waits for a slot on
// the light item's XCD.  Within a residue class the largest j (the lightest
// extra, finishing first) frees the slot of the first late workgroup, which
// holds the heaviest late item.  A unit's total work is unchanged.  Used
// when the geometry fits: the period (compute units) a multiple of 8
// dividing S into an even number of blocks (MINB 2 or 4 on 256 units), E at
// most one block.
constexpr int kPairMaxFrac = 8;
constexpr int kXcds = 8;

struct SchedLds {
  int hist[kSortBins];
  int off[kSegLds + 1];
  int wmax[16], wbad[16];
  int wave[17];
  double wsum[16];
  int nparts, nsplit;
  int cst[kSegLds + 1];   // first cell of each segment (cells enumerated segment by segment)
};

// Parts of an item of w key tiles with fair share F: count P, length L; part
// p covers [max(0, w - (P - p) L), w - (P - 1 - p) L).
NAMOH_DEV void split_parts(int w, int F, int& P, int& L) {
  if (w > F && w >= kSplitMinTiles) {
    const int P0 = min(kSplitMaxParts, (w + F - 1) / F);
    L = (w + P0 - 1) / P0;
    P = (w + L - 1) / L;
  } else {
    P = 1;
    L = w;
  }
}

// Serpentine placement: the hardware puts workgroup i on the compute unit of
// workgroup i mod (number of compute units) as long as every unit has room,
// so in heaviest-first order unit u would receive ranks u, P + u, 2P + u, ...
// (P units), all near the top of their block of P ranks.  Reversing every
// other block of P ranks gives unit u the ranks u, 2P - 1 - u, 2P + u, ...,
// whose sums are nearly equal.  The map is a permutation of [0, total).
NAMOH_DEV int serpentine(int rank, int total, int period) {
  if (period <= 1) return rank;
  const int blk = rank / period;
  if ((blk & 1) == 0) return rank;
  const int first = blk * period;
  const int len = min(period, total - first);
  return first + len - 1 - (rank - first);
}

// Dispatch position of rank `rank` among `total` items when `slots`
// workgroups are resident at once.  Only the first round is placed by the
// hardware's fixed unit order, so only ranks below `slots` are reversed in
// alternate blocks; later workgroups start on whichever unit (of their XCD)
// frees a slot first, in index order, so they keep the heaviest-first order
// (a reversed block would start its heaviest item last).  slots <= 0: every
// block alternates.
NAMOH_DEV int resident_pos(int rank, int total, int slots, int period) {
  if (slots <= 0 || total <= slots) return serpentine(rank, total, period);
  return rank < slots ? serpentine(rank, slots, period) : rank;
}

NAMOH_DEV bool late_pairs_fit(int slots, int extra, int period) {
  return extra > 0 && period > 1 && period % kXcds == 0 && slots % period == 0 &&
         (slots / period) % 2 == 0 && extra <= slots / kPairMaxFrac && extra <= period;
}

// Dispatch position of rank `rank` with `extra` late pairs over `slots`
// resident slots (see kPairMaxFrac); a permutation of [0, slots + extra).
NAMOH_DEV int late_pair_pos(int rank, int slots, int extra, int period) {
  const int S = slots, E = extra;
  if (rank < S - E) {
    const int p = serpentine(rank, S, period);
    return p % period < E ? p + period : p;   // one block younger on a paired unit
  }
  if (rank >= S) return rank - S;       // the light item of pair rank - S
  // late item of pair j: residue a = j mod 8, t = j / 8; the class holds
  // ceil((E - a) / 8) pairs, taken largest t first
  const int j = S - 1 - rank;
  const int a = j % kXcds, t = j / kXcds;
  const int Ta = (E - a + kXcds - 1) / kXcds;
  return S + kXcds * (Ta - 1 - t) + a;
}

template <int NT>
NAMOH_DEV void attn_schedule(const int32_t* __restrict__ seg_offsets_g, int BH, int T, int BM,
                             int Nr, int max_items, int period, int G,
                             WorkItem* __restrict__ items, int32_t* __restrict__ meta,
                             SchedLds& L, int split_slots = 0,
                             SplitItem* __restrict__ splits = nullptr, int resident_slots = 0) {
  static_assert(NT % kWave == 0 && NT / kWave <= 16 && kSortBins % NT == 0, "block size");
  const int tid = thread_x();
  const int lane = tid % kWave, wave = tid / kWave;
  const int per_qb = BM / kBN;           // key tiles added per query block
  const bool in_lds = BH <= kSegLds;
  if (in_lds)
    for (int i = tid; i <= BH; i += NT) L.off[i] = seg_offsets_g[i];
  for (int i = tid; i < kSortBins; i += NT) L.hist[i] = 0;
  if (tid == 0) L.nparts = L.nsplit = 0;
  __syncthreads();
  const int32_t* off = in_lds ? L.off : seg_offsets_g;
  // validity and the longest segment
  int mx = 0, bad = 0;
  for (int s = tid; s < BH; s += NT) {
    const int n = off[s + 1] - off[s];
    mx = max(mx, n);
    bad |= n < 0 || n > T;
  }
  mx = wave_max_i(mx);
  bad = __ballot(bad) != 0;
  if (lane == 0) {
    L.wmax[wave] = mx;
    L.wbad[wave] = bad;
  }
  __syncthreads();
  int maxn = 0;
  bad = off[0] != 0 || off[BH] != Nr;
#pragma unroll
  for (int w = 0; w < NT / kWave; ++w) {
    maxn = max(maxn, L.wmax[w]);
    bad |= L.wbad[w];
  }
  if (bad) {
    if (tid == 0) {
      meta[kMetaItems] = 0;
      meta[kMetaBad] = 1;
      meta[kMetaSplit] = 0;
    }
    return;
  }
  // The cells (segment, query block), w: a cell's key tiles; with key/value
  // groups each cell stands for G items (query heads u < G) of the same
  // work, which take G consecutive ranks.  With the segment table in LDS
  // only the real cells are visited, numbered segment by segment (cst[s]:
  // the first cell of segment s, found back by binary search).  Otherwise,
  // or when the full (query block, segment) grid holds at most twice the
  // real cells, the grid is visited qb-major (cells past a segment's end
  // inactive; a thread steps its (qb, s) by NT cells without dividing).
  const int grid_cells = (maxn + BM - 1) / BM * BH;   // below 2^31 (checked on the host)
  bool compact = in_lds;
  int ncells = grid_cells;
  if (compact) {
    constexpr int SPT = (kSegLds + NT - 1) / NT;
    int cnt[SPT];
    int csum = 0;
#pragma unroll
    for (int i = 0; i < SPT; ++i) {
      const int sg = tid * SPT + i;
      cnt[i] = sg < BH ? (off[sg + 1] - off[sg] + BM - 1) / BM : 0;
      csum += cnt[i];
    }
    int ctot = 0;
    int crun = block_exclusive_scan<NT>(csum, L.wave, ctot);
#pragma unroll
    for (int i = 0; i < SPT; ++i) {
      const int sg = tid * SPT + i;
      if (sg < BH) L.cst[sg] = crun;
      crun += cnt[i];
    }
    __syncthreads();
    // the grid when it holds at most twice the real cells (no search needed)
    if (grid_cells > 2 * ctot) ncells = ctot;
    else compact = false;
  }
  // a thread's cells are tid, tid + NT, ...; in grid order cell c is
  // (qb, s) = (c / BH, c mod BH), advanced by (NT / BH, NT mod BH) per round
  const int dq = NT / BH, ds = NT - (NT / BH) * BH;
  const int qb_first = tid / BH, s_first = tid - (tid / BH) * BH;
  auto cell = [&](int c, int& s, int& qb, int& seg0, int& n, int& w) {
    if (compact) {
      int lo = 0, hi = BH - 1;   // the last segment whose first cell is at most c
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (L.cst[mid] <= c) lo = mid; else hi = mid - 1;
      }
      s = lo;
      qb = c - L.cst[lo];
    }   // else (s, qb) are the caller's stepped values
    seg0 = off[s];
    n = off[s + 1] - seg0;
    w = min((n + kBN - 1) / kBN, (qb + 1) * per_qb);
    return qb * BM < n;
  };
  auto step = [&](int& s, int& qb) {
    s += ds;
    qb += dq;
    if (s >= BH) {
      s -= BH;
      ++qb;
    }
  };
  // rank of the first of `cnt` items of key `key` among those placed so far
  // (one LDS atomic per lane: the LDS serves the lanes of one instruction
  // together, conflicts on one key in turn)
  auto bin_add = [&](int key, int cnt) { return atomicAdd(&L.hist[key], cnt); };
  auto key_of = [](int tiles) { return kSortBins - 1 - min(tiles, kSortBins - 1); };
  // the fair share of a slot (no parts without split_slots); a segment of
  // nt key tiles and nq query blocks holds sum over q < nq of
  // min(nt, per_qb (q + 1)) key tiles of work per query head
  int F = 0x7fffffff;
  if (split_slots > 0) {
    long work = 0;
    for (int sg = tid; sg < BH; sg += NT) {
      const int n = off[sg + 1] - off[sg];
      const int nt = (n + kBN - 1) / kBN, nq = (n + BM - 1) / BM;
      const long m = min(nq, nt / per_qb);
      work += per_qb * m * (m + 1) / 2 + static_cast<long>(nq - m) * nt;
    }
    work *= G;
    // exact total (the bounds on parts and partial slots rest on it): the
    // per-lane counts are integers far below 2^53, summed in double
    const double wsum = wave_sum_d(static_cast<double>(work));
    if (lane == 0) L.wsum[wave] = wsum;
    __syncthreads();
    double wt = 0.0;
#pragma unroll
    for (int w = 0; w < NT / kWave; ++w) wt += L.wsum[w];
    const long wtot = static_cast<long>(wt);
    F = static_cast<int>(min((wtot + split_slots - 1) / split_slots, 0x7fffffffL));
    F = max(F, 1);
  }
  {
    int sg = s_first, qb = qb_first;
    for (int c0 = 0; c0 < ncells; c0 += NT) {
      const int c = c0 + tid;
      int seg0 = 0, n = 0, w = 0;
      const bool act = c < ncells && cell(c, sg, qb, seg0, n, w);
      int P = 1, Lp = w;
      if (act) {
        // part 0 holds w - (P - 1) L tiles, parts 1 .. P - 1 L each
        split_parts(w, F, P, Lp);
        bin_add(key_of(w - (P - 1) * Lp), G);
        if (P > 1) bin_add(key_of(Lp), (P - 1) * G);
      }
      if (!compact) step(sg, qb);
    }
  }
  __syncthreads();
  // exclusive scan of the histogram -> insertion cursors (heaviest first)
  constexpr int PER = kSortBins / NT;
  int h[PER];
  int sum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    h[i] = L.hist[tid * PER + i];
    sum += h[i];
  }
  int total;
  int run = block_exclusive_scan<NT>(sum, L.wave, total);
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    L.hist[tid * PER + i] = run;
    run += h[i];
  }
  __syncthreads();
  const int placed = min(total, max_items);
  const int extra = split_slots > 0 && late_pairs_fit(split_slots, placed - split_slots, period)
                        ? placed - split_slots
                        : 0;
  {
    int sg = s_first, qb = qb_first;
    for (int c0 = 0; c0 < ncells; c0 += NT) {
      const int c = c0 + tid;
      int seg0 = 0, n = 0, w = 0;
      const bool act = c < ncells && cell(c, sg, qb, seg0, n, w);
      int P = 1, Lp = w;
      if (act) split_parts(w, F, P, Lp);
      // a split cell: G split items (one per query head u) with partial slots
      // [base + u P, base + (u + 1) P)
      int base = -1;
      if (act && P > 1) {
        base = atomicAdd(&L.nparts, P * G);
        const int j = atomicAdd(&L.nsplit, G);
        for (int u = 0; u < G; ++u) {
          SplitItem si;
          si.s = sg;
          si.qb = qb;
          si.seg0 = seg0;
          si.n = n;
          si.qh = u;
          si.P = P;
          si.base = base + u * P;
          si.pad = 0;
          splits[j + u] = si;
        }
      }
      // ranks: part 0 of query head u at r0 + u, part p >= 1 at
      // rL + (p - 1) G + u
      int r0 = 0, rL = 0;
      if (act) {
        r0 = bin_add(key_of(w - (P - 1) * Lp), G);
        if (P > 1) rL = bin_add(key_of(Lp), (P - 1) * G);
      }
      for (int p = 0; p < kSplitMaxParts; ++p) {
        if (!__any(act && p < P)) break;
        const int hi = w - (P - 1 - p) * Lp;
        const int lo = max(0, hi - Lp);
        const int rank = p == 0 ? r0 : rL + (p - 1) * G;
        if (act && p < P) {
          for (int u = 0; u < G; ++u) {
            const int r = rank + u;
            if (r >= placed) break;
            const int pos = extra > 0 ? late_pair_pos(r, split_slots, extra, period)
                                      : resident_pos(r, placed, resident_slots, period);
            WorkItem wi;
            wi.s = sg;
            wi.qb = qb;
            wi.seg0 = seg0;
            wi.n = n;
            wi.tile0 = seg_tile0(seg0, sg);
            wi.qh = u | ((P > 1 ? base + u * P + p + 1 : 0) << kQhBits) |
                    ((P > 1 ? P : 0) << kQhPartsShift) | ((P > 1 ? p : 0) << kQhPartShift);
            wi.kt_lo = lo;
            wi.kt_hi = hi;
            items[pos] = wi;
          }
        }
      }
      if (!compact) step(sg, qb);
    }
  }
  __syncthreads();
  if (tid == 0) {
    meta[kMetaItems] = placed;
    meta[kMetaBad] = 0;
    meta[kMetaSplit] = L.nsplit;
  }
}

}  // namespace namoh
