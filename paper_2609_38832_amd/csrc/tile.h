// Shared pieces of the MFMA attention kernels (forward and backward): the
// packed 64-row tile layout, the work-item record, bf16 packing, the LDS
// granule swizzle and the direct HBM -> LDS tile loads.  Internal to libnamoh.
//
// v_mfma_f32_32x32x16_bf16 operand order used throughout (wave64, lane =
// 32*g + c): A (32 x 16): lane holds row c, reduction slots 8g..8g+7;
// B (16 x 32): lane holds column c, the same reduction slots; C (32 x 32):
// lane holds column c, rows 8j + 4g + i in accumulator 4j + i.  A 16-slot
// reduction step fed from accumulators 8s..8s+7 of a C tile therefore covers
// its rows 8a + 4g + i (a = 0, 1); a transposed tile stores, inside each
// 16-row group, row 8a + 4g + i at position 8g + 4a + i (vt_key_of_pos), so
// one 16-byte LDS read gives the matching A operand.
#pragma once

#include "common.h"

namespace namoh {

constexpr int kBN = 64;            // keys per tile

enum Meta { kMetaItems = 0, kMetaBad = 1, kMetaSplit = 2, kMetaCount = 4 };

// Packed key tiles of segment s (first packed row seg0, length n) are
// numbered from seg_tile0 = floor(seg0 / 64) + s.  The ranges of successive
// segments are disjoint and increasing, because
// floor((seg0 + n) / 64) - floor(seg0 / 64) + 1 >= ceil(n / 64), and every
// index stays below Nr / 64 + BH + 1, so no running sum is needed.
NAMOH_DEV int seg_tile0(int seg0, int s) { return seg0 / kBN + s; }

// One work item, a (segment, query block) pair, or one key-range part of
// one, with everything the attention workgroup needs before its first load,
// so an item costs one dependent global read.
struct __attribute__((aligned(32))) WorkItem {
  int s, qb, seg0, n;            // segment b*H + h, query block, first packed row, length
  int tile0;                     // first packed key tile of the segment
  int qh;                        // bits 0-2: query head of the item within its key/value
                                 // group (0 without groups); bits 3-19: 1 + partial slot of
                                 // a key-range part, 0 for a whole item; bits 20-23: the
                                 // part count of a split item (0 for a whole item); bits
                                 // 24-26: the part's index
  int kt_lo, kt_hi;              // key tiles [kt_lo, kt_hi) of the segment the item covers
};
constexpr int kQhBits = 3;
constexpr int kQhSlotMask = (1 << 17) - 1;   // (qh >> kQhBits) & mask: 1 + partial slot
constexpr int kQhPartsShift = 20;            // (qh >> shift) & 15: part count P (0: whole)
constexpr int kQhPartShift = 24;             // (qh >> shift) & 7: part index p
NAMOH_DEV int item_slot(int qh) { return ((qh >> kQhBits) & kQhSlotMask) - 1; }
NAMOH_DEV int item_parts(int qh) { return (qh >> kQhPartsShift) & 15; }
NAMOH_DEV int item_part(int qh) { return (qh >> kQhPartShift) & 7; }

// A split item (a query block run as key-range parts): its parts' partial
// slots are [base, base + P); qh is the query head.
struct SplitItem {
  int s, qb, seg0, n, qh, P, base, pad;
};

// Work item of this workgroup, or false if it has none.  The record is read
// together with the item count (the grid has max_items workgroups, so the
// read is in bounds either way).
NAMOH_DEV bool my_item(const WorkItem* __restrict__ items, const int32_t* __restrict__ meta,
                       WorkItem& it) {
  const int cnt = meta[kMetaItems];
  const WorkItem v = items[block_x()];
  // the record is the same for the whole workgroup: keep it in scalar registers
  it.s = __builtin_amdgcn_readfirstlane(v.s);
  it.qb = __builtin_amdgcn_readfirstlane(v.qb);
  it.seg0 = __builtin_amdgcn_readfirstlane(v.seg0);
  it.n = __builtin_amdgcn_readfirstlane(v.n);
  it.tile0 = __builtin_amdgcn_readfirstlane(v.tile0);
  it.qh = __builtin_amdgcn_readfirstlane(v.qh);
  it.kt_lo = __builtin_amdgcn_readfirstlane(v.kt_lo);
  it.kt_hi = __builtin_amdgcn_readfirstlane(v.kt_hi);
  return block_x() < __builtin_amdgcn_readfirstlane(cnt);
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
NAMOH_DEV void load_rope8(float4 (&c4)[4], const float2* __restrict__ cs) {
  const float4* p = reinterpret_cast<const float4*>(cs);
#pragma unroll
  for (int e = 0; e < 4; ++e) c4[e] = p[e];
}

NAMOH_DEV void rope8(float* x1, float* x2, const float4 (&c4)[4]) {
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

// (cos, sin) of the RoPE angle pos * theta_j, given f = theta_j / (2 pi) in
// double: the fraction of a revolution is formed in double and the hardware
// cosine/sine take their argument in revolutions.  Against double-precision
// cos/sin the absolute error stays below 3e-7 (measured on MI355X for
// positions below 32768, d <= 128, bases 1e4 and 5e5), far below the bf16
// rounding (2^-9 relative) the rotated rows then take.
NAMOH_DEV float2 rope_cs_rev(double pos, double f) {
  const double rev = pos * f;
  const float fr = static_cast<float>(rev - floor(rev));
  return make_float2(__builtin_amdgcn_cosf(fr), __builtin_amdgcn_sinf(fr));
}

// Rotation factors of 8 consecutive pairs j0 .. j0 + 7 in the layout of
// load_rope8: c4[e] = (cos, sin) of pair j0 + 2e, then of pair j0 + 2e + 1.
NAMOH_DEV void rope8_rev(float4 (&c4)[4], double pos, const double* f) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float2 a = rope_cs_rev(pos, f[2 * e]);
    const float2 b = rope_cs_rev(pos, f[2 * e + 1]);
    c4[e] = make_float4(a.x, a.y, b.x, b.y);
  }
}

// Position of key `p16` within a 16-key group of the transposed value tile:
// bits 2 and 3 swapped (see k_attn_mfma, P.V operand order).
NAMOH_DEV int vt_key_of_pos(int p) {
  return (p & ~12) | ((p & 4) << 1) | ((p & 8) >> 1);
}

// LDS granule swizzle.  gfx950 LDS serves 256 bytes (64 banks) per clock,
// i.e. 16 lanes of a 16-byte read at once; the operand reads below have 16
// consecutive lanes read the same logical 16-byte granule of 16 consecutive
// rows.  XOR-ing the granule index with row bits makes those 16 reads cover
// all 64 banks: rows of 16 granules (256 B) use row & 15; rows of 8 granules
// (128 B, two rows per bank sweep) use x = (row >> 1) & 7 with bit 2 flipped
// for odd x (still one value per row pair).  The flip serves the transposing
// reads of the backward, where a read covers four granules of eight
// consecutive rows: the row pairs then alternate between the two halves of
// the granule range and every bank is hit twice (the minimum for 512 bytes),
// not four times.
template <int GPR>
NAMOH_DEV int swz(int row, int gr) {
  static_assert(GPR == 8 || GPR == 16, "granules per row");
  return GPR == 16 ? (gr ^ (row & 15)) : (gr ^ (((row >> 1) & 7) ^ ((row & 2) << 1)));
}

// Tile staging, direct HBM -> LDS (buffer_load_dwordx4 ... lds): KPT 16-byte
// granules per thread of one packed key tile or one transposed value tile
// (contiguous in HBM).  Lane l of a wave instruction writes LDS granule
// base + l, so the swizzle is applied on the source side: the lane that
// fills physical granule P = row * GPR + phys fetches logical granule
// swz(row, phys) of that row (the XOR is its own inverse).  The buffer
// resource covers the item's key (or value) tiles and the tile is selected
// by the scalar offset, so a tile costs no vector address arithmetic; the
// LDS base goes through M0 from scalar registers.  Completion is tracked by
// vmcnt; a tile is published by wait_vmcnt<0>() and a barrier (a partial
// wait, meant to leave only the newest loads in flight, let a transposed
// tile be read before all of it had landed in LDS: these loads are not
// relied on to complete in issue order).

// Byte offset (inside one tile) of the first granule this lane fetches.  The
// lane's i-th granule lies i * NT granules further: NT / GPR rows is a
// multiple of the 16-row period of the swizzle, so the XOR term does not
// change with i and one register serves all KPT loads.
template <int GPR, int NT>
NAMOH_DEV uint32_t tile_voffset(int tid) {
  static_assert((NT / GPR) % 16 == 0, "rows per load must be a multiple of the swizzle period");
  const int row = tid / GPR, phys = tid % GPR;
  return static_cast<uint32_t>((row * GPR + swz<GPR>(row, phys)) * 16);
}

// Raw buffer resource (stride 0, num_records = nbytes) in scalar registers;
// the item's values are wave uniform, readfirstlane says so.
typedef int i32x4 __attribute__((ext_vector_type(4)));
NAMOH_DEV i32x4 buffer_rsrc(const uint16_t* base, uint32_t nbytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r.x = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(a)));
  r.y = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(a >> 32) & 0xFFFF));
  r.z = __builtin_amdgcn_readfirstlane(static_cast<int>(nbytes));
  r.w = 0x00020000;
  return r;
}

// LDS byte address of a __shared__ object (the address-space cast of a
// shared variable needs no null check).
template <typename T>
NAMOH_DEV uint32_t lds_address(T* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) T*)p));
}

// The loads are written as inline assembly (M0, the LDS base, is an input
// operand the compiler sets): the compiler's wait-count pass cannot tell the
// ring's LDS stages apart and, for its own builtin form of these loads,
// waits for every tile load in flight before any LDS read, which would
// serialise the ring.  Here the explicit vmcnt waits are the only ones, and
// the memory clobber keeps the compiler from moving LDS accesses across.
NAMOH_DEV void lds_dma16(i32x4 rsrc, uint32_t lds, uint32_t voff, int soff) {
  asm volatile("buffer_load_dwordx4 %1, %2, %3 offen lds" ::"{m0}"(lds), "v"(voff), "s"(rsrc),
               "s"(soff)
               : "memory");
}

// One tile.  base/nbytes: the buffer (the item's key or value tiles);
// tile_bytes: byte offset of the tile in it (wave uniform, in range);
// lds_wave: LDS address of the stage's tile plus this wave's first granule
// (wave uniform).
template <int KPT, int NT>
NAMOH_DEV void tile_dma(const uint16_t* base, uint32_t nbytes, uint32_t tile_bytes,
                        uint32_t lds_wave, uint32_t voff) {
  const i32x4 rsrc = buffer_rsrc(base, nbytes);
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    // wave-uniform scalar offset (readfirstlane keeps it out of vector
    // registers, which would force a loop over distinct values)
    const int tb = __builtin_amdgcn_readfirstlane(static_cast<int>(tile_bytes) + i * NT * 16);
    lds_dma16(rsrc, __builtin_amdgcn_readfirstlane(lds_wave + i * NT * 16), voff, tb);
  }
}

// s_waitcnt vmcnt(N) (expcnt and lgkmcnt left at their "no wait" values);
// the 6-bit count is split over bits 3:0 and 15:14 of the immediate.
template <int N>
NAMOH_DEV void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

}  // namespace namoh
