// Internal launch interface between the C ABI (api.cpp) and the kernels.
// Every launcher enqueues on `st` and returns the first HIP error it sees.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace namoh {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }

// Carves consecutive aligned regions out of one workspace block.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* p) : base(static_cast<char*>(p)) {}
  template <class T>
  T* take(size_t count) {
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += align_up(count * sizeof(T));
    return p;
  }
};

// ---- opt-in event timing (profile.cpp) ------------------------------------
void prof_mark(const char* section, bool begin, hipStream_t st);
// The next pair of events of `section` for a launch through hipExtLaunchKernel
// (false, and null events, when timing is off or the section is full).
bool prof_pair(const char* section, hipEvent_t* start, hipEvent_t* stop);

// ---- routing (route.hip) -------------------------------------------------
constexpr int kRouteChunk = 64;   // tokens per routing workgroup (one wave)
size_t route_workspace_bytes(int B, int T, int H, int K);
hipError_t launch_route_bias_update(const int32_t* head_len, int B, int T, int H, int K,
                                   float eta, float* bias, hipStream_t st);
// bias: NULL for the plain selection, else [H] per-head selection biases
hipError_t launch_route(const float* logits, const float* bias, int B, int T, int H, int K,
                        int gate_mode, int32_t* topk_idx, float* gates,
                        int32_t* head_len, int32_t* seg_offsets,
                        int32_t* perm_token, int32_t* slot_pos, void* ws,
                        hipStream_t st);

// ---- prefill attention (attn.hip) ----------------------------------------
// H, K: key/value heads and selected key/value heads per token; G query heads
// per key/value head (key/value-group routing; 1 = one query head per head).
size_t attn_workspace_bytes(int B, int T, int H, int K, int d, int dtype, int G = 1);
hipError_t launch_attn(const void* q, const void* k, const void* v, int dtype,
                       int B, int T, int H, int K, int d, float rope_base,
                       int rope_mode, float scale, const float* gates,
                       const int32_t* seg_offsets, const int32_t* perm_token,
                       const int32_t* slot_pos, void* out, int out_dtype,
                       float* head_out, void* ws, hipStream_t st, int G = 1);

struct WorkItem;
struct SplitItem;
// Where launch_attn_stats leaves the forward's pieces inside its workspace.
struct AttnTiles {
  const uint16_t* Kp;      // rotated keys, bf16, 64-row tiles [max_tiles * 64, d]
  const uint16_t* Vt;      // values, bf16, per tile transposed [max_tiles, d, 64]
  const double* freq;      // RoPE theta_j / (2 pi), double [d / 2] (as the forward rotates)
  const WorkItem* items;   // (segment, query block) work list, heaviest first, with
                           // key-range parts for blocks heavier than a fair share
  const int32_t* meta;     // item count, validity flag, split-item count
  const SplitItem* splits; // the split blocks and their parts' partial slots
  float* part;             // partial rows [part_rows, d] f32 (free once the forward merged)
  float* h;                // head outputs, f32 packed [Nr, d]
  int max_items, max_tiles, BM, part_rows;
};
hipError_t launch_attn_stats(const void* q, const void* k, const void* v, int B, int T, int H,
                             int K, int d, float rope_base, int rope_mode, float scale,
                             const int32_t* seg_offsets, const int32_t* perm_token, float* lse,
                             void* ws, AttnTiles& tiles, hipStream_t st);
// The tiles a launch_attn_stats on the same workspace and sizes left there
// (nothing is launched).
void attn_stats_tiles(void* ws, int B, int T, int H, int K, int d, AttnTiles& tiles);
// out[t] = sum over k of gates[t, k] * rows[slot_pos[t, k]] with f32 rows.
hipError_t launch_combine_f32(const float* rows, const float* gates, const int32_t* slot_pos,
                              long BT, int K, int D, int Nr, void* out, int out_dtype,
                              hipStream_t st);

// Always-active shared heads (attn.hip): Hs heads over all T tokens, causal
// (window 0) or inside a window of `window` tokens; out (+)= sum of the heads.
size_t shared_workspace_bytes(int B, int T, int Hs, int d);
hipError_t launch_shared(const void* q, const void* k, const void* v, int B, int T, int Hs, int d,
                         int window, float rope_base, int rope_mode, float scale, void* out,
                         int out_dtype, int accumulate, float* head_out, void* ws,
                         hipStream_t st);

// Gated combine of bf16 rows [Nr, D]: out[t] = sum_k gates[t,k] rows[slot_pos[t,k]]
// (attn.hip; D a multiple of 8).
hipError_t launch_combine_rows(const uint16_t* rows, const float* gates, const int32_t* slot_pos,
                               long BT, int K, int D, int Nr, void* out, int out_dtype,
                               hipStream_t st);

// ---- routed projections (proj.hip) ---------------------------------------
hipError_t launch_qkv_proj(const void* x, const void* w_qkv, int B, int T, int H, int K, int d,
                           int d_model, const int32_t* seg_offsets, const int32_t* perm_token,
                           void* q, void* k, void* v, hipStream_t st);
size_t out_proj_workspace_bytes(int B, int T, int H, int K, int d, int d_model);
bool out_proj_dense(int H, int K, int d);
hipError_t launch_out_proj(const void* head_out, int head_out_dtype, const void* w_o,
                           const float* gates, const int32_t* slot_pos,
                           const int32_t* seg_offsets, int B, int T, int H, int K, int d,
                           int d_model, void* out, int out_dtype, void* ws, hipStream_t st);

// ---- decode (decode.hip) --------------------------------------------------
size_t decode_workspace_bytes(int B, int H, int K, int d, int cap, int G = 1);
// bias: NULL for the plain selection, else [H] loss-free balancing biases
hipError_t launch_decode(const float* logits, const float* bias, const void* q, const void* k,
                         const void* v, int dtype, void* k_cache,
                         void* v_cache, int32_t* cache_len,
                         const int32_t* seq_pos, int B, int H, int K, int d,
                         int cap, float rope_base, int rope_mode,
                         int gate_mode, float scale, int32_t* topk_idx,
                         float* gates, void* out, int out_dtype,
                         int32_t* dev_status, void* ws, hipStream_t st);
// The no-allocation decode step's scratch: its size, and the device address
// of the current device's copy (resolved once per device).
size_t decode_scratch_bytes();
hipError_t decode_scratch(void** ptr);
// bf16, d in {64, 128}, G in {1, 2, 4, 8} query heads per key/value head
hipError_t launch_decode_grouped(const float* logits, const void* q, const void* k, const void* v,
                                 void* k_cache, void* v_cache, int32_t* cache_len,
                                 const int32_t* seq_pos, int B, int H, int K, int G, int d, int cap,
                                 float rope_base, int rope_mode, int gate_mode, float scale,
                                 int32_t* topk_idx, float* gates, void* out, int out_dtype,
                                 int32_t* dev_status, void* ws, hipStream_t st);
// Shared heads in the decode step: Hs always-active heads per sequence, caches
// [B, Hs, cap, d] (rings of the most recent cap tokens when window > 0),
// cache_len [B] = tokens so far; out (+)= the ungated sum of the heads.
size_t shared_decode_workspace_bytes(int B, int Hs, int d, int cap);
hipError_t launch_shared_decode(const void* q, const void* k, const void* v, int dtype,
                                void* k_cache, void* v_cache, int32_t* cache_len, int B, int Hs,
                                int d, int cap, int window, float rope_base, int rope_mode,
                                float scale, void* out, int out_dtype, int accumulate,
                                int32_t* dev_status, void* ws, hipStream_t st);
hipError_t launch_shared_prefill_cache(const void* k, const void* v, int dtype, int B, int T,
                                       int Hs, int d, int cap, float rope_base, int rope_mode,
                                       void* k_cache, void* v_cache, int32_t* cache_len,
                                       hipStream_t st);
hipError_t launch_prefill_cache(const void* k, const void* v, int dtype, int B, int T, int H,
                                int K, int d, float rope_base, int rope_mode,
                                const int32_t* seg_offsets, const int32_t* perm_token,
                                void* k_cache, void* v_cache, int32_t* cache_len, int cap,
                                hipStream_t st);

// ---- backward (bwd.hip) ---------------------------------------------------
size_t attn_bwd_workspace_bytes(int B, int T, int H, int K, int d);
hipError_t launch_attn_bwd(const void* q, const void* k, const void* v, int dtype, int B, int T,
                           int H, int K, int d, float rope_base, int rope_mode, float scale,
                           const int32_t* topk_idx, const float* gates,
                           const int32_t* seg_offsets, const int32_t* perm_token,
                           const float* dout, float* dq, float* dk, float* dv, float* dgates,
                           void* ws, hipStream_t st, bool packed = false, bool saved = false);
// The training forward (matrix-core path: bf16, d = 64 or 128): output plus
// the state launch_attn_bwd(saved = true) reuses from the same workspace.
bool attn_train_supported(int dtype, int d);
hipError_t launch_train_fwd(const void* q, const void* k, const void* v, int dtype, int B,
                            int T, int H, int K, int d, float rope_base, int rope_mode,
                            float scale, const float* gates, const int32_t* seg_offsets,
                            const int32_t* perm_token, const int32_t* slot_pos, void* out,
                            int out_dtype, void* ws, hipStream_t st);
hipError_t launch_route_bwd(const float* logits, const int32_t* topk_idx, const float* gates,
                            const float* dgates, int B, int T, int H, int K, int gate_mode,
                            float* dlogits, hipStream_t st);

}  // namespace namoh
