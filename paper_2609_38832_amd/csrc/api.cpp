// C ABI of libnamoh: host-side validation, workspace checks, dispatch.
// Every argument is checked before anything is enqueued, so a call that
// returns an error has launched nothing.  The semantics of each call are
// documented in include/namoh.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "../../include/namoh.h"
#include "internal.h"

namespace {

thread_local char g_err[512] = "";

namoh_status fail(namoh_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

namoh_status ok() {
  g_err[0] = '\0';
  return NAMOH_OK;
}

bool aligned(const void* p, size_t a) {
  return (reinterpret_cast<uintptr_t>(p) % a) == 0;
}

#define REQUIRE(cond, ...)                                   \
  do {                                                       \
    if (!(cond)) return fail(NAMOH_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)

#define REQUIRE_PTR(p, a)                                                      \
  do {                                                                         \
    if ((p) == nullptr) return fail(NAMOH_ERR_INVALID_ARG, #p " is NULL");     \
    if (!aligned((p), (a)))                                                    \
      return fail(NAMOH_ERR_INVALID_ARG, #p " is not %d-byte aligned", (int)(a)); \
  } while (0)

namoh_status check_sizes(int B, int T, int H, int K) {
  REQUIRE(B >= 1, "B must be >= 1 (got %d)", B);
  REQUIRE(T >= 1, "T must be >= 1 (got %d)", T);
  REQUIRE(H >= 1 && H <= 64, "H must be in [1, 64] (got %d)", H);
  REQUIRE(K >= 1 && K <= H, "K must be in [1, H] (got K=%d, H=%d)", K, H);
  const long long nr = static_cast<long long>(B) * T * K;
  REQUIRE(nr < (1ll << 31), "B*T*K must be < 2^31 (got %lld)", nr);
  // the attention work list's (64-query block, segment) grid is indexed in int
  const long long cells = (static_cast<long long>(T) + 63) / 64 * B * H;
  REQUIRE(cells < (1ll << 31), "ceil(T/64)*B*H must be < 2^31 (got %lld)", cells);
  return NAMOH_OK;
}

// The MFMA kernels address one segment's packed key/value tiles with 32-bit
// buffer offsets.
namoh_status check_segment_bytes(int dtype, int T, int d_head) {
  if (dtype == NAMOH_BF16 && (d_head == 64 || d_head == 128)) {
    const long long seg_bytes = (static_cast<long long>(T) + 63) / 64 * 64 * d_head * 2;
    if (seg_bytes >= (1ll << 32))
      return fail(NAMOH_ERR_UNSUPPORTED, "T = %d too long for d_head = %d on the bf16 path", T,
                  d_head);
  }
  return NAMOH_OK;
}

namoh_status check_head_width(int d) {
  if (d != 32 && d != 64 && d != 128)
    return fail(NAMOH_ERR_UNSUPPORTED, "d_head must be 32, 64 or 128 (got %d)", d);
  return NAMOH_OK;
}

namoh_status check_workspace(void* ws, size_t have, size_t need) {
  if (need == 0) return NAMOH_OK;
  if (ws == nullptr) return fail(NAMOH_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
  if (!aligned(ws, 256)) return fail(NAMOH_ERR_INVALID_ARG, "workspace is not 256-byte aligned");
  if (have < need)
    return fail(NAMOH_ERR_WORKSPACE, "workspace too small: %zu bytes given, %zu needed", have, need);
  return NAMOH_OK;
}

namoh_status hip_status(hipError_t e) {
  if (e == hipSuccess) return ok();
  return fail(NAMOH_ERR_HIP, "HIP error %d: %s", static_cast<int>(e), hipGetErrorString(e));
}

// NAMOH_SYNC_CHECK=1 in the environment (read once): every call that
// launched work synchronises its stream and reports an asynchronous error of
// its kernels as NAMOH_ERR_HIP (debugging aid; the calls otherwise never
// synchronise).
bool sync_check_on() {
  static const bool on = [] {
    const char* v = std::getenv("NAMOH_SYNC_CHECK");
    return v != nullptr && v[0] != '\0' && v[0] != '0';
  }();
  return on;
}

// Status of a call whose launches returned e.
namoh_status launched(void* stream, hipError_t e) {
  if (e != hipSuccess || !sync_check_on()) return hip_status(e);
  const hipError_t se = hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (se != hipSuccess)
    return fail(NAMOH_ERR_HIP, "NAMOH_SYNC_CHECK: error in the call's kernels: HIP error %d: %s",
                static_cast<int>(se), hipGetErrorString(se));
  return ok();
}

// Clears a sticky error left by an earlier unrelated call so that the
// launches below report their own status.
void clear_hip_error() { (void)hipGetLastError(); }

}  // namespace

extern "C" {

const char* namoh_status_string(int s) {
  switch (s) {
    case NAMOH_OK: return "NAMOH_OK";
    case NAMOH_ERR_INVALID_ARG: return "NAMOH_ERR_INVALID_ARG";
    case NAMOH_ERR_UNSUPPORTED: return "NAMOH_ERR_UNSUPPORTED";
    case NAMOH_ERR_WORKSPACE: return "NAMOH_ERR_WORKSPACE";
    case NAMOH_ERR_HIP: return "NAMOH_ERR_HIP";
    default: return "NAMOH_UNKNOWN_STATUS";
  }
}

const char* namoh_last_error(void) { return g_err; }

const char* namoh_version(void) { return "namoh-gfx950 0.1"; }

size_t namoh_route_workspace_size(int B, int T, int H, int K) {
  if (check_sizes(B, T, H, K) != NAMOH_OK) return 0;
  return namoh::route_workspace_bytes(B, T, H, K);
}

namoh_status namoh_route(const float* logits, int B, int T, int H, int K,
                         int gate_mode, int32_t* topk_idx, float* gates,
                         int32_t* head_len, int32_t* seg_offsets,
                         int32_t* perm_token, int32_t* slot_pos,
                         void* workspace, size_t workspace_bytes, void* stream) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  REQUIRE(gate_mode == NAMOH_GATE_SOFTMAX_SELECTED || gate_mode == NAMOH_GATE_SOFTMAX_ALL,
          "unknown gate_mode %d", gate_mode);
  REQUIRE_PTR(logits, 4);
  REQUIRE_PTR(topk_idx, 4);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(head_len, 4);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(perm_token, 4);
  REQUIRE_PTR(slot_pos, 4);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::route_workspace_bytes(B, T, H, K))) != NAMOH_OK)
    return s;
  clear_hip_error();
  return launched(stream, namoh::launch_route(logits, nullptr, B, T, H, K, gate_mode, topk_idx, gates,
                                        head_len, seg_offsets, perm_token, slot_pos,
                                        workspace, static_cast<hipStream_t>(stream)));
}

namoh_status namoh_route_biased(const float* logits, const float* bias, int B, int T, int H,
                                int K, int32_t* topk_idx, float* gates, int32_t* head_len,
                                int32_t* seg_offsets, int32_t* perm_token, int32_t* slot_pos,
                                void* workspace, size_t workspace_bytes, void* stream) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  REQUIRE_PTR(logits, 4);
  REQUIRE_PTR(bias, 4);
  REQUIRE_PTR(topk_idx, 4);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(head_len, 4);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(perm_token, 4);
  REQUIRE_PTR(slot_pos, 4);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::route_workspace_bytes(B, T, H, K))) != NAMOH_OK)
    return s;
  clear_hip_error();
  return launched(stream, namoh::launch_route(logits, bias, B, T, H, K, NAMOH_GATE_SOFTMAX_ALL,
                                        topk_idx, gates, head_len, seg_offsets, perm_token,
                                        slot_pos, workspace, static_cast<hipStream_t>(stream)));
}

namoh_status namoh_route_bias_update(const int32_t* head_len, int B, int T, int H, int K,
                                     float eta, float* bias, void* stream) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  REQUIRE(std::isfinite(eta), "eta must be finite");
  REQUIRE_PTR(head_len, 4);
  REQUIRE_PTR(bias, 4);
  clear_hip_error();
  return launched(stream, namoh::launch_route_bias_update(head_len, B, T, H, K, eta, bias,
                                                    static_cast<hipStream_t>(stream)));
}

size_t namoh_attn_fwd_workspace_size(int B, int T, int H, int K, int d_head, int dtype) {
  if (check_sizes(B, T, H, K) != NAMOH_OK || check_head_width(d_head) != NAMOH_OK) return 0;
  if (dtype != NAMOH_F32 && dtype != NAMOH_BF16) return 0;
  return namoh::attn_workspace_bytes(B, T, H, K, d_head, dtype);
}

namoh_status namoh_attn_fwd(const void* q, const void* k, const void* v, int dtype,
                            int B, int T, int H, int K, int d_head, float rope_base,
                            int rope_mode, float softmax_scale, const float* gates,
                            const int32_t* seg_offsets, const int32_t* perm_token,
                            const int32_t* slot_pos, void* out, int out_dtype,
                            float* head_out, void* workspace, size_t workspace_bytes,
                            void* stream) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  if ((s = check_head_width(d_head)) != NAMOH_OK) return s;
  REQUIRE(dtype == NAMOH_F32 || dtype == NAMOH_BF16, "unknown dtype %d", dtype);
  REQUIRE(out_dtype == NAMOH_F32 || out_dtype == NAMOH_BF16, "unknown out_dtype %d", out_dtype);
  REQUIRE(rope_mode == NAMOH_ROPE_HEAD_RELATIVE || rope_mode == NAMOH_ROPE_GLOBAL ||
              rope_mode == NAMOH_ROPE_NONE,
          "unknown rope_mode %d", rope_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_NONE || (std::isfinite(rope_base) && rope_base > 0.f),
          "rope_base must be finite and > 0 (got %g)", static_cast<double>(rope_base));
  REQUIRE(!std::isnan(softmax_scale) && !std::isinf(softmax_scale), "softmax_scale must be finite");
  const long long dense = static_cast<long long>(B) * H * T * d_head;
  REQUIRE(dense < (1ll << 40), "q/k/v too large");
  if ((s = check_segment_bytes(dtype, T, d_head)) != NAMOH_OK) return s;
  REQUIRE_PTR(q, 16);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(perm_token, 4);
  REQUIRE_PTR(slot_pos, 4);
  REQUIRE(out != nullptr || head_out != nullptr, "out and head_out are both NULL");
  if (out != nullptr) REQUIRE_PTR(out, 16);
  if (head_out != nullptr) REQUIRE_PTR(head_out, 16);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::attn_workspace_bytes(B, T, H, K, d_head, dtype))) != NAMOH_OK)
    return s;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt(static_cast<float>(d_head));
  clear_hip_error();
  return launched(stream, namoh::launch_attn(q, k, v, dtype, B, T, H, K, d_head, rope_base, rope_mode,
                                       scale, gates, seg_offsets, perm_token, slot_pos, out,
                                       out_dtype, head_out, workspace,
                                       static_cast<hipStream_t>(stream)));
}

namoh_status namoh_prefill_cache(const void* k, const void* v, int dtype, int B, int T, int H,
                                 int K, int d_head, float rope_base, int rope_mode,
                                 const int32_t* seg_offsets, const int32_t* perm_token,
                                 void* k_cache, void* v_cache, int32_t* cache_len, int cap,
                                 void* stream) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  if ((s = check_head_width(d_head)) != NAMOH_OK) return s;
  REQUIRE(dtype == NAMOH_F32 || dtype == NAMOH_BF16, "unknown dtype %d", dtype);
  REQUIRE(rope_mode == NAMOH_ROPE_HEAD_RELATIVE || rope_mode == NAMOH_ROPE_GLOBAL ||
              rope_mode == NAMOH_ROPE_NONE,
          "unknown rope_mode %d", rope_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_NONE || (std::isfinite(rope_base) && rope_base > 0.f),
          "rope_base must be finite and > 0 (got %g)", static_cast<double>(rope_base));
  REQUIRE(cap >= T, "cap (%d) must hold a whole prompt (T = %d)", cap, T);
  REQUIRE(static_cast<long long>(B) * H * cap * d_head < (1ll << 40), "caches too large");
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(perm_token, 4);
  REQUIRE_PTR(k_cache, 16);
  REQUIRE_PTR(v_cache, 16);
  REQUIRE_PTR(cache_len, 4);
  clear_hip_error();
  return launched(stream, namoh::launch_prefill_cache(k, v, dtype, B, T, H, K, d_head, rope_base,
                                                rope_mode, seg_offsets, perm_token, k_cache,
                                                v_cache, cache_len, cap,
                                                static_cast<hipStream_t>(stream)));
}

namespace {
namoh_status check_shared(int B, int T, int Hs, int d_head) {
  REQUIRE(B >= 1, "B must be >= 1 (got %d)", B);
  REQUIRE(T >= 1, "T must be >= 1 (got %d)", T);
  REQUIRE(Hs >= 1 && Hs <= 1024, "Hs must be in [1, 1024] (got %d)", Hs);
  REQUIRE(static_cast<long long>(B) * Hs * T < (1ll << 31), "B*Hs*T must be < 2^31");
  if (d_head != 64 && d_head != 128)
    return fail(NAMOH_ERR_UNSUPPORTED, "shared heads need d_head 64 or 128 (got %d)", d_head);
  if ((static_cast<long long>(T) + 63) / 64 * 64 * d_head * 2 >= (1ll << 32))
    return fail(NAMOH_ERR_UNSUPPORTED, "T = %d too long for d_head = %d on the bf16 path", T,
                d_head);
  return NAMOH_OK;
}
}  // namespace

size_t namoh_shared_attn_workspace_size(int B, int T, int Hs, int d_head) {
  if (check_shared(B, T, Hs, d_head) != NAMOH_OK) return 0;
  return namoh::shared_workspace_bytes(B, T, Hs, d_head);
}

namoh_status namoh_shared_attn(const void* q, const void* k, const void* v, int dtype, int B,
                               int T, int Hs, int d_head, int window, float rope_base,
                               int rope_mode, float softmax_scale, void* out, int out_dtype,
                               int accumulate, float* head_out, void* workspace,
                               size_t workspace_bytes, void* stream) {
  namoh_status s;
  if ((s = check_shared(B, T, Hs, d_head)) != NAMOH_OK) return s;
  REQUIRE(dtype == NAMOH_F32 || dtype == NAMOH_BF16, "unknown dtype %d", dtype);
  if (dtype != NAMOH_BF16) return fail(NAMOH_ERR_UNSUPPORTED, "shared heads need bf16 inputs");
  REQUIRE(window >= 0, "window must be >= 0 (got %d)", window);
  REQUIRE(out_dtype == NAMOH_F32 || out_dtype == NAMOH_BF16, "unknown out_dtype %d", out_dtype);
  REQUIRE(rope_mode == NAMOH_ROPE_HEAD_RELATIVE || rope_mode == NAMOH_ROPE_GLOBAL ||
              rope_mode == NAMOH_ROPE_NONE,
          "unknown rope_mode %d", rope_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_NONE || (std::isfinite(rope_base) && rope_base > 0.f),
          "rope_base must be finite and > 0 (got %g)", static_cast<double>(rope_base));
  REQUIRE(!std::isnan(softmax_scale) && !std::isinf(softmax_scale), "softmax_scale must be finite");
  REQUIRE_PTR(q, 16);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE(out != nullptr || head_out != nullptr, "out and head_out are both NULL");
  if (out != nullptr) REQUIRE_PTR(out, 16);
  if (head_out != nullptr) REQUIRE_PTR(head_out, 16);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::shared_workspace_bytes(B, T, Hs, d_head))) != NAMOH_OK)
    return s;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt(static_cast<float>(d_head));
  clear_hip_error();
  return launched(stream, namoh::launch_shared(q, k, v, B, T, Hs, d_head, window, rope_base,
                                         rope_mode == NAMOH_ROPE_NONE ? 2 : 1, scale, out,
                                         out_dtype, accumulate, head_out, workspace,
                                         static_cast<hipStream_t>(stream)));
}

namespace {
namoh_status check_shared_decode(int B, int Hs, int d_head, int cap, int window, int dtype,
                                 int rope_mode, float rope_base) {
  namoh_status s;
  REQUIRE(B >= 1, "B must be >= 1 (got %d)", B);
  REQUIRE(Hs >= 1 && Hs <= 1024, "Hs must be in [1, 1024] (got %d)", Hs);
  if ((s = check_head_width(d_head)) != NAMOH_OK) return s;
  REQUIRE(dtype == NAMOH_F32 || dtype == NAMOH_BF16, "unknown dtype %d", dtype);
  REQUIRE(cap >= 1, "cap must be >= 1 (got %d)", cap);
  REQUIRE(window >= 0, "window must be >= 0 (got %d)", window);
  REQUIRE(window == 0 || cap >= window, "cap (%d) must hold the window (%d)", cap, window);
  REQUIRE(static_cast<long long>(B) * Hs * ((cap + 511) / 512) < (1ll << 31),
          "B*Hs*ceil(cap/512) must be < 2^31");
  REQUIRE(static_cast<long long>(B) * Hs * cap * d_head < (1ll << 40), "caches too large");
  REQUIRE(rope_mode == NAMOH_ROPE_HEAD_RELATIVE || rope_mode == NAMOH_ROPE_GLOBAL ||
              rope_mode == NAMOH_ROPE_NONE,
          "unknown rope_mode %d", rope_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_NONE || (std::isfinite(rope_base) && rope_base > 0.f),
          "rope_base must be finite and > 0 (got %g)", static_cast<double>(rope_base));
  return NAMOH_OK;
}
}  // namespace

size_t namoh_shared_decode_workspace_size(int B, int Hs, int d_head, int cap) {
  if (check_shared_decode(B, Hs, d_head, cap, 0, NAMOH_BF16, NAMOH_ROPE_NONE, 1.f) != NAMOH_OK)
    return 0;
  return namoh::shared_decode_workspace_bytes(B, Hs, d_head, cap);
}

namoh_status namoh_shared_decode_step(const void* q, const void* k, const void* v, int dtype,
                                      int B, int Hs, int d_head, int cap, int window,
                                      float rope_base, int rope_mode, float softmax_scale,
                                      void* k_cache, void* v_cache, int32_t* cache_len, void* out,
                                      int out_dtype, int accumulate, int32_t* dev_status,
                                      void* workspace, size_t workspace_bytes, void* stream) {
  namoh_status s;
  if ((s = check_shared_decode(B, Hs, d_head, cap, window, dtype, rope_mode, rope_base)) !=
      NAMOH_OK)
    return s;
  REQUIRE(!std::isnan(softmax_scale) && !std::isinf(softmax_scale), "softmax_scale must be finite");
  REQUIRE(out_dtype == NAMOH_F32 || out_dtype == NAMOH_BF16, "unknown out_dtype %d", out_dtype);
  REQUIRE(accumulate == 0 || accumulate == 1, "accumulate must be 0 or 1 (got %d)", accumulate);
  REQUIRE_PTR(q, 16);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE_PTR(k_cache, 16);
  REQUIRE_PTR(v_cache, 16);
  REQUIRE_PTR(cache_len, 4);
  REQUIRE_PTR(out, 16);
  if (dev_status != nullptr) REQUIRE_PTR(dev_status, 4);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::shared_decode_workspace_bytes(B, Hs, d_head, cap))) != NAMOH_OK)
    return s;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt(static_cast<float>(d_head));
  clear_hip_error();
  return launched(stream, namoh::launch_shared_decode(
                              q, k, v, dtype, k_cache, v_cache, cache_len, B, Hs, d_head, cap,
                              window, rope_base, rope_mode == NAMOH_ROPE_NONE ? 2 : 1, scale, out,
                              out_dtype, accumulate, dev_status, workspace,
                              static_cast<hipStream_t>(stream)));
}

namoh_status namoh_shared_prefill_cache(const void* k, const void* v, int dtype, int B, int T,
                                        int Hs, int d_head, int cap, int window, float rope_base,
                                        int rope_mode, void* k_cache, void* v_cache,
                                        int32_t* cache_len, void* stream) {
  namoh_status s;
  if ((s = check_shared_decode(B, Hs, d_head, cap, window, dtype, rope_mode, rope_base)) !=
      NAMOH_OK)
    return s;
  REQUIRE(T >= 1, "T must be >= 1 (got %d)", T);
  REQUIRE(static_cast<long long>(B) * Hs * T < (1ll << 31), "B*Hs*T must be < 2^31");
  REQUIRE(window > 0 || cap >= T, "without a window cap (%d) must hold the prompt (T = %d)", cap,
          T);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE_PTR(k_cache, 16);
  REQUIRE_PTR(v_cache, 16);
  REQUIRE_PTR(cache_len, 4);
  clear_hip_error();
  return launched(stream, namoh::launch_shared_prefill_cache(
                              k, v, dtype, B, T, Hs, d_head, cap, rope_base,
                              rope_mode == NAMOH_ROPE_NONE ? 2 : 1, k_cache, v_cache, cache_len,
                              static_cast<hipStream_t>(stream)));
}

size_t namoh_attn_fwd_grouped_workspace_size(int B, int T, int H_kv, int K_kv, int group_size,
                                             int d_head, int dtype) {
  if (check_sizes(B, T, H_kv, K_kv) != NAMOH_OK || group_size < 1 || group_size > 16 ||
      (d_head != 64 && d_head != 128) || dtype != NAMOH_BF16)
    return 0;
  return namoh::attn_workspace_bytes(B, T, H_kv, K_kv, d_head, dtype, group_size);
}

namoh_status namoh_attn_fwd_grouped(const void* q, const void* k, const void* v, int dtype,
                                    int B, int T, int H_kv, int K_kv, int group_size, int d_head,
                                    float rope_base, int rope_mode, float softmax_scale,
                                    const float* gates, const int32_t* seg_offsets,
                                    const int32_t* perm_token, const int32_t* slot_pos,
                                    void* out, int out_dtype, float* head_out, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  namoh_status s;
  if ((s = check_sizes(B, T, H_kv, K_kv)) != NAMOH_OK) return s;
  REQUIRE(group_size >= 1 && group_size <= 16, "group_size must be in [1, 16] (got %d)",
          group_size);
  REQUIRE(dtype == NAMOH_F32 || dtype == NAMOH_BF16, "unknown dtype %d", dtype);
  if (dtype != NAMOH_BF16 || (d_head != 64 && d_head != 128))
    return fail(NAMOH_ERR_UNSUPPORTED, "key/value groups need bf16 and d_head 64 or 128");
  REQUIRE(out_dtype == NAMOH_F32 || out_dtype == NAMOH_BF16, "unknown out_dtype %d", out_dtype);
  REQUIRE(rope_mode == NAMOH_ROPE_HEAD_RELATIVE || rope_mode == NAMOH_ROPE_GLOBAL ||
              rope_mode == NAMOH_ROPE_NONE,
          "unknown rope_mode %d", rope_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_NONE || (std::isfinite(rope_base) && rope_base > 0.f),
          "rope_base must be finite and > 0 (got %g)", static_cast<double>(rope_base));
  REQUIRE(!std::isnan(softmax_scale) && !std::isinf(softmax_scale), "softmax_scale must be finite");
  REQUIRE(static_cast<long long>(B) * H_kv * group_size * T * d_head < (1ll << 40),
          "q too large");
  // the MFMA path addresses one segment's key tiles with 32-bit byte offsets
  if ((static_cast<long long>(T) + 63) / 64 * 64 * d_head * 2 >= (1ll << 32))
    return fail(NAMOH_ERR_UNSUPPORTED, "T = %d too long for d_head = %d on the bf16 path", T,
                d_head);
  REQUIRE_PTR(q, 16);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(perm_token, 4);
  REQUIRE_PTR(slot_pos, 4);
  REQUIRE(out != nullptr || head_out != nullptr, "out and head_out are both NULL");
  if (out != nullptr) REQUIRE_PTR(out, 16);
  if (head_out != nullptr) REQUIRE_PTR(head_out, 16);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::attn_workspace_bytes(B, T, H_kv, K_kv, d_head, dtype,
                                                       group_size))) != NAMOH_OK)
    return s;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt(static_cast<float>(d_head));
  clear_hip_error();
  return launched(stream, namoh::launch_attn(q, k, v, dtype, B, T, H_kv, K_kv, d_head, rope_base,
                                       rope_mode, scale, gates, seg_offsets, perm_token,
                                       slot_pos, out, out_dtype, head_out, workspace,
                                       static_cast<hipStream_t>(stream), group_size));
}

namespace {
namoh_status check_proj(int B, int T, int H, int K, int d_head, int d_model) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  if (d_head != 64 && d_head != 128)
    return fail(NAMOH_ERR_UNSUPPORTED, "projections need d_head 64 or 128 (got %d)", d_head);
  if (d_model < 128 || d_model % 128 != 0 || d_model > 65536)
    return fail(NAMOH_ERR_UNSUPPORTED, "d_model must be a multiple of 128 in [128, 65536] (got %d)",
                d_model);
  REQUIRE(static_cast<long long>(B) * T * K * d_model < (1ll << 40), "projection too large");
  REQUIRE(static_cast<long long>(B) * H * T * d_head < (1ll << 40), "q/k/v too large");
  return NAMOH_OK;
}
}  // namespace

namoh_status namoh_qkv_proj(const void* x, const void* w_qkv, int B, int T, int H, int K,
                            int d_head, int d_model, const int32_t* seg_offsets,
                            const int32_t* perm_token, void* q, void* k, void* v, void* stream) {
  namoh_status s;
  if ((s = check_proj(B, T, H, K, d_head, d_model)) != NAMOH_OK) return s;
  REQUIRE_PTR(x, 16);
  REQUIRE_PTR(w_qkv, 16);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(perm_token, 4);
  REQUIRE_PTR(q, 16);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  clear_hip_error();
  return launched(stream, namoh::launch_qkv_proj(x, w_qkv, B, T, H, K, d_head, d_model, seg_offsets,
                                           perm_token, q, k, v, static_cast<hipStream_t>(stream)));
}

size_t namoh_out_proj_workspace_size(int B, int T, int H, int K, int d_head, int d_model) {
  if (check_proj(B, T, H, K, d_head, d_model) != NAMOH_OK) return 0;
  return namoh::out_proj_workspace_bytes(B, T, H, K, d_head, d_model);
}

namoh_status namoh_out_proj(const void* head_out, int head_out_dtype, const void* w_o,
                            const float* gates, const int32_t* slot_pos,
                            const int32_t* seg_offsets, int B, int T, int H, int K, int d_head,
                            int d_model, void* out, int out_dtype, void* workspace,
                            size_t workspace_bytes, void* stream) {
  namoh_status s;
  if ((s = check_proj(B, T, H, K, d_head, d_model)) != NAMOH_OK) return s;
  REQUIRE(head_out_dtype == NAMOH_F32 || head_out_dtype == NAMOH_BF16,
          "unknown head_out_dtype %d", head_out_dtype);
  REQUIRE(out_dtype == NAMOH_F32 || out_dtype == NAMOH_BF16, "unknown out_dtype %d", out_dtype);
  REQUIRE_PTR(head_out, 16);
  REQUIRE_PTR(w_o, 16);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(slot_pos, 4);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(out, 16);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::out_proj_workspace_bytes(B, T, H, K, d_head, d_model))) != NAMOH_OK)
    return s;
  clear_hip_error();
  return launched(stream, namoh::launch_out_proj(head_out, head_out_dtype, w_o, gates, slot_pos,
                                           seg_offsets, B, T, H, K, d_head, d_model, out,
                                           out_dtype, workspace,
                                           static_cast<hipStream_t>(stream)));
}

size_t namoh_attn_bwd_workspace_size(int B, int T, int H, int K, int d_head) {
  if (check_sizes(B, T, H, K) != NAMOH_OK || check_head_width(d_head) != NAMOH_OK) return 0;
  return namoh::attn_bwd_workspace_bytes(B, T, H, K, d_head);
}

static namoh_status attn_bwd_common(const void* q, const void* k, const void* v, int dtype,
                                    int B, int T, int H, int K, int d_head, float rope_base,
                                    int rope_mode, float softmax_scale, const int32_t* topk_idx,
                                    const float* gates, const int32_t* seg_offsets,
                                    const int32_t* perm_token, const float* dout, float* dq,
                                    float* dk, float* dv, float* dgates, void* workspace,
                                    size_t workspace_bytes, void* stream, bool packed,
                                    bool saved = false) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  if ((s = check_head_width(d_head)) != NAMOH_OK) return s;
  REQUIRE(dtype == NAMOH_F32 || dtype == NAMOH_BF16, "unknown dtype %d", dtype);
  REQUIRE(rope_mode == NAMOH_ROPE_HEAD_RELATIVE || rope_mode == NAMOH_ROPE_GLOBAL ||
              rope_mode == NAMOH_ROPE_NONE,
          "unknown rope_mode %d", rope_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_NONE || (std::isfinite(rope_base) && rope_base > 0.f),
          "rope_base must be finite and > 0 (got %g)", static_cast<double>(rope_base));
  REQUIRE(!std::isnan(softmax_scale) && !std::isinf(softmax_scale), "softmax_scale must be finite");
  REQUIRE(static_cast<long long>(B) * H * T * d_head < (1ll << 40), "q/k/v too large");
  REQUIRE(B * H <= 65535, "B*H = %d segments exceed the backward grid", B * H);
  if ((s = check_segment_bytes(dtype, T, d_head)) != NAMOH_OK) return s;
  if (saved && !namoh::attn_train_supported(dtype, d_head))
    return fail(NAMOH_ERR_UNSUPPORTED,
                "namoh_attn_bwd_saved needs dtype bf16 and d_head 64 or 128 (got dtype %d, "
                "d_head %d)", dtype, d_head);
  REQUIRE_PTR(q, 16);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE_PTR(topk_idx, 4);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(perm_token, 4);
  REQUIRE_PTR(dout, 16);
  REQUIRE_PTR(dq, 16);
  REQUIRE_PTR(dk, 16);
  REQUIRE_PTR(dv, 16);
  REQUIRE_PTR(dgates, 4);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::attn_bwd_workspace_bytes(B, T, H, K, d_head))) != NAMOH_OK)
    return s;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt(static_cast<float>(d_head));
  clear_hip_error();
  return launched(stream, namoh::launch_attn_bwd(q, k, v, dtype, B, T, H, K, d_head, rope_base,
                                           rope_mode, scale, topk_idx, gates, seg_offsets,
                                           perm_token, dout, dq, dk, dv, dgates, workspace,
                                           static_cast<hipStream_t>(stream), packed, saved));
}

namoh_status namoh_attn_bwd(const void* q, const void* k, const void* v, int dtype, int B, int T,
                            int H, int K, int d_head, float rope_base, int rope_mode,
                            float softmax_scale, const int32_t* topk_idx, const float* gates,
                            const int32_t* seg_offsets, const int32_t* perm_token,
                            const float* dout, float* dq, float* dk, float* dv, float* dgates,
                            void* workspace, size_t workspace_bytes, void* stream) {
  return attn_bwd_common(q, k, v, dtype, B, T, H, K, d_head, rope_base, rope_mode, softmax_scale,
                         topk_idx, gates, seg_offsets, perm_token, dout, dq, dk, dv, dgates,
                         workspace, workspace_bytes, stream, false);
}

namoh_status namoh_attn_bwd_packed(const void* q, const void* k, const void* v, int dtype, int B,
                                   int T, int H, int K, int d_head, float rope_base,
                                   int rope_mode, float softmax_scale, const int32_t* topk_idx,
                                   const float* gates, const int32_t* seg_offsets,
                                   const int32_t* perm_token, const float* dout, float* dq,
                                   float* dk, float* dv, float* dgates, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  return attn_bwd_common(q, k, v, dtype, B, T, H, K, d_head, rope_base, rope_mode, softmax_scale,
                         topk_idx, gates, seg_offsets, perm_token, dout, dq, dk, dv, dgates,
                         workspace, workspace_bytes, stream, true);
}

namoh_status namoh_attn_bwd_saved(const void* q, const void* k, const void* v, int dtype, int B,
                                  int T, int H, int K, int d_head, float rope_base,
                                  int rope_mode, float softmax_scale, const int32_t* topk_idx,
                                  const float* gates, const int32_t* seg_offsets,
                                  const int32_t* perm_token, const float* dout, float* dq,
                                  float* dk, float* dv, float* dgates, int packed,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  REQUIRE(packed == 0 || packed == 1, "packed must be 0 or 1 (got %d)", packed);
  return attn_bwd_common(q, k, v, dtype, B, T, H, K, d_head, rope_base, rope_mode, softmax_scale,
                         topk_idx, gates, seg_offsets, perm_token, dout, dq, dk, dv, dgates,
                         workspace, workspace_bytes, stream, packed == 1, true);
}

namoh_status namoh_attn_fwd_train(const void* q, const void* k, const void* v, int dtype, int B,
                                  int T, int H, int K, int d_head, float rope_base,
                                  int rope_mode, float softmax_scale, const float* gates,
                                  const int32_t* seg_offsets, const int32_t* perm_token,
                                  const int32_t* slot_pos, void* out, int out_dtype,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  if ((s = check_head_width(d_head)) != NAMOH_OK) return s;
  REQUIRE(dtype == NAMOH_F32 || dtype == NAMOH_BF16, "unknown dtype %d", dtype);
  REQUIRE(out_dtype == NAMOH_F32 || out_dtype == NAMOH_BF16, "unknown out_dtype %d", out_dtype);
  REQUIRE(rope_mode == NAMOH_ROPE_HEAD_RELATIVE || rope_mode == NAMOH_ROPE_GLOBAL ||
              rope_mode == NAMOH_ROPE_NONE,
          "unknown rope_mode %d", rope_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_NONE || (std::isfinite(rope_base) && rope_base > 0.f),
          "rope_base must be finite and > 0 (got %g)", static_cast<double>(rope_base));
  REQUIRE(!std::isnan(softmax_scale) && !std::isinf(softmax_scale), "softmax_scale must be finite");
  REQUIRE(static_cast<long long>(B) * H * T * d_head < (1ll << 40), "q/k/v too large");
  if ((s = check_segment_bytes(dtype, T, d_head)) != NAMOH_OK) return s;
  if (!namoh::attn_train_supported(dtype, d_head))
    return fail(NAMOH_ERR_UNSUPPORTED,
                "namoh_attn_fwd_train needs dtype bf16 and d_head 64 or 128 (got dtype %d, "
                "d_head %d)", dtype, d_head);
  REQUIRE_PTR(q, 16);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(seg_offsets, 4);
  REQUIRE_PTR(perm_token, 4);
  REQUIRE_PTR(slot_pos, 4);
  REQUIRE_PTR(out, 16);
  if ((s = check_workspace(workspace, workspace_bytes,
                           namoh::attn_bwd_workspace_bytes(B, T, H, K, d_head))) != NAMOH_OK)
    return s;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt(static_cast<float>(d_head));
  clear_hip_error();
  return launched(stream, namoh::launch_train_fwd(q, k, v, dtype, B, T, H, K, d_head, rope_base,
                                                  rope_mode, scale, gates, seg_offsets,
                                                  perm_token, slot_pos, out, out_dtype,
                                                  workspace, static_cast<hipStream_t>(stream)));
}

namoh_status namoh_route_bwd(const float* logits, const int32_t* topk_idx, const float* gates,
                             const float* dgates, int B, int T, int H, int K, int gate_mode,
                             float* dlogits, void* stream) {
  namoh_status s;
  if ((s = check_sizes(B, T, H, K)) != NAMOH_OK) return s;
  REQUIRE(gate_mode == NAMOH_GATE_SOFTMAX_SELECTED || gate_mode == NAMOH_GATE_SOFTMAX_ALL,
          "unknown gate_mode %d", gate_mode);
  REQUIRE_PTR(logits, 4);
  REQUIRE_PTR(topk_idx, 4);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(dgates, 4);
  REQUIRE_PTR(dlogits, 4);
  clear_hip_error();
  return launched(stream, namoh::launch_route_bwd(logits, topk_idx, gates, dgates, B, T, H, K,
                                            gate_mode, dlogits,
                                            static_cast<hipStream_t>(stream)));
}

size_t namoh_decode_workspace_size(int B, int H, int K, int d_head, int cap) {
  if (check_sizes(B, 1, H, K) != NAMOH_OK || check_head_width(d_head) != NAMOH_OK || cap < 1)
    return 0;
  return namoh::decode_workspace_bytes(B, H, K, d_head, cap);
}

size_t namoh_decode_grouped_workspace_size(int B, int H_kv, int K_kv, int group_size, int d_head,
                                           int cap) {
  if (check_sizes(B, 1, H_kv, K_kv) != NAMOH_OK || (d_head != 64 && d_head != 128) || cap < 1 ||
      (group_size != 1 && group_size != 2 && group_size != 4 && group_size != 8))
    return 0;
  return namoh::decode_workspace_bytes(B, H_kv, K_kv, d_head, cap, group_size);
}

static namoh_status decode_common(const float* logits, const float* bias, const void* q,
                                  const void* k, const void* v, int dtype, void* k_cache,
                                  void* v_cache, int32_t* cache_len, const int32_t* seq_pos,
                                  int B, int H, int K, int d_head, int cap, float rope_base,
                                  int rope_mode, int gate_mode, float softmax_scale,
                                  int32_t* topk_idx, float* gates, void* out, int out_dtype,
                                  int32_t* dev_status, void* workspace, size_t workspace_bytes,
                                  void* stream, int group_size = 0, bool noalloc = false) {
  // group_size 0: the per-head step; >= 1: key/value groups of that many
  // query heads (namoh_decode_step_grouped).  noalloc: the workspace is the
  // library's fixed scratch (namoh_decode_step_noalloc), resolved after every
  // other argument has been checked.
  namoh_status s;
  if ((s = check_sizes(B, 1, H, K)) != NAMOH_OK) return s;
  if ((s = check_head_width(d_head)) != NAMOH_OK) return s;
  if (group_size != 0) {
    REQUIRE(group_size == 1 || group_size == 2 || group_size == 4 || group_size == 8,
            "group_size must be 1, 2, 4 or 8 (got %d)", group_size);
    if (dtype != NAMOH_BF16 || (d_head != 64 && d_head != 128))
      return fail(NAMOH_ERR_UNSUPPORTED, "grouped decode needs bf16 and d_head 64 or 128");
  }
  REQUIRE(cap >= 1, "cap must be >= 1 (got %d)", cap);
  REQUIRE(dtype == NAMOH_F32 || dtype == NAMOH_BF16, "unknown dtype %d", dtype);
  REQUIRE(out_dtype == NAMOH_F32 || out_dtype == NAMOH_BF16, "unknown out_dtype %d", out_dtype);
  REQUIRE(gate_mode == NAMOH_GATE_SOFTMAX_SELECTED || gate_mode == NAMOH_GATE_SOFTMAX_ALL,
          "unknown gate_mode %d", gate_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_HEAD_RELATIVE || rope_mode == NAMOH_ROPE_GLOBAL ||
              rope_mode == NAMOH_ROPE_NONE,
          "unknown rope_mode %d", rope_mode);
  REQUIRE(rope_mode == NAMOH_ROPE_NONE || (std::isfinite(rope_base) && rope_base > 0.f),
          "rope_base must be finite and > 0 (got %g)", static_cast<double>(rope_base));
  REQUIRE(!std::isnan(softmax_scale) && !std::isinf(softmax_scale), "softmax_scale must be finite");
  REQUIRE_PTR(logits, 4);
  REQUIRE_PTR(q, 16);
  REQUIRE_PTR(k, 16);
  REQUIRE_PTR(v, 16);
  REQUIRE_PTR(k_cache, 16);
  REQUIRE_PTR(v_cache, 16);
  REQUIRE_PTR(cache_len, 4);
  if (rope_mode == NAMOH_ROPE_GLOBAL) REQUIRE_PTR(seq_pos, 4);
  REQUIRE_PTR(topk_idx, 4);
  REQUIRE_PTR(gates, 4);
  REQUIRE_PTR(out, 16);
  if (dev_status != nullptr) REQUIRE_PTR(dev_status, 4);
  const size_t need =
      namoh::decode_workspace_bytes(B, H, K, d_head, cap, group_size > 0 ? group_size : 1);
  if (noalloc) {
    workspace_bytes = namoh::decode_scratch_bytes();
    if (need > workspace_bytes)
      return fail(NAMOH_ERR_WORKSPACE,
                  "namoh_decode_step_noalloc: B=%d K=%d d_head=%d cap=%d needs %zu bytes of "
                  "scratch, above its fixed %zu bytes (use namoh_decode_step with a workspace)",
                  B, K, d_head, cap, need, workspace_bytes);
    clear_hip_error();
    const hipError_t e = namoh::decode_scratch(&workspace);
    if (e != hipSuccess) return hip_status(e);
  }
  if ((s = check_workspace(workspace, workspace_bytes, need)) != NAMOH_OK) return s;
  const float scale = softmax_scale > 0.f ? softmax_scale : 1.f / std::sqrt(static_cast<float>(d_head));
  clear_hip_error();
  if (group_size != 0)
    return launched(stream, namoh::launch_decode_grouped(
        logits, q, k, v, k_cache, v_cache, cache_len, seq_pos, B, H, K, group_size, d_head, cap,
        rope_base, rope_mode, gate_mode, scale, topk_idx, gates, out, out_dtype, dev_status,
        workspace, static_cast<hipStream_t>(stream)));
  return launched(stream, namoh::launch_decode(logits, bias, q, k, v, dtype, k_cache, v_cache,
                                         cache_len, seq_pos, B, H, K, d_head, cap, rope_base,
                                         rope_mode, gate_mode, scale, topk_idx, gates, out,
                                         out_dtype, dev_status, workspace,
                                         static_cast<hipStream_t>(stream)));
}

namoh_status namoh_decode_step(const float* logits, const void* q, const void* k,
                               const void* v, int dtype, void* k_cache, void* v_cache,
                               int32_t* cache_len, const int32_t* seq_pos, int B, int H,
                               int K, int d_head, int cap, float rope_base, int rope_mode,
                               int gate_mode, float softmax_scale, int32_t* topk_idx,
                               float* gates, void* out, int out_dtype, int32_t* dev_status,
                               void* workspace, size_t workspace_bytes, void* stream) {
  return decode_common(logits, nullptr, q, k, v, dtype, k_cache, v_cache, cache_len, seq_pos, B,
                       H, K, d_head, cap, rope_base, rope_mode, gate_mode, softmax_scale,
                       topk_idx, gates, out, out_dtype, dev_status, workspace, workspace_bytes,
                       stream);
}

namoh_status namoh_decode_step_noalloc(const float* logits, const void* q, const void* k,
                                       const void* v, int dtype, void* k_cache, void* v_cache,
                                       int32_t* cache_len, const int32_t* seq_pos, int B, int H,
                                       int K, int d_head, int cap, float rope_base, int rope_mode,
                                       int gate_mode, float softmax_scale, int32_t* topk_idx,
                                       float* gates, void* out, int out_dtype, int32_t* dev_status,
                                       void* stream) {
  return decode_common(logits, nullptr, q, k, v, dtype, k_cache, v_cache, cache_len, seq_pos, B,
                       H, K, d_head, cap, rope_base, rope_mode, gate_mode, softmax_scale,
                       topk_idx, gates, out, out_dtype, dev_status, nullptr, 0, stream, 0, true);
}

namoh_status namoh_decode_step_biased(const float* logits, const float* bias, const void* q,
                                      const void* k, const void* v, int dtype, void* k_cache,
                                      void* v_cache, int32_t* cache_len, const int32_t* seq_pos,
                                      int B, int H, int K, int d_head, int cap, float rope_base,
                                      int rope_mode, float softmax_scale, int32_t* topk_idx,
                                      float* gates, void* out, int out_dtype,
                                      int32_t* dev_status, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  REQUIRE_PTR(bias, 4);
  return decode_common(logits, bias, q, k, v, dtype, k_cache, v_cache, cache_len, seq_pos, B, H,
                       K, d_head, cap, rope_base, rope_mode, NAMOH_GATE_SOFTMAX_ALL,
                       softmax_scale, topk_idx, gates, out, out_dtype, dev_status, workspace,
                       workspace_bytes, stream);
}

namoh_status namoh_decode_step_grouped(const float* logits, const void* q, const void* k,
                                       const void* v, int dtype, void* k_cache, void* v_cache,
                                       int32_t* cache_len, const int32_t* seq_pos, int B, int H_kv,
                                       int K_kv, int group_size, int d_head, int cap,
                                       float rope_base, int rope_mode, int gate_mode,
                                       float softmax_scale, int32_t* topk_idx, float* gates,
                                       void* out, int out_dtype, int32_t* dev_status,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  if (group_size < 1) return fail(NAMOH_ERR_INVALID_ARG, "group_size must be >= 1 (got %d)",
                                  group_size);
  return decode_common(logits, nullptr, q, k, v, dtype, k_cache, v_cache, cache_len, seq_pos, B,
                       H_kv, K_kv, d_head, cap, rope_base, rope_mode, gate_mode, softmax_scale,
                       topk_idx, gates, out, out_dtype, dev_status, workspace, workspace_bytes,
                       stream, group_size);
}

}  // extern "C"
