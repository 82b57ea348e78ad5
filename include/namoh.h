/*
 * namoh.h — C ABI of the MI355X (gfx950) routed mixture-of-head attention
 * library (libnamoh.so).
 *
 * The layer follows NAMOH ("Native Sparse Attention from Mixture-of-Head"):
 * every token picks K of H heads from its router logits (Sec. 3.1,
 * Eq. namoh-gates), each head runs causal scaled dot-product attention only
 * over the tokens routed to it (Sec. 3.1, Eq. namoh-attention), with RoPE at
 * the token's rank inside that head's subsequence (Sec. 3.2,
 * Eq. namoh-head-rope), and the gated per-head outputs are summed per token.
 * The per-head output projection W_O^(i) is taken as the identity, so the
 * layer output has the head width d.
 *
 * Conventions shared by every call
 *  - Every pointer argument is a DEVICE pointer to contiguous memory owned by
 *    the caller.  The library allocates nothing, frees nothing, never
 *    synchronises, and enqueues all its work on `stream` (a hipStream_t;
 *    NULL = the default stream), in order.
 *  - Arguments are validated on the host before anything is enqueued; a call
 *    that returns an error has launched nothing.  namoh_last_error() then
 *    gives a thread-local message.
 *  - Floating-point tensors are 16-byte aligned; int32 / float32 index and
 *    gate arrays are 4-byte aligned.
 *  - Limits: 1 <= K <= H <= 64; d_head in {32, 64, 128}; B, T >= 1;
 *    B*T*K < 2^31.
 *  - No floating-point atomics are used: results are bit-identical from run
 *    to run for the same inputs.
 *  - Workspace: query its size with the matching *_workspace_size() call;
 *    pass at least that many bytes, 256-byte aligned (NULL allowed when the
 *    size is 0).  Its contents need not be initialised and are garbage after.
 *  - Debugging: with NAMOH_SYNC_CHECK=1 in the environment (read once per
 *    process), every call that launched work synchronises its stream before
 *    returning and reports an error of its kernels as NAMOH_ERR_HIP.
 */
#ifndef NAMOH_H_
#define NAMOH_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum namoh_status {
  NAMOH_OK = 0,
  NAMOH_ERR_INVALID_ARG = 1,  /* NULL pointer, bad size, bad enum, misalignment */
  NAMOH_ERR_UNSUPPORTED = 2,  /* valid request outside the supported set      */
  NAMOH_ERR_WORKSPACE = 3,    /* workspace smaller than the size query        */
  NAMOH_ERR_HIP = 4           /* a HIP runtime/launch error (e.g. no device)  */
} namoh_status;

typedef enum namoh_dtype { NAMOH_F32 = 0, NAMOH_BF16 = 1 } namoh_dtype;

/* Gate definition.  SOFTMAX_SELECTED: g = softmax over the K selected logits
 * (gates sum to one).  SOFTMAX_ALL: g_i = softmax over all H logits at the
 * selected heads, not renormalised (Eq. namoh-gates as printed). */
typedef enum namoh_gate_mode {
  NAMOH_GATE_SOFTMAX_SELECTED = 0,
  NAMOH_GATE_SOFTMAX_ALL = 1
} namoh_gate_mode;

/* Position used by RoPE.  HEAD_RELATIVE: the token's zero-based rank inside
 * the head's routed subsequence (Eq. namoh-head-rope).  GLOBAL: the token's
 * index t (Sec. 3.2, last sentence of the head-relative paragraph).  NONE:
 * no rotation.  Rotation pairs element j with j + d/2, angle
 * p * base^(-2j/d), V is never rotated. */
typedef enum namoh_rope_mode {
  NAMOH_ROPE_HEAD_RELATIVE = 0,
  NAMOH_ROPE_GLOBAL = 1,
  NAMOH_ROPE_NONE = 2
} namoh_rope_mode;

/* ------------------------------------------------------------------------
 * Routing and dispatch (Sec. 3.1, Eq. namoh-gates and the definition of the
 * ordered index sets I_i; Sec. 3.2 "Efficient execution": packing of each
 * (batch, head) subsequence).
 *
 * In:  logits    float32 [B, T, H]   router logits (finite; NaN is outside
 *                                    the contract).
 * Out: topk_idx  int32 [B, T, K]     selected heads ordered by logit
 *                                    descending, equal logits by head index
 *                                    ascending (-0.0 equals +0.0).
 *      gates     float32 [B, T, K]   gate of topk_idx[b,t,k] (gate_mode).
 *      head_len  int32 [B, H]        n_i of every (b, h).
 *      seg_offsets int32 [B*H + 1]   segment s = b*H + h occupies packed
 *                                    positions [seg_offsets[s], seg_offsets[s+1]).
 *      perm_token int32 [B*T*K]      packed position -> token t; tokens are
 *                                    ascending inside a segment, so the rank
 *                                    rho_h(t) = position - seg_offsets[s].
 *      slot_pos  int32 [B, T, K]     packed position of (b, t, topk_idx[b,t,k]).
 * All outputs are exact integers / deterministic floats.
 * ---------------------------------------------------------------------- */
size_t namoh_route_workspace_size(int B, int T, int H, int K);

namoh_status namoh_route(const float* logits, int B, int T, int H, int K,
                         int gate_mode, int32_t* topk_idx, float* gates,
                         int32_t* head_len, int32_t* seg_offsets,
                         int32_t* perm_token, int32_t* slot_pos,
                         void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Routing with loss-free balancing biases (App. "Auxiliary-Loss-Free
 * Balancing", Eq. namoh-biased-routing): the heads are selected by their
 * affinity plus a per-head bias, the gates keep the affinity alone.
 *
 * In:  logits    float32 [B, T, H]   as for namoh_route.
 *      bias      float32 [H]         per-head selection bias (finite).
 * Out: as namoh_route, with
 *      topk_idx  the K heads of largest score s_i = float(a_i + b_i),
 *                ordered by score descending, equal scores by head index
 *                ascending, where a = softmax over the H logits is formed
 *                in double (exp of l - max over the token) and the sum
 *                a_i + b_i is rounded once to float;
 *      gates     g_k = a of the selected head, rounded to float, not
 *                renormalised.
 * Same workspace as namoh_route (namoh_route_workspace_size).
 * ---------------------------------------------------------------------- */
namoh_status namoh_route_biased(const float* logits, const float* bias, int B, int T,
                                int H, int K, int32_t* topk_idx, float* gates,
                                int32_t* head_len, int32_t* seg_offsets,
                                int32_t* perm_token, int32_t* slot_pos,
                                void* workspace, size_t workspace_bytes,
                                void* stream);

/* ------------------------------------------------------------------------
 * Loss-free balancing bias step after a batch (App. "Auxiliary-Loss-Free
 * Balancing", Eq. namoh-loss-free): with c_i = sum over b of head_len[b, i]
 * and c_bar = B*T*K / H, bias[i] += eta * sign(c_bar - c_i) (sign(0) = 0,
 * taken exactly in integers; one float add).
 *
 * In:  head_len  int32 [B, H] of the batch (namoh_route's output).
 *      eta       the update rate (finite).
 * In/out: bias   float32 [H].  No workspace.
 * ---------------------------------------------------------------------- */
namoh_status namoh_route_bias_update(const int32_t* head_len, int B, int T, int H, int K,
                                     float eta, float* bias, void* stream);

/* ------------------------------------------------------------------------
 * Routed causal attention and gated combine (Sec. 3.1 Eq. namoh-attention,
 * Sec. 3.2 Eq. namoh-head-rope).  Consumes namoh_route's outputs.
 *
 * In:  q, k, v     [B, H, T, d] of `dtype` (dense per head; only the rows of
 *                  routed (t, h) pairs are read).
 *      rope_base   > 0 unless rope_mode == NONE.
 *      softmax_scale  <= 0 selects 1/sqrt(d).
 *      gates, seg_offsets, perm_token, slot_pos: as produced by namoh_route.
 * Out: out         [B, T, d] of `out_dtype`:
 *                  o_t = sum_k gates[b,t,k] * h(t, topk_idx[b,t,k]);
 *                  may be NULL when head_out is given (the combine is then
 *                  skipped, e.g. before namoh_out_proj).
 *      head_out    optional float32 [B*T*K, d]: ungated head outputs h at
 *                  their packed positions; NULL to skip.
 * bf16 with d in {64, 128} runs on bf16 MFMA (float32 accumulation and
 * softmax; rotated q/k and the probabilities are rounded to bf16 before
 * their products); every other combination runs in float32 arithmetic.
 * The bf16 MFMA path needs ceil(T/64)*64*d*2 < 2^32 bytes per segment
 * (T below 2^24 at d = 128); longer T returns NAMOH_ERR_UNSUPPORTED.
 * ---------------------------------------------------------------------- */
size_t namoh_attn_fwd_workspace_size(int B, int T, int H, int K, int d_head,
                                     int dtype);

namoh_status namoh_attn_fwd(const void* q, const void* k, const void* v,
                            int dtype, int B, int T, int H, int K, int d_head,
                            float rope_base, int rope_mode, float softmax_scale,
                            const float* gates, const int32_t* seg_offsets,
                            const int32_t* perm_token, const int32_t* slot_pos,
                            void* out, int out_dtype, float* head_out,
                            void* workspace, size_t workspace_bytes,
                            void* stream);

/* ------------------------------------------------------------------------
 * Backward of the layer (training path; Sec. 3.2 "Efficient execution":
 * training runs the same packed varlen attention).  The exact gradient of
 * o = namoh_attn_fwd(q, k, v, routing) with the selection held fixed, for
 * an upstream gradient dout:
 *   per (b, h) segment, with the rotated rows Q~, K~, S = Q~ K~^T scale
 *   (causal), P = softmax(S), O = P V, dO_r = g_r dout_t:
 *   dV = P^T dO, dS = P (dO V^T - rowsum(dO O)), dQ~ = dS K~ scale,
 *   dK~ = dS^T Q~ scale, dq = dQ~ R^T (the rotation by minus the angle);
 *   dgates[b,t,k] = <h(t, topk_idx[b,t,k]), dout_t>.
 * The forward statistics are recomputed (fp32 arithmetic throughout), so
 * nothing from the forward call is needed.
 *
 * In:  q, k, v [B, H, T, d] `dtype`; rope and scale as for namoh_attn_fwd;
 *      topk_idx, gates, seg_offsets, perm_token from namoh_route (any gate
 *      mode, or namoh_route_biased); dout float32 [B, T, d].
 * Out: dq, dk, dv float32 [B, H, T, d] (rows of tokens not routed to the
 *      head are zero); dgates float32 [B, T, K].  B*H <= 65535.
 * ---------------------------------------------------------------------- */
size_t namoh_attn_bwd_workspace_size(int B, int T, int H, int K, int d_head);

namoh_status namoh_attn_bwd(const void* q, const void* k, const void* v, int dtype,
                            int B, int T, int H, int K, int d_head, float rope_base,
                            int rope_mode, float softmax_scale, const int32_t* topk_idx,
                            const float* gates, const int32_t* seg_offsets,
                            const int32_t* perm_token, const float* dout, float* dq,
                            float* dk, float* dv, float* dgates, void* workspace,
                            size_t workspace_bytes, void* stream);

/* The same backward with the gradients of the routed (token, head) pairs
 * only, in the routing's packed order: dq, dk, dv float32 [B*T*K, d], row
 * seg_offsets[b*H + h] + rho of the pair (token perm_token[row], head h);
 * that is the layout a routed projection's backward consumes (Sec. 3.1,
 * Eq. namoh-qkv: only routed pairs are projected), and it needs no zero fill
 * of the unrouted rows.  Same inputs, workspace and limits as
 * namoh_attn_bwd; dgates as there. */
namoh_status namoh_attn_bwd_packed(const void* q, const void* k, const void* v, int dtype,
                                   int B, int T, int H, int K, int d_head, float rope_base,
                                   int rope_mode, float softmax_scale, const int32_t* topk_idx,
                                   const float* gates, const int32_t* seg_offsets,
                                   const int32_t* perm_token, const float* dout, float* dq,
                                   float* dk, float* dv, float* dgates, void* workspace,
                                   size_t workspace_bytes, void* stream);

/* Training forward, Sec. 3.2 "Efficient execution" (training runs the same
 * packed varlen attention as prefill) with Sec. 3.1, Eq. namoh-attention:
 * the layer output of namoh_attn_fwd (same inputs; out [B, T, d] in
 * out_dtype, combined from float32 head outputs) and, in `workspace`, what
 * the backward needs from the forward: every routed row's log-sum-exp and
 * head output, the rotated key / value tiles and the work list.
 * namoh_attn_bwd_saved then takes them from there instead of running the
 * forward a second time.  dtype must be NAMOH_BF16 and d_head 64 or 128
 * (otherwise NAMOH_ERR_UNSUPPORTED).  Workspace: at least
 * namoh_attn_bwd_workspace_size(B, T, H, K, d_head) bytes, 256-byte
 * aligned; the caller keeps it unchanged until the backward has run. */
namoh_status namoh_attn_fwd_train(const void* q, const void* k, const void* v, int dtype,
                                  int B, int T, int H, int K, int d_head, float rope_base,
                                  int rope_mode, float softmax_scale, const float* gates,
                                  const int32_t* seg_offsets, const int32_t* perm_token,
                                  const int32_t* slot_pos, void* out, int out_dtype,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* namoh_attn_bwd (packed = 0) or namoh_attn_bwd_packed (packed = 1) on the
 * state a namoh_attn_fwd_train with the same inputs, sizes and routing left
 * in `workspace`: the gradients are those of the stateless calls, bit for
 * bit.  dtype NAMOH_BF16, d_head 64 or 128 (otherwise
 * NAMOH_ERR_UNSUPPORTED); other arguments, outputs and limits as there.
 * The workspace may not have been used by another call in between.  The
 * work records read from it are range-checked on the device before they
 * address anything (a record outside the packed arrays is skipped), so a
 * workspace that did not come from namoh_attn_fwd_train gives undefined
 * gradients but no out-of-range access. */
namoh_status namoh_attn_bwd_saved(const void* q, const void* k, const void* v, int dtype, int B,
                                  int T, int H, int K, int d_head, float rope_base,
                                  int rope_mode, float softmax_scale, const int32_t* topk_idx,
                                  const float* gates, const int32_t* seg_offsets,
                                  const int32_t* perm_token, const float* dout, float* dq,
                                  float* dk, float* dv, float* dgates, int packed,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* Gradient of the gates with respect to the router logits, the selection
 * held fixed (Sec. 3.1, Eq. namoh-gates; the router learns through the
 * gates).  gate_mode SOFTMAX_SELECTED: dl_j = g_j (dg_j - sum_k g_k dg_k)
 * on the selected heads, 0 elsewhere; SOFTMAX_ALL (also the gates of
 * namoh_route_biased): dl = a (da - <a, da>), a = softmax of all H logits,
 * da = dgates placed at the selected heads.
 * In:  logits float32 [B, T, H], topk_idx, gates, dgates [B, T, K].
 * Out: dlogits float32 [B, T, H].  No workspace. */
namoh_status namoh_route_bwd(const float* logits, const int32_t* topk_idx,
                             const float* gates, const float* dgates, int B, int T,
                             int H, int K, int gate_mode, float* dlogits, void* stream);

/* ------------------------------------------------------------------------
 * Key/value-group routing (App. "GQA+NAMOH", adopted KV-group routing): the
 * H = H_kv * g query heads form H_kv groups of g consecutive heads (group j:
 * heads j*g .. j*g + g - 1) that share one key/value head.  The router
 * selects K_kv of the H_kv groups per token (namoh_route on group logits
 * [B, T, H_kv] with K = K_kv); every query head of a selected group attends
 * causally over the group's routed subsequence (RoPE at the group-local
 * rank for the queries and the shared key), and the g head outputs are
 * summed with the group's gate:
 *   o_t = sum_k gates[b,t,k] * sum_{u<g} h(t, topk_idx[b,t,k] * g + u).
 * In:  q [B, H_kv*g, T, d], k, v [B, H_kv, T, d]: bf16, d in {64, 128}
 *      (else NAMOH_ERR_UNSUPPORTED); 1 <= group_size <= 16.
 *      rope/scale and the routing arrays as for namoh_attn_fwd (routing of
 *      the groups).
 * Out: out [B, T, d] of out_dtype (may be NULL when head_out is given);
 *      head_out optional float32 [B*T*K_kv, g, d]: head u of the pair at
 *      packed row p is row p*g + u.
 * group_size 1 computes exactly what namoh_attn_fwd computes.
 * ---------------------------------------------------------------------- */
size_t namoh_attn_fwd_grouped_workspace_size(int B, int T, int H_kv, int K_kv, int group_size,
                                             int d_head, int dtype);

namoh_status namoh_attn_fwd_grouped(const void* q, const void* k, const void* v, int dtype,
                                    int B, int T, int H_kv, int K_kv, int group_size, int d_head,
                                    float rope_base, int rope_mode, float softmax_scale,
                                    const float* gates, const int32_t* seg_offsets,
                                    const int32_t* perm_token, const int32_t* slot_pos,
                                    void* out, int out_dtype, float* head_out, void* workspace,
                                    size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * One decoding step with key/value-group routing (App. "GQA+NAMOH", adopted
 * KV-group routing; the decode counterpart of namoh_attn_fwd_grouped): the
 * new token selects K_kv of the H_kv groups from its group logits (as
 * namoh_decode_step selects heads), appends one rotated key and its value
 * to each selected group's cache at rank n = cache_len (RoPE at the
 * group-local rank, the global position, or none), and each of the group's
 * g query heads attends over the group's n + 1 rows; the step reads each
 * cached row once for all g heads.
 *   out[b] = sum_k gates[b,k] * sum_{u<g} h(query head topk_idx[b,k]*g + u).
 * In:  logits [B, H_kv] f32; q [B, H_kv*g, d]; k, v [B, H_kv, d] (only the
 *      selected groups read); caches [B, H_kv, cap, d], cache_len [B, H_kv]
 *      as for namoh_decode_step.  bf16, d in {64, 128}, group_size in
 *      {1, 2, 4, 8} (else UNSUPPORTED / INVALID_ARG).  With 4 or 8 heads
 *      per group the scores and the probability-weighted values run on the
 *      matrix cores: the rotated, scaled queries and the probabilities are
 *      rounded to bf16 before their products (float32 accumulation and
 *      softmax, as in the bf16 prefill); with 1 or 2 they stay float32.
 * Out: topk_idx, gates [B, K_kv]; out [B, d] of out_dtype; caches and
 *      cache_len updated; dev_status as for namoh_decode_step.
 * Workspace: namoh_decode_grouped_workspace_size bytes.
 * ---------------------------------------------------------------------- */
size_t namoh_decode_grouped_workspace_size(int B, int H_kv, int K_kv, int group_size, int d_head,
                                           int cap);

namoh_status namoh_decode_step_grouped(const float* logits, const void* q, const void* k,
                                       const void* v, int dtype, void* k_cache, void* v_cache,
                                       int32_t* cache_len, const int32_t* seq_pos, int B, int H_kv,
                                       int K_kv, int group_size, int d_head, int cap,
                                       float rope_base, int rope_mode, int gate_mode,
                                       float softmax_scale, int32_t* topk_idx, float* gates,
                                       void* out, int out_dtype, int32_t* dev_status,
                                       void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Always-active shared heads (Sec. 4.4, "shared heads for local context"):
 * Hs heads outside the routing, each attending for every token either to
 * the full causal prefix (window = 0, or window >= T) or to the most recent
 * `window` tokens including the token itself (t - window < s <= t), with
 * RoPE at the global position t (rope_mode GLOBAL; HEAD_RELATIVE is the same
 * position here, since every token is in every shared head; NONE: no
 * rotation).  Their outputs are added to the layer output without a gate:
 *   out[b, t] = (accumulate ? out[b, t] : 0) + sum_{s < Hs} h_s(b, t),
 * with the heads summed in order (call it after namoh_attn_fwd to add the
 * shared heads to the routed output).
 * In:  q, k, v [B, Hs, T, d] bf16 (d in {64, 128}, else UNSUPPORTED).
 * Out: out [B, T, d] of out_dtype (may be NULL when head_out is given);
 *      head_out optional float32 [B, Hs, T, d] (the per-head outputs).
 * Limits: Hs >= 1, B*Hs*T < 2^31, window >= 0.
 * ---------------------------------------------------------------------- */
size_t namoh_shared_attn_workspace_size(int B, int T, int Hs, int d_head);

namoh_status namoh_shared_attn(const void* q, const void* k, const void* v, int dtype, int B,
                               int T, int Hs, int d_head, int window, float rope_base,
                               int rope_mode, float softmax_scale, void* out, int out_dtype,
                               int accumulate, float* head_out, void* workspace,
                               size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Shared heads in the decode step (Sec. 4.4 "Shared heads for local
 * context"; Sec. 3.2: decoding extends the caches one token at a time).
 * The new token of sequence b, at global position p = cache_len[b] (the
 * number of tokens before it), enters every one of the Hs always-active
 * heads: its key, rotated at p (HEAD_RELATIVE and GLOBAL both mean the
 * position p here, every token being in every shared head; NONE: no
 * rotation), and its value are written to row p mod cap of the head's
 * caches, and its query (rotated at p) attends over the keys at positions
 * max(0, p + 1 - window) .. p (window 0: 0 .. p), itself included.  The head
 * outputs are added without a gate:
 *   out[b] = (accumulate ? out[b] : 0) + sum_{s < Hs} h_s(b),
 * so after namoh_decode_step (accumulate = 1) out holds the routed heads
 * plus the shared ones; cache_len[b] = p + 1.
 * In:  q, k, v [B, Hs, d] of `dtype` (f32 or bf16; d 32, 64 or 128).
 * In/out: k_cache, v_cache [B, Hs, cap, d] `dtype` (keys stored rotated);
 *      with window > 0 they are rings that keep the most recent cap tokens
 *      (cap >= window, else NAMOH_ERR_INVALID_ARG), row t mod cap holding
 *      token t; with window = 0 row t holds token t and a step with p >= cap
 *      skips the sequence: nothing is written, cache_len[b] stays, out[b]
 *      gets no shared-head term and *dev_status (if non-NULL) is set to 1.
 *      cache_len int32 [B].
 * Out: out [B, d] of out_dtype.  Workspace: namoh_shared_decode_workspace_size
 *      bytes (rotated queries, history extents, per-512-row partials).
 * Limits: Hs <= 1024, B*Hs*ceil(cap/512) < 2^31.
 * ---------------------------------------------------------------------- */
size_t namoh_shared_decode_workspace_size(int B, int Hs, int d_head, int cap);

namoh_status namoh_shared_decode_step(const void* q, const void* k, const void* v, int dtype,
                                      int B, int Hs, int d_head, int cap, int window,
                                      float rope_base, int rope_mode, float softmax_scale,
                                      void* k_cache, void* v_cache, int32_t* cache_len, void* out,
                                      int out_dtype, int accumulate, int32_t* dev_status,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* Prefill -> decode hand-off of the shared heads (the counterpart of
 * namoh_prefill_cache): for every sequence b and shared head s, the prompt's
 * tokens t (keys rotated at t as above, values as given) go to row t mod cap
 * of the head's caches, for the last min(T, cap) tokens; cache_len[b] = T.
 * window as in namoh_shared_decode_step (0: cap >= T required, else
 * NAMOH_ERR_INVALID_ARG).  In: k, v [B, Hs, T, d] of `dtype`.  No workspace;
 * allocates nothing. */
namoh_status namoh_shared_prefill_cache(const void* k, const void* v, int dtype, int B, int T,
                                        int Hs, int d_head, int cap, int window, float rope_base,
                                        int rope_mode, void* k_cache, void* v_cache,
                                        int32_t* cache_len, void* stream);

/* ------------------------------------------------------------------------
 * Routed per-head projections (Sec. 3.1, Eq. namoh-qkv: tokens are
 * dispatched to their heads before projection, and only active (token, head)
 * pairs compute q, k, v; Eq. namoh-attention: o_t = sum over the selected
 * heads of g_{t,i} h_{t,i} W_O^(i)).  With these two calls around
 * namoh_attn_fwd the layer keeps its per-head output projections instead of
 * taking them as the identity.
 *
 * Weights are stored as linear maps (out x in), bf16, 16-byte aligned:
 *   w_qkv [H, 3, d, d_model]: rows 0 / 1 / 2 of head i are its query, key
 *     and value maps, q_{t,i} = x_t w_qkv[i, 0]^T (the paper's x_t W_Q^(i));
 *   w_o   [H, d_model, d]: h_{t,i} W_O^(i) = h_{t,i} w_o[i]^T.
 * Supported: bf16 x and weights, d_head in {64, 128}, d_model a multiple
 * of 128 (else NAMOH_ERR_UNSUPPORTED).  fp32 accumulation on the matrix
 * cores; q/k/v rounded to bf16.  The output projection takes one of two
 * forms, chosen from H, K and d (the dense form when H * d <= 384 * K and
 * H <= 64):
 *   per-pair: every routed pair's row h W_O^(i) is formed (rounded to bf16)
 *     and the K rows of a token are summed with their gates in k order;
 *   dense:    each token's gated head rows g h (rounded to bf16) enter one
 *     product with the stacked W_O over all H heads (unselected heads
 *     contribute exact zeros) and are summed in head order in fp32: H/K
 *     times the multiply-adds, no per-pair rows.
 * ---------------------------------------------------------------------- */

/* In:  x [B, T, d_model] bf16; w_qkv as above; seg_offsets, perm_token from
 *      namoh_route.
 * Out: q, k, v [B, H, T, d] bf16: the row (b, i, t) is written for every
 *      routed pair (token t of sequence b selected head i) and no other row
 *      is touched (namoh_attn_fwd reads only routed rows).  No workspace. */
namoh_status namoh_qkv_proj(const void* x, const void* w_qkv, int B, int T, int H, int K,
                            int d_head, int d_model, const int32_t* seg_offsets,
                            const int32_t* perm_token, void* q, void* k, void* v,
                            void* stream);

size_t namoh_out_proj_workspace_size(int B, int T, int H, int K, int d_head, int d_model);

/* In:  head_out [B*T*K, d] packed ungated head outputs (as namoh_attn_fwd
 *      writes them to its head_out argument), float32 (head_out_dtype
 *      NAMOH_F32) or bf16; w_o as above; gates, slot_pos, seg_offsets from
 *      namoh_route.
 * Out: out [B, T, d_model] of out_dtype: o_t = sum over the token's k of
 *      gates[b,t,k] * (h W_O^(topk_idx[b,t,k])) at the pair's packed row
 *      (the head of a packed row is that of its segment).
 * Workspace: namoh_out_proj_workspace_size bytes: per-pair form, the
 *      projected rows (bf16 [B*T*K, d_model]); dense form, the per-token head
 *      map (int32 pairs [B*T, H]). */
namoh_status namoh_out_proj(const void* head_out, int head_out_dtype, const void* w_o,
                            const float* gates, const int32_t* slot_pos,
                            const int32_t* seg_offsets, int B, int T, int H, int K, int d_head,
                            int d_model, void* out, int out_dtype, void* workspace,
                            size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Prefill -> decode hand-off (Sec. 3.2, efficient execution: decoding reads
 * and extends only the active heads' caches; Eq. namoh-head-rope: keys are
 * cached after rotation, in rank order).  For every (b, h) with n = n_{b,h}
 * prompt tokens routed to head h, rows [0, n) of the caches receive, in
 * rank order, the rotated keys (RoPE at the rank, the global position, or
 * none, as in namoh_attn_fwd) and the values of those tokens, and
 * cache_len[b,h] = n; rows [n, cap) are not touched.  namoh_decode_step can
 * then continue the sequences.
 *
 * In:  k, v        [B, H, T, d] of `dtype` (the prompt's dense keys/values).
 *      seg_offsets, perm_token: as produced by namoh_route for the prompt.
 * Out: k_cache, v_cache [B, H, cap, d] `dtype`; cache_len int32 [B, H].
 * cap >= T (every head's prompt fits).  No workspace; allocates nothing.
 * Offsets that are not a packing of [0, B*T*K) leave the rows they do not
 * describe unwritten.
 * ---------------------------------------------------------------------- */
namoh_status namoh_prefill_cache(const void* k, const void* v, int dtype, int B, int T,
                                 int H, int K, int d_head, float rope_base,
                                 int rope_mode, const int32_t* seg_offsets,
                                 const int32_t* perm_token, void* k_cache,
                                 void* v_cache, int32_t* cache_len, int cap,
                                 void* stream);

/* ------------------------------------------------------------------------
 * One decoding step for B sequences (Sec. 3.1: prefill and incremental
 * decoding compute the same thing; Sec. 3.2: decoding launches only the
 * active heads and reads/updates only their caches; Eq. namoh-kv-cost).
 *
 * In:  logits     float32 [B, H]     the new token's router logits.
 *      q, k, v    [B, H, d] `dtype`  the new token's projections; only the
 *                                    K selected heads are read.
 *      k_cache, v_cache [B, H, cap, d] `dtype`: rows [0, cache_len[b,h]) hold
 *                 head h's rotated keys / values in rank order.
 *      cache_len  int32 [B, H]       in/out.
 *      seq_pos    int32 [B]          the new token's global index; read only
 *                                    when rope_mode == GLOBAL (else NULL ok).
 * Out: topk_idx int32 [B, K], gates float32 [B, K], out [B, d] `out_dtype`.
 *      For each selected head h with n = cache_len[b,h] < cap, the rotated
 *      key (rank n) and the value are written to row n, cache_len becomes
 *      n + 1, and the token attends to rows [0, n] (itself included).
 *      If n == cap the append is skipped, *dev_status (if non-NULL) is set
 *      to 1 and that head contributes nothing to out.  *dev_status is never
 *      cleared by the library.
 * ---------------------------------------------------------------------- */
size_t namoh_decode_workspace_size(int B, int H, int K, int d_head, int cap);

namoh_status namoh_decode_step(const float* logits, const void* q,
                               const void* k, const void* v, int dtype,
                               void* k_cache, void* v_cache, int32_t* cache_len,
                               const int32_t* seq_pos, int B, int H, int K,
                               int d_head, int cap, float rope_base,
                               int rope_mode, int gate_mode,
                               float softmax_scale, int32_t* topk_idx,
                               float* gates, void* out, int out_dtype,
                               int32_t* dev_status, void* workspace,
                               size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * namoh_decode_step for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same step, the same arguments and results, but no
 * workspace argument.  The step's workspace lives in a fixed device array
 * inside the library: NAMOH_DECODE_NOALLOC_SCRATCH_BYTES (32 MiB) per GPU,
 * held from the first call on that GPU until the process ends.  Calls whose
 * workspace would exceed it (namoh_decode_workspace_size(B, H, K, d_head,
 * cap) > 32 MiB) return NAMOH_ERR_WORKSPACE and launch nothing.  Every call
 * on one GPU uses that GPU's array: calls that overlap on one GPU (several
 * streams or host threads) race, so serialise them.  The call allocates
 * nothing; its first call on a device looks up the array's address there.
 * ---------------------------------------------------------------------- */
#define NAMOH_DECODE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

namoh_status namoh_decode_step_noalloc(const float* logits, const void* q, const void* k,
                                       const void* v, int dtype, void* k_cache, void* v_cache,
                                       int32_t* cache_len, const int32_t* seq_pos, int B, int H,
                                       int K, int d_head, int cap, float rope_base, int rope_mode,
                                       int gate_mode, float softmax_scale, int32_t* topk_idx,
                                       float* gates, void* out, int out_dtype, int32_t* dev_status,
                                       void* stream);

/* The same step with loss-free balancing biases (App. "Auxiliary-Loss-Free
 * Balancing", Eq. namoh-biased-routing; the biases stay fixed during
 * inference): heads selected by float(a + b) and gated by the affinity a
 * exactly as in namoh_route_biased.  bias: float32 [H].  Other arguments and
 * the workspace as for namoh_decode_step (no gate_mode). */
namoh_status namoh_decode_step_biased(const float* logits, const float* bias,
                                      const void* q, const void* k, const void* v,
                                      int dtype, void* k_cache, void* v_cache,
                                      int32_t* cache_len, const int32_t* seq_pos,
                                      int B, int H, int K, int d_head, int cap,
                                      float rope_base, int rope_mode,
                                      float softmax_scale, int32_t* topk_idx,
                                      float* gates, void* out, int out_dtype,
                                      int32_t* dev_status, void* workspace,
                                      size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Diagnostics (not part of the layer's computation).  Opt-in timing of the
 * dominant kernels with HIP events recorded on the call's stream: sections
 * "attn" (routed attention kernel), "pack" (key/value packing), "combine",
 * "decode_attn" (decode history attention).  namoh_profile_enable(n) keeps
 * up to n launches per section (n = 0 stops and clears); it creates HIP
 * events, so it allocates.  namoh_profile_read waits for the recorded events
 * and returns the summed milliseconds and the launch count; it returns -1 for
 * a section that was never timed.  Not for concurrent use from several host
 * threads.
 * ---------------------------------------------------------------------- */
int namoh_profile_enable(int capacity);
int namoh_profile_read(const char* section, double* total_ms, int* count);

/* Static description of a status code. */
const char* namoh_status_string(int status);
/* Thread-local detail of the last non-OK return on this thread ("" if none). */
const char* namoh_last_error(void);
/* Library version string. */
const char* namoh_version(void);

#ifdef __cplusplus
}
#endif
#endif /* NAMOH_H_ */
