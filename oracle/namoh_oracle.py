"""Plain float64 CPU oracle of NAMOH routed mixture-of-head attention.

TEST INFRASTRUCTURE ONLY (see the package docstring): slow, obviously
correct, shares no code with the GPU library.

Paper passages followed (NAMOH, "Native Sparse Attention from
Mixture-of-Head"):

* Sec. 3.1, Eq. (namoh-gates): TopK head selection, mask m, gates g.
* Sec. 3.1, the paragraph on sparse projection: ordered index sets I_i and
  lengths n_i; routing before projection.
* Sec. 3.1, Eq. (namoh-attention): causal scaled dot-product attention of a
  routed query over keys/values of earlier-or-equal tokens routed to the same
  head; output o_t = sum over selected heads of g_{t,i} h_{t,i} W_O^(i).
* Sec. 3.2, Eq. (namoh-head-rope): head-relative rank rho_i(t) = (number of
  tokens s <= t routed to head i) - 1, RoPE at that rank; global RoPE
  replaces rho_i(t) by t.
* Sec. 3.2, "Efficient execution": each (batch, head) subsequence is an
  independent packed sequence; decoding touches only the selected heads.
* App. B.5 (NAMOH complexity), Eqs. (app-assignment-count),
  (app-routed-kv), (app-routed-interactions): sum_i n_i = TK, M_KV = TK,
  A_KV = sum over the next token's heads of n_i, C_attn = 1/2 sum n_i(n_i+1).

Readings where the paper is silent (each also listed in the design notes):

* R1 selection ranks the raw float32 router logits (softmax is monotone, so
  the set equals TopK of the affinities); equal logits go to the lower head
  index; -0.0 equals +0.0.  ``topk_idx[t, :]`` lists the heads in that order.
* R2 gates: ``GATE_SOFTMAX_SELECTED`` (softmax over the K selected logits,
  the workloads' wording) or ``GATE_SOFTMAX_ALL`` (g = softmax over all H
  logits, not renormalised: Eq. namoh-gates as printed).
* R3 W_O^(i) is the identity, so o_t lives in the head width d.
* R4 RoPE uses the rotate-half pairing (element j with j + d/2),
  theta_j = base^(-2j/d), x'_j = x_j cos - x_{j+d/2} sin,
  x'_{j+d/2} = x_{j+d/2} cos + x_j sin.  V is not rotated.
* R5 softmax scale 1/sqrt(d) unless given.
* R6 decode caches hold keys after rotation, in rank order; the new token
  takes rank n (its head's current length) and attends to itself.
* R7 sequences of a batch are independent (ranks restart per sequence).
* R16 routed projections (Eq. namoh-qkv and the output aggregation of Eq.
  namoh-attention with W_O^(i) kept): per-head weights are stored as linear
  maps out x in, W_QKV [H, 3, d, d_model] (rows 0 / 1 / 2: query, key,
  value; q_{t,i} = x_t W_QKV[i, 0]^T, the paper's x_t W_Q^(i)) and
  W_O [H, d_model, d] (h_{t,i} W_O^(i) = h_{t,i} W_O[i]^T).  Only routed
  (token, head) pairs are projected.
* R17 KV-group routing (App. "GQA+NAMOH", adopted KV-group routing): the
  H query heads form H/g groups of g consecutive heads (group j holds heads
  j*g .. j*g + g - 1) sharing one key/value head; the router selects K/g of
  the H/g groups (same selection rule), all g query heads of a selected
  group attend over the group's subsequence with the group's gate, and RoPE
  uses the group-local rank for the queries and the shared key.
* R18 always-active shared heads (Sec. 4.4, shared heads for local context):
  H_s heads outside the routing attend, for every token, to the full causal
  prefix or to the most recent w original tokens including the token itself
  (t - w < s <= t), with RoPE at the global position; their outputs are
  added to the routed output without a gate (W_O = I, R3).
* R12 loss-free balancing selects by float32(a + b) with the affinities a
  formed in float64; equal scores go to the lower head index; the gates are
  a (the paper fixes no precision for the selection; one rounding step both
  sides take keeps the decision reproducible).
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "GATE_SOFTMAX_SELECTED", "GATE_SOFTMAX_ALL",
    "ROPE_HEAD_RELATIVE", "ROPE_GLOBAL", "ROPE_NONE",
    "select_heads", "route_gates", "select_heads_biased", "bias_update",
    "membership", "head_ranks", "permutation",
    "rope_rotate", "visibility_mask", "attention_definition",
    "attention_gathered", "combine_packed", "combine_dense", "prefill",
    "prefill_rows", "prefill_cache", "decode_step", "brute_force_layer", "interaction_count",
    "attention_backward", "gates_backward",
    "qkv_projection", "output_projection",
    "attention_kv_groups", "combine_kv_groups", "decode_step_kv_groups",
    "always_active_heads",
    "shared_head_counts",
]

GATE_SOFTMAX_SELECTED = 0
GATE_SOFTMAX_ALL = 1
ROPE_HEAD_RELATIVE = 0
ROPE_GLOBAL = 1
ROPE_NONE = 2


# ----------------------------------------------------------------------------
# Routing: Sec. 3.1 Eq. (namoh-gates)

def select_heads(logits: np.ndarray, K: int) -> np.ndarray:
    """S_K(t): the K highest-scoring heads of every token.

    ``logits`` [..., H] (float32 values, compared exactly in float64).  Heads
    are ordered by logit descending, then head index ascending (reading R1);
    the first K are returned as int32 [..., K] in that order.
    """
    l = np.asarray(logits, dtype=np.float64)
    if np.isnan(l).any():
        raise ValueError("router logits must not be NaN")
    H = l.shape[-1]
    if not 1 <= K <= H:
        raise ValueError("need 1 <= K <= H")
    # np.lexsort: last key is primary.  Primary: -logit ascending; secondary:
    # head index ascending.  Float comparison makes -0.0 == +0.0.
    idx = np.broadcast_to(np.arange(H), l.shape)
    order = np.lexsort((idx, -l), axis=-1)
    return order[..., :K].astype(np.int32)


def route_gates(logits: np.ndarray, topk_idx: np.ndarray, mode: int) -> np.ndarray:
    """Gates g_{t,i} of the selected heads, float64 [..., K] (reading R2)."""
    l = np.asarray(logits, dtype=np.float64)
    if mode == GATE_SOFTMAX_SELECTED:
        sel = np.take_along_axis(l, topk_idx.astype(np.int64), axis=-1)
        e = np.exp(sel - sel.max(axis=-1, keepdims=True))
        return e / e.sum(axis=-1, keepdims=True)
    if mode == GATE_SOFTMAX_ALL:
        e = np.exp(l - l.max(axis=-1, keepdims=True))
        a = e / e.sum(axis=-1, keepdims=True)          # affinities a_t
        return np.take_along_axis(a, topk_idx.astype(np.int64), axis=-1)  # g = m * a
    raise ValueError("unknown gate mode")


# ----------------------------------------------------------------------------
# Loss-free balancing: App. "Auxiliary-Loss-Free Balancing",
# Eqs. (namoh-biased-routing), (namoh-loss-free); reading R12

def select_heads_biased(logits: np.ndarray, bias: np.ndarray, K: int):
    """S_K(t) = TopK_i(a_{t,i} + b_i) with a_t = softmax over the H logits;
    gates g = a of the selected heads, not renormalised.

    The score is decided in one fixed precision on every side (reading R12):
    a in float64 (exp of l - max, divided by the sum), then a + b rounded
    once to float32; heads ordered by score descending, then head index
    ascending.  Returns topk int32 [..., K] and gates float64 [..., K]."""
    l = np.asarray(logits, dtype=np.float64)
    if np.isnan(l).any():
        raise ValueError("router logits must not be NaN")
    H = l.shape[-1]
    if not 1 <= K <= H:
        raise ValueError("need 1 <= K <= H")
    b = np.asarray(bias, dtype=np.float32).astype(np.float64)
    e = np.exp(l - l.max(axis=-1, keepdims=True))
    a = e / e.sum(axis=-1, keepdims=True)
    score = (a + b).astype(np.float32).astype(np.float64)
    idx = np.broadcast_to(np.arange(H), l.shape)
    topk = np.lexsort((idx, -score), axis=-1)[..., :K].astype(np.int32)
    return topk, np.take_along_axis(a, topk.astype(np.int64), axis=-1)


def bias_update(head_len: np.ndarray, bias: np.ndarray, eta: float, T: int, K: int):
    """b_i <- b_i + eta sign(c_bar - c_i), c_i = sum over the batch of n_{b,i},
    c_bar = N K / H with N = B T tokens (sign(0) = 0), as float32 [H]."""
    n = np.asarray(head_len, dtype=np.int64)
    B, H = n.shape
    c = n.sum(axis=0)
    sgn = np.sign(B * T * K - H * c)            # sign(c_bar - c_i), exact in integers
    step = np.float32(eta) * sgn.astype(np.float32)
    return (np.asarray(bias, dtype=np.float32) + step).astype(np.float32)


def membership(topk_idx: np.ndarray, H: int) -> np.ndarray:
    """m_{t,i} = 1{i in S_K(t)}: bool [B, T, H]."""
    B, T, K = topk_idx.shape
    m = np.zeros((B, T, H), dtype=bool)
    for k in range(K):
        np.put_along_axis(m, topk_idx[..., k:k + 1].astype(np.int64), True, axis=-1)
    return m


def head_ranks(m: np.ndarray) -> np.ndarray:
    """rho_i(t) = sum_{s<=t} m_{s,i} - 1 (Eq. namoh-head-rope), int64 [B,T,H].

    Meaningful only where m is set."""
    return np.cumsum(m.astype(np.int64), axis=1) - 1


def permutation(topk_idx: np.ndarray, H: int):
    """Packed varlen layout of the ordered index sets I_i (Sec. 3.1, 3.2).

    Returns ``head_len`` int32 [B,H] (n_i per sequence), ``seg_offsets``
    int32 [B*H+1] (segment b*H+h starts there; exclusive running sum of the
    lengths in segment order), ``perm_token`` int32 [B*T*K] (packed position
    -> token t, tokens ascending inside a segment) and ``slot_pos`` int32
    [B,T,K] (packed position of the pair (t, topk_idx[b,t,k])).
    """
    B, T, K = topk_idx.shape
    m = membership(topk_idx, H)
    n = m.sum(axis=1)                                     # [B, H]
    flat = n.reshape(-1)
    seg_offsets = np.concatenate([[0], np.cumsum(flat)]).astype(np.int64)
    perm = np.empty(int(seg_offsets[-1]), dtype=np.int64)
    for b in range(B):
        for h in range(H):
            s = b * H + h
            perm[seg_offsets[s]:seg_offsets[s + 1]] = np.nonzero(m[b, :, h])[0]
    rho = head_ranks(m)
    slot = np.empty((B, T, K), dtype=np.int64)
    for b in range(B):
        for k in range(K):
            hk = topk_idx[b, :, k].astype(np.int64)
            slot[b, :, k] = seg_offsets[b * H + hk] + rho[b, np.arange(T), hk]
    return (n.astype(np.int32), seg_offsets.astype(np.int32),
            perm.astype(np.int32), slot.astype(np.int32))


# ----------------------------------------------------------------------------
# Positional encoding: Sec. 3.2 Eq. (namoh-head-rope), reading R4

def rope_rotate(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """x R(p) for rows x [..., n, d] at positions p [..., n] (float64)."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    j = np.arange(half, dtype=np.float64)
    theta = np.power(float(base), -2.0 * j / d)
    ang = np.asarray(positions, dtype=np.float64)[..., None] * theta
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def _positions(rank: np.ndarray, t: np.ndarray, rope_mode: int):
    if rope_mode == ROPE_HEAD_RELATIVE:
        return rank
    if rope_mode == ROPE_GLOBAL:
        return t
    return None


def _rotate(x, pos, base):
    return x if pos is None else rope_rotate(x, pos, base)


# ----------------------------------------------------------------------------
# Attention, definition form (O1): explicit visibility mask

def visibility_mask(m_bh: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """Vis_i[t, s] = m_{t,i} and m_{s,i} and s <= t over global indices
    (Eq. namoh-attention), for the query tokens ``rows``: bool [len(rows), T]."""
    T = m_bh.shape[0]
    s = np.arange(T)
    return m_bh[rows][:, None] & m_bh[None, :] & (s[None, :] <= rows[:, None])


def attention_definition(q, k, v, topk_idx, H, rope_base, rope_mode=ROPE_HEAD_RELATIVE,
                         scale=None, block=512):
    """h_{t,i} for every routed pair from the definition, float64 [B,H,T,d]
    (zero where m_{t,i} = 0).  q, k, v: float64 [B,H,T,d]."""
    B, _, T, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    m = membership(topk_idx, H)
    rho = head_ranks(m)
    out = np.zeros((B, H, T, d))
    t_all = np.arange(T)
    for b in range(B):
        for h in range(H):
            mb = m[b, :, h]
            tok = np.nonzero(mb)[0]
            if tok.size == 0:
                continue
            pos = _positions(rho[b, :, h], t_all, rope_mode)
            # rotate every token's key at its own rank; non-routed keys are
            # never visible, so their (meaningless) rotation is never used.
            kt = _rotate(k[b, h], pos, rope_base)
            qt = _rotate(q[b, h], pos, rope_base)
            for i0 in range(0, tok.size, block):
                rows = tok[i0:i0 + block]
                vis = visibility_mask(mb, rows)
                sc = (qt[rows] @ kt.T) * scale
                sc = np.where(vis, sc, -np.inf)
                sc = sc - sc.max(axis=1, keepdims=True)
                p = np.where(vis, np.exp(sc), 0.0)
                p /= p.sum(axis=1, keepdims=True)
                out[b, h, rows] = p @ v[b, h]
    return out


def combine_dense(h_dense, topk_idx, gates):
    """o_t = sum_{i in S_K(t)} g_{t,i} h_{t,i} (Eq. namoh-attention, R3)."""
    B, H, T, d = h_dense.shape
    o = np.zeros((B, T, d))
    for kk in range(topk_idx.shape[-1]):
        hk = topk_idx[:, :, kk].astype(np.int64)
        sel = h_dense[np.arange(B)[:, None], hk, np.arange(T)[None, :]]
        o += gates[:, :, kk, None] * sel
    return o


# ----------------------------------------------------------------------------
# Routed projections: Sec. 3.1, Eq. (namoh-qkv) and the output aggregation of
# Eq. (namoh-attention), R16

def qkv_projection(x, w_qkv, topk_idx):
    """Queries, keys and values of the routed (token, head) pairs only.

    x [B, T, d_model]; w_qkv [H, 3, d, d_model] (linear maps out x in).
    Returns q, k, v [B, H, T, d] and the membership mask m [B, T, H]; rows of
    pairs with m = 0 are NaN (such pairs produce no vectors, Eq. namoh-qkv)."""
    B, T, dm = x.shape
    H, three, d, dm2 = w_qkv.shape
    assert three == 3 and dm2 == dm
    m = membership(topk_idx, H)
    out = [np.full((B, H, T, d), np.nan) for _ in range(3)]
    for b in range(B):
        for i in range(H):
            rows = np.nonzero(m[b, :, i])[0]          # the ordered index set I_i
            if rows.size == 0:
                continue
            xi = x[b, rows]                             # dispatch before projection
            for j in range(3):
                out[j][b, i, rows] = xi @ w_qkv[i, j].T
    return out[0], out[1], out[2], m


def output_projection(h_dense, topk_idx, gates, w_o):
    """o_t = sum over the selected heads i of g_{t,i} h_{t,i} W_O^(i).

    h_dense [B, H, T, d] (rows of unselected pairs are never read);
    w_o [H, d_model, d].  Returns o [B, T, d_model]."""
    B, H, T, d = h_dense.shape
    dm = w_o.shape[1]
    o = np.zeros((B, T, dm))
    for b in range(B):
        for t in range(T):
            for kk in range(topk_idx.shape[-1]):
                i = int(topk_idx[b, t, kk])
                o[b, t] += gates[b, t, kk] * (w_o[i] @ h_dense[b, i, t])
    return o


# ----------------------------------------------------------------------------
# KV-group routing (App. GQA+NAMOH, adopted KV-group routing), R17

def attention_kv_groups(q, k, v, topk_groups, g, rope_base, rope_mode=ROPE_HEAD_RELATIVE,
                        scale=None, form="gathered"):
    """Ungated head outputs [B, H, T, d] (NaN where the token's group is not
    selected) for query heads q [B, H, T, d] and group keys/values
    k, v [B, H/g, T, d]; topk_groups [B, T, K/g] are the selected groups.

    form 'definition': the explicit visibility mask of each group over
    global indices, Vis_j[t, s] = m_{t,j} m_{s,j} [s <= t], applied to every
    query head of the group; 'gathered': each group's routed rows as one
    causal sequence."""
    B, H, T, d = q.shape
    G = H // g
    assert k.shape[1] == G and v.shape[1] == G
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    m = membership(topk_groups, G)                  # [B, T, G]
    rank = head_ranks(m)                            # group-local ranks
    out = np.full((B, H, T, d), np.nan)
    tpos = np.arange(T)
    for b in range(B):
        for j in range(G):
            rows = np.nonzero(m[b, :, j])[0]
            if rows.size == 0:
                continue
            if form == "definition":
                pos = _positions(rank[b, :, j], tpos, rope_mode)
                kt = _rotate(k[b, j], pos, rope_base)
                vis = visibility_mask(m[b, :, j], rows)        # [n, T]
                for u in range(g):
                    h = j * g + u
                    qt = _rotate(q[b, h, rows], None if pos is None else pos[rows], rope_base)
                    sc = np.where(vis, (qt @ kt.T) * scale, -np.inf)
                    sc = sc - sc.max(axis=1, keepdims=True)
                    p = np.where(vis, np.exp(sc), 0.0)
                    p /= p.sum(axis=1, keepdims=True)
                    out[b, h, rows] = p @ v[b, j]
            else:
                n = rows.size
                pos = _positions(np.arange(n), rows, rope_mode)
                kt = _rotate(k[b, j, rows], pos, rope_base)
                vv = v[b, j, rows]
                causal = np.arange(n)[None, :] <= np.arange(n)[:, None]
                for u in range(g):
                    h = j * g + u
                    qt = _rotate(q[b, h, rows], pos, rope_base)
                    sc = np.where(causal, (qt @ kt.T) * scale, -np.inf)
                    sc = sc - sc.max(axis=1, keepdims=True)
                    p = np.exp(sc)
                    p /= p.sum(axis=1, keepdims=True)
                    out[b, h, rows] = p @ vv
    return out


def combine_kv_groups(h_dense, topk_groups, gates, g):
    """o_t = sum over the selected groups j of g_{t,j} sum_u h_{t, j*g + u}
    (the group's query heads share its gate; W_O = I, R3)."""
    B, H, T, d = h_dense.shape
    o = np.zeros((B, T, d))
    for kk in range(topk_groups.shape[-1]):
        j = topk_groups[:, :, kk].astype(np.int64)
        for u in range(g):
            sel = h_dense[np.arange(B)[:, None], j * g + u, np.arange(T)[None, :]]
            o += gates[:, :, kk, None] * sel
    return o


# ----------------------------------------------------------------------------
# Always-active shared heads (Sec. 4.4, shared heads for local context), R18

def always_active_heads(q, k, v, window, rope_base, rope_mode=ROPE_GLOBAL, scale=None):
    """Outputs [B, Hs, T, d] of always-active heads: token t attends to
    tokens s with s <= t (window 0) or t - window < s <= t, through the
    explicit visibility mask; RoPE at the global position t (or none)."""
    B, Hs, T, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    t = np.arange(T)
    vis = t[None, :] <= t[:, None]
    if window > 0:
        vis &= t[None, :] > t[:, None] - window
    pos = None if rope_mode == ROPE_NONE else t
    out = np.empty((B, Hs, T, d))
    for b in range(B):
        for h in range(Hs):
            qt = _rotate(q[b, h], pos, rope_base)
            kt = _rotate(k[b, h], pos, rope_base)
            sc = np.where(vis, (qt @ kt.T) * scale, -np.inf)
            sc = sc - sc.max(axis=1, keepdims=True)
            p = np.where(vis, np.exp(sc), 0.0)
            p /= p.sum(axis=1, keepdims=True)
            out[b, h] = p @ v[b, h]
    return out


# ----------------------------------------------------------------------------
# Attention, gathered form (O2): per packed segment

def attention_gathered(q, k, v, head_len, seg_offsets, perm_token, H, rope_base,
                       rope_mode=ROPE_HEAD_RELATIVE, scale=None, block=1024,
                       segments=None):
    """Packed ungated head outputs float64 [B*T*K, d].

    Each (batch, head) segment is an independent causal sequence of its
    routed tokens in order (Sec. 3.2, efficient execution).  ``segments``
    limits the work to a subset of segment ids (rows of other segments stay
    zero)."""
    B, _, T, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    N = int(seg_offsets[-1])
    out = np.zeros((N, d))
    segs = range(B * H) if segments is None else segments
    for sid in segs:
        b, h = divmod(int(sid), H)
        a, e = int(seg_offsets[sid]), int(seg_offsets[sid + 1])
        n = e - a
        if n == 0:
            continue
        tok = perm_token[a:e].astype(np.int64)
        pos = _positions(np.arange(n), tok, rope_mode)
        qt = _rotate(q[b, h, tok], pos, rope_base)
        kt = _rotate(k[b, h, tok], pos, rope_base)
        vv = v[b, h, tok]
        for r0 in range(0, n, block):
            r1 = min(n, r0 + block)
            sc = (qt[r0:r1] @ kt[:r1].T) * scale
            causal = np.arange(r1)[None, :] <= np.arange(r0, r1)[:, None]
            sc = np.where(causal, sc, -np.inf)
            sc -= sc.max(axis=1, keepdims=True)
            p = np.exp(sc)
            p /= p.sum(axis=1, keepdims=True)
            out[a + r0:a + r1] = p @ vv[:r1]
    return out


def combine_packed(h_packed, slot_pos, gates):
    """o_t = sum_k g_{t,k} h[slot_pos[t,k]] in k order."""
    B, T, K = slot_pos.shape
    o = np.zeros((B, T, h_packed.shape[-1]))
    for kk in range(K):
        o += gates[:, :, kk, None] * h_packed[slot_pos[:, :, kk].astype(np.int64)]
    return o


def prefill(logits, q, k, v, K, rope_base, rope_mode=ROPE_HEAD_RELATIVE,
            gate_mode=GATE_SOFTMAX_SELECTED, scale=None, form="gathered", bias=None):
    """Whole layer: routing, permutation, attention, combine.

    q, k, v float64 [B,H,T,d].  ``form`` = 'gathered' (O2) or 'definition'
    (O1).  With ``bias`` [H] the routing is select_heads_biased (gate_mode
    ignored).  Returns a dict of every intermediate the GPU library exposes."""
    H = logits.shape[-1]
    if bias is None:
        topk = select_heads(logits, K)
        g = route_gates(logits, topk, gate_mode)
    else:
        topk, g = select_heads_biased(logits, bias, K)
    head_len, seg_offsets, perm, slot = permutation(topk, H)
    if form == "definition":
        hd = attention_definition(q, k, v, topk, H, rope_base, rope_mode, scale)
        o = combine_dense(hd, topk, g)
        # pack the dense per-head outputs at the permutation's positions
        B, _, T, d = q.shape
        hp = np.zeros((int(seg_offsets[-1]), d))
        for b in range(B):
            for kk in range(K):
                hp[slot[b, :, kk]] = hd[b, topk[b, :, kk], np.arange(T)]
    else:
        hp = attention_gathered(q, k, v, head_len, seg_offsets, perm, H, rope_base,
                                rope_mode, scale)
        o = combine_packed(hp, slot, g)
    return {"topk_idx": topk, "gates": g, "head_len": head_len,
            "seg_offsets": seg_offsets, "perm_token": perm, "slot_pos": slot,
            "head_out": hp, "out": o}


def prefill_rows(q, k, v, topk_idx, gates, H, rope_base, b, tokens,
                 rope_mode=ROPE_HEAD_RELATIVE, scale=None):
    """Layer output o_t for a few tokens of sequence b, each computed on its
    own from the definition (used to sample outputs at full size).

    q, k, v are indexable [B,H,T,d] arrays in any float dtype (converted
    row by row); returns float64 [len(tokens), d] and the per-head outputs
    float64 [len(tokens), K, d]."""
    topk_b = topk_idx[b]
    T, K = topk_b.shape
    d = q.shape[-1]
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    m = membership(topk_idx[b:b + 1], H)[0]
    o = np.zeros((len(tokens), d))
    hs = np.zeros((len(tokens), K, d))
    for r, t in enumerate(tokens):
        for kk in range(K):
            h = int(topk_b[t, kk])
            src = np.nonzero(m[:t + 1, h])[0]       # s in I_h, s <= t
            ranks = np.arange(src.size)             # rho_h(s)
            pos = _positions(ranks, src, rope_mode)
            kt = _rotate(np.asarray(k[b, h][src], dtype=np.float64), pos, rope_base)
            qpos = None if pos is None else pos[-1:]
            qt = _rotate(np.asarray(q[b, h][t:t + 1], dtype=np.float64), qpos, rope_base)
            sc = (kt @ qt[0]) * scale
            p = np.exp(sc - sc.max())
            p /= p.sum()
            hs[r, kk] = p @ np.asarray(v[b, h][src], dtype=np.float64)
            o[r] += gates[b, t, kk] * hs[r, kk]
    return o, hs


# ----------------------------------------------------------------------------
# Backward of the layer (training path): the exact gradient of Eqs.
# (namoh-gates), (namoh-head-rope), (namoh-attention) with the selection S_K
# held fixed (it is piecewise constant), for the packed varlen attention of
# Sec. 3.2 "Efficient execution" that training also uses.

def _unrotate(dx, pos, base):
    """Gradient through x -> x R(p): dx R(p)^T, i.e. the rotation by -p."""
    return dx if pos is None else rope_rotate(dx, -np.asarray(pos, dtype=np.float64), base)


def attention_backward(q, k, v, gates, seg_offsets, perm_token, slot_pos, H, rope_base,
                       dout, rope_mode=ROPE_HEAD_RELATIVE, scale=None):
    """Gradients of o = combine(attention(q, k, v), gates) for the upstream
    gradient dout [B,T,d].

    Per segment, with the rotated rows Q~, K~ and S = Q~ K~^T scale (causal),
    P = softmax(S), O = P V, dO_r = g_r dout_t (g_r the gate of packed row r):
    dV = P^T dO, dP = dO V^T, dS = P (dP - rowsum(dO O)), dQ~ = dS K~ scale,
    dK~ = dS^T Q~ scale, then dq = dQ~ R^T (rotation by minus the angle)
    scattered to the token rows; dgates[t,k] = <h(t, topk_k), dout_t>.
    Returns dq, dk, dv float64 [B,H,T,d] (zero where the token is not routed
    to the head) and dgates float64 [B,T,K]."""
    B, _, T, d = q.shape
    K = slot_pos.shape[-1]
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    N = int(seg_offsets[-1])
    dout = np.asarray(dout, dtype=np.float64)
    # packed gate and upstream row of every packed position
    g_pack = np.zeros(N)
    t_pack = np.zeros(N, dtype=np.int64)
    b_pack = np.zeros(N, dtype=np.int64)
    for b in range(B):
        for kk in range(K):
            sl = slot_pos[b, :, kk].astype(np.int64)
            g_pack[sl] = gates[b, :, kk]
            t_pack[sl] = np.arange(T)
            b_pack[sl] = b
    do_pack = g_pack[:, None] * dout[b_pack, t_pack]
    dq = np.zeros((B, H, T, d))
    dk = np.zeros((B, H, T, d))
    dv = np.zeros((B, H, T, d))
    h_pack = np.zeros((N, d))
    for sid in range(B * H):
        b, h = divmod(sid, H)
        a, e = int(seg_offsets[sid]), int(seg_offsets[sid + 1])
        n = e - a
        if n == 0:
            continue
        tok = perm_token[a:e].astype(np.int64)
        pos = _positions(np.arange(n), tok, rope_mode)
        qt = _rotate(q[b, h, tok], pos, rope_base)
        kt = _rotate(k[b, h, tok], pos, rope_base)
        vv = np.asarray(v[b, h, tok], dtype=np.float64)
        sc = (qt @ kt.T) * scale
        causal = np.tril(np.ones((n, n), dtype=bool))
        sc = np.where(causal, sc, -np.inf)
        p = np.exp(sc - sc.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        o = p @ vv
        h_pack[a:e] = o
        dO = do_pack[a:e]
        dv_s = p.T @ dO
        dp = dO @ vv.T
        ds = p * (dp - (dO * o).sum(axis=1, keepdims=True))
        dqt = ds @ kt * scale
        dkt = ds.T @ qt * scale
        dq[b, h, tok] = _unrotate(dqt, pos, rope_base)
        dk[b, h, tok] = _unrotate(dkt, pos, rope_base)
        dv[b, h, tok] = dv_s
    dgates = np.zeros((B, T, K))
    for kk in range(K):
        dgates[:, :, kk] = (h_pack[slot_pos[:, :, kk].astype(np.int64)] * dout).sum(axis=-1)
    return dq, dk, dv, dgates


def gates_backward(logits, topk_idx, dgates, mode):
    """Gradient of the gates (reading R2, or loss-free balancing's affinity
    gates, which are GATE_SOFTMAX_ALL's) with respect to the router logits,
    the selection held fixed: SOFTMAX_SELECTED g = softmax of the selected
    logits, dl_j = g_j (dg_j - sum_k g_k dg_k) on the selected heads, 0
    elsewhere; SOFTMAX_ALL g_k = a(topk_k), a = softmax of all H logits,
    dl = a (da - <a, da>) with da the gate gradients placed at their heads.
    Returns float64 [..., H]."""
    l = np.asarray(logits, dtype=np.float64)
    idx = topk_idx.astype(np.int64)
    dg = np.asarray(dgates, dtype=np.float64)
    dl = np.zeros_like(l)
    if mode == GATE_SOFTMAX_SELECTED:
        g = route_gates(l, topk_idx, mode)
        val = g * (dg - (g * dg).sum(axis=-1, keepdims=True))
        np.put_along_axis(dl, idx, val, axis=-1)
        return dl
    if mode == GATE_SOFTMAX_ALL:
        e = np.exp(l - l.max(axis=-1, keepdims=True))
        a = e / e.sum(axis=-1, keepdims=True)
        da = np.zeros_like(l)
        np.put_along_axis(da, idx, dg, axis=-1)
        return a * (da - (a * da).sum(axis=-1, keepdims=True))
    raise ValueError("unknown gate mode")


# ----------------------------------------------------------------------------
# Prefill -> decode hand-off: Sec. 3.2 (decoding reads and extends only the
# active heads' caches), reading R6 (caches hold rotated keys in rank order)

def prefill_cache(k, v, topk_idx, H, rope_base, rope_mode=ROPE_HEAD_RELATIVE):
    """Decode caches after a prompt: for each (b, h), the keys of the tokens
    routed to h rotated at their rank (or global position), and their
    values, in rank order.

    k, v [B,H,T,d] (any float dtype); returns k_cache, v_cache float64
    [B,H,T,d] (rows [n_{b,h}, T) zero) and cache_len int [B,H]."""
    B, _, T, d = k.shape
    m = membership(topk_idx, H)
    kc = np.zeros((B, H, T, d))
    vc = np.zeros((B, H, T, d))
    n = np.zeros((B, H), dtype=np.int64)
    for b in range(B):
        for h in range(H):
            src = np.nonzero(m[b, :, h])[0]         # I_h in token order = rank order
            n[b, h] = src.size
            if src.size == 0:
                continue
            pos = _positions(np.arange(src.size), src, rope_mode)
            kc[b, h, :src.size] = _rotate(np.asarray(k[b, h][src], dtype=np.float64), pos,
                                          rope_base)
            vc[b, h, :src.size] = np.asarray(v[b, h][src], dtype=np.float64)
    return kc, vc, n


# ----------------------------------------------------------------------------
# Decode: Sec. 3.1 (prefill and incremental decoding compute the same thing),
# Sec. 3.2 (decoding reads/updates only the selected caches), reading R6

def decode_step(logits, q, k, v, cache_k, cache_v, cache_len, K, rope_base,
                rope_mode=ROPE_HEAD_RELATIVE, gate_mode=GATE_SOFTMAX_SELECTED,
                seq_pos=None, scale=None, bias=None):
    """One decoding step for B sequences.

    logits [B,H]; q,k,v float64 [B,H,d]; ``cache_k(b, h, n)`` and
    ``cache_v(b, h, n)`` return rows [0, n) of the post-RoPE key / value
    cache of head h (float64 [n, d]); cache_len int [B,H].

    Returns topk_idx [B,K], gates [B,K], out [B,d], the ungated head outputs
    [B,K,d], the appended rotated keys [B,K,d] and the updated lengths.  Only
    the selected heads' caches are read.  With ``bias`` [H] the heads are
    selected and gated as in select_heads_biased (gate_mode ignored)."""
    B, H, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if bias is None:
        topk = select_heads(logits, K)
        g = route_gates(logits, topk, gate_mode)
    else:
        topk, g = select_heads_biased(logits, bias, K)
    out = np.zeros((B, d))
    heads = np.zeros((B, K, d))
    new_k = np.zeros((B, K, d))
    new_len = np.array(cache_len, dtype=np.int64, copy=True)
    for b in range(B):
        for kk in range(K):
            h = int(topk[b, kk])
            n = int(cache_len[b, h])
            p = n if rope_mode == ROPE_HEAD_RELATIVE else (
                None if rope_mode == ROPE_NONE else int(seq_pos[b]))
            pos = None if p is None else np.array([p])
            qt = _rotate(q[b, h][None], pos, rope_base)[0]
            kt = _rotate(k[b, h][None], pos, rope_base)[0]
            Kc = np.concatenate([np.asarray(cache_k(b, h, n), dtype=np.float64).reshape(n, d), kt[None]])
            Vc = np.concatenate([np.asarray(cache_v(b, h, n), dtype=np.float64).reshape(n, d), v[b, h][None]])
            sc = (Kc @ qt) * scale
            w = np.exp(sc - sc.max())
            w /= w.sum()
            heads[b, kk] = w @ Vc
            out[b] += g[b, kk] * heads[b, kk]
            new_k[b, kk] = kt
            new_len[b, h] = n + 1
    return {"topk_idx": topk, "gates": g, "out": out, "head_out": heads,
            "new_k": new_k, "cache_len": new_len}


def decode_step_kv_groups(logits, q, k, v, cache_k, cache_v, cache_len, K_kv, g, rope_base,
                          rope_mode=ROPE_HEAD_RELATIVE, gate_mode=GATE_SOFTMAX_SELECTED,
                          seq_pos=None, scale=None):
    """One decoding step with key/value-group routing (R17).

    logits [B, H_kv] (group logits); q float64 [B, H_kv*g, d]; k, v float64
    [B, H_kv, d]; ``cache_k(b, j, n)`` / ``cache_v(b, j, n)`` return rows
    [0, n) of group j's rotated keys / values; cache_len [B, H_kv].  The new
    token takes rank n_j in each selected group j, appends one key/value row
    there, and each of the group's g query heads attends over the group's
    n_j + 1 rows.  Returns topk_idx [B, K_kv], gates, out [B, d] (the gated
    sum over selected groups of the sum of their g head outputs), head_out
    [B, K_kv, g, d] and the updated lengths."""
    B, Hq, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    topk = select_heads(logits, K_kv)
    gt = route_gates(logits, topk, gate_mode)
    out = np.zeros((B, d))
    heads = np.zeros((B, K_kv, g, d))
    new_len = np.array(cache_len, dtype=np.int64, copy=True)
    for b in range(B):
        for kk in range(K_kv):
            j = int(topk[b, kk])
            n = int(cache_len[b, j])
            p = n if rope_mode == ROPE_HEAD_RELATIVE else (
                None if rope_mode == ROPE_NONE else int(seq_pos[b]))
            pos = None if p is None else np.array([p])
            kt = _rotate(k[b, j][None], pos, rope_base)[0]
            Kc = np.concatenate([np.asarray(cache_k(b, j, n), dtype=np.float64).reshape(n, d), kt[None]])
            Vc = np.concatenate([np.asarray(cache_v(b, j, n), dtype=np.float64).reshape(n, d), v[b, j][None]])
            for u in range(g):
                qt = _rotate(q[b, j * g + u][None], pos, rope_base)[0]
                sc = (Kc @ qt) * scale
                w = np.exp(sc - sc.max())
                w /= w.sum()
                heads[b, kk, u] = w @ Vc
                out[b] += gt[b, kk] * heads[b, kk, u]
            new_len[b, j] = n + 1
    return {"topk_idx": topk, "gates": gt, "out": out, "head_out": heads, "cache_len": new_len}


# ----------------------------------------------------------------------------
# O0: brute force with scalar loops (tiny inputs only)

def brute_force_layer(logits, q, k, v, K, rope_base, rope_mode=ROPE_HEAD_RELATIVE,
                      gate_mode=GATE_SOFTMAX_SELECTED, scale=None):
    """Scalar-loop evaluation of Eqs. (namoh-gates), (namoh-head-rope),
    (namoh-attention) for one sequence: logits [T,H], q/k/v [H,T,d] (nested
    lists or arrays).  Returns (selected heads per token, gates, o [T][d])."""
    T, H = len(logits), len(logits[0])
    d = len(q[0][0])
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    sel, gat = [], []
    for t in range(T):
        row = [float(x) for x in logits[t]]
        heads = sorted(range(H), key=lambda i: (-row[i], i))[:K]
        if gate_mode == GATE_SOFTMAX_SELECTED:
            mx = max(row[i] for i in heads)
            ex = [math.exp(row[i] - mx) for i in heads]
            gat.append([e / sum(ex) for e in ex])
        else:
            mx = max(row)
            z = sum(math.exp(x - mx) for x in row)
            gat.append([math.exp(row[i] - mx) / z for i in heads])
        sel.append(heads)

    def rot(vec, p):
        if rope_mode == ROPE_NONE:
            return list(vec)
        half = d // 2
        outv = [0.0] * d
        for j in range(half):
            ang = p * float(rope_base) ** (-2.0 * j / d)
            c, s = math.cos(ang), math.sin(ang)
            outv[j] = vec[j] * c - vec[j + half] * s
            outv[j + half] = vec[j + half] * c + vec[j] * s
        return outv

    o = [[0.0] * d for _ in range(T)]
    for t in range(T):
        for kk, i in enumerate(sel[t]):
            hist = [s for s in range(t + 1) if i in sel[s]]     # I_i, s <= t
            def pos_of(s):
                rank = sum(1 for u in range(s + 1) if i in sel[u]) - 1
                return rank if rope_mode == ROPE_HEAD_RELATIVE else s
            qt = rot([float(x) for x in q[i][t]], pos_of(t))
            scores = []
            for s in hist:
                ks = rot([float(x) for x in k[i][s]], pos_of(s))
                scores.append(sum(a * b for a, b in zip(qt, ks)) * scale)
            mx = max(scores)
            w = [math.exp(x - mx) for x in scores]
            z = sum(w)
            for j in range(d):
                acc = sum(w[u] / z * float(v[i][s][j]) for u, s in enumerate(hist))
                o[t][j] += gat[t][kk] * acc
    return sel, gat, o


# ----------------------------------------------------------------------------
# Cost accounting: App. B.5

def interaction_count(head_len) -> int:
    """C_attn = 1/2 sum_i n_i (n_i + 1) (Eq. app-routed-interactions)."""
    n = np.asarray(head_len, dtype=np.int64)
    return int((n * (n + 1)).sum() // 2)


def shared_head_counts(m_b: np.ndarray) -> np.ndarray:
    """R = tril(M M^T) for one sequence's mask M [T,H] (Sec. 4.3): the number
    of active heads shared by token t and an earlier-or-equal token s."""
    M = m_b.astype(np.int64)
    return np.tril(M @ M.T)
