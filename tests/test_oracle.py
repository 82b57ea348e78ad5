"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: values the
paper prints for its worked example, closed forms of App. B.5, library
routines (numpy stable sort, scipy softmax, torch scaled-dot-product
attention), an independent complex-number form of RoPE, brute force with
scalar loops, and invariants.  No GPU is touched.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle as O
from paper_2609_38832_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
rng = np.random.default_rng(1234)


def _rand_logits(B, T, H, seed=0):
    return np.random.default_rng(seed).standard_normal((B, T, H)).astype(np.float32)


# ----------------------------------------------------------------------------
# selection (Eq. namoh-gates TopK; ties -> lower head index)

def test_select_matches_scalar_sort():
    l = _rand_logits(2, 50, 7, seed=1)
    got = O.select_heads(l, 3)
    for b in range(2):
        for t in range(50):
            row = [float(x) for x in l[b, t]]
            want = sorted(range(7), key=lambda i: (-row[i], i))[:3]
            assert list(got[b, t]) == want


def test_select_matches_numpy_stable_argsort_with_ties():
    # integer-valued logits: many exact ties
    l = np.random.default_rng(2).integers(-3, 4, size=(3, 200, 16)).astype(np.float32)
    got = O.select_heads(l, 5)
    want = np.argsort(-l.astype(np.float64), axis=-1, kind="stable")[..., :5]
    np.testing.assert_array_equal(got, want)


def test_select_forced_ties_and_specials():
    assert list(O.select_heads(np.zeros((1, 6), np.float32), 3)[0]) == [0, 1, 2]
    # -0.0 equals +0.0: lower index wins
    z = np.array([[0.0, -0.0, 0.0, -0.0]], np.float32)
    assert list(O.select_heads(z, 2)[0]) == [0, 1]
    z2 = np.array([[-0.0, 0.0, -1.0]], np.float32)
    assert list(O.select_heads(z2, 2)[0]) == [0, 1]
    inf = np.array([[-np.inf, np.inf, np.inf, 1.0, -np.inf]], np.float32)
    assert list(O.select_heads(inf, 4)[0]) == [1, 2, 3, 0]
    with pytest.raises(ValueError):
        O.select_heads(np.array([[np.nan, 0.0]], np.float32), 1)


def test_each_token_has_exactly_K_distinct_heads():
    l = _rand_logits(2, 300, 12, seed=3)
    topk = O.select_heads(l, 4)
    m = O.membership(topk, 12)
    assert (m.sum(-1) == 4).all()
    assert all(len(set(r)) == 4 for r in topk.reshape(-1, 4).tolist())


# ----------------------------------------------------------------------------
# gates

def test_gates_softmax_selected_and_all():
    l = _rand_logits(1, 40, 10, seed=4)
    topk = O.select_heads(l, 3)
    g = O.route_gates(l, topk, O.GATE_SOFTMAX_SELECTED)
    sel = np.take_along_axis(l.astype(np.float64), topk.astype(np.int64), -1)
    np.testing.assert_allclose(g, scipy.special.softmax(sel, axis=-1), rtol=1e-13)
    np.testing.assert_allclose(g.sum(-1), 1.0, rtol=1e-13)
    assert (np.diff(g, axis=-1) <= 1e-15).all()         # ordered by logit
    ga = O.route_gates(l, topk, O.GATE_SOFTMAX_ALL)
    a = scipy.special.softmax(l.astype(np.float64), axis=-1)
    np.testing.assert_allclose(ga, np.take_along_axis(a, topk.astype(np.int64), -1), rtol=1e-13)
    assert (ga.sum(-1) < 1.0).all()


def test_gates_K_equals_H_modes_agree():
    l = _rand_logits(1, 20, 6, seed=5)
    topk = O.select_heads(l, 6)
    np.testing.assert_allclose(O.route_gates(l, topk, 0), O.route_gates(l, topk, 1), rtol=1e-13)


# ----------------------------------------------------------------------------
# membership, ranks, permutation: worked example of Fig. 2 and App. B.5

def test_worked_example_fig2():
    fx = json.load(open(os.path.join(HERE, "golden", "worked_example_fig2.json")))
    pr = fx["printed"]
    H, K = pr["H"], pr["K"]
    asg = fx["assignment"]
    T = len(asg)
    logits = np.zeros((1, T, H), np.float32)
    for t, heads in enumerate(asg):
        logits[0, t, heads] = 1.0
    topk = O.select_heads(logits, K)
    m = O.membership(topk, H)
    rho = O.head_ranks(m)
    head0 = np.nonzero(m[0, :8, 0])[0]
    assert list(head0) == pr["head0_global_positions_prefill"]
    assert list(rho[0, head0, 0]) == pr["head0_local_indices"]
    assert sorted(topk[0, 8]) == pr["token8_heads"]
    assert rho[0, 8, 0] == pr["token8_head0_index"]
    assert sorted(topk[0, 9]) == pr["token9_heads"]
    # the permutation places head 0's tokens first, at their local indices
    n, off, perm, slot = O.permutation(topk[:, :8], H)
    assert list(perm[off[0]:off[1]]) == pr["head0_global_positions_prefill"]


def test_permutation_invariants():
    B, T, H, K = 3, 257, 10, 3
    topk = O.select_heads(_rand_logits(B, T, H, seed=6), K)
    n, off, perm, slot = O.permutation(topk, H)
    assert n.sum() == B * T * K                                 # sum n_i = TK
    assert (n.sum(1) == T * K).all()
    assert off[0] == 0 and off[-1] == B * T * K
    np.testing.assert_array_equal(np.diff(off), n.reshape(-1))
    for s in range(B * H):
        seg = perm[off[s]:off[s + 1]]
        assert (np.diff(seg) > 0).all()                         # ascending t
    for b in range(B):
        for t in range(T):
            for kk in range(K):
                p = slot[b, t, kk]
                assert perm[p] == t
                sid = np.searchsorted(off, p, side="right") - 1
                assert sid == b * H + topk[b, t, kk]
    assert len(set(slot.reshape(-1).tolist())) == B * T * K       # bijection


def test_rank_is_running_count():
    topk = O.select_heads(_rand_logits(1, 64, 5, seed=7), 2)
    m = O.membership(topk, 5)
    rho = O.head_ranks(m)
    for h in range(5):
        toks = np.nonzero(m[0, :, h])[0]
        assert list(rho[0, toks, h]) == list(range(len(toks)))


@pytest.mark.parametrize("H", [8, 16, 32, 64])
def test_kv_storage_unchanged_as_H_grows(H):
    T, K = 1000, 8
    topk = O.select_heads(_rand_logits(1, T, H, seed=H), K)
    n, *_ = O.permutation(topk, H)
    assert n.sum() == T * K                                     # M_KV = TK


# ----------------------------------------------------------------------------
# visibility mask and interaction counts (Sec. 4.3, App. B.5)

def _all_vis(m_b):
    T, H = m_b.shape
    return [O.visibility_mask(m_b[:, h], np.arange(T)) for h in range(H)]


def test_mask_sum_equals_tril_MMt_and_interactions():
    T, H, K = 90, 6, 2
    topk = O.select_heads(_rand_logits(1, T, H, seed=8), K)
    m = O.membership(topk, H)[0]
    vis = _all_vis(m)
    R = sum(v.astype(np.int64) for v in vis)
    np.testing.assert_array_equal(R, O.shared_head_counts(m))
    n = m.sum(0)
    pop = sum(int(v.sum()) for v in vis)
    assert pop == O.interaction_count(n)
    # second-moment form, Eq. (app-load-second-moment) / (namoh-attention-work)
    nbar = T * K / H
    cv2 = ((n - nbar) ** 2).mean() / nbar ** 2
    assert math.isclose(pop, T * T * K * K / (2 * H) * (1 + cv2) + T * K / 2, rel_tol=1e-12)


def test_interaction_bounds_attained():
    T, H, K = 48, 8, 2
    # exactly balanced: token t takes heads (tK + j) mod H
    bal = np.array([[(t * K + j) % H for j in range(K)] for t in range(T)])[None]
    n, *_ = O.permutation(bal.astype(np.int32), H)
    assert O.interaction_count(n) == T * T * K * K // (2 * H) + T * K // 2
    # every token picks the same heads: upper bound K T (T+1) / 2
    same = np.tile(np.array([[3, 5]]), (T, 1))[None].astype(np.int32)
    n2, *_ = O.permutation(same, H)
    assert O.interaction_count(n2) == K * T * (T + 1) // 2
    m = O.membership(same, H)[0]
    pop = sum(int(v.sum()) for v in _all_vis(m))
    assert pop == K * T * (T + 1) // 2


# ----------------------------------------------------------------------------
# RoPE (Eq. namoh-head-rope, reading R4)

def test_rope_matches_complex_rotation():
    d, base = 16, 500.0
    x = rng.standard_normal((7, d))
    p = np.array([0, 1, 2, 5, 77, 1000, 123456])
    got = O.rope_rotate(x, p, base)
    half = d // 2
    z = x[:, :half] + 1j * x[:, half:]
    freqs = np.array([base ** (-(2 * j) / d) for j in range(half)])
    zr = z * np.exp(1j * np.outer(p, freqs))
    np.testing.assert_allclose(got, np.concatenate([zr.real, zr.imag], -1), atol=1e-12)


def test_rope_hand_values_and_properties():
    # d = 4, base 100: theta = (1, 0.1).  Element 1 pairs with element 3.
    e1 = np.array([[0.0, 1.0, 0.0, 0.0]])
    r = O.rope_rotate(e1, np.array([1]), 100.0)[0]
    np.testing.assert_allclose(r, [0.0, math.cos(0.1), 0.0, math.sin(0.1)], atol=1e-15)
    e0 = np.array([[1.0, 0.0]])
    np.testing.assert_allclose(O.rope_rotate(e0, np.array([math.pi / 2]), 7.0)[0], [0, 1], atol=1e-15)
    x = rng.standard_normal((5, 32))
    np.testing.assert_allclose(O.rope_rotate(x, np.zeros(5), 1e4), x)   # identity at 0
    np.testing.assert_allclose(np.linalg.norm(O.rope_rotate(x, np.arange(5) * 37, 1e4), axis=1),
                               np.linalg.norm(x, axis=1), rtol=1e-13)
    # scores depend on the position difference only
    q, k = rng.standard_normal(32), rng.standard_normal(32)
    for a, b in [(3, 10), (100, 107), (1000, 1007)]:
        s = O.rope_rotate(q[None], np.array([b]), 1e4)[0] @ O.rope_rotate(k[None], np.array([a]), 1e4)[0]
        s0 = O.rope_rotate(q[None], np.array([b - a]), 1e4)[0] @ k
        assert math.isclose(s, s0, rel_tol=1e-10, abs_tol=1e-12)


# ----------------------------------------------------------------------------
# attention: K = H reduces to dense causal MHA with standard RoPE

def test_K_equals_H_is_dense_causal_mha_torch_sdpa():
    torch = pytest.importorskip("torch")
    import torch.nn.functional as F
    B, T, H, d, base = 2, 37, 4, 8, 1e4
    g = np.random.default_rng(9)
    q, k, v = (g.standard_normal((B, H, T, d)) for _ in range(3))
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    for form in ("definition", "gathered"):
        res = O.prefill(logits, q, k, v, H, base, O.ROPE_HEAD_RELATIVE, O.GATE_SOFTMAX_ALL, form=form)
        pos = np.arange(T)
        qr = O.rope_rotate(q, np.broadcast_to(pos, (B, H, T)), base)
        kr = O.rope_rotate(k, np.broadcast_to(pos, (B, H, T)), base)
        ref = F.scaled_dot_product_attention(torch.from_numpy(qr), torch.from_numpy(kr),
                                             torch.from_numpy(v), is_causal=True).numpy()
        a = scipy.special.softmax(logits.astype(np.float64), -1)           # [B,T,H]
        o_ref = np.einsum("bth,bhtd->btd", a, ref)
        np.testing.assert_allclose(res["out"], o_ref, atol=1e-12)
        # head-relative and global RoPE coincide when K = H
        res_g = O.prefill(logits, q, k, v, H, base, O.ROPE_GLOBAL, O.GATE_SOFTMAX_ALL, form=form)
        np.testing.assert_allclose(res_g["out"], res["out"], atol=1e-12)


def test_attention_special_cases():
    B, T, H, K, d = 1, 30, 5, 2, 6
    g = np.random.default_rng(10)
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    # head 4 selected by token 7 only: that head's output there is v itself
    logits[..., 4] = -10.0
    logits[0, 7, 4] = 10.0
    q, k, v = (g.standard_normal((B, H, T, d)) for _ in range(3))
    res = O.prefill(logits, q, k, v, K, 1e4, form="definition")
    slot = res["slot_pos"][0, 7, 0]
    assert res["topk_idx"][0, 7, 0] == 4
    np.testing.assert_allclose(res["head_out"][slot], v[0, 4, 7], atol=1e-14)
    # q = 0: uniform weights -> prefix mean of the head's routed values
    res0 = O.prefill(logits, np.zeros_like(q), k, v, K, 1e4, form="gathered")
    n, off, perm = res0["head_len"], res0["seg_offsets"], res0["perm_token"]
    for h in range(H):
        toks = perm[off[h]:off[h + 1]]
        for r in range(len(toks)):
            np.testing.assert_allclose(res0["head_out"][off[h] + r],
                                       v[0, h, toks[:r + 1]].mean(0), atol=1e-13)
    # constant V -> constant output (gates sum to one)
    vc = np.full_like(v, 0.375)
    resc = O.prefill(logits, q, k, vc, K, 1e4, form="gathered")
    np.testing.assert_allclose(resc["out"], 0.375, atol=1e-13)


@pytest.mark.parametrize("rope_mode", [O.ROPE_HEAD_RELATIVE, O.ROPE_GLOBAL, O.ROPE_NONE])
@pytest.mark.parametrize("gate_mode", [O.GATE_SOFTMAX_SELECTED, O.GATE_SOFTMAX_ALL])
def test_brute_force_equals_definition_equals_gathered(rope_mode, gate_mode):
    T, H, K, d, base = 24, 5, 2, 6, 100.0
    g = np.random.default_rng(11 + rope_mode + 3 * gate_mode)
    logits = g.integers(-2, 3, size=(1, T, H)).astype(np.float32)   # ties included
    q, k, v = (g.standard_normal((1, H, T, d)) for _ in range(3))
    sel, gat, o0 = O.brute_force_layer(logits[0], q[0], k[0], v[0], K, base, rope_mode, gate_mode)
    r1 = O.prefill(logits, q, k, v, K, base, rope_mode, gate_mode, form="definition")
    r2 = O.prefill(logits, q, k, v, K, base, rope_mode, gate_mode, form="gathered")
    assert r1["topk_idx"][0].tolist() == sel
    np.testing.assert_allclose(r1["gates"][0], np.array(gat), atol=1e-15)
    np.testing.assert_allclose(r1["out"][0], np.array(o0), atol=1e-12)
    np.testing.assert_allclose(r2["out"], r1["out"], atol=1e-12)
    np.testing.assert_allclose(r2["head_out"], r1["head_out"], atol=1e-12)


def test_definition_equals_gathered_medium():
    B, T, H, K, d = 2, 300, 6, 3, 16
    g = np.random.default_rng(12)
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    q, k, v = (g.standard_normal((B, H, T, d)) for _ in range(3))
    r1 = O.prefill(logits, q, k, v, K, 1e4, form="definition")
    r2 = O.prefill(logits, q, k, v, K, 1e4, form="gathered")
    np.testing.assert_allclose(r2["out"], r1["out"], atol=1e-12)
    # sampled rows computed one by one agree too
    toks = [0, 1, 150, 299]
    o, hs = O.prefill_rows(q, k, v, r1["topk_idx"], r1["gates"], H, 1e4, 1, toks)
    np.testing.assert_allclose(o, r1["out"][1, toks], atol=1e-12)
    for i, t in enumerate(toks):
        np.testing.assert_allclose(hs[i], r1["head_out"][r1["slot_pos"][1, t]], atol=1e-12)


# ----------------------------------------------------------------------------
# decode (Sec. 3.1: prefill and incremental decoding are the same computation)

def _cache_from_prefill(q, k, logits, K, base, Tp):
    """Post-RoPE key cache of each head after Tp tokens, in rank order."""
    B, H, T, d = q.shape
    topk = O.select_heads(logits[:, :Tp], K)
    m = O.membership(topk, H)
    rho = O.head_ranks(m)
    caches = {}
    for b in range(B):
        for h in range(H):
            toks = np.nonzero(m[b, :, h])[0]
            caches[(b, h)] = toks, O.rope_rotate(k[b, h, toks], rho[b, toks, h], base)
    return caches


@pytest.mark.parametrize("gate_mode", [O.GATE_SOFTMAX_SELECTED, O.GATE_SOFTMAX_ALL])
def test_prefill_equals_incremental_decode(gate_mode):
    B, T, H, K, d, base = 2, 41, 6, 3, 8, 1e4
    g = np.random.default_rng(13)
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    q, k, v = (g.standard_normal((B, H, T, d)) for _ in range(3))
    full = O.prefill(logits, q, k, v, K, base, gate_mode=gate_mode, form="definition")
    for Tp in (0, 1, 20, T - 1):
        caches = _cache_from_prefill(q, k, logits, K, base, Tp)
        lens = np.array([[len(caches[(b, h)][0]) for h in range(H)] for b in range(B)])
        res = O.decode_step(logits[:, Tp], q[:, :, Tp], k[:, :, Tp], v[:, :, Tp],
                            lambda b, h, n: caches[(b, h)][1][:n],
                            lambda b, h, n: v[b, h, caches[(b, h)][0][:n]],
                            lens, K, base, gate_mode=gate_mode)
        np.testing.assert_allclose(res["out"], full["out"][:, Tp], atol=1e-12)
        np.testing.assert_array_equal(res["topk_idx"], full["topk_idx"][:, Tp])
        for b in range(B):
            for kk in range(K):
                assert res["cache_len"][b, res["topk_idx"][b, kk]] == lens[b, res["topk_idx"][b, kk]] + 1


@pytest.mark.parametrize("rope_mode", [O.ROPE_HEAD_RELATIVE, O.ROPE_GLOBAL, O.ROPE_NONE])
def test_prefill_cache_continues_as_the_definition(rope_mode):
    # prefill_cache of a prompt followed by one decode step gives the layer's
    # definition (explicit visibility mask) at the next token: a wrong rank
    # order, rotation position or missing row would not
    B, T, H, K, d, base = 2, 37, 5, 2, 8, 1e4
    g = np.random.default_rng(21)
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    q, k, v = (g.standard_normal((B, H, T, d)) for _ in range(3))
    full = O.prefill(logits, q, k, v, K, base, rope_mode=rope_mode, form="definition")
    for Tp in (0, 1, 17, T - 1):
        topk = O.select_heads(logits[:, :Tp], K)
        kc, vc, n = O.prefill_cache(k[:, :, :Tp], v[:, :, :Tp], topk, H, base, rope_mode)
        np.testing.assert_array_equal(n, O.permutation(topk, H)[0])
        res = O.decode_step(logits[:, Tp], q[:, :, Tp], k[:, :, Tp], v[:, :, Tp],
                            lambda b, h, nn: kc[b, h, :nn], lambda b, h, nn: vc[b, h, :nn],
                            n, K, base, rope_mode=rope_mode, seq_pos=np.full(B, Tp))
        np.testing.assert_allclose(res["out"], full["out"][:, Tp], atol=1e-12)


def test_biased_prefill_continues_as_biased_decode():
    # with loss-free balancing biases, prefill_cache + one biased decode step
    # is the biased layer's definition at the next token
    B, T, H, K, d, base = 2, 29, 6, 2, 8, 1e4
    g = np.random.default_rng(22)
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    bias = (g.standard_normal(H) * 0.1).astype(np.float32)
    q, k, v = (g.standard_normal((B, H, T, d)) for _ in range(3))
    full = O.prefill(logits, q, k, v, K, base, form="definition", bias=bias)
    assert (full["topk_idx"] != O.select_heads(logits, K)).any()
    for Tp in (0, 9, T - 1):
        topk, _ = O.select_heads_biased(logits[:, :Tp], bias, K)
        kc, vc, n = O.prefill_cache(k[:, :, :Tp], v[:, :, :Tp], topk, H, base)
        res = O.decode_step(logits[:, Tp], q[:, :, Tp], k[:, :, Tp], v[:, :, Tp],
                            lambda b, h, nn: kc[b, h, :nn], lambda b, h, nn: vc[b, h, :nn],
                            n, K, base, bias=bias)
        np.testing.assert_allclose(res["out"], full["out"][:, Tp], atol=1e-12)
        np.testing.assert_array_equal(res["topk_idx"], full["topk_idx"][:, Tp])


def test_decode_reads_only_selected_caches_and_counts():
    B, H, K, d = 3, 8, 2, 4
    g = np.random.default_rng(14)
    logits = g.standard_normal((B, H)).astype(np.float32)
    q, k, v = (g.standard_normal((B, H, d)) for _ in range(3))
    lens = g.integers(0, 9, size=(B, H))
    store_k = g.standard_normal((B, H, 10, d))
    store_v = g.standard_normal((B, H, 10, d))
    reads = []

    def ck(b, h, n):
        reads.append((b, h, n))
        return store_k[b, h, :n]
    r1 = O.decode_step(logits, q, k, v, ck, lambda b, h, n: store_v[b, h, :n], lens, K, 1e4)
    topk = r1["topk_idx"]
    assert sorted((b, h) for b, h, _ in reads) == sorted((b, int(h)) for b in range(B) for h in topk[b])
    # A_KV = sum of the selected heads' lengths (Eq. namoh-kv-cost)
    assert sum(n for *_, n in reads) == sum(int(lens[b, h]) for b in range(B) for h in topk[b])
    # perturb every non-selected cache: output unchanged
    sk2, sv2 = store_k.copy(), store_v.copy()
    for b in range(B):
        for h in range(H):
            if h not in topk[b]:
                sk2[b, h] += 100.0
                sv2[b, h] -= 50.0
    r2 = O.decode_step(logits, q, k, v, lambda b, h, n: sk2[b, h, :n],
                       lambda b, h, n: sv2[b, h, :n], lens, K, 1e4)
    np.testing.assert_array_equal(r2["out"], r1["out"])


# ----------------------------------------------------------------------------
# input generator: determinism and format (no layer arithmetic)

def test_workload_generator_is_deterministic_and_rounds_bf16():
    w = W.WORKLOADS[1].with_(T=64)
    a, b = W.prefill_inputs(w), W.prefill_inputs(w)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5e-3, 3.0e5], np.float32)
    bits = W.f32_to_bf16_bits(x)
    # 1 + 2^-8 is a tie -> even (1.0); 1 + 3*2^-8 is a tie -> even (1 + 2^-6)
    np.testing.assert_array_equal(W.bf16_bits_to_f32(bits)[:3], [1.0, 1.0, 1.015625])
    assert abs(W.bf16_bits_to_f32(bits)[3] / x[3] - 1) < 2 ** -8


# ----------------------------------------------------------------------------
# Loss-free balancing (App. "Auxiliary-Loss-Free Balancing")

def test_biased_selection_without_bias_is_the_plain_selection():
    # softmax is monotone, so TopK of the affinities is TopK of the logits
    g = np.random.default_rng(31)
    logits = g.standard_normal((3, 50, 16)).astype(np.float32)
    for K in (1, 4, 16):
        topk, gates = O.select_heads_biased(logits, np.zeros(16), K)
        np.testing.assert_array_equal(topk, O.select_heads(logits, K))
        np.testing.assert_allclose(gates, O.route_gates(logits, topk, O.GATE_SOFTMAX_ALL),
                                   rtol=1e-14)


def test_biased_selection_bias_moves_selection_not_gates():
    g = np.random.default_rng(32)
    H, K = 12, 3
    logits = g.standard_normal((2, 40, H)).astype(np.float32)
    bias = np.zeros(H)
    bias[7] = 2.0                        # above any affinity: always selected, first
    topk, gates = O.select_heads_biased(logits, bias, K)
    assert (topk[..., 0] == 7).all()
    np.testing.assert_allclose(gates, O.route_gates(logits, topk, O.GATE_SOFTMAX_ALL),
                               rtol=1e-14)   # gates keep the unbiased affinities
    bias = np.full(H, -2.0)
    bias[[2, 5, 9]] = 0.0                # only these three can win
    topk, _ = O.select_heads_biased(logits, bias, K)
    assert (np.sort(topk, axis=-1) == [2, 5, 9]).all()
    # the three kept heads come in affinity order
    a = O.route_gates(logits, topk, O.GATE_SOFTMAX_ALL)
    assert (np.diff(a, axis=-1) <= 0).all()


def test_biased_selection_worked_example():
    # logits (0, ln 2, 0, 0): a = (0.2, 0.4, 0.2, 0.2); bias (0.125, 0, 0.0625, 0)
    # -> scores (0.325, 0.4, 0.2625, 0.2): heads 1 then 0, gates 0.4 and 0.2
    logits = np.array([[[0.0, np.log(2.0), 0.0, 0.0]]], dtype=np.float32)
    topk, gates = O.select_heads_biased(logits, np.array([0.125, 0.0, 0.0625, 0.0]), 2)
    assert topk.tolist() == [[[1, 0]]]
    np.testing.assert_allclose(gates[0, 0], [0.4, 0.2], rtol=1e-6)
    # equal scores: the lower head index first
    topk, _ = O.select_heads_biased(np.zeros((1, 1, 5), np.float32), np.zeros(5), 3)
    assert topk.tolist() == [[[0, 1, 2]]]


def test_bias_update_step():
    # c = (5, 3, 2, 2), c_bar = T K / H = 6 * 2 / 4 = 3: the overloaded head
    # steps down, the balanced one stays, the underloaded ones step up
    b = O.bias_update(np.array([[5, 3, 2, 2]]), np.array([0.5, 0.0, -0.25, 0.0]), 0.125, 6, 2)
    assert b.dtype == np.float32
    assert b.tolist() == [0.375, 0.0, -0.125, 0.125]
    # counts over a routed batch sum to N K (Eq. app-assignment-count); a
    # non-integer c_bar never gives a zero step
    g = np.random.default_rng(33)
    logits = g.standard_normal((3, 37, 7)).astype(np.float32)
    topk, _ = O.select_heads_biased(logits, g.standard_normal(7) * 0.05, 2)
    n = O.permutation(topk, 7)[0]
    assert n.sum() == 3 * 37 * 2
    b = O.bias_update(n, np.zeros(7), 0.5, 37, 2)
    assert set(np.unique(b)) <= {-0.5, 0.5}


# ----------------------------------------------------------------------------
# Backward (training path): the exact gradient, pinned by finite differences
# of the forward oracle and by torch autograd (float64, CPU)

def _bwd_case(seed, B=2, T=11, H=4, K=2, d=8):
    g = np.random.default_rng(seed)
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    q, k, v = (g.standard_normal((B, H, T, d)) for _ in range(3))
    topk = O.select_heads(logits, K)
    gates = O.route_gates(logits, topk, O.GATE_SOFTMAX_SELECTED)
    n, off, perm, slot = O.permutation(topk, H)
    dout = g.standard_normal((B, T, d))
    return logits, q, k, v, topk, gates, n, off, perm, slot, dout


def _layer(q, k, v, gates, n, off, perm, slot, H, base, rope_mode):
    hp = O.attention_gathered(q, k, v, n, off, perm, H, base, rope_mode)
    return O.combine_packed(hp, slot, gates)


@pytest.mark.parametrize("rope_mode", [O.ROPE_HEAD_RELATIVE, O.ROPE_GLOBAL, O.ROPE_NONE])
def test_attention_backward_finite_differences(rope_mode):
    base = 1e4
    logits, q, k, v, topk, gates, n, off, perm, slot, dout = _bwd_case(41 + rope_mode)
    H = q.shape[1]
    dq, dk, dv, dg = O.attention_backward(q, k, v, gates, off, perm, slot, H, base, dout,
                                          rope_mode)
    loss = lambda q_, k_, v_, g_: float((_layer(q_, k_, v_, g_, n, off, perm, slot, H, base,
                                                 rope_mode) * dout).sum())
    rng = np.random.default_rng(5)
    eps = 1e-6
    for name, x, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv), ("g", gates, dg)):
        for _ in range(12):
            idx = tuple(rng.integers(0, s) for s in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            args = {"q": q, "k": k, "v": v, "g": gates}
            fp = loss(*[xp if a == name else args[a] for a in ("q", "k", "v", "g")])
            fm = loss(*[xm if a == name else args[a] for a in ("q", "k", "v", "g")])
            fd = (fp - fm) / (2 * eps)
            assert abs(fd - grad[idx]) <= 1e-7 + 1e-6 * abs(fd), (name, idx, fd, grad[idx])
    # rows of tokens not routed to a head get no gradient
    m = O.membership(topk, H)
    assert not dq[~m.transpose(0, 2, 1)].any() and not dk[~m.transpose(0, 2, 1)].any()


@pytest.mark.parametrize("mode", [O.GATE_SOFTMAX_SELECTED, O.GATE_SOFTMAX_ALL])
def test_gates_backward_finite_differences(mode):
    g = np.random.default_rng(43 + mode)
    B, T, H, K = 2, 7, 6, 3
    logits = g.standard_normal((B, T, H))
    topk = O.select_heads(logits.astype(np.float32), K)
    dg = g.standard_normal((B, T, K))
    dl = O.gates_backward(logits, topk, dg, mode)
    eps = 1e-6
    for b in range(B):
        for t in range(T):
            for h in range(H):
                lp, lm = logits.copy(), logits.copy()
                lp[b, t, h] += eps
                lm[b, t, h] -= eps
                fd = ((O.route_gates(lp, topk, mode) - O.route_gates(lm, topk, mode)) * dg).sum()
                assert abs(fd / (2 * eps) - dl[b, t, h]) <= 1e-8


def test_attention_backward_matches_autograd():
    torch = pytest.importorskip("torch")
    base = 5e5
    logits, q, k, v, topk, gates, n, off, perm, slot, dout = _bwd_case(44, B=2, T=37, H=5, K=2,
                                                                         d=16)
    H, d = q.shape[1], q.shape[-1]
    dq, dk, dv, dg = O.attention_backward(q, k, v, gates, off, perm, slot, H, base, dout)
    tq, tk, tv, tg = (torch.tensor(x, dtype=torch.float64, requires_grad=True)
                      for x in (q, k, v, gates))
    theta = base ** (-2.0 * torch.arange(d // 2, dtype=torch.float64) / d)

    def rot(x, p):
        ang = p[:, None].to(torch.float64) * theta
        c, s = torch.cos(ang), torch.sin(ang)
        x1, x2 = x[:, :d // 2], x[:, d // 2:]
        return torch.cat([x1 * c - x2 * s, x2 * c + x1 * s], dim=1)

    hp = [None] * int(off[-1])
    for sid in range(len(off) - 1):
        b, h = divmod(sid, H)
        a, e = int(off[sid]), int(off[sid + 1])
        if a == e:
            continue
        tok = torch.tensor(perm[a:e].astype(np.int64))
        pos = torch.arange(e - a)
        qq, kk = rot(tq[b, h, tok], pos), rot(tk[b, h, tok], pos)
        sc = qq @ kk.T / np.sqrt(d)
        sc = sc.masked_fill(~torch.tril(torch.ones(e - a, e - a, dtype=torch.bool)), float("-inf"))
        o = torch.softmax(sc, dim=1) @ tv[b, h, tok]
        for r in range(e - a):
            hp[a + r] = o[r]
    hp = torch.stack(hp)
    out = sum(tg[:, :, kk, None] * hp[torch.tensor(slot[:, :, kk].astype(np.int64))]
              for kk in range(slot.shape[-1]))
    (out * torch.tensor(dout)).sum().backward()
    np.testing.assert_allclose(tq.grad.numpy(), dq, atol=1e-11)
    np.testing.assert_allclose(tk.grad.numpy(), dk, atol=1e-11)
    np.testing.assert_allclose(tv.grad.numpy(), dv, atol=1e-11)
    np.testing.assert_allclose(tg.grad.numpy(), dg, atol=1e-11)


# ----------------------------------------------------------------------------
# routed projections (Eq. namoh-qkv; output aggregation of Eq. namoh-attention)

def _proj_case(seed, B=2, T=9, H=4, K=2, d=4, dm=6):
    g = np.random.default_rng(seed)
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    x = g.standard_normal((B, T, dm))
    w_qkv = g.standard_normal((H, 3, d, dm))
    w_o = g.standard_normal((H, dm, d))
    return logits, x, w_qkv, w_o


def test_qkv_projection_all_heads_is_dense_multihead_projection():
    # K = H: every pair is routed, so the projections are those of standard
    # multi-head attention, computed here with the concatenated weight matrix
    logits, x, w_qkv, _ = _proj_case(71, H=3, K=3, d=5, dm=7)
    B, T, dm = x.shape
    H, d = 3, 5
    topk = O.select_heads(logits, 3)
    q, k, v, m = O.qkv_projection(x, w_qkv, topk)
    assert m.all()
    for j, got in enumerate((q, k, v)):
        w_cat = w_qkv[:, j].reshape(H * d, dm)           # [H*d, d_model]
        dense = (x.reshape(B * T, dm) @ w_cat.T).reshape(B, T, H, d).transpose(0, 2, 1, 3)
        np.testing.assert_allclose(got, dense, rtol=1e-12, atol=1e-12)


def test_qkv_projection_brute_force_and_unrouted_pairs():
    logits, x, w_qkv, _ = _proj_case(72)
    topk = O.select_heads(logits, 2)
    q, k, v, m = O.qkv_projection(x, w_qkv, topk)
    B, T, dm = x.shape
    H, _, d, _ = w_qkv.shape
    for b in range(B):
        for t in range(T):
            sel = [int(i) for i in topk[b, t]]
            for i in range(H):
                for j, arr in enumerate((q, k, v)):
                    if i in sel:
                        for c in range(d):
                            want = sum(x[b, t, e] * w_qkv[i, j, c, e] for e in range(dm))
                            assert abs(arr[b, i, t, c] - want) < 1e-12
                    else:
                        assert np.isnan(arr[b, i, t]).all()   # no vectors for inactive pairs
    # each token is projected into exactly K heads
    assert (m.sum(-1) == 2).all()


def test_output_projection_identity_is_the_combine():
    # W_O^(i) = I (d_model = d) reduces the aggregation to the gated combine
    logits, x, w_qkv, _ = _proj_case(73, d=4, dm=4)
    topk = O.select_heads(logits, 2)
    gates = O.route_gates(logits, topk, O.GATE_SOFTMAX_SELECTED)
    h = np.random.default_rng(5).standard_normal((2, 4, 9, 4))
    eye = np.broadcast_to(np.eye(4), (4, 4, 4)).copy()
    np.testing.assert_allclose(O.output_projection(h, topk, gates, eye),
                               O.combine_dense(h, topk, gates), rtol=1e-13, atol=1e-13)


def test_output_projection_all_heads_is_dense_output_projection():
    # K = H: o_t = concat_i(g_{t,i} h_{t,i}) W_O, the standard output
    # projection with the concatenated [d_model, H*d] weight
    logits, x, _, w_o = _proj_case(74, H=3, K=3, d=5, dm=7)
    B, T = 2, 9
    H, d, dm = 3, 5, 7
    topk = O.select_heads(logits, 3)
    gates = O.route_gates(logits, topk, O.GATE_SOFTMAX_SELECTED)
    h = np.random.default_rng(6).standard_normal((B, H, T, d))
    g_dense = np.zeros((B, T, H))
    np.put_along_axis(g_dense, topk.astype(np.int64), gates, axis=-1)
    gh = (h * g_dense.transpose(0, 2, 1)[..., None]).transpose(0, 2, 1, 3).reshape(B, T, H * d)
    w_cat = w_o.transpose(1, 0, 2).reshape(dm, H * d)
    np.testing.assert_allclose(O.output_projection(h, topk, gates, w_o), gh @ w_cat.T,
                               rtol=1e-12, atol=1e-12)


def test_projected_layer_reads_only_routed_pairs():
    # the unrouted rows of q/k/v are NaN: a layer that read any of them would
    # return NaN; the gathered attention and the aggregation read none
    logits, x, w_qkv, w_o = _proj_case(75, B=2, T=13, H=5, K=2, d=4, dm=6)
    topk = O.select_heads(logits, 2)
    q, k, v, _ = O.qkv_projection(x, w_qkv, topk)
    ref = O.prefill(logits, q, k, v, 2, 1e4)
    H = 5
    h = np.full(q.shape, np.nan)
    n, off, perm, slot = O.permutation(topk, H)
    for sid in range(2 * H):
        b, i = divmod(sid, H)
        a, e = int(off[sid]), int(off[sid + 1])
        h[b, i, perm[a:e]] = ref["head_out"][a:e]
    o = O.output_projection(h, topk, ref["gates"], w_o)
    assert np.isfinite(o).all()
    # and the aggregation equals the packed form: per routed row h W_O^(i),
    # then the gated combine over the K slots
    y = np.zeros((int(off[-1]), w_o.shape[1]))
    for sid in range(2 * H):
        b, i = divmod(sid, H)
        a, e = int(off[sid]), int(off[sid + 1])
        y[a:e] = ref["head_out"][a:e] @ w_o[i].T
    np.testing.assert_allclose(O.combine_packed(y, slot, ref["gates"]), o, rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------------------
# KV-group routing (App. GQA+NAMOH, adopted KV-group routing)

def _gqa_case(seed, B=2, T=23, G=4, Kg=2, g=2, d=8):
    r = np.random.default_rng(seed)
    logits = r.standard_normal((B, T, G)).astype(np.float32)
    q = r.standard_normal((B, G * g, T, d))
    k = r.standard_normal((B, G, T, d))
    v = r.standard_normal((B, G, T, d))
    return logits, q, k, v, O.select_heads(logits, Kg)


@pytest.mark.parametrize("rope_mode", [O.ROPE_HEAD_RELATIVE, O.ROPE_GLOBAL, O.ROPE_NONE])
def test_kv_groups_of_one_are_the_routed_heads(rope_mode):
    # g = 1: every query head has its own key/value head; the result is the
    # per-head routed attention
    logits, q, k, v, topk = _gqa_case(81, G=5, Kg=2, g=1)
    h = O.attention_kv_groups(q, k, v, topk, 1, 1e4, rope_mode)
    n, off, perm, slot = O.permutation(topk, 5)
    hp = O.attention_gathered(q, k, v, n, off, perm, 5, 1e4, rope_mode)
    for sid in range(2 * 5):
        b, i = divmod(sid, 5)
        a, e = int(off[sid]), int(off[sid + 1])
        np.testing.assert_allclose(h[b, i, perm[a:e]], hp[a:e], rtol=1e-12, atol=1e-12)


def test_kv_groups_all_selected_is_dense_gqa():
    # all H/g groups selected: standard causal grouped-query attention with
    # standard RoPE (torch scaled_dot_product_attention, float64, keys and
    # values repeated for the g query heads of each group)
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    logits, q, k, v, topk = _gqa_case(82, B=2, T=19, G=3, Kg=3, g=2, d=6)
    B, H, T, d = q.shape
    base = 1e4
    pos = np.arange(T)
    qr = O.rope_rotate(q, np.broadcast_to(pos, (B, H, T)), base)
    kr = O.rope_rotate(k, np.broadcast_to(pos, (B, 3, T)), base)
    kt = torch.from_numpy(kr).repeat_interleave(2, dim=1)
    vt = torch.from_numpy(v).repeat_interleave(2, dim=1)
    ref = F.scaled_dot_product_attention(torch.from_numpy(qr), kt, vt, is_causal=True).numpy()
    for form in ("definition", "gathered"):
        got = O.attention_kv_groups(q, k, v, topk, 2, base, O.ROPE_HEAD_RELATIVE, form=form)
        np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("rope_mode", [O.ROPE_HEAD_RELATIVE, O.ROPE_GLOBAL, O.ROPE_NONE])
def test_kv_groups_definition_equals_gathered(rope_mode):
    logits, q, k, v, topk = _gqa_case(83, B=2, T=31, G=4, Kg=2, g=3, d=8)
    a = O.attention_kv_groups(q, k, v, topk, 3, 1e4, rope_mode, form="definition")
    b = O.attention_kv_groups(q, k, v, topk, 3, 1e4, rope_mode, form="gathered")
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12, equal_nan=True)
    # unselected (token, group) pairs produce nothing; selected ones are finite
    m = O.membership(topk, 4)
    for j in range(4):
        for u in range(3):
            assert np.isnan(a[:, j * 3 + u][~m[:, :, j]]).all()
            assert np.isfinite(a[:, j * 3 + u][m[:, :, j]]).all()


def test_kv_groups_interaction_count_closed_form():
    # Eq. app-group-prefill: C_attn = g/2 sum n_j^2 + g/2 sum n_j, counted
    # here from the explicit visibility masks of every query head
    logits, q, k, v, topk = _gqa_case(84, B=1, T=40, G=4, Kg=2, g=3, d=4)
    G, g = 4, 3
    m = O.membership(topk, G)
    pairs = 0
    for j in range(G):
        rows = np.nonzero(m[0, :, j])[0]
        pairs += g * int(O.visibility_mask(m[0, :, j], rows).sum())
    n = m[0].sum(0)
    assert n.sum() == 40 * 2                     # sum_j n_j = T K/g (K/g = 2 groups per token)
    assert pairs == g * (n * n).sum() // 2 + g * n.sum() // 2


def test_kv_groups_brute_force_and_combine():
    # scalar loops over (t, head, s) for one tiny sequence, then the gated
    # group combine against its definition
    logits, q, k, v, topk = _gqa_case(85, B=1, T=9, G=3, Kg=2, g=2, d=4)
    base = 1e4
    sel = [[int(j) for j in topk[0, t]] for t in range(9)]

    def rot(vec, p):
        half = 2
        out = [0.0] * 4
        for jj in range(half):
            ang = p * base ** (-2.0 * jj / 4)
            c, s_ = math.cos(ang), math.sin(ang)
            out[jj] = vec[jj] * c - vec[jj + half] * s_
            out[jj + half] = vec[jj + half] * c + vec[jj] * s_
        return out

    h = O.attention_kv_groups(q, k, v, topk, 2, base)
    gates = O.route_gates(logits, topk, O.GATE_SOFTMAX_SELECTED)
    o = O.combine_kv_groups(h, topk, gates, 2)
    for t in range(9):
        want_o = [0.0] * 4
        for kk, j in enumerate(sel[t]):
            hist = [s for s in range(t + 1) if j in sel[s]]
            rank = {s: r for r, s in enumerate(hist)}
            for u in range(2):
                qv = rot(list(q[0, j * 2 + u, t]), rank[t])
                sc = [sum(a * b for a, b in zip(qv, rot(list(k[0, j, s]), rank[s]))) / 2.0
                      for s in hist]
                mx = max(sc)
                e = [math.exp(x - mx) for x in sc]
                hv = [sum(e[i] * v[0, j, s, c] for i, s in enumerate(hist)) / sum(e) for c in range(4)]
                np.testing.assert_allclose(h[0, j * 2 + u, t], hv, rtol=1e-12, atol=1e-12)
                for c in range(4):
                    want_o[c] += gates[0, t, kk] * hv[c]
        np.testing.assert_allclose(o[0, t], want_o, rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------------------
# always-active shared heads (Sec. 4.4, shared heads for local context)

def _shared_case(seed, B=2, Hs=2, T=40, d=8):
    r = np.random.default_rng(seed)
    return (r.standard_normal((B, Hs, T, d)) for _ in range(3))


def test_shared_full_prefix_is_causal_attention_with_rope():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    q, k, v = _shared_case(91)
    B, Hs, T, d = q.shape
    pos = np.broadcast_to(np.arange(T), (B, Hs, T))
    ref = F.scaled_dot_product_attention(torch.from_numpy(O.rope_rotate(q, pos, 1e4)),
                                         torch.from_numpy(O.rope_rotate(k, pos, 1e4)),
                                         torch.from_numpy(v), is_causal=True).numpy()
    np.testing.assert_allclose(O.always_active_heads(q, k, v, 0, 1e4), ref, rtol=1e-12, atol=1e-12)
    # a window at least as long as the sequence is the full prefix
    np.testing.assert_allclose(O.always_active_heads(q, k, v, T, 1e4), ref, rtol=1e-12, atol=1e-12)


def test_shared_sliding_window_against_a_library_mask():
    # the band mask t - w < s <= t handed to torch's attention as a boolean mask
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    q, k, v = _shared_case(92, T=37)
    B, Hs, T, d = q.shape
    w = 5
    pos = np.broadcast_to(np.arange(T), (B, Hs, T))
    i = torch.arange(T)
    band = (i[None, :] <= i[:, None]) & (i[None, :] > i[:, None] - w)
    ref = F.scaled_dot_product_attention(torch.from_numpy(O.rope_rotate(q, pos, 1e4)),
                                         torch.from_numpy(O.rope_rotate(k, pos, 1e4)),
                                         torch.from_numpy(v), attn_mask=band).numpy()
    np.testing.assert_allclose(O.always_active_heads(q, k, v, w, 1e4), ref, rtol=1e-12, atol=1e-12)


def test_shared_window_special_cases():
    q, k, v = _shared_case(93, T=20)
    # w = 1: every token attends to itself only
    np.testing.assert_allclose(O.always_active_heads(q, k, v, 1, 1e4), v, rtol=1e-13, atol=1e-13)
    # constant values give that constant, whatever the window
    c = np.full_like(v, 0.75)
    np.testing.assert_allclose(O.always_active_heads(q, k, c, 4, 1e4), c, rtol=1e-13, atol=1e-13)
    # q = 0: the mean of the window's values (closed form)
    z = np.zeros_like(q)
    got = O.always_active_heads(z, k, v, 3, 1e4, O.ROPE_NONE)
    for t in range(20):
        lo = max(0, t - 2)
        np.testing.assert_allclose(got[:, :, t], v[:, :, lo:t + 1].mean(axis=2), rtol=1e-12,
                                   atol=1e-12)
    # global RoPE: shifting every position by the same amount leaves the
    # output unchanged (scores depend on position differences only)
    a = O.always_active_heads(q, k, v, 6, 1e4, O.ROPE_GLOBAL)
    B, Hs, T, d = q.shape
    pos = np.broadcast_to(np.arange(T) + 9, (B, Hs, T))
    qs, ks = O.rope_rotate(q, pos, 1e4), O.rope_rotate(k, pos, 1e4)
    b = O.always_active_heads(qs, ks, v, 6, 1e4, O.ROPE_NONE)
    np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-10)


def test_kv_group_decode_of_one_is_the_decode_step():
    r = np.random.default_rng(86)
    B, H, K, d, cap = 2, 5, 2, 8, 12
    logits = r.standard_normal((B, H)).astype(np.float32)
    q, k, v = (r.standard_normal((B, H, d)) for _ in range(3))
    ck, cv = r.standard_normal((B, H, cap, d)), r.standard_normal((B, H, cap, d))
    n = r.integers(0, cap - 1, size=(B, H))
    a = O.decode_step(logits, q, k, v, lambda b, h, m: ck[b, h, :m], lambda b, h, m: cv[b, h, :m],
                      n, K, 1e4)
    b_ = O.decode_step_kv_groups(logits, q, k, v, lambda b, h, m: ck[b, h, :m],
                                 lambda b, h, m: cv[b, h, :m], n, K, 1, 1e4)
    np.testing.assert_allclose(b_["out"], a["out"], rtol=1e-13, atol=1e-13)
    np.testing.assert_array_equal(b_["cache_len"], a["cache_len"])


@pytest.mark.parametrize("rope_mode", [O.ROPE_HEAD_RELATIVE, O.ROPE_GLOBAL, O.ROPE_NONE])
def test_kv_group_prefill_then_decode_is_the_definition(rope_mode):
    # decoding token T from the grouped prefill's caches gives the grouped
    # attention (definition form) of T + 1 tokens at its last row
    r = np.random.default_rng(87)
    B, T, G, Kg, g, d = 2, 17, 4, 2, 3, 8
    base = 1e4
    logits = r.standard_normal((B, T + 1, G)).astype(np.float32)
    q = r.standard_normal((B, G * g, T + 1, d))
    k = r.standard_normal((B, G, T + 1, d))
    v = r.standard_normal((B, G, T + 1, d))
    topk = O.select_heads(logits, Kg)
    full = O.attention_kv_groups(q, k, v, topk, g, base, rope_mode, form="definition")
    gates = O.route_gates(logits, topk, O.GATE_SOFTMAX_SELECTED)
    o_full = O.combine_kv_groups(full, topk, gates, g)[:, T]
    # caches of the first T tokens: each group's rotated keys and values in rank order
    m = O.membership(topk[:, :T], G)
    rank = O.head_ranks(m)
    caches_k, caches_v, n = {}, {}, np.zeros((B, G), dtype=np.int64)
    for b in range(B):
        for j in range(G):
            rows = np.nonzero(m[b, :, j])[0]
            n[b, j] = rows.size
            pos = {O.ROPE_HEAD_RELATIVE: rank[b, rows, j], O.ROPE_GLOBAL: rows,
                   O.ROPE_NONE: None}[rope_mode]
            caches_k[b, j] = k[b, j, rows] if pos is None else O.rope_rotate(k[b, j, rows], pos, base)
            caches_v[b, j] = v[b, j, rows]
    res = O.decode_step_kv_groups(logits[:, T], q[:, :, T], k[:, :, T], v[:, :, T],
                                  lambda b, j, nn: caches_k[b, j][:nn],
                                  lambda b, j, nn: caches_v[b, j][:nn], n, Kg, g, base, rope_mode,
                                  seq_pos=np.full(B, T))
    np.testing.assert_array_equal(res["topk_idx"], topk[:, T])
    np.testing.assert_allclose(res["out"], o_full, rtol=1e-11, atol=1e-11)
