"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Routing and permutation indices are compared bit for bit; outputs within
max abs 1e-4 (fp32) or 2e-2 + 1e-2*|ref| (bf16) of the float64 oracle.
Full-size workloads compare every index and every output row (against the
gathered oracle run one segment at a time, plus a sample of rows that the
oracle computes one token at a time); mid-sized cases (several tiles and
ragged tails) compare every output.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
from paper_2609_38832_amd import workloads as W  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_38832_amd import _lib
    _lib.lib()   # fail loudly if the library is missing


from gpu_util import (DEV, assert_routing_exact, check_out, from_dev, run_prefill,  # noqa: E402
                      say, to_dev)
from paper_2609_38832_amd import _lib as L  # noqa: E402


def _f64(inp, w):
    return {k: W.as_float64(inp[k], w.dtype) for k in ("q", "k", "v")}


def _oracle_routing(inp, w, gate_mode=0):
    topk = O.select_heads(inp["logits"], w.K)
    g = O.route_gates(inp["logits"], topk, gate_mode)
    n, off, perm, slot = O.permutation(topk, w.H)
    return {"topk_idx": topk, "gates": g, "head_len": n, "seg_offsets": off,
            "perm_token": perm, "slot_pos": slot}


# ----------------------------------------------------------------------------
# routing

@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_route_full_size_bit_exact(cfg):
    w = W.WORKLOADS[cfg]
    say(f"route full size: {w.name}")
    logits = W.prefill_logits(w)
    r = L.route(torch.from_numpy(logits).to(DEV), w.K)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in r.items()}
    assert_routing_exact(got, _oracle_routing({"logits": logits}, w))


@pytest.mark.parametrize("case", ["integers", "all_equal", "signed_zero", "infinities"])
@pytest.mark.parametrize("gate_mode", [0, 1])
def test_route_forced_ties(case, gate_mode):
    g = np.random.default_rng(5)
    B, T, H, K = 2, 700, 16, 5
    if case == "integers":
        lg = g.integers(-2, 3, size=(B, T, H)).astype(np.float32)
    elif case == "all_equal":
        lg = np.full((B, T, H), 0.25, np.float32)
    elif case == "signed_zero":
        lg = np.where(g.random((B, T, H)) < 0.5, np.float32(0.0), np.float32(-0.0)).astype(np.float32)
        lg[:, ::3, 2] = 1.0
    else:
        lg = g.choice(np.array([-np.inf, -1.0, 0.0, 2.0], np.float32), size=(B, T, H))
    say(f"route ties: {case} gate_mode={gate_mode}")
    r = L.route(torch.from_numpy(lg).to(DEV), K, gate_mode)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in r.items()}
    w = W.WORKLOADS[1].with_(B=B, T=T, H=H, K=K)
    ref = _oracle_routing({"logits": lg}, w, gate_mode)
    for key in ("topk_idx", "head_len", "seg_offsets", "perm_token", "slot_pos"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)
    if case != "infinities":
        np.testing.assert_allclose(got["gates"], ref["gates"], rtol=2e-6, atol=1e-7)


@pytest.mark.parametrize("H,K,T", [(1, 1, 5), (3, 3, 1), (64, 64, 130), (64, 1, 1000), (7, 3, 257)])
def test_route_shapes(H, K, T):
    lg = np.random.default_rng(H * 100 + K).standard_normal((3, T, H)).astype(np.float32)
    say(f"route shapes H={H} K={K} T={T}")
    r = L.route(torch.from_numpy(lg).to(DEV), K)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in r.items()}
    w = W.WORKLOADS[1].with_(B=3, T=T, H=H, K=K)
    assert_routing_exact(got, _oracle_routing({"logits": lg}, w))


@pytest.mark.parametrize("H,K,T", [(8, 2, 300), (32, 8, 1000), (64, 8, 700), (16, 9, 200),
                                   (64, 12, 130), (5, 5, 65)])
def test_route_biased_bit_exact(H, K, T):
    # loss-free balancing selection: biases of the size of the affinity gaps
    B = 2
    g = np.random.default_rng(100 + H + K)
    logits = g.standard_normal((B, T, H)).astype(np.float32)
    bias = (g.standard_normal(H) * (0.5 / H)).astype(np.float32)
    say(f"route biased H={H} K={K} T={T}")
    r = L.route(torch.from_numpy(logits).to(DEV), K, bias=torch.from_numpy(bias).to(DEV))
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in r.items()}
    topk, gates = O.select_heads_biased(logits, bias, K)
    n, off, perm, slot = O.permutation(topk, H)
    ref = {"topk_idx": topk, "gates": gates, "head_len": n, "seg_offsets": off,
           "perm_token": perm, "slot_pos": slot}
    assert_routing_exact(got, ref)
    # the bias changed the selection somewhere (the case is not vacuous)
    assert K == H or (topk != O.select_heads(logits, K)).any()


def test_route_biased_ties_and_bias_update():
    # equal logits and equal biases: every score ties, the lowest heads win
    B, T, H, K = 2, 100, 16, 4
    logits = np.zeros((B, T, H), np.float32)
    r = L.route(torch.from_numpy(logits).to(DEV), K, bias=torch.zeros(H, device=DEV))
    torch.cuda.synchronize()
    assert (r["topk_idx"].cpu().numpy() == np.arange(K)).all()
    np.testing.assert_allclose(r["gates"].cpu().numpy(), 1.0 / H, rtol=1e-6)
    # the bias step on a skewed batch, bit for bit, over several batches
    g = np.random.default_rng(7)
    bias = np.zeros(H, np.float32)
    bias_d = torch.zeros(H, device=DEV)
    for step in range(4):
        lg = (g.standard_normal((B, T, H)) + np.log(1.0 / (np.arange(H) + 1.0))).astype(np.float32)
        rr = L.route(torch.from_numpy(lg).to(DEV), K, bias=bias_d)
        L.route_bias_update(rr["head_len"], T, K, 0.01, bias_d)
        torch.cuda.synchronize()
        topk, _ = O.select_heads_biased(lg, bias, K)
        n = O.permutation(topk, H)[0]
        np.testing.assert_array_equal(rr["head_len"].cpu().numpy(), n)
        bias = O.bias_update(n, bias, 0.01, T, K)
        np.testing.assert_array_equal(bias_d.cpu().numpy(), bias)
    say(f"  bias after 4 steps: {bias.round(3).tolist()}")


def test_prefill_biased_routing():
    # the whole layer on a loss-free-balancing routing
    w = W.WORKLOADS[2].with_(B=2, T=900)
    say("prefill with biased routing")
    inp = W.prefill_inputs(w)
    bias = (np.random.default_rng(5).standard_normal(w.H) * 0.02).astype(np.float32)
    lg = torch.from_numpy(inp["logits"]).to(DEV)
    q, k, v = (to_dev(inp[x], w.dtype) for x in ("q", "k", "v"))
    r = L.route(lg, w.K, bias=torch.from_numpy(bias).to(DEV))
    o = L.attn_fwd(q, k, v, r, w.K, w.rope_base, out_dtype=torch.float32)
    torch.cuda.synchronize()
    f = _f64(inp, w)
    topk, gates = O.select_heads_biased(inp["logits"], bias, w.K)
    n, off, perm, slot = O.permutation(topk, w.H)
    np.testing.assert_array_equal(r["topk_idx"].cpu().numpy(), topk)
    hp = O.attention_gathered(f["q"], f["k"], f["v"], n, off, perm, w.H, w.rope_base)
    ref = O.combine_packed(hp, slot, gates)
    e = check_out(from_dev(o), ref, w.dtype)
    say(f"  max err {e:.2e}")


# ----------------------------------------------------------------------------
# backward (training path)

def _check_grad(got, ref, what, rel=2e-4, rel_l2=None):
    # within rel of the tensor's largest gradient plus rel of the element,
    # and (bf16 products) a relative L2 bound over the whole tensor
    got = np.asarray(got, dtype=np.float64)
    assert np.isfinite(got).all(), f"{what}: non-finite"
    scale = np.abs(ref).max() + 1e-30
    err = np.abs(got - ref)
    bad = err > rel * scale + rel * np.abs(ref)
    assert not bad.any(), f"{what}: {bad.sum()} elements off, max err {err.max():.3e} (scale {scale:.3e})"
    if rel_l2 is not None:
        l2 = np.linalg.norm(got - ref) / (np.linalg.norm(ref) + 1e-30)
        assert l2 <= rel_l2, f"{what}: relative L2 error {l2:.3e}"
    return float(err.max() / scale)


# Gradient tolerances.  fp32 path: fp32 arithmetic on exact inputs, sums of
# up to a few thousand terms.  bf16 MFMA path (d = 64, 128): the rotated
# q/k, the probabilities, dS and g*dout are rounded to bf16 (2^-9 relative
# each) before their products, accumulation in fp32; the errors are those of
# the forward's bf16 path, so the same bounds apply, taken relative to the
# tensor's largest gradient.
GRAD_TOL_F32 = dict(rel=2e-4)
GRAD_TOL_BF16 = dict(rel=2e-2, rel_l2=1e-2)


def _grad_tol(w):
    return GRAD_TOL_BF16 if w.dtype == "bf16" and w.d in (64, 128) else GRAD_TOL_F32


BWD = {
    "bf16_d64_rel": (W.WORKLOADS[2].with_(B=2, T=700, H=4, K=2), O.ROPE_HEAD_RELATIVE),
    "bf16_d128_global": (W.WORKLOADS[3].with_(B=1, T=900, H=4, K=2), O.ROPE_GLOBAL),
    "bf16_d128_rel": (W.WORKLOADS[3].with_(B=2, T=500, H=8, K=3), O.ROPE_HEAD_RELATIVE),
    "f32_d32_none": (W.WORKLOADS[1].with_(B=2, T=400, H=4, K=2), O.ROPE_NONE),
    "bf16_d32_rel": (W.WORKLOADS[1].with_(B=1, T=300, H=4, K=2, dtype="bf16"), O.ROPE_HEAD_RELATIVE),
    "bf16_d64_none": (W.WORKLOADS[2].with_(B=1, T=600, H=3, K=3), O.ROPE_NONE),
    "f32_d64_dense": (W.WORKLOADS[2].with_(B=1, T=300, H=4, K=4, dtype="f32"), O.ROPE_HEAD_RELATIVE),
    "skewed_long": (W.WORKLOADS[4].with_(B=1, T=1600, H=8, K=1), O.ROPE_HEAD_RELATIVE),
    # the balanced workload's shape with two sequences (64 segments of ~1024
    # rows), and 16 heads of ~4096 rows at d = 128
    "balanced_b2": (W.WORKLOADS[2].with_(B=2), O.ROPE_HEAD_RELATIVE),
    "long_d128": (W.WORKLOADS[3].with_(T=8192, H=16), O.ROPE_HEAD_RELATIVE),
    # long segments: query blocks far heavier than a workgroup's fair share
    # run as key-range parts (up to eight), on the query side summed by the
    # merge, on the key side taken once
    "parts_d64": (W.WORKLOADS[2].with_(B=1, T=4500, H=4, K=2), O.ROPE_HEAD_RELATIVE),
    "parts_d128_global": (W.WORKLOADS[3].with_(B=1, T=6000, H=2, K=1), O.ROPE_GLOBAL),
    # more (batch, head) segments than the packing and the key-side work list
    # stage in LDS (2112 > 2048): both search the offsets in global memory
    "many_segments_d64": (W.WORKLOADS[2].with_(B=33, T=64, H=64, K=2), O.ROPE_HEAD_RELATIVE),
    "many_segments_d128": (W.WORKLOADS[3].with_(B=33, T=96, H=64, K=4), O.ROPE_GLOBAL),
}


@pytest.mark.parametrize("name", list(BWD))
def test_attn_bwd_parity(name):
    w, rope_mode = BWD[name]
    say(f"backward {name}: {w}")
    inp = W.prefill_inputs(w)
    lg = torch.from_numpy(inp["logits"]).to(DEV)
    q, k, v = (to_dev(inp[x], w.dtype) for x in ("q", "k", "v"))
    r = L.route(lg, w.K)
    dout = np.random.default_rng(77).standard_normal((w.B, w.T, w.d)).astype(np.float32)
    g = L.attn_bwd(q, k, v, r, w.K, w.rope_base, torch.from_numpy(dout).to(DEV), rope_mode)
    torch.cuda.synchronize()
    f = _f64(inp, w)
    ref = _oracle_routing(inp, w)
    dq, dk, dv, dg = O.attention_backward(f["q"], f["k"], f["v"], ref["gates"], ref["seg_offsets"],
                                          ref["perm_token"], ref["slot_pos"], w.H, w.rope_base,
                                          dout.astype(np.float64), rope_mode)
    tol = _grad_tol(w)
    errs = [_check_grad(g["dq"].cpu().numpy(), dq, "dq", **tol),
            _check_grad(g["dk"].cpu().numpy(), dk, "dk", **tol),
            _check_grad(g["dv"].cpu().numpy(), dv, "dv", **tol),
            _check_grad(g["dgates"].cpu().numpy(), dg, "dgates", **tol)]
    say(f"  rel max err dq {errs[0]:.1e} dk {errs[1]:.1e} dv {errs[2]:.1e} dgates {errs[3]:.1e}")
    # rows of tokens not routed to the head are exactly zero
    m = O.membership(ref["topk_idx"], w.H).transpose(0, 2, 1)
    assert not g["dq"].cpu().numpy()[~m].any()


@pytest.mark.parametrize("name", ["bf16_d64_rel", "bf16_d128_global", "f32_d32_none",
                                  "bf16_d32_rel", "balanced_b2", "long_d128", "parts_d64",
                                  "many_segments_d128"])
def test_attn_bwd_packed(name):
    # namoh_attn_bwd_packed: the routed pairs' gradients in the routing's
    # packed order, against the oracle's gradients at those pairs, and bit
    # for bit the dense call's rows gathered at the same pairs
    w, rope_mode = BWD[name]
    say(f"backward, packed gradients {name}: {w}")
    inp = W.prefill_inputs(w)
    lg = torch.from_numpy(inp["logits"]).to(DEV)
    q, k, v = (to_dev(inp[x], w.dtype) for x in ("q", "k", "v"))
    r = L.route(lg, w.K)
    dout = np.random.default_rng(77).standard_normal((w.B, w.T, w.d)).astype(np.float32)
    dd = torch.from_numpy(dout).to(DEV)
    gp = L.attn_bwd(q, k, v, r, w.K, w.rope_base, dd, rope_mode, packed=True)
    gd = L.attn_bwd(q, k, v, r, w.K, w.rope_base, dd, rope_mode)
    torch.cuda.synchronize()
    off = r["seg_offsets"].cpu().numpy().astype(np.int64)
    perm = r["perm_token"].cpu().numpy().astype(np.int64)
    seg = np.repeat(np.arange(w.B * w.H), np.diff(off))
    bb, hh = seg // w.H, seg % w.H
    f = _f64(inp, w)
    ref = _oracle_routing(inp, w)
    dq, dk, dv, dg = O.attention_backward(f["q"], f["k"], f["v"], ref["gates"], ref["seg_offsets"],
                                          ref["perm_token"], ref["slot_pos"], w.H, w.rope_base,
                                          dout.astype(np.float64), rope_mode)
    tol = _grad_tol(w)
    for key, full in (("dq", dq), ("dk", dk), ("dv", dv)):
        got = gp[key].cpu().numpy()
        assert got.shape == (w.B * w.T * w.K, w.d)
        _check_grad(got, full[bb, hh, perm], key, **tol)
        np.testing.assert_array_equal(got, gd[key].cpu().numpy()[bb, hh, perm], err_msg=key)
    np.testing.assert_array_equal(gp["dgates"].cpu().numpy(), gd["dgates"].cpu().numpy())
    _check_grad(gp["dgates"].cpu().numpy(), dg, "dgates", **tol)


@pytest.mark.parametrize("name", ["bf16_d64_rel", "bf16_d128_global", "bf16_d128_rel",
                                  "bf16_d64_none", "balanced_b2", "long_d128", "parts_d64",
                                  "parts_d128_global", "many_segments_d64"])
def test_attn_train_saved(name):
    # namoh_attn_fwd_train: the layer output against the oracle; then
    # namoh_attn_bwd_saved on its workspace: bit for bit the gradients of the
    # stateless calls (dense and packed), which rerun the forward themselves
    w, rope_mode = BWD[name]
    say(f"training forward + saved backward {name}: {w}")
    inp = W.prefill_inputs(w)
    lg = torch.from_numpy(inp["logits"]).to(DEV)
    q, k, v = (to_dev(inp[x], w.dtype) for x in ("q", "k", "v"))
    r = L.route(lg, w.K)
    dout = np.random.default_rng(77).standard_normal((w.B, w.T, w.d)).astype(np.float32)
    dd = torch.from_numpy(dout).to(DEV)
    ws = L.workspace(int(L.lib().namoh_attn_bwd_workspace_size(w.B, w.T, w.H, w.K, w.d)), DEV)
    o = L.attn_fwd_train(q, k, v, r, w.K, w.rope_base, ws, rope_mode, out_dtype=torch.float32)
    gs = L.attn_bwd(q, k, v, r, w.K, w.rope_base, dd, rope_mode, ws=ws, saved=True)
    gsp = L.attn_bwd(q, k, v, r, w.K, w.rope_base, dd, rope_mode, ws=ws, saved=True, packed=True)
    gd = L.attn_bwd(q, k, v, r, w.K, w.rope_base, dd, rope_mode)
    gp = L.attn_bwd(q, k, v, r, w.K, w.rope_base, dd, rope_mode, packed=True)
    torch.cuda.synchronize()
    for key in ("dq", "dk", "dv", "dgates"):
        np.testing.assert_array_equal(gs[key].cpu().numpy(), gd[key].cpu().numpy(), err_msg=key)
        np.testing.assert_array_equal(gsp[key].cpu().numpy(), gp[key].cpu().numpy(),
                                      err_msg=key)
    ref = _oracle_routing(inp, w)
    f = _f64(inp, w)
    hp = O.attention_gathered(f["q"], f["k"], f["v"], ref["head_len"], ref["seg_offsets"],
                              ref["perm_token"], w.H, w.rope_base, rope_mode)
    want = O.combine_packed(hp, ref["slot_pos"], ref["gates"])
    e = check_out(o.cpu().numpy().astype(np.float64), want, w.dtype)
    say(f"  output max err {e:.2e}")


@pytest.mark.parametrize("gate_mode", [O.GATE_SOFTMAX_SELECTED, O.GATE_SOFTMAX_ALL])
def test_route_bwd_parity(gate_mode):
    # router gradient fed by the GPU's own gate gradients (the training chain)
    w = W.WORKLOADS[2].with_(B=2, T=300)
    say(f"route backward gate_mode={gate_mode}")
    inp = W.prefill_inputs(w)
    lg = torch.from_numpy(inp["logits"]).to(DEV)
    q, k, v = (to_dev(inp[x], w.dtype) for x in ("q", "k", "v"))
    r = L.route(lg, w.K, gate_mode)
    dout = np.random.default_rng(78).standard_normal((w.B, w.T, w.d)).astype(np.float32)
    g = L.attn_bwd(q, k, v, r, w.K, w.rope_base, torch.from_numpy(dout).to(DEV))
    dl = L.route_bwd(lg, r, g["dgates"], gate_mode)
    torch.cuda.synchronize()
    f = _f64(inp, w)
    ref = _oracle_routing(inp, w, gate_mode)
    _, _, _, dg = O.attention_backward(f["q"], f["k"], f["v"], ref["gates"], ref["seg_offsets"],
                                       ref["perm_token"], ref["slot_pos"], w.H, w.rope_base,
                                       dout.astype(np.float64))
    dl_ref = O.gates_backward(inp["logits"], ref["topk_idx"], dg, gate_mode)
    e = _check_grad(dl.cpu().numpy(), dl_ref, "dlogits", **_grad_tol(w))
    say(f"  rel max err dlogits {e:.1e}")


# ----------------------------------------------------------------------------
# prefill: whole outputs at sizes the oracle finishes quickly

MID = {
    "tiny_fp32_full": W.WORKLOADS[1],
    "balanced_d64_mid": W.WORKLOADS[2].with_(B=2, T=1500),
    "long_d128_mid": W.WORKLOADS[3].with_(T=2600, H=16),
    "skewed_d128_mid": W.WORKLOADS[4].with_(B=1, T=3000),
    "peaky_d128": W.WORKLOADS[3].with_(T=1100, H=8, K=3, qkv_scale=1.0),
    "peaky_d64": W.WORKLOADS[2].with_(B=1, T=900, qkv_scale=1.0),
    "fp32_d64": W.WORKLOADS[2].with_(B=1, T=700, dtype="f32"),
    "fp32_d128": W.WORKLOADS[3].with_(T=600, H=8, dtype="f32"),
    "bf16_d32": W.WORKLOADS[1].with_(T=800, dtype="bf16"),
    # more than 1024 (batch, head) segments: segment offsets read from global
    # memory by the work list and the packing (not staged in LDS)
    "many_segments_d64": W.WORKLOADS[2].with_(B=20, T=300, H=64, K=4),
    "many_segments_d128": W.WORKLOADS[3].with_(B=20, T=300, K=4),
}


@pytest.mark.parametrize("name", list(MID))
def test_prefill_parity_mid(name):
    w = MID[name]
    say(f"prefill mid: {name} {w}")
    inp = W.prefill_inputs(w)
    got = run_prefill(w, inp, head_out=True)
    f = _f64(inp, w)
    ref = O.prefill(inp["logits"], f["q"], f["k"], f["v"], w.K, w.rope_base)
    assert_routing_exact(got, ref)
    e1 = check_out(got["out"], ref["out"], w.dtype)
    e2 = check_out(got["head_out"], ref["head_out"], w.dtype, "head_out")
    say(f"  max err out {e1:.2e} head_out {e2:.2e}")


@pytest.mark.parametrize("rope_mode", [O.ROPE_GLOBAL, O.ROPE_NONE])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_prefill_rope_modes(rope_mode, dtype):
    w = W.WORKLOADS[3].with_(T=1000, H=8, K=2, dtype=dtype, rope_base=1e4)
    say(f"prefill rope_mode={rope_mode} dtype={dtype}")
    inp = W.prefill_inputs(w)
    got = run_prefill(w, inp, rope_mode=rope_mode)
    f = _f64(inp, w)
    ref = O.prefill(inp["logits"], f["q"], f["k"], f["v"], w.K, w.rope_base, rope_mode)
    check_out(got["out"], ref["out"], dtype)


def test_prefill_gate_all_and_bf16_out():
    w = W.WORKLOADS[2].with_(B=1, T=777)
    say("prefill gate_mode=ALL, bf16 output")
    inp = W.prefill_inputs(w)
    got = run_prefill(w, inp, gate_mode=O.GATE_SOFTMAX_ALL, out_dtype=torch.bfloat16)
    f = _f64(inp, w)
    ref = O.prefill(inp["logits"], f["q"], f["k"], f["v"], w.K, w.rope_base,
                    gate_mode=O.GATE_SOFTMAX_ALL)
    check_out(got["out"], ref["out"], "bf16")


@pytest.mark.parametrize("dtype,d", [("bf16", 64), ("bf16", 128), ("f32", 32)])
def test_prefill_edge_cases(dtype, d):
    # T = 1; K = H (dense causal attention); one head; every token on the
    # same K heads (empty segments); a length that is not a tile multiple.
    cases = [dict(T=1, H=4, K=2), dict(T=200, H=4, K=4), dict(T=65, H=1, K=1),
             dict(T=321, H=8, K=3, same=True), dict(T=127, H=5, K=2)]
    for c in cases:
        same = c.pop("same", False)
        w = W.WORKLOADS[2].with_(B=2, d=d, dtype=dtype, qkv_scale=d ** -0.5, **c)
        say(f"prefill edge {dtype} d={d} {c} same_heads={same}")
        inp = W.prefill_inputs(w)
        if same:
            inp["logits"] = inp["logits"].copy()
            inp["logits"][:, :, :w.K] += 100.0
        got = run_prefill(w, inp, head_out=True)
        f = _f64(inp, w)
        ref = O.prefill(inp["logits"], f["q"], f["k"], f["v"], w.K, w.rope_base)
        assert_routing_exact(got, ref)
        check_out(got["out"], ref["out"], dtype)


@pytest.mark.parametrize("d,K,scale", [(64, 2, None), (128, 1, None), (128, 1, 1.0),
                                        (64, 1, 1.0)])
def test_prefill_long_segment(d, K, scale):
    # Every token on the same K heads: one 4500-row segment per head (ragged
    # last tile, query blocks of up to 71 key tiles) and empty segments for
    # the others; both head-output paths (fp32 rows handed in, bf16 internal
    # rows), and two runs that agree bit for bit.  The few heavy query blocks
    # far exceed a workgroup's fair share of the work, so they run as up to 8
    # key-range parts merged afterwards; scale 1.0 gives peaky scores, so the
    # parts take the exact-maximum path and their running maxima differ.
    w = W.WORKLOADS[2 if d == 64 else 4].with_(B=1, T=4500, H=4, K=K, d=d,
                                               qkv_scale=d ** -0.5 if scale is None else scale,
                                               zipf_bias=0.0)
    say(f"prefill long segment d={d} K={K} scale={scale}")
    inp = W.prefill_inputs(w)
    inp["logits"] = inp["logits"].copy()
    inp["logits"][:, :, :K] += 100.0
    f = _f64(inp, w)
    ref = O.prefill(inp["logits"], f["q"], f["k"], f["v"], w.K, w.rope_base)
    got = run_prefill(w, inp, head_out=True)
    assert_routing_exact(got, ref)
    e1 = check_out(got["out"], ref["out"], w.dtype)
    e2 = check_out(got["head_out"], ref["head_out"], w.dtype, "head_out")
    got2 = run_prefill(w, inp)
    e3 = check_out(got2["out"], ref["out"], w.dtype)
    got3 = run_prefill(w, inp)
    np.testing.assert_array_equal(got2["out"], got3["out"])
    say(f"  max err out {e1:.2e} head_out {e2:.2e} out(bf16 rows) {e3:.2e}")


@pytest.mark.parametrize("dtype,d,rope_mode", [("bf16", 64, O.ROPE_HEAD_RELATIVE),
                                                ("bf16", 128, O.ROPE_GLOBAL),
                                                ("bf16", 128, O.ROPE_NONE),
                                                ("f32", 32, O.ROPE_HEAD_RELATIVE)])
def test_prefill_cache_then_decode(dtype, d, rope_mode):
    # prompt of T tokens -> route, attention, hand-off to the decode caches;
    # the caches against the oracle's (keys within the rounding of one
    # rotation, values and lengths exact), then one GPU decode step for token
    # T against the oracle's prefill of T + 1 tokens at that token
    T, cap = 700, 720
    w = W.WORKLOADS[2].with_(B=2, T=T + 1, H=8, K=2, d=d, dtype=dtype, qkv_scale=d ** -0.5)
    say(f"prefill -> cache -> decode {dtype} d={d} rope_mode={rope_mode}")
    inp = W.prefill_inputs(w)
    wp = w.with_(T=T)
    pin = {"logits": np.ascontiguousarray(inp["logits"][:, :T])}
    for x in ("q", "k", "v"):
        pin[x] = np.ascontiguousarray(inp[x][:, :, :T])
    lg = torch.from_numpy(pin["logits"]).to(DEV)
    q, k, v = (to_dev(pin[x], dtype) for x in ("q", "k", "v"))
    r = L.route(lg, w.K)
    L.attn_fwd(q, k, v, r, w.K, w.rope_base, rope_mode)
    tdt = k.dtype
    kc = torch.zeros(w.B, w.H, cap, d, dtype=tdt, device=DEV)
    vc = torch.zeros(w.B, w.H, cap, d, dtype=tdt, device=DEV)
    cl = torch.full((w.B, w.H), -7, dtype=torch.int32, device=DEV)
    L.prefill_cache(k, v, r, w.K, w.rope_base, kc, vc, cl, rope_mode)
    torch.cuda.synchronize()
    f = _f64(pin, wp)
    topk = O.select_heads(pin["logits"], w.K)
    rk, rv, rn = O.prefill_cache(f["k"], f["v"], topk, w.H, w.rope_base, rope_mode)
    np.testing.assert_array_equal(cl.cpu().numpy(), rn)
    kcg, vcg = from_dev(kc), from_dev(vc)
    for b in range(w.B):
        for h in range(w.H):
            n = int(rn[b, h])
            gk = np.asarray(kcg[b, h, :n], dtype=np.float64)
            tol = 2.0 ** -8 * np.abs(rk[b, h, :n]) + 1e-6 if dtype == "bf16" else 2e-6
            assert (np.abs(gk - rk[b, h, :n]) <= tol).all(), f"k cache b={b} h={h}"
            np.testing.assert_array_equal(np.asarray(vcg[b, h, :n], dtype=np.float64), rv[b, h, :n])
            assert not np.asarray(kcg[b, h, n:], dtype=np.float64).any()   # rows past n untouched
    # one decode step for token T
    lg1 = torch.from_numpy(np.ascontiguousarray(inp["logits"][:, T])).to(DEV)
    q1, k1, v1 = (to_dev(np.ascontiguousarray(inp[x][:, :, T]), dtype) for x in ("q", "k", "v"))
    seq_pos = torch.full((w.B,), T, dtype=torch.int32, device=DEV) if rope_mode == O.ROPE_GLOBAL else None
    res = L.decode_step(lg1, q1, k1, v1, kc, vc, cl, w.K, w.rope_base, rope_mode, seq_pos=seq_pos,
                        out_dtype=torch.float32)
    torch.cuda.synchronize()
    topk_full = O.select_heads(inp["logits"], w.K)
    g_full = O.route_gates(inp["logits"], topk_full, O.GATE_SOFTMAX_SELECTED)
    ff = _f64(inp, w)
    for b in range(w.B):
        o, _ = O.prefill_rows(ff["q"], ff["k"], ff["v"], topk_full, g_full, w.H, w.rope_base, b,
                              [T], rope_mode)
        e = check_out(from_dev(res["out"])[b:b + 1], o, dtype)
        say(f"  b={b} decode after hand-off: max err {e:.2e}")


def test_biased_prefill_cache_then_biased_decode():
    # loss-free balancing end to end: biased routing of the prompt, hand-off,
    # one biased decode step against the oracle's biased layer at token T
    T, cap = 500, 512
    w = W.WORKLOADS[3].with_(B=3, T=T + 1, H=16, K=4)
    say("biased prefill -> cache -> biased decode")
    inp = W.prefill_inputs(w)
    bias = (np.random.default_rng(9).standard_normal(w.H) * 0.03).astype(np.float32)
    bias_d = torch.from_numpy(bias).to(DEV)
    lg = torch.from_numpy(np.ascontiguousarray(inp["logits"][:, :T])).to(DEV)
    k, v = (to_dev(np.ascontiguousarray(inp[x][:, :, :T]), w.dtype) for x in ("k", "v"))
    r = L.route(lg, w.K, bias=bias_d)
    kc = torch.zeros(w.B, w.H, cap, w.d, dtype=k.dtype, device=DEV)
    vc = torch.zeros_like(kc)
    cl = torch.zeros(w.B, w.H, dtype=torch.int32, device=DEV)
    L.prefill_cache(k, v, r, w.K, w.rope_base, kc, vc, cl)
    lg1 = torch.from_numpy(np.ascontiguousarray(inp["logits"][:, T])).to(DEV)
    q1, k1, v1 = (to_dev(np.ascontiguousarray(inp[x][:, :, T]), w.dtype) for x in ("q", "k", "v"))
    res = L.decode_step(lg1, q1, k1, v1, kc, vc, cl, w.K, w.rope_base, out_dtype=torch.float32,
                        bias=bias_d)
    torch.cuda.synchronize()
    topk, gates = O.select_heads_biased(inp["logits"], bias, w.K)
    np.testing.assert_array_equal(res["topk_idx"].cpu().numpy(), topk[:, T])
    np.testing.assert_allclose(res["gates"].cpu().numpy(), gates[:, T], rtol=2e-6, atol=1e-7)
    ff = _f64(inp, w)
    for b in range(w.B):
        o, _ = O.prefill_rows(ff["q"], ff["k"], ff["v"], topk, gates, w.H, w.rope_base, b, [T])
        e = check_out(from_dev(res["out"])[b:b + 1], o, w.dtype)
        say(f"  b={b} max err {e:.2e}")


def test_prefill_deterministic():
    w = W.WORKLOADS[4].with_(B=1, T=2048)
    say("prefill determinism")
    inp = W.prefill_inputs(w)
    a = run_prefill(w, inp, head_out=True)
    b = run_prefill(w, inp, head_out=True)
    np.testing.assert_array_equal(a["out"], b["out"])
    np.testing.assert_array_equal(a["head_out"], b["head_out"])


# ----------------------------------------------------------------------------
# prefill at the full workload sizes: every index and every output row

class _Rows:
    """Lazy float64 view of a dense [B,H,T,d] input, converted per (b, h)."""

    def __init__(self, x, dtype):
        self.x, self.dtype, self.cache = x, dtype, {}
        self.shape = x.shape

    def __getitem__(self, bh):
        if bh not in self.cache:
            self.cache[bh] = W.as_float64(self.x[bh], self.dtype)
        return self.cache[bh]


def _oracle_by_segment(inp, w, ref):
    """The gathered oracle (O2) run one (batch, head) segment at a time, each
    segment's rows converted to float64 on their own (the whole float64
    tensors of the long workloads would take gigabytes); segments run in a
    thread pool (numpy releases the interpreter lock in its kernels)."""
    off, perm = ref["seg_offsets"], ref["perm_token"]
    hp = np.zeros((int(off[-1]), w.d))

    def seg(sid):
        b, h = divmod(sid, w.H)
        a, e = int(off[sid]), int(off[sid + 1])
        if e == a:
            return
        sub = {x: W.as_float64(inp[x][b:b + 1, h:h + 1], w.dtype) for x in ("q", "k", "v")}
        hp[a:e] = O.attention_gathered(sub["q"], sub["k"], sub["v"], None,
                                       np.array([0, e - a]), perm[a:e], 1, w.rope_base)

    with ThreadPoolExecutor(max(1, min(16, len(os.sched_getaffinity(0))))) as ex:
        list(ex.map(seg, range(w.B * w.H)))
    return hp, O.combine_packed(hp, ref["slot_pos"], ref["gates"])


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_prefill_full_size_elementwise(cfg):
    # Every output row and every ungated head-output row of the full
    # workload against the gathered oracle: all work items of the heaviest-
    # first schedule, including the items past the resident workgroup slots
    # and the reversed (serpentine) blocks of ranks.
    w = W.WORKLOADS[cfg]
    say(f"prefill full size, element-wise: {w.name}")
    inp = W.prefill_inputs(w)
    ref = _oracle_routing(inp, w)
    # the benchmark's launch: bf16 output, head rows kept in bf16 inside
    got = run_prefill(w, inp, out_dtype=torch.bfloat16)
    assert_routing_exact(got, ref)
    hp, o = _oracle_by_segment(inp, w, ref)
    e1 = check_out(got["out"], o, w.dtype)
    # float32 head rows handed in by the caller
    got2 = run_prefill(w, inp, head_out=True)
    assert_routing_exact(got2, ref)
    e2 = check_out(got2["head_out"], hp, w.dtype, "head_out")
    e3 = check_out(got2["out"], o, w.dtype)
    say(f"  max err out(bf16) {e1:.2e} head_out {e2:.2e} out(f32) {e3:.2e}")
    # a sample of tokens from the one-token-at-a-time form, an independent
    # evaluation of the same definition
    g = np.random.default_rng(cfg)
    for b in range(w.B):
        toks = sorted(set([0, 1, w.T - 1] + list(g.choice(w.T, 5, replace=False))))
        o1, _ = O.prefill_rows(_Rows(inp["q"], w.dtype), _Rows(inp["k"], w.dtype),
                               _Rows(inp["v"], w.dtype), ref["topk_idx"], ref["gates"],
                               w.H, w.rope_base, b, toks)
        check_out(got2["out"][b, toks], o1, w.dtype)


# ----------------------------------------------------------------------------
# decode

def _decode_case(w, lengths, cap, seed=0):
    """Host caches (numpy) for a small decode test."""
    B, H, d = w.B, w.H, w.d
    kc = np.zeros((B, H, cap, d), W.storage_dtype(w.dtype))
    vc = np.zeros_like(kc)
    for b in range(B):
        for h in range(H):
            kc[b, h] = W.decode_cache_block(w, b, h, cap, "k")
            vc[b, h] = W.decode_cache_block(w, b, h, cap, "v")
    return kc, vc


def _run_decode(w, step, kc, vc, lengths, rope_mode=0, gate_mode=0, seq_pos=None):
    dt = w.dtype
    kcd, vcd = to_dev(kc, dt), to_dev(vc, dt)
    cl = torch.from_numpy(lengths.astype(np.int32)).to(DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    sp = None if seq_pos is None else torch.from_numpy(seq_pos.astype(np.int32)).to(DEV)
    res = L.decode_step(torch.from_numpy(step["logits"]).to(DEV), to_dev(step["q"], dt),
                        to_dev(step["k"], dt), to_dev(step["v"], dt), kcd, vcd, cl, w.K,
                        w.rope_base, rope_mode, gate_mode, seq_pos=sp,
                        out_dtype=torch.float32, dev_status=st)
    torch.cuda.synchronize()
    return res, kcd, vcd, cl, st


@pytest.mark.parametrize("dtype,d,rope_mode,gate_mode", [
    ("bf16", 128, 0, 0), ("bf16", 64, 0, 1), ("f32", 32, 0, 0), ("bf16", 128, 1, 0),
    ("f32", 128, 2, 0), ("bf16", 32, 0, 0)])
def test_decode_parity_small(dtype, d, rope_mode, gate_mode):
    w = W.WORKLOADS[5].with_(B=5, H=12, K=4, d=d, dtype=dtype, qkv_scale=d ** -0.5)
    g = np.random.default_rng(d + rope_mode)
    lengths = g.integers(0, 1300, size=(w.B, w.H))
    lengths[0, :] = 0
    cap = 1400
    say(f"decode small {dtype} d={d} rope={rope_mode} gate={gate_mode}")
    kc, vc = _decode_case(w, lengths, cap)
    step = W.decode_step_inputs(w)
    seq_pos = g.integers(1000, 5000, size=w.B) if rope_mode == 1 else None
    res, kcd, vcd, cl, st = _run_decode(w, step, kc, vc, lengths, rope_mode, gate_mode, seq_pos)
    kf, vf = W.as_float64(kc, dtype), W.as_float64(vc, dtype)
    sf = {k: W.as_float64(step[k], dtype) for k in ("q", "k", "v")}
    ref = O.decode_step(step["logits"], sf["q"], sf["k"], sf["v"],
                        lambda b, h, n: kf[b, h, :n], lambda b, h, n: vf[b, h, :n],
                        lengths, w.K, w.rope_base, rope_mode, gate_mode, seq_pos=seq_pos)
    np.testing.assert_array_equal(res["topk_idx"].cpu().numpy(), ref["topk_idx"])
    np.testing.assert_allclose(res["gates"].cpu().numpy(), ref["gates"], rtol=2e-6, atol=1e-7)
    np.testing.assert_array_equal(cl.cpu().numpy(), ref["cache_len"])
    assert int(st.item()) == 0
    check_out(from_dev(res["out"]), ref["out"], dtype)
    # the appended rows: rotated key (rounded to the cache dtype) and value
    kd, vd = from_dev(kcd), from_dev(vcd)
    for b in range(w.B):
        for kk in range(w.K):
            h = ref["topk_idx"][b, kk]
            n = lengths[b, h]
            check_out(kd[b, h, n], ref["new_k"][b, kk], dtype, "appended key")
            np.testing.assert_array_equal(vd[b, h, n], sf["v"][b, h])
            np.testing.assert_array_equal(kd[b, h, :n], kf[b, h, :n])     # history untouched


def test_decode_isolation_and_overflow():
    w = W.WORKLOADS[5].with_(B=4, H=10, K=3, d=128)
    lengths = np.random.default_rng(3).integers(1, 600, size=(w.B, w.H))
    cap = 640
    kc, vc = _decode_case(w, lengths, cap)
    step = W.decode_step_inputs(w)
    topk = O.select_heads(step["logits"], w.K)
    say("decode isolation")
    r1, *_ = _run_decode(w, step, kc, vc, lengths)
    kc2, vc2 = kc.copy(), vc.copy()
    for b in range(w.B):
        for h in range(w.H):
            if h not in topk[b]:
                kc2[b, h] = W.f32_to_bf16_bits(np.full((cap, w.d), 3.0, np.float32))
                vc2[b, h] = W.f32_to_bf16_bits(np.full((cap, w.d), -7.0, np.float32))
    r2, *_ = _run_decode(w, step, kc2, vc2, lengths)
    np.testing.assert_array_equal(r1["out"].cpu().numpy(), r2["out"].cpu().numpy())
    # a full head: status set, its cache untouched, it contributes nothing
    say("decode capacity overflow")
    l3 = lengths.copy()
    h_full = topk[1, 0]
    l3[1, h_full] = cap
    r3, kcd, vcd, cl, st = _run_decode(w, step, kc, vc, l3)
    assert int(st.item()) == 1
    assert cl.cpu().numpy()[1, h_full] == cap
    kf, vf = W.as_float64(kc, "bf16"), W.as_float64(vc, "bf16")
    sf = {k: W.as_float64(step[k], "bf16") for k in ("q", "k", "v")}
    l_or = l3.copy()
    l_or[1, h_full] = cap - 1        # oracle stand-in; its head output is dropped below
    ref = O.decode_step(step["logits"], sf["q"], sf["k"], sf["v"],
                        lambda b, h, n: kf[b, h, :n], lambda b, h, n: vf[b, h, :n],
                        l_or, w.K, w.rope_base)
    exp = ref["out"].copy()
    exp[1] -= ref["gates"][1, 0] * ref["head_out"][1, 0]
    check_out(r3["out"].cpu().numpy(), exp, "bf16")


def test_decode_full_size():
    w = W.WORKLOADS[5]
    say(f"decode full size: {w.name}")
    from paper_2609_38832_amd import device_inputs as DI
    lengths = W.decode_prior_lengths(w)
    cap = W.decode_cache_capacity(lengths)
    kc, vc = DI.decode_caches(w.B, w.H, cap, w.d, w.dtype, w.seed, w.qkv_scale, DEV)
    step = W.decode_step_inputs(w)
    topk = O.select_heads(step["logits"], w.K)
    # host copies of the rows the step reads, taken before the step runs
    hist = {}
    for b in range(w.B):
        for h in topk[b]:
            n = int(lengths[b, h])
            hist[(b, int(h))] = (from_dev(kc[b, h, :n]), from_dev(vc[b, h, :n]))
    say("  caches ready, running the step")
    cl = torch.from_numpy(lengths).to(DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    res = L.decode_step(torch.from_numpy(step["logits"]).to(DEV), to_dev(step["q"], "bf16"),
                        to_dev(step["k"], "bf16"), to_dev(step["v"], "bf16"), kc, vc, cl, w.K,
                        w.rope_base, out_dtype=torch.float32, dev_status=st)
    torch.cuda.synchronize()
    sf = {k: W.as_float64(step[k], "bf16") for k in ("q", "k", "v")}
    ref = O.decode_step(step["logits"], sf["q"], sf["k"], sf["v"],
                        lambda b, h, n: hist[(b, h)][0], lambda b, h, n: hist[(b, h)][1],
                        lengths, w.K, w.rope_base)
    np.testing.assert_array_equal(res["topk_idx"].cpu().numpy(), ref["topk_idx"])
    np.testing.assert_array_equal(cl.cpu().numpy(), ref["cache_len"])
    assert int(st.item()) == 0
    e = check_out(res["out"].cpu().numpy(), ref["out"], "bf16")
    say(f"  max err {e:.2e}")
    del kc, vc
    torch.cuda.empty_cache()
