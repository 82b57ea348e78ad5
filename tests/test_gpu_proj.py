"""GPU parity of the routed projections (Eq. namoh-qkv; output aggregation
of Eq. namoh-attention with W_O^(i) kept) through the C ABI, against the
float64 oracle.

Tolerance: the bf16 bound of the other parity tests, |got - ref| <= 2e-2 +
1e-2 |ref| and relative L2 <= 1e-2 (operands are bf16, products accumulate
in fp32; the only roundings are the bf16 results, 2^-9 relative, and for the
output projection the bf16 per-pair rows before the gated sum).
"""
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


from gpu_util import DEV, check_out, from_dev, say, to_dev  # noqa: E402
from paper_2609_38832_amd import _lib as L  # noqa: E402

SENTINEL = 12288.0   # exact in bf16 (3 * 2^12); rows the projection must not touch keep it

CASES = {
    "d64_dm256": dict(B=2, T=300, H=8, K=2, d=64, d_model=256),
    "d128_dm384_ragged": dict(B=1, T=257, H=5, K=3, d=128, d_model=384),
    "all_heads": dict(B=2, T=200, H=4, K=4, d=64, d_model=128),
    "one_head": dict(B=1, T=130, H=1, K=1, d=64, d_model=128),
    # H d > 384 K: the per-pair form of the output projection
    "pairs_d64_h16_k2": dict(B=2, T=200, H=16, K=2, d=64, d_model=256),
    "pairs_d128_h8_k2_ragged": dict(B=1, T=333, H=8, K=2, d=128, d_model=384),
    # more than 1024 (b, h) segments: segment offsets read from global memory
    "many_segments_dense": dict(B=17, T=40, H=64, K=11, d=64, d_model=128),
    "many_segments_pairs": dict(B=20, T=70, H=64, K=4, d=64, d_model=128),
    # K > 32, d = 128
    "k40_d128": dict(B=2, T=150, H=64, K=40, d=128, d_model=256),
}


def _dense_form(w):
    # the library's choice between the dense and the per-pair output projection
    return w.H * w.d <= 384 * w.K and w.H <= 64


def _case(name):
    return W.WORKLOADS[6].with_(**CASES[name])


def _f64(bits):
    return W.as_float64(bits, "bf16")


def _route(inp, w):
    lg = torch.from_numpy(inp["logits"]).to(DEV)
    r = L.route(lg, w.K)
    topk = O.select_heads(inp["logits"], w.K)
    np.testing.assert_array_equal(r["topk_idx"].cpu().numpy(), topk)
    return r, topk


@pytest.mark.parametrize("name", list(CASES))
def test_qkv_proj_parity(name):
    w = _case(name)
    say(f"qkv projection {name}: {w}")
    inp = W.projection_inputs(w)
    r, topk = _route(inp, w)
    x, wq = to_dev(inp["x"], "bf16"), to_dev(inp["w_qkv"], "bf16")
    out = {n: torch.full((w.B, w.H, w.T, w.d), SENTINEL, dtype=torch.bfloat16, device=DEV)
           for n in ("q", "k", "v")}
    L.qkv_proj(x, wq, r, w.H, w.K, out=out)
    torch.cuda.synchronize()
    rq, rk, rv, m = O.qkv_projection(_f64(inp["x"]), _f64(inp["w_qkv"]), topk)
    routed = m.transpose(0, 2, 1)               # [B, H, T]
    for n, ref in (("q", rq), ("k", rk), ("v", rv)):
        got = from_dev(out[n])
        check_out(got[routed], ref[routed], "bf16", what=f"{name} {n}")
        assert (got[~routed] == SENTINEL).all(), f"{name} {n}: an unrouted row was written"


def _packed_to_dense(hp, topk, H, T, d):
    B = topk.shape[0]
    n, off, perm, slot = O.permutation(topk, H)
    h = np.full((B, H, T, d), np.nan)
    for sid in range(B * H):
        b, i = divmod(sid, H)
        a, e = int(off[sid]), int(off[sid + 1])
        h[b, i, perm[a:e]] = hp[a:e]
    return h


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("hdt,odt", [("f32", torch.float32), ("bf16", torch.bfloat16)])
def test_out_proj_parity(name, hdt, odt):
    w = _case(name)
    form = "dense" if _dense_form(w) else "per-pair"
    say(f"output projection {name} ({form} form) head_out={hdt} out={odt}")
    ws_bytes = L.out_proj_workspace_size(w.B, w.T, w.H, w.K, w.d, w.d_model)
    need = (w.B * w.T * w.H * 4 + w.B * w.T * w.K * w.d * 2 if form == "dense"
            else w.B * w.T * w.K * w.d_model * 2)
    assert need <= ws_bytes < need + 4096
    inp = W.projection_inputs(w)
    r, topk = _route(inp, w)
    Nr = w.B * w.T * w.K
    hp = np.random.default_rng(17).standard_normal((Nr, w.d)).astype(np.float32)
    if hdt == "bf16":
        hp_bits = W.f32_to_bf16_bits(hp)
        hdev, hp64 = to_dev(hp_bits, "bf16"), _f64(hp_bits)
    else:
        hdev, hp64 = to_dev(hp, "f32"), hp.astype(np.float64)
    wo = to_dev(inp["w_o"], "bf16")
    o = L.out_proj(hdev, wo, r, w.B, w.T, w.H, w.K, out_dtype=odt)
    torch.cuda.synchronize()
    gates = r["gates"].cpu().numpy().astype(np.float64)
    ref = O.output_projection(_packed_to_dense(hp64, topk, w.H, w.T, w.d), topk, gates,
                              _f64(inp["w_o"]))
    check_out(from_dev(o), ref, "bf16", what=f"{name} out_proj")


@pytest.mark.parametrize("K", [2, 3])   # per-pair form, dense form
def test_out_proj_skewed_routing(K):
    # a few heads take most tokens: segments of very different lengths
    w = _case("pairs_d64_h16_k2").with_(T=700, K=K)
    say(f"output projection, skewed routing ({'dense' if _dense_form(w) else 'per-pair'}): {w}")
    inp = W.projection_inputs(w)
    inp["logits"][..., :2] += 2.5
    r, topk = _route(inp, w)
    n = np.bincount(topk.reshape(-1), minlength=w.H)
    assert n.max() > 4 * max(1, n.min())
    Nr = w.B * w.T * w.K
    hp_bits = W.f32_to_bf16_bits(np.random.default_rng(18).standard_normal((Nr, w.d)).astype(np.float32))
    wo = to_dev(inp["w_o"], "bf16")
    o = L.out_proj(to_dev(hp_bits, "bf16"), wo, r, w.B, w.T, w.H, w.K)
    torch.cuda.synchronize()
    gates = r["gates"].cpu().numpy().astype(np.float64)
    ref = O.output_projection(_packed_to_dense(_f64(hp_bits), topk, w.H, w.T, w.d), topk, gates,
                              _f64(inp["w_o"]))
    check_out(from_dev(o), ref, "bf16", what="skewed out_proj")


def test_projected_layer():
    # x -> routed q/k/v -> routed attention -> routed output projections,
    # against the oracle chain in float64
    w = _case("d64_dm256").with_(B=1, T=600)
    say(f"projected layer: {w}")
    inp = W.projection_inputs(w)
    r, topk = _route(inp, w)
    x, wq, wo = (to_dev(inp[n], "bf16") for n in ("x", "w_qkv", "w_o"))
    qkv = L.qkv_proj(x, wq, r, w.H, w.K)
    ho = torch.empty(w.B * w.T * w.K, w.d, dtype=torch.float32, device=DEV)
    L.attn_fwd(qkv["q"], qkv["k"], qkv["v"], r, w.K, w.rope_base, head_out=ho, out=False)
    o = L.out_proj(ho, wo, r, w.B, w.T, w.H, w.K)
    torch.cuda.synchronize()
    q, k, v, _ = O.qkv_projection(_f64(inp["x"]), _f64(inp["w_qkv"]), topk)
    ref = O.prefill(inp["logits"], q, k, v, w.K, w.rope_base)
    h = _packed_to_dense(ref["head_out"], topk, w.H, w.T, w.d)
    o_ref = O.output_projection(h, topk, ref["gates"], _f64(inp["w_o"]))
    check_out(from_dev(o), o_ref, "bf16", what="projected layer")


def test_layer_workload_full_size_sampled():
    # the full layer workload (B4 T4096 H32 K8 d64, d_model 2048): every stage
    # at full size, checked on sampled rows the oracle computes one by one
    w = W.WORKLOADS[6]
    say(f"projected layer, full size: {w.name}")
    inp = W.projection_inputs(w)
    r, topk = _route(inp, w)
    x, wq, wo = (to_dev(inp[n], "bf16") for n in ("x", "w_qkv", "w_o"))
    qkv = L.qkv_proj(x, wq, r, w.H, w.K)
    ho = torch.empty(w.B * w.T * w.K, w.d, dtype=torch.float32, device=DEV)
    L.attn_fwd(qkv["q"], qkv["k"], qkv["v"], r, w.K, w.rope_base, head_out=ho, out=False)
    o = L.out_proj(ho, wo, r, w.B, w.T, w.H, w.K)
    torch.cuda.synchronize()
    g = np.random.default_rng(3)
    xs, wqs, wos = _f64(inp["x"]), _f64(inp["w_qkv"]), _f64(inp["w_o"])
    gates = r["gates"].cpu().numpy().astype(np.float64)
    slot = r["slot_pos"].cpu().numpy()
    hp = ho.cpu().numpy().astype(np.float64)
    qg, kg, vg = (from_dev(qkv[n]) for n in ("q", "k", "v"))
    og = from_dev(o)
    got_q, ref_q, got_o, ref_o = [], [], [], []
    for _ in range(48):
        b, t = int(g.integers(w.B)), int(g.integers(w.T))
        for kk in range(w.K):
            i = int(topk[b, t, kk])
            for j, arr in enumerate((qg, kg, vg)):
                got_q.append(arr[b, i, t])
                ref_q.append(wqs[i, j] @ xs[b, t])
        # the aggregation of the GPU's own head outputs (the attention is
        # checked at full size by the forward parity tests)
        got_o.append(og[b, t])
        ref_o.append(sum(gates[b, t, kk] * (wos[int(topk[b, t, kk])] @ hp[slot[b, t, kk]])
                         for kk in range(w.K)))
    check_out(np.array(got_q), np.array(ref_q), "bf16", what="sampled q/k/v rows")
    check_out(np.array(got_o), np.array(ref_o), "bf16", what="sampled output rows")
