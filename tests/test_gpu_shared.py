"""GPU parity of always-active shared heads (Sec. 4.4, shared heads for local
context) through the C ABI, against the float64 oracle: full causal prefix
or a sliding window of w tokens, global RoPE, outputs added to the routed
layer output.  bf16 bound |got - ref| <= 2e-2 + 1e-2 |ref|, relative L2
<= 1e-2.
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

# (B, T, Hs, d, window, RoPE mode, query/key scale factor)
CASES = {
    "d64_w128": (2, 700, 2, 64, 128, O.ROPE_GLOBAL, 1.0),
    "d128_full": (1, 900, 4, 128, 0, O.ROPE_GLOBAL, 1.0),
    "d64_w1": (2, 300, 1, 64, 1, O.ROPE_GLOBAL, 1.0),
    "d128_w200_none_peaky": (1, 650, 2, 128, 200, O.ROPE_NONE, 12.0),
    "d64_w_longer_than_T": (1, 100, 2, 64, 500, O.ROPE_GLOBAL, 1.0),
    "d64_w64_ragged": (1, 333, 3, 64, 64, O.ROPE_GLOBAL, 1.0),
}


def _qkv(B, T, Hs, d, scale):
    base = W.WORKLOADS[2] if d == 64 else W.WORKLOADS[3]
    w = base.with_(B=B, T=T, H=Hs, K=1, d=d, seed=base.seed + 100)
    q, k, v = (W.prefill_qkv(w, n) for n in ("q", "k", "v"))
    if scale != 1.0:
        q = W.f32_to_bf16_bits(W.bf16_bits_to_f32(q) * np.float32(scale))
        k = W.f32_to_bf16_bits(W.bf16_bits_to_f32(k) * np.float32(scale))
    return w, q, k, v


@pytest.mark.parametrize("name", list(CASES))
def test_shared_heads_parity(name):
    B, T, Hs, d, window, rope, scale = CASES[name]
    say(f"shared heads {name}")
    w, q, k, v = _qkv(B, T, Hs, d, scale)
    qd, kd, vd = (to_dev(x, "bf16") for x in (q, k, v))
    ho = torch.empty(B, Hs, T, d, dtype=torch.float32, device=DEV)
    out = L.shared_attn(qd, kd, vd, window, w.rope_base, rope, out_dtype=torch.float32,
                        head_out=ho)
    torch.cuda.synchronize()
    f64 = [W.as_float64(x, "bf16") for x in (q, k, v)]
    ref = O.always_active_heads(*f64, window, w.rope_base, rope)
    check_out(ho.cpu().numpy(), ref, "bf16", what=f"{name} head outputs")
    check_out(from_dev(out), ref.sum(axis=1), "bf16", what=f"{name} out")


def test_shared_heads_added_to_the_routed_layer():
    # routed layer (H 8, K 2) plus two sliding-window shared heads (w 128)
    w = W.WORKLOADS[2].with_(B=2, T=800, H=8, K=2)
    say("routed layer plus shared heads")
    inp = W.prefill_inputs(w)
    r = L.route(torch.from_numpy(inp["logits"]).to(DEV), w.K)
    q, k, v = (to_dev(inp[n], "bf16") for n in ("q", "k", "v"))
    out = L.attn_fwd(q, k, v, r, w.K, w.rope_base, out_dtype=torch.float32)
    _, qs, ks, vs = _qkv(w.B, w.T, 2, w.d, 1.0)
    L.shared_attn(*(to_dev(x, "bf16") for x in (qs, ks, vs)), 128, w.rope_base, out=out,
                  accumulate=True)
    torch.cuda.synchronize()
    f = {n: W.as_float64(inp[n], "bf16") for n in ("q", "k", "v")}
    ref = O.prefill(inp["logits"], f["q"], f["k"], f["v"], w.K, w.rope_base)["out"]
    ref = ref + O.always_active_heads(*(W.as_float64(x, "bf16") for x in (qs, ks, vs)), 128,
                                      w.rope_base).sum(axis=1)
    check_out(from_dev(out), ref, "bf16", what="routed + shared")


# ----------------------------------------------------------------------------
# decode step of the shared heads: the prompt's keys/values handed to the
# caches, then one token at a time; step i must equal row T + i of the
# oracle's prefill over all tokens (the same causal computation)

# (B, T, Hs, d, window, cap, decode steps, RoPE mode, dtype)
SDEC = {
    "d64_w16_ring": (2, 50, 2, 64, 16, 24, 4, O.ROPE_GLOBAL, "bf16"),
    "d128_full": (1, 300, 3, 128, 0, 310, 3, O.ROPE_GLOBAL, "bf16"),
    "d64_w128_none": (2, 200, 2, 64, 128, 128, 2, O.ROPE_NONE, "bf16"),
    "d64_w8_f32": (2, 40, 2, 64, 8, 8, 5, O.ROPE_GLOBAL, "f32"),
    "d32_full_f32": (1, 100, 1, 32, 0, 120, 2, O.ROPE_GLOBAL, "f32"),
    "d128_full_long": (1, 2600, 2, 128, 0, 2700, 1, O.ROPE_GLOBAL, "bf16"),
}


def _decode_inputs(B, T, Hs, d, steps, dtype):
    w, q, k, v = _qkv(B, T + steps, Hs, d, 1.0)
    if dtype == "f32":   # the same values, exact in float32
        q, k, v = (W.bf16_bits_to_f32(x) for x in (q, k, v))
        f64 = [x.astype(np.float64) for x in (q, k, v)]
    else:
        f64 = [W.as_float64(x, "bf16") for x in (q, k, v)]
    return w, (q, k, v), f64


@pytest.mark.parametrize("name", list(SDEC))
def test_shared_decode_parity(name):
    B, T, Hs, d, window, cap, steps, rope, dtype = SDEC[name]
    say(f"shared-head decode {name}")
    w, (q, k, v), f64 = _decode_inputs(B, T, Hs, d, steps, dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    qd, kd, vd = (to_dev(x, dtype) for x in (q, k, v))
    kc = torch.zeros(B, Hs, cap, d, dtype=tdt, device=DEV)
    vc = torch.zeros_like(kc)
    clen = torch.zeros(B, dtype=torch.int32, device=DEV)
    L.shared_prefill_cache(kd[:, :, :T].contiguous(), vd[:, :, :T].contiguous(), kc, vc, clen,
                           window, w.rope_base, rope)
    ref = O.always_active_heads(*f64, window, w.rope_base, rope).sum(axis=1)   # [B, T+steps, d]
    for i in range(steps):
        t = T + i
        out = L.shared_decode_step(qd[:, :, t].contiguous(), kd[:, :, t].contiguous(),
                                   vd[:, :, t].contiguous(), kc, vc, clen, window, w.rope_base,
                                   rope, out_dtype=torch.float32)
        torch.cuda.synchronize()
        check_out(from_dev(out), ref[:, t], dtype, what=f"{name} step {i}")
    assert (clen.cpu().numpy() == T + steps).all()


def test_shared_decode_accumulates_and_reports_overflow():
    B, T, Hs, d = 2, 60, 2, 64
    w, (q, k, v), f64 = _decode_inputs(B, T, Hs, d, 1, "bf16")
    qd, kd, vd = (to_dev(x, "bf16") for x in (q, k, v))
    ref = O.always_active_heads(*f64, 0, w.rope_base, O.ROPE_GLOBAL).sum(axis=1)[:, T]
    base = np.random.default_rng(5).standard_normal((B, d)).astype(np.float32)
    for cap, expect_over in ((T + 1, False), (T, True)):
        kc = torch.zeros(B, Hs, cap, d, dtype=torch.bfloat16, device=DEV)
        vc = torch.zeros_like(kc)
        clen = torch.zeros(B, dtype=torch.int32, device=DEV)
        st = torch.zeros(1, dtype=torch.int32, device=DEV)
        L.shared_prefill_cache(kd[:, :, :T].contiguous(), vd[:, :, :T].contiguous(), kc, vc, clen,
                               0, w.rope_base)
        out = torch.from_numpy(base.copy()).to(DEV)
        L.shared_decode_step(qd[:, :, T].contiguous(), kd[:, :, T].contiguous(),
                             vd[:, :, T].contiguous(), kc, vc, clen, 0, w.rope_base, out=out,
                             accumulate=True, dev_status=st)
        torch.cuda.synchronize()
        say(f"  cap {cap}: status {int(st.item())}")
        if expect_over:   # no room for row T: nothing added, nothing appended, reported
            assert int(st.item()) == 1
            np.testing.assert_array_equal(out.cpu().numpy(), base)
            assert (clen.cpu().numpy() == T).all()
        else:
            assert int(st.item()) == 0
            check_out(out.cpu().numpy().astype(np.float64), base + ref, "bf16",
                      what="accumulated shared decode")
            assert (clen.cpu().numpy() == T + 1).all()
