"""The decode step without a workspace (namoh_decode_step_noalloc, for callers
that cannot allocate) against namoh_decode_step with one: two calls in a
row, the second on a smaller input, every result compared bit for bit (the
same kernels run on the same inputs; only the workspace's address differs),
and a call above the fixed scratch rejected before anything runs."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2609_38832_amd import workloads as W  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_38832_amd import _lib
    _lib.lib()


def _case(B, H, K, d, cap, seed):
    from gpu_util import DEV, to_dev
    w = W.WORKLOADS[5].with_(B=B, H=H, K=K, d=d, qkv_scale=d ** -0.5)
    lengths = np.random.default_rng(seed).integers(0, cap - 1, size=(B, H))
    kc = np.stack([np.stack([W.decode_cache_block(w, b, h, cap, "k") for h in range(H)])
                   for b in range(B)])
    vc = np.stack([np.stack([W.decode_cache_block(w, b, h, cap, "v") for h in range(H)])
                   for b in range(B)])
    st = W.decode_step_inputs(w)
    dev = {"logits": torch.from_numpy(st["logits"]).to(DEV),
           "q": to_dev(st["q"], "bf16"), "k": to_dev(st["k"], "bf16"), "v": to_dev(st["v"], "bf16"),
           "kc": to_dev(kc, "bf16"), "vc": to_dev(vc, "bf16"),
           "len": torch.from_numpy(lengths.astype(np.int32)).to(DEV)}
    return w, dev


def _outs(B, K, d, dev):
    return {"topk_idx": torch.empty(B, K, dtype=torch.int32, device=dev),
            "gates": torch.empty(B, K, dtype=torch.float32, device=dev),
            "out": torch.empty(B, d, dtype=torch.float32, device=dev)}


@pytest.mark.parametrize("shapes", [((8, 16, 4, 128, 3000), (3, 8, 2, 64, 700))])
def test_noalloc_matches_workspace_step(shapes):
    from gpu_util import DEV, say
    from paper_2609_38832_amd import _lib as L
    for i, (B, H, K, d, cap) in enumerate(shapes):
        say(f"noalloc decode call {i}: B={B} H={H} K={K} d={d} cap={cap}")
        w, x = _case(B, H, K, d, cap, seed=11 + i)
        kc2, vc2, len2 = x["kc"].clone(), x["vc"].clone(), x["len"].clone()
        st1 = torch.zeros(1, dtype=torch.int32, device=DEV)
        st2 = torch.zeros(1, dtype=torch.int32, device=DEV)
        ref = L.decode_step(x["logits"], x["q"], x["k"], x["v"], x["kc"], x["vc"], x["len"], K,
                            w.rope_base, out=_outs(B, K, d, DEV), dev_status=st1)
        got = L.decode_step_noalloc(x["logits"], x["q"], x["k"], x["v"], kc2, vc2, len2, K,
                                    w.rope_base, dev_status=st2, out=_outs(B, K, d, DEV))
        torch.cuda.synchronize()
        for key in ("topk_idx", "gates", "out"):
            assert torch.equal(got[key], ref[key]), key
        assert torch.equal(len2, x["len"])
        assert torch.equal(kc2, x["kc"]) and torch.equal(vc2, x["vc"])
        assert int(st1.item()) == 0 and int(st2.item()) == 0
        assert torch.isfinite(got["out"]).all() and got["out"].abs().sum() > 0


def test_noalloc_rejects_above_scratch():
    # 64 sequences, 8 of 64 heads, d = 128, 70000 rows of capacity: the step's
    # workspace is above the fixed 32 MiB; the call is rejected on the host,
    # before anything is launched (the pointers are real but small: nothing
    # behind them is read)
    from gpu_util import DEV
    from paper_2609_38832_amd import _lib as L
    B, H, K, d, cap = 64, 64, 8, 128, 70000
    buf = torch.zeros(1 << 16, dtype=torch.float32, device=DEV)
    p = buf.data_ptr()
    rc = L.lib().namoh_decode_step_noalloc(p, p, p, p, L.BF16, p, p, p, None, B, H, K, d, cap,
                                           5e5, L.ROPE_HEAD_RELATIVE, L.GATE_SOFTMAX_SELECTED,
                                           0.0, p, p, p, L.F32, None, None)
    torch.cuda.synchronize()
    assert rc == L.NAMOH_ERR_WORKSPACE
    assert "scratch" in L.last_error()
    assert not buf.any()
