"""C-ABI tests that need no GPU: the library loads, exports every symbol the
header declares, and rejects invalid arguments on the host before launching
anything."""
import ctypes
import os
import re

import pytest

from paper_2609_38832_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "namoh.h")

P = ctypes.c_void_p
A = 0x7f0000000000          # fake, well-aligned device addresses: never dereferenced


def fake(i):
    return P(A + i * 0x100000)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("libnamoh.so not built")
    return L.lib()


def test_exports_match_header(lib):
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(namoh_[a-z_]+)\s*\(", text))
    assert declared == set(L.EXPORTED)
    for name in declared:
        assert hasattr(lib, name)
    out = os.popen(f"nm -D --defined-only {L.LIB_PATH}").read()
    exported = set(re.findall(r"\bT (namoh_[a-z_]+)\b", out))
    assert declared <= exported


def test_status_strings(lib):
    assert L.status_string(0) == "NAMOH_OK"
    assert L.status_string(3) == "NAMOH_ERR_WORKSPACE"
    assert lib.namoh_version().startswith(b"namoh-gfx950")


def _route(lib, logits=fake(0), B=1, T=64, H=8, K=2, gate=0, ws=fake(9), wsb=1 << 20, **over):
    args = dict(topk=fake(1), gates=fake(2), hl=fake(3), so=fake(4), pt=fake(5), sp=fake(6))
    args.update(over)
    return lib.namoh_route(logits, B, T, H, K, gate, args["topk"], args["gates"], args["hl"],
                           args["so"], args["pt"], args["sp"], ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(logits=None), 1), (dict(topk=None), 1), (dict(sp=None), 1),
    (dict(B=0), 1), (dict(T=0), 1), (dict(H=65), 1), (dict(K=0), 1), (dict(K=9), 1),
    (dict(gate=7), 1), (dict(logits=P(A + 2)), 1),
    (dict(B=1 << 20, T=1 << 10, K=2), 1),        # B*T*K >= 2^31
    (dict(wsb=16), 3), (dict(ws=None), 3), (dict(ws=P(A + 64)), 1),
])
def test_route_rejects(lib, kw, code):
    assert _route(lib, **kw) == code
    assert L.last_error() != ""


def _route_b(lib, bias=fake(8), B=1, T=64, H=8, K=2, ws=fake(9), wsb=1 << 20, logits=fake(0)):
    return lib.namoh_route_biased(logits, bias, B, T, H, K, fake(1), fake(2), fake(3), fake(4),
                                  fake(5), fake(6), ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(bias=None), 1), (dict(bias=P(A + 2)), 1), (dict(logits=None), 1), (dict(K=9), 1),
    (dict(H=65), 1), (dict(wsb=16), 3),
])
def test_route_biased_rejects(lib, kw, code):
    assert _route_b(lib, **kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(eta=float("nan")), 1), (dict(eta=float("inf")), 1), (dict(hl=None), 1),
    (dict(bias=None), 1), (dict(bias=P(A + 1)), 1), (dict(K=0), 1), (dict(H=65), 1),
])
def test_route_bias_update_rejects(lib, kw, code):
    a = dict(hl=fake(0), B=2, T=64, H=8, K=2, eta=0.01, bias=fake(1))
    a.update(kw)
    assert lib.namoh_route_bias_update(a["hl"], a["B"], a["T"], a["H"], a["K"], a["eta"],
                                       a["bias"], None) == code


def _attn(lib, dtype=1, B=1, T=64, H=8, K=2, d=64, base=1e4, rope=0, scale=0.0, out_dt=0,
          q=fake(0), out=fake(7), head_out=None, ws=fake(9), wsb=1 << 30, gates=fake(3)):
    return lib.namoh_attn_fwd(q, fake(1), fake(2), dtype, B, T, H, K, d, base, rope, scale,
                              gates, fake(4), fake(5), fake(6), out, out_dt, head_out,
                              ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(d=48), 2), (dict(d=256), 2), (dict(dtype=5), 1), (dict(out_dt=3), 1),
    (dict(rope=4), 1), (dict(base=0.0), 1), (dict(base=float("inf")), 1),
    (dict(scale=float("nan")), 1), (dict(q=None), 1), (dict(q=P(A + 8)), 1),
    (dict(gates=None), 1), (dict(out=P(A + 4)), 1), (dict(head_out=P(A + 4)), 1),
    (dict(wsb=100), 3), (dict(K=9), 1),
    (dict(T=1 << 24, d=128), 2),                 # segment tiles past 32-bit offsets
])
def test_attn_rejects(lib, kw, code):
    assert _attn(lib, **kw) == code


def test_attn_rope_none_ignores_base(lib):
    # base is not validated when rope is off: the call passes validation and
    # then fails only because there is no device here (or succeeds on a GPU
    # box with fake pointers — never run there).
    if os.environ.get("HIP_VISIBLE_DEVICES") or _has_gpu():
        pytest.skip("would launch on a real GPU with fake pointers")
    assert _attn(lib, rope=2, base=0.0) == 4


def _has_gpu():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


def _dec(lib, B=2, H=8, K=2, d=64, cap=128, dtype=1, rope=0, gate=0, seq_pos=None,
         kc=fake(4), wsb=1 << 30, status=None):
    return lib.namoh_decode_step(fake(0), fake(1), fake(2), fake(3), dtype, kc, fake(5),
                                 fake(6), seq_pos, B, H, K, d, cap, 1e4, rope, gate, 0.0,
                                 fake(7), fake(8), fake(10), 0, status, fake(9), wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(cap=0), 1), (dict(d=16), 2), (dict(K=9), 1), (dict(rope=1), 1),  # GLOBAL needs seq_pos
    (dict(gate=2), 1), (dict(kc=None), 1), (dict(kc=P(A + 2)), 1), (dict(status=P(A + 2)), 1),
    (dict(wsb=8), 3),
])
def test_decode_rejects(lib, kw, code):
    assert _dec(lib, **kw) == code


def _dec_na(lib, B=2, H=8, K=2, d=64, cap=128, dtype=1, rope=0, kc=fake(4)):
    return lib.namoh_decode_step_noalloc(fake(0), fake(1), fake(2), fake(3), dtype, kc, fake(5),
                                         fake(6), None, B, H, K, d, cap, 1e4, rope, 0, 0.0,
                                         fake(7), fake(8), fake(10), 0, None, None)


@pytest.mark.parametrize("kw,code", [
    (dict(cap=0), 1), (dict(d=16), 2), (dict(K=9), 1), (dict(rope=1), 1), (dict(kc=None), 1),
    (dict(kc=P(A + 2)), 1),
    # the step's workspace above the fixed scratch (64 sequences, 8 heads, d = 128, 70000 rows)
    (dict(B=64, H=64, K=8, d=128, cap=70000), 3),
])
def test_decode_noalloc_rejects(lib, kw, code):
    assert _dec_na(lib, **kw) == code
    if code == 3:
        assert "noalloc" in L.last_error() and "scratch" in L.last_error()


def test_decode_noalloc_scratch_limit(lib):
    # the decode workload's step (64 sequences, 8 of 64 heads, d = 128, about
    # 17k rows of history) fits in the 32 MiB scratch; 70000 rows do not
    assert lib.namoh_decode_workspace_size(64, 64, 8, 128, 17152) <= 32 << 20
    assert lib.namoh_decode_workspace_size(64, 64, 8, 128, 70000) > 32 << 20


def test_decode_noalloc_without_device(lib):
    if _has_gpu():
        pytest.skip("a GPU is visible")
    assert _dec_na(lib) == 4     # valid arguments; no device to hold the scratch


def _pcache(lib, dtype=1, B=2, T=64, H=8, K=2, d=64, base=1e4, rope=0, cap=64, k=fake(0),
            kc=fake(4), cl=fake(6), so=fake(2)):
    return lib.namoh_prefill_cache(k, fake(1), dtype, B, T, H, K, d, base, rope, so, fake(3),
                                   kc, fake(5), cl, cap, None)


@pytest.mark.parametrize("kw,code", [
    (dict(cap=63), 1), (dict(d=48), 2), (dict(K=9), 1), (dict(dtype=3), 1), (dict(rope=5), 1),
    (dict(base=-1.0), 1), (dict(k=None), 1), (dict(kc=P(A + 4)), 1), (dict(cl=None), 1),
    (dict(so=P(A + 2)), 1), (dict(B=0), 1),
    (dict(B=64, H=64, T=1 << 16, cap=1 << 22, d=128), 1),   # caches past 2^40 elements
])
def test_prefill_cache_rejects(lib, kw, code):
    assert _pcache(lib, **kw) == code
    assert L.last_error() != ""


def test_decode_biased_rejects(lib):
    # same checks as namoh_decode_step plus the bias pointer
    args = [fake(0), fake(11), fake(1), fake(2), fake(3), 1, fake(4), fake(5), fake(6), None,
            2, 8, 2, 64, 128, 1e4, 0, 0.0, fake(7), fake(8), fake(10), 0, None, fake(9), 8, None]
    assert lib.namoh_decode_step_biased(*args) == 3            # workspace too small
    bad = list(args)
    bad[1] = None
    assert lib.namoh_decode_step_biased(*bad) == 1              # no bias
    bad = list(args)
    bad[1] = P(A + 2)
    assert lib.namoh_decode_step_biased(*bad) == 1              # misaligned bias
    bad = list(args)
    bad[16] = 1
    assert lib.namoh_decode_step_biased(*bad) == 1              # GLOBAL needs seq_pos


def _bwd(lib, dtype=1, B=2, T=64, H=8, K=2, d=64, base=1e4, rope=0, scale=0.0, q=fake(0),
         dout=fake(5), dq=fake(6), dg=fake(9), wsb=1 << 30, ws=fake(10)):
    return lib.namoh_attn_bwd(q, fake(1), fake(2), dtype, B, T, H, K, d, base, rope, scale,
                              fake(3), fake(4), fake(11), fake(12), dout, dq, fake(7), fake(8),
                              dg, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(d=48), 2), (dict(dtype=4), 1), (dict(rope=3), 1), (dict(base=0.0), 1),
    (dict(scale=float("inf")), 1), (dict(q=None), 1), (dict(dout=P(A + 4)), 1), (dict(dq=None), 1),
    (dict(dg=P(A + 1)), 1), (dict(wsb=64), 3), (dict(ws=None), 3), (dict(K=9), 1),
    (dict(B=64, H=1025, K=1), 1), (dict(B=1024, H=64, T=8, K=1), 1),   # H > 64; B*H > 65535
])
def test_attn_bwd_rejects(lib, kw, code):
    assert _bwd(lib, **kw) == code


def _bwd_saved(lib, dtype=1, B=2, T=64, H=8, K=2, d=64, base=1e4, rope=0, scale=0.0,
               q=fake(0), dout=fake(5), dq=fake(6), dg=fake(9), packed=0, wsb=1 << 30,
               ws=fake(10)):
    return lib.namoh_attn_bwd_saved(q, fake(1), fake(2), dtype, B, T, H, K, d, base, rope, scale,
                                    fake(3), fake(4), fake(11), fake(12), dout, dq, fake(7),
                                    fake(8), dg, packed, ws, wsb, None)


def _fwd_train(lib, dtype=1, B=2, T=64, H=8, K=2, d=64, base=1e4, rope=0, scale=0.0,
               q=fake(0), slot=fake(6), out=fake(7), odt=1, wsb=1 << 30, ws=fake(10)):
    return lib.namoh_attn_fwd_train(q, fake(1), fake(2), dtype, B, T, H, K, d, base, rope,
                                    scale, fake(3), fake(4), fake(5), slot, out, odt, ws, wsb,
                                    None)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=0), 2), (dict(d=32), 2), (dict(d=48), 2), (dict(dtype=4), 1), (dict(packed=2), 1),
    (dict(rope=3), 1), (dict(q=None), 1), (dict(dout=P(A + 4)), 1), (dict(dg=None), 1),
    (dict(wsb=64), 3), (dict(K=9), 1),
])
def test_attn_bwd_saved_rejects(lib, kw, code):
    assert _bwd_saved(lib, **kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=0), 2), (dict(d=32), 2), (dict(odt=3), 1), (dict(base=-1.0), 1),
    (dict(q=None), 1), (dict(slot=None), 1), (dict(out=None), 1), (dict(out=P(A + 8)), 1),
    (dict(wsb=64), 3), (dict(ws=None), 3), (dict(T=1 << 25, B=1, H=2, K=1, d=128), 2),
])
def test_attn_fwd_train_rejects(lib, kw, code):
    assert _fwd_train(lib, **kw) == code


def test_train_calls_without_device(lib):
    if _has_gpu():
        pytest.skip("a GPU is present")
    need = lib.namoh_attn_bwd_workspace_size(2, 64, 8, 2, 64)
    assert _fwd_train(lib, wsb=need) == L.NAMOH_ERR_HIP
    assert _bwd_saved(lib, wsb=need) == L.NAMOH_ERR_HIP


@pytest.mark.parametrize("kw,code", [
    (dict(gate=2), 1), (dict(logits=None), 1), (dict(dl=P(A + 2)), 1), (dict(K=0), 1),
])
def test_route_bwd_rejects(lib, kw, code):
    a = dict(logits=fake(0), gate=0, dl=fake(4), K=2)
    a.update(kw)
    assert lib.namoh_route_bwd(a["logits"], fake(1), fake(2), fake(3), 2, 16, 8, a["K"],
                               a["gate"], a["dl"], None) == code


def _qkv(lib, B=2, T=64, H=8, K=2, d=64, dm=256, x=fake(0), w=fake(1), so=fake(2), q=fake(4)):
    return lib.namoh_qkv_proj(x, w, B, T, H, K, d, dm, so, fake(3), q, fake(5), fake(6), None)


@pytest.mark.parametrize("kw,code", [
    (dict(d=32), 2), (dict(d=48), 2), (dict(dm=192), 2), (dict(dm=0), 2), (dict(x=None), 1),
    (dict(w=P(A + 8)), 1), (dict(so=None), 1), (dict(q=P(A + 2)), 1), (dict(K=9), 1),
    (dict(H=65, K=1), 1),
])
def test_qkv_proj_rejects(lib, kw, code):
    assert _qkv(lib, **kw) == code


def _oproj(lib, B=2, T=64, H=8, K=2, d=64, dm=256, h=fake(0), hdt=0, odt=0, out=fake(5),
           wsb=1 << 30, ws=fake(6)):
    return lib.namoh_out_proj(h, hdt, fake(1), fake(2), fake(3), fake(4), B, T, H, K, d, dm, out,
                              odt, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(d=32), 2), (dict(dm=200), 2), (dict(hdt=2), 1), (dict(odt=5), 1), (dict(h=None), 1),
    (dict(out=P(A + 4)), 1), (dict(wsb=1024), 3), (dict(ws=None), 3), (dict(K=0), 1),
])
def test_out_proj_rejects(lib, kw, code):
    assert _oproj(lib, **kw) == code


def test_out_proj_workspace_size(lib):
    # dense form (H d <= 384 K): the per-token head map and the gated bf16 rows
    assert lib.namoh_out_proj_workspace_size(4, 4096, 32, 8, 64, 2048) >= \
        4 * 4096 * 32 * 4 + 4 * 4096 * 8 * 64 * 2
    assert lib.namoh_out_proj_workspace_size(4, 4096, 32, 8, 64, 2048) < 4 * 4096 * 8 * 2048 * 2
    # per-pair form: the bf16 per-pair rows
    assert lib.namoh_out_proj_workspace_size(4, 4096, 64, 8, 128, 2048) >= 4 * 4096 * 8 * 2048 * 2
    assert lib.namoh_out_proj_workspace_size(4, 4096, 32, 8, 64, 100) == 0
    assert lib.namoh_out_proj_workspace_size(4, 4096, 32, 8, 96, 2048) == 0


def _grp(lib, dtype=1, B=2, T=64, H=8, K=2, g=2, d=64, base=1e4, rope=0, q=fake(0), out=fake(7),
         ho=None, wsb=1 << 30, ws=fake(9)):
    return lib.namoh_attn_fwd_grouped(q, fake(1), fake(2), dtype, B, T, H, K, g, d, base, rope, 0.0,
                                      fake(3), fake(4), fake(5), fake(6), out, 0, ho, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(g=0), 1), (dict(g=17), 1), (dict(dtype=0), 2), (dict(d=32), 2), (dict(dtype=3), 1),
    (dict(rope=7), 1), (dict(base=-1.0), 1), (dict(q=None), 1), (dict(out=None), 1),
    (dict(out=P(A + 8)), 1), (dict(wsb=16), 3), (dict(K=9), 1), (dict(T=1 << 25, d=128), 2),
])
def test_attn_fwd_grouped_rejects(lib, kw, code):
    assert _grp(lib, **kw) == code


def test_grouped_workspace_grows_with_the_group(lib):
    a = lib.namoh_attn_fwd_grouped_workspace_size(2, 1024, 8, 2, 1, 64, 1)
    b = lib.namoh_attn_fwd_grouped_workspace_size(2, 1024, 8, 2, 4, 64, 1)
    assert a == lib.namoh_attn_fwd_workspace_size(2, 1024, 8, 2, 64, 1)
    assert b > a
    assert lib.namoh_attn_fwd_grouped_workspace_size(2, 1024, 8, 2, 4, 64, 0) == 0


def _shared(lib, dtype=1, B=2, T=300, Hs=2, d=64, window=128, base=1e4, rope=1, q=fake(0),
            out=fake(3), odt=0, ho=None, wsb=1 << 30, ws=fake(5)):
    return lib.namoh_shared_attn(q, fake(1), fake(2), dtype, B, T, Hs, d, window, base, rope, 0.0,
                                 out, odt, 1, ho, ws, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=0), 2), (dict(d=32), 2), (dict(dtype=2), 1), (dict(window=-1), 1),
    (dict(Hs=0), 1), (dict(B=0), 1), (dict(rope=4), 1), (dict(base=0.0), 1), (dict(q=None), 1),
    (dict(out=None), 1), (dict(out=P(A + 2)), 1), (dict(odt=3), 1), (dict(wsb=8), 3),
    (dict(B=1 << 20, T=1 << 12, Hs=1), 1),
])
def test_shared_attn_rejects(lib, kw, code):
    assert _shared(lib, **kw) == code


def _sdec(lib, dtype=1, B=2, Hs=2, d=64, cap=256, window=128, base=1e4, rope=1, q=fake(0),
          kc=fake(3), clen=fake(5), out=fake(6), odt=0, acc=1, st=None, wsb=1 << 30, ws=fake(8)):
    return lib.namoh_shared_decode_step(q, fake(1), fake(2), dtype, B, Hs, d, cap, window, base,
                                        rope, 0.0, kc, fake(4), clen, out, odt, acc, st, ws, wsb,
                                        None)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=2), 1), (dict(d=48), 2), (dict(B=0), 1), (dict(Hs=0), 1), (dict(Hs=1025), 1),
    (dict(cap=0), 1), (dict(window=-1), 1), (dict(cap=100, window=128), 1), (dict(rope=3), 1),
    (dict(base=-1.0), 1), (dict(q=None), 1), (dict(kc=P(A + 8)), 1), (dict(clen=None), 1),
    (dict(out=None), 1), (dict(odt=2), 1), (dict(acc=2), 1), (dict(st=P(A + 2)), 1),
    (dict(wsb=64), 3), (dict(ws=None), 3), (dict(B=1 << 20, Hs=1024, cap=1 << 20), 1),
])
def test_shared_decode_rejects(lib, kw, code):
    assert _sdec(lib, **kw) == code


def _spc(lib, dtype=1, B=2, T=300, Hs=2, d=64, cap=512, window=0, base=1e4, rope=1, k=fake(0),
         clen=fake(4)):
    return lib.namoh_shared_prefill_cache(k, fake(1), dtype, B, T, Hs, d, cap, window, base, rope,
                                          fake(2), fake(3), clen, None)


@pytest.mark.parametrize("kw,code", [
    (dict(cap=200), 1), (dict(cap=100, window=128), 1), (dict(T=0), 1), (dict(d=16), 2),
    (dict(k=None), 1), (dict(clen=None), 1), (dict(dtype=5), 1), (dict(B=1 << 20, T=1 << 12), 1),
])
def test_shared_prefill_cache_rejects(lib, kw, code):
    assert _spc(lib, **kw) == code


def test_shared_decode_sizes_and_calls_without_device(lib):
    a = lib.namoh_shared_decode_workspace_size(4, 2, 128, 1000)
    # rotated queries, four int/float words per head, two 512-row partials per head
    assert a >= 4 * 2 * (128 * 4 + 16 + 2 * (128 * 4 + 8))
    assert lib.namoh_shared_decode_workspace_size(4, 2, 96, 1000) == 0
    assert _sdec(lib, wsb=a, B=4, d=128, cap=1000) == L.NAMOH_ERR_HIP
    assert _spc(lib, cap=128, window=128) == L.NAMOH_ERR_HIP   # window: the last 128 tokens


def _gdec(lib, dtype=1, B=2, H=8, K=2, g=4, d=64, cap=100, q=fake(1), wsb=1 << 30):
    return lib.namoh_decode_step_grouped(fake(0), q, fake(2), fake(3), dtype, fake(4), fake(5),
                                         fake(6), None, B, H, K, g, d, cap, 1e4, 0, 0, 0.0,
                                         fake(7), fake(8), fake(9), 0, None, fake(10), wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(g=0), 1), (dict(g=3), 1), (dict(g=16), 1), (dict(dtype=0), 2), (dict(d=32), 2),
    (dict(cap=0), 1), (dict(q=None), 1), (dict(wsb=4), 3), (dict(K=9), 1),
])
def test_decode_step_grouped_rejects(lib, kw, code):
    assert _gdec(lib, **kw) == code


def test_workspace_queries(lib):
    assert lib.namoh_route_workspace_size(0, 10, 8, 2) == 0
    assert lib.namoh_route_workspace_size(1, 10, 8, 2) > 0
    assert lib.namoh_attn_fwd_workspace_size(1, 64, 8, 2, 48, 1) == 0
    a = lib.namoh_attn_fwd_workspace_size(4, 4096, 32, 8, 64, 1)
    assert a > 4 * 4096 * 8 * 64 * 4                 # holds the packed head outputs
    assert lib.namoh_decode_workspace_size(64, 64, 8, 128, 17000) > 0
    assert lib.namoh_decode_workspace_size(64, 64, 8, 128, 0) == 0


def test_valid_call_without_device_reports_hip_error(lib):
    if _has_gpu():
        pytest.skip("a GPU is present")
    need = lib.namoh_route_workspace_size(1, 64, 8, 2)
    assert _route(lib, wsb=need) == L.NAMOH_ERR_HIP
    assert "HIP error" in L.last_error()


def test_missing_library_raises(monkeypatch, tmp_path):
    monkeypatch.setattr(L, "_lib", None)
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "nope.so"))
    with pytest.raises(ImportError):
        L.lib()
