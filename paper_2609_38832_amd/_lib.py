"""ctypes binding of libnamoh.so (C ABI declared in include/namoh.h).

Only argument marshalling happens here: torch supplies device memory (outputs
and workspace are ``torch.empty`` on the inputs' device) and the current
stream; every step of the layer runs in the library's HIP kernels.  There is
no fallback: if the library is missing or a call fails, an exception is
raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# NAMOH_LIB selects another build of the same library (the host-sanitizer
# build the CPU tests use); by default the in-tree libnamoh.so
LIB_PATH = os.environ.get("NAMOH_LIB") or os.path.join(_HERE, "libnamoh.so")

NAMOH_OK = 0
NAMOH_ERR_INVALID_ARG = 1
NAMOH_ERR_UNSUPPORTED = 2
NAMOH_ERR_WORKSPACE = 3
NAMOH_ERR_HIP = 4

F32, BF16 = 0, 1
GATE_SOFTMAX_SELECTED, GATE_SOFTMAX_ALL = 0, 1
ROPE_HEAD_RELATIVE, ROPE_GLOBAL, ROPE_NONE = 0, 1, 2

EXPORTED = (
    "namoh_route_workspace_size", "namoh_route", "namoh_route_biased", "namoh_route_bias_update",
    "namoh_attn_fwd_workspace_size", "namoh_attn_fwd",
    "namoh_prefill_cache", "namoh_attn_bwd_workspace_size", "namoh_attn_bwd",
    "namoh_attn_bwd_packed", "namoh_attn_fwd_train", "namoh_attn_bwd_saved", "namoh_route_bwd",
    "namoh_decode_workspace_size", "namoh_decode_step", "namoh_decode_step_biased",
    "namoh_decode_step_noalloc",
    "namoh_qkv_proj", "namoh_out_proj_workspace_size", "namoh_out_proj",
    "namoh_attn_fwd_grouped_workspace_size", "namoh_attn_fwd_grouped",
    "namoh_shared_attn_workspace_size", "namoh_shared_attn",
    "namoh_shared_decode_workspace_size", "namoh_shared_decode_step", "namoh_shared_prefill_cache",
    "namoh_decode_grouped_workspace_size", "namoh_decode_step_grouped",
    "namoh_status_string", "namoh_last_error", "namoh_version",
    "namoh_profile_enable", "namoh_profile_read",
)

_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float
_S = ctypes.c_size_t

_SIGS = {
    "namoh_route_workspace_size": (_S, [_I, _I, _I, _I]),
    "namoh_route": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "namoh_route_biased": (_I, [_P, _P, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "namoh_route_bias_update": (_I, [_P, _I, _I, _I, _I, _F, _P, _P]),
    "namoh_attn_fwd_workspace_size": (_S, [_I, _I, _I, _I, _I, _I]),
    "namoh_attn_fwd": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _F,
                            _P, _P, _P, _P, _P, _I, _P, _P, _S, _P]),
    "namoh_prefill_cache": (_I, [_P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _P, _P, _P, _P, _P,
                                 _I, _P]),
    "namoh_attn_bwd_workspace_size": (_S, [_I, _I, _I, _I, _I]),
    "namoh_attn_bwd": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _F, _P, _P, _P, _P, _P,
                            _P, _P, _P, _P, _P, _S, _P]),
    "namoh_attn_bwd_packed": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _F, _P, _P, _P,
                                   _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "namoh_attn_fwd_train": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _F,
                                  _P, _P, _P, _P, _P, _I, _P, _S, _P]),
    "namoh_attn_bwd_saved": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _F, _P, _P, _P,
                                  _P, _P, _P, _P, _P, _P, _I, _P, _S, _P]),
    "namoh_route_bwd": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P]),
    "namoh_decode_workspace_size": (_S, [_I, _I, _I, _I, _I]),
    "namoh_decode_step": (_I, [_P, _P, _P, _P, _I, _P, _P, _P, _P, _I, _I, _I, _I, _I,
                               _F, _I, _I, _F, _P, _P, _P, _I, _P, _P, _S, _P]),
    "namoh_decode_step_noalloc": (_I, [_P, _P, _P, _P, _I, _P, _P, _P, _P, _I, _I, _I, _I, _I,
                                       _F, _I, _I, _F, _P, _P, _P, _I, _P, _P]),
    "namoh_decode_step_biased": (_I, [_P, _P, _P, _P, _P, _I, _P, _P, _P, _P, _I, _I, _I, _I,
                                      _I, _F, _I, _F, _P, _P, _P, _I, _P, _P, _S, _P]),
    "namoh_attn_fwd_grouped_workspace_size": (_S, [_I, _I, _I, _I, _I, _I, _I]),
    "namoh_attn_fwd_grouped": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _I, _F,
                                    _P, _P, _P, _P, _P, _I, _P, _P, _S, _P]),
    "namoh_shared_attn_workspace_size": (_S, [_I, _I, _I, _I]),
    "namoh_shared_attn": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _F, _P, _I, _I, _P,
                               _P, _S, _P]),
    "namoh_shared_decode_workspace_size": (_S, [_I, _I, _I, _I]),
    "namoh_shared_decode_step": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _I, _F, _I, _F, _P, _P, _P,
                                      _P, _I, _I, _P, _P, _S, _P]),
    "namoh_shared_prefill_cache": (_I, [_P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _I, _P, _P, _P,
                                        _P]),
    "namoh_decode_grouped_workspace_size": (_S, [_I, _I, _I, _I, _I, _I]),
    "namoh_decode_step_grouped": (_I, [_P, _P, _P, _P, _I, _P, _P, _P, _P, _I, _I, _I, _I, _I,
                                       _I, _F, _I, _I, _F, _P, _P, _P, _I, _P, _P, _S, _P]),
    "namoh_qkv_proj": (_I, [_P, _P, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P]),
    "namoh_out_proj_workspace_size": (_S, [_I, _I, _I, _I, _I, _I]),
    "namoh_out_proj": (_I, [_P, _I, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _P, _S, _P]),
    "namoh_status_string": (ctypes.c_char_p, [_I]),
    "namoh_last_error": (ctypes.c_char_p, []),
    "namoh_version": (ctypes.c_char_p, []),
    "namoh_profile_enable": (_I, [_I]),
    "namoh_profile_read": (_I, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                ctypes.POINTER(ctypes.c_int)]),
}

_lib = None


class NamohError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} [{status_string(status)}]")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load the HIP library (built in-tree by ``build()``); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                              "(python -m paper_2609_38832_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def status_string(s: int) -> str:
    return lib().namoh_status_string(int(s)).decode()


def last_error() -> str:
    return lib().namoh_last_error().decode()


def check(status: int) -> None:
    if status != NAMOH_OK:
        raise NamohError(status, last_error())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def dtype_code(dt: torch.dtype) -> int:
    if dt == torch.float32:
        return F32
    if dt == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {dt}")


def torch_dtype(code: int) -> torch.dtype:
    return torch.float32 if code == F32 else torch.bfloat16


def workspace(nbytes: int, device) -> torch.Tensor:
    """A device byte buffer whose data pointer is 256-byte aligned.  The
    returned tensor is a view starting at the aligned address."""
    raw = torch.empty(max(int(nbytes), 1) + 256, dtype=torch.uint8, device=device)
    off = (-raw.data_ptr()) % 256
    return raw[off:off + max(int(nbytes), 1)]


def _need_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("tensors must live on the GPU")
        if t is not None and not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


# ----------------------------------------------------------------------------
def route_workspace_size(B, T, H, K) -> int:
    return int(lib().namoh_route_workspace_size(B, T, H, K))


def route(logits: torch.Tensor, K: int, gate_mode: int = GATE_SOFTMAX_SELECTED,
          out: Optional[dict] = None, ws: Optional[torch.Tensor] = None,
          bias: Optional[torch.Tensor] = None) -> dict:
    """namoh_route on float32 logits [B, T, H]; with a float32 [H] `bias`,
    namoh_route_biased (loss-free balancing; gate_mode is then ignored)."""
    _need_cuda(logits, bias)
    if bias is not None and (bias.dtype != torch.float32 or bias.shape != (logits.shape[-1],)):
        raise ValueError("bias must be float32 [H]")
    if logits.dtype != torch.float32 or logits.dim() != 3:
        raise ValueError("logits must be float32 [B, T, H]")
    B, T, H = logits.shape
    dev = logits.device
    if out is None:
        i32 = dict(dtype=torch.int32, device=dev)
        out = {
            "topk_idx": torch.empty(B, T, K, **i32),
            "gates": torch.empty(B, T, K, dtype=torch.float32, device=dev),
            "head_len": torch.empty(B, H, **i32),
            "seg_offsets": torch.empty(B * H + 1, **i32),
            "perm_token": torch.empty(B * T * K, **i32),
            "slot_pos": torch.empty(B, T, K, **i32),
        }
    nbytes = route_workspace_size(B, T, H, K)
    if ws is None:
        ws = workspace(nbytes, dev)
    outs = (_ptr(out["topk_idx"]), _ptr(out["gates"]), _ptr(out["head_len"]),
            _ptr(out["seg_offsets"]), _ptr(out["perm_token"]), _ptr(out["slot_pos"]))
    if bias is None:
        check(lib().namoh_route(_ptr(logits), B, T, H, K, gate_mode, *outs, _ptr(ws),
                                ws.numel(), _stream(dev)))
    else:
        check(lib().namoh_route_biased(_ptr(logits), _ptr(bias), B, T, H, K, *outs, _ptr(ws),
                                       ws.numel(), _stream(dev)))
    return out


def route_bias_update(head_len: torch.Tensor, T: int, K: int, eta: float,
                      bias: torch.Tensor) -> None:
    """namoh_route_bias_update: bias [H] += eta * sign(B*T*K/H - sum_b head_len[b])."""
    _need_cuda(head_len, bias)
    B, H = head_len.shape
    if head_len.dtype != torch.int32 or bias.dtype != torch.float32 or bias.shape != (H,):
        raise ValueError("head_len int32 [B, H], bias float32 [H]")
    check(lib().namoh_route_bias_update(_ptr(head_len), B, T, H, K, float(eta), _ptr(bias),
                                        _stream(head_len.device)))


def attn_workspace_size(B, T, H, K, d, dtype_c) -> int:
    return int(lib().namoh_attn_fwd_workspace_size(B, T, H, K, d, dtype_c))


def attn_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, routing: dict, K: int,
             rope_base: float, rope_mode: int = ROPE_HEAD_RELATIVE,
             softmax_scale: float = 0.0, out_dtype: Optional[torch.dtype] = None,
             head_out: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
             ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """namoh_attn_fwd on dense q/k/v [B, H, T, d]; returns out [B, T, d].
    With out_dtype=None and head_out given, pass out=False to skip the
    combine (returns head_out)."""
    _need_cuda(q, k, v, head_out, None if out is False else out)
    B, H, T, d = q.shape
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("q, k, v must share shape and dtype")
    dt = dtype_code(q.dtype)
    odt = q.dtype if out_dtype is None else out_dtype
    skip = out is False
    if skip and head_out is None:
        raise ValueError("out=False needs head_out")
    if out is None:
        out = torch.empty(B, T, d, dtype=odt, device=q.device)
    if ws is None:
        ws = workspace(attn_workspace_size(B, T, H, K, d, dt), q.device)
    check(lib().namoh_attn_fwd(_ptr(q), _ptr(k), _ptr(v), dt, B, T, H, K, d,
                               float(rope_base), rope_mode, float(softmax_scale),
                               _ptr(routing["gates"]), _ptr(routing["seg_offsets"]),
                               _ptr(routing["perm_token"]), _ptr(routing["slot_pos"]),
                               None if skip else _ptr(out),
                               dtype_code(odt) if skip else dtype_code(out.dtype),
                               _ptr(head_out), _ptr(ws), ws.numel(), _stream(q.device)))
    return head_out if skip else out


def attn_fwd_grouped(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, routing: dict,
                     K_kv: int, rope_base: float, rope_mode: int = ROPE_HEAD_RELATIVE,
                     softmax_scale: float = 0.0, out_dtype: Optional[torch.dtype] = None,
                     head_out: Optional[torch.Tensor] = None, out=None,
                     ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """namoh_attn_fwd_grouped: query heads q [B, H_kv*g, T, d] over
    key/value groups k, v [B, H_kv, T, d] (bf16) with the groups' routing;
    returns out [B, T, d] (or head_out [B*T*K_kv, g, d] with out=False)."""
    _need_cuda(q, k, v, head_out, None if out is False else out)
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    if k.shape != v.shape or k.shape[0] != B or k.shape[2:] != q.shape[2:] or Hq % Hkv:
        raise ValueError("q [B, H_kv*g, T, d], k and v [B, H_kv, T, d]")
    g = Hq // Hkv
    dt = dtype_code(q.dtype)
    odt = q.dtype if out_dtype is None else out_dtype
    skip = out is False
    if skip and head_out is None:
        raise ValueError("out=False needs head_out")
    if out is None:
        out = torch.empty(B, T, d, dtype=odt, device=q.device)
    if ws is None:
        ws = workspace(int(lib().namoh_attn_fwd_grouped_workspace_size(B, T, Hkv, K_kv, g, d, dt)),
                       q.device)
    check(lib().namoh_attn_fwd_grouped(
        _ptr(q), _ptr(k), _ptr(v), dt, B, T, Hkv, K_kv, g, d, float(rope_base), rope_mode,
        float(softmax_scale), _ptr(routing["gates"]), _ptr(routing["seg_offsets"]),
        _ptr(routing["perm_token"]), _ptr(routing["slot_pos"]), None if skip else _ptr(out),
        dtype_code(odt) if skip else dtype_code(out.dtype), _ptr(head_out), _ptr(ws), ws.numel(),
        _stream(q.device)))
    return head_out if skip else out


def shared_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, window: int,
                rope_base: float, rope_mode: int = ROPE_GLOBAL, softmax_scale: float = 0.0,
                out=None, accumulate: bool = False, out_dtype: Optional[torch.dtype] = None,
                head_out: Optional[torch.Tensor] = None,
                ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """namoh_shared_attn: always-active heads q, k, v [B, Hs, T, d] (bf16),
    causal (window 0) or inside a sliding window; out [B, T, d] (+)= the sum
    of the heads (accumulate adds to the given out).  out=False with
    head_out given skips the sum (returns head_out [B, Hs, T, d] float32)."""
    skip = out is False
    _need_cuda(q, k, v, None if skip else out, head_out)
    B, Hs, T, d = q.shape
    if k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must share [B, Hs, T, d]")
    if skip and head_out is None:
        raise ValueError("out=False needs head_out")
    if out is None:
        out = torch.zeros(B, T, d, dtype=q.dtype if out_dtype is None else out_dtype,
                          device=q.device)
    if ws is None:
        ws = workspace(int(lib().namoh_shared_attn_workspace_size(B, T, Hs, d)), q.device)
    check(lib().namoh_shared_attn(_ptr(q), _ptr(k), _ptr(v), dtype_code(q.dtype), B, T, Hs, d,
                                  int(window), float(rope_base), rope_mode, float(softmax_scale),
                                  None if skip else _ptr(out),
                                  F32 if skip else dtype_code(out.dtype), int(bool(accumulate)),
                                  _ptr(head_out), _ptr(ws), ws.numel(), _stream(q.device)))
    return head_out if skip else out


def _shared_caches(k_cache, v_cache, cache_len, B, Hs, d, dtype):
    cap = k_cache.shape[2]
    if tuple(k_cache.shape) != (B, Hs, cap, d) or tuple(v_cache.shape) != (B, Hs, cap, d):
        raise ValueError("caches must be [B, Hs, cap, d]")
    if k_cache.dtype != dtype or v_cache.dtype != dtype:
        raise ValueError("the caches must have the inputs' dtype")
    if tuple(cache_len.shape) != (B,) or cache_len.dtype != torch.int32:
        raise ValueError("cache_len must be int32 [B]")
    return cap


def shared_decode_step(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                       k_cache: torch.Tensor, v_cache: torch.Tensor, cache_len: torch.Tensor,
                       window: int, rope_base: float, rope_mode: int = ROPE_GLOBAL,
                       softmax_scale: float = 0.0, out: Optional[torch.Tensor] = None,
                       accumulate: bool = False, out_dtype: Optional[torch.dtype] = None,
                       dev_status: Optional[torch.Tensor] = None,
                       ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """namoh_shared_decode_step: the new token's q, k, v [B, Hs, d] for the Hs
    shared heads; caches [B, Hs, cap, d] (rings of the last cap tokens when
    window > 0), cache_len int32 [B]; out [B, d] (+)= the heads' sum."""
    _need_cuda(q, k, v, k_cache, v_cache, cache_len, out, dev_status, ws)
    B, Hs, d = q.shape
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("q, k, v must share [B, Hs, d] and dtype")
    cap = _shared_caches(k_cache, v_cache, cache_len, B, Hs, d, q.dtype)
    if out is None:
        out = torch.zeros(B, d, dtype=q.dtype if out_dtype is None else out_dtype, device=q.device)
    if ws is None:
        ws = workspace(int(lib().namoh_shared_decode_workspace_size(B, Hs, d, cap)), q.device)
    check(lib().namoh_shared_decode_step(_ptr(q), _ptr(k), _ptr(v), dtype_code(q.dtype), B, Hs, d,
                                         cap, int(window), float(rope_base), rope_mode,
                                         float(softmax_scale), _ptr(k_cache), _ptr(v_cache),
                                         _ptr(cache_len), _ptr(out), dtype_code(out.dtype),
                                         int(bool(accumulate)), _ptr(dev_status), _ptr(ws),
                                         ws.numel(), _stream(q.device)))
    return out


def shared_prefill_cache(k: torch.Tensor, v: torch.Tensor, k_cache: torch.Tensor,
                         v_cache: torch.Tensor, cache_len: torch.Tensor, window: int,
                         rope_base: float, rope_mode: int = ROPE_GLOBAL) -> None:
    """namoh_shared_prefill_cache: the prompt's shared-head keys (rotated) and
    values k, v [B, Hs, T, d] into the decode caches; cache_len [B] = T."""
    _need_cuda(k, v, k_cache, v_cache, cache_len)
    B, Hs, T, d = k.shape
    if v.shape != k.shape or v.dtype != k.dtype:
        raise ValueError("k and v must share [B, Hs, T, d] and dtype")
    cap = _shared_caches(k_cache, v_cache, cache_len, B, Hs, d, k.dtype)
    check(lib().namoh_shared_prefill_cache(_ptr(k), _ptr(v), dtype_code(k.dtype), B, T, Hs, d,
                                           cap, int(window), float(rope_base), rope_mode,
                                           _ptr(k_cache), _ptr(v_cache), _ptr(cache_len),
                                           _stream(k.device)))


def prefill_cache(k: torch.Tensor, v: torch.Tensor, r: dict, K: int, rope_base: float,
                  k_cache: torch.Tensor, v_cache: torch.Tensor, cache_len: torch.Tensor,
                  rope_mode: int = ROPE_HEAD_RELATIVE) -> None:
    """namoh_prefill_cache: the prompt's rotated keys / values, per head in rank
    order, into caches [B, H, cap, d]; cache_len [B, H] = the head lengths."""
    _need_cuda(k, v, k_cache, v_cache, cache_len)
    B, H, T, d = k.shape
    cap = k_cache.shape[2]
    if tuple(k_cache.shape) != (B, H, cap, d) or tuple(v_cache.shape) != (B, H, cap, d):
        raise ValueError("caches must be [B, H, cap, d]")
    if k_cache.dtype != k.dtype or v_cache.dtype != k.dtype or v.dtype != k.dtype:
        raise ValueError("k, v and the caches must share one dtype")
    if tuple(cache_len.shape) != (B, H) or cache_len.dtype != torch.int32:
        raise ValueError("cache_len must be int32 [B, H]")
    check(lib().namoh_prefill_cache(_ptr(k), _ptr(v), dtype_code(k.dtype), B, T, H, K, d,
                                    float(rope_base), rope_mode, _ptr(r["seg_offsets"]),
                                    _ptr(r["perm_token"]), _ptr(k_cache), _ptr(v_cache),
                                    _ptr(cache_len), cap, _stream(k.device)))


def attn_fwd_train(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, routing: dict, K: int,
                   rope_base: float, ws: torch.Tensor, rope_mode: int = ROPE_HEAD_RELATIVE,
                   softmax_scale: float = 0.0, out_dtype: Optional[torch.dtype] = None,
                   out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """namoh_attn_fwd_train: the layer output [B, T, d]; `ws` (at least
    namoh_attn_bwd_workspace_size bytes) keeps the state attn_bwd(...,
    saved=True) reads back."""
    _need_cuda(q, k, v, out, ws)
    B, H, T, d = q.shape
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("q, k, v must share shape and dtype")
    odt = q.dtype if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty(B, T, d, dtype=odt, device=q.device)
    check(lib().namoh_attn_fwd_train(_ptr(q), _ptr(k), _ptr(v), dtype_code(q.dtype), B, T, H, K,
                                     d, float(rope_base), rope_mode, float(softmax_scale),
                                     _ptr(routing["gates"]), _ptr(routing["seg_offsets"]),
                                     _ptr(routing["perm_token"]), _ptr(routing["slot_pos"]),
                                     _ptr(out), dtype_code(out.dtype), _ptr(ws), ws.numel(),
                                     _stream(q.device)))
    return out


def attn_bwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, routing: dict, K: int,
             rope_base: float, dout: torch.Tensor, rope_mode: int = ROPE_HEAD_RELATIVE,
             softmax_scale: float = 0.0, ws: Optional[torch.Tensor] = None,
             out: Optional[dict] = None, packed: bool = False, saved: bool = False) -> dict:
    """namoh_attn_bwd: gradients dq, dk, dv [B, H, T, d] and dgates [B, T, K]
    (float32) for the upstream gradient dout float32 [B, T, d]; `out` may
    hold preallocated tensors of those shapes under the same keys.  With
    packed=True, namoh_attn_bwd_packed: dq, dk, dv [B*T*K, d] in the
    routing's packed order.  With saved=True, namoh_attn_bwd_saved on the
    state attn_fwd_train left in `ws`."""
    _need_cuda(q, k, v, dout)
    B, H, T, d = q.shape
    if k.shape != q.shape or v.shape != q.shape or k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("q, k, v must share shape and dtype")
    if dout.dtype != torch.float32 or tuple(dout.shape) != (B, T, d):
        raise ValueError("dout must be float32 [B, T, d]")
    dev = q.device
    f32 = dict(dtype=torch.float32, device=dev)
    gshape = (B * T * K, d) if packed else (B, H, T, d)
    if out is None:
        out = {"dq": torch.empty(*gshape, **f32), "dk": torch.empty(*gshape, **f32),
               "dv": torch.empty(*gshape, **f32), "dgates": torch.empty(B, T, K, **f32)}
    for key, shape in (("dq", gshape), ("dk", gshape), ("dv", gshape), ("dgates", (B, T, K))):
        if out[key].dtype != torch.float32 or tuple(out[key].shape) != shape \
                or not out[key].is_contiguous():
            raise ValueError(f"out[{key!r}] must be contiguous float32 {shape}")
    if ws is None:
        if saved:
            raise ValueError("saved=True needs the workspace attn_fwd_train used")
        ws = workspace(int(lib().namoh_attn_bwd_workspace_size(B, T, H, K, d)), dev)
    args = (_ptr(q), _ptr(k), _ptr(v), dtype_code(q.dtype), B, T, H, K, d, float(rope_base),
            rope_mode, float(softmax_scale), _ptr(routing["topk_idx"]), _ptr(routing["gates"]),
            _ptr(routing["seg_offsets"]), _ptr(routing["perm_token"]), _ptr(dout),
            _ptr(out["dq"]), _ptr(out["dk"]), _ptr(out["dv"]), _ptr(out["dgates"]))
    if saved:
        check(lib().namoh_attn_bwd_saved(*args, 1 if packed else 0, _ptr(ws), ws.numel(),
                                         _stream(dev)))
    else:
        fn = lib().namoh_attn_bwd_packed if packed else lib().namoh_attn_bwd
        check(fn(*args, _ptr(ws), ws.numel(), _stream(dev)))
    return out


def route_bwd(logits: torch.Tensor, routing: dict, dgates: torch.Tensor,
              gate_mode: int = GATE_SOFTMAX_SELECTED) -> torch.Tensor:
    """namoh_route_bwd: d logits [B, T, H] from the gate gradients."""
    _need_cuda(logits, dgates)
    B, T, H = logits.shape
    K = dgates.shape[-1]
    dl = torch.empty(B, T, H, dtype=torch.float32, device=logits.device)
    check(lib().namoh_route_bwd(_ptr(logits), _ptr(routing["topk_idx"]), _ptr(routing["gates"]),
                                _ptr(dgates), B, T, H, K, gate_mode, _ptr(dl),
                                _stream(logits.device)))
    return dl


def decode_step_grouped(logits: torch.Tensor, q: torch.Tensor, k: torch.Tensor,
                        v: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                        cache_len: torch.Tensor, K_kv: int, rope_base: float,
                        rope_mode: int = ROPE_HEAD_RELATIVE,
                        gate_mode: int = GATE_SOFTMAX_SELECTED, softmax_scale: float = 0.0,
                        seq_pos: Optional[torch.Tensor] = None,
                        out_dtype: Optional[torch.dtype] = None,
                        dev_status: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None) -> dict:
    """namoh_decode_step_grouped: group logits [B, H_kv], q [B, H_kv*g, d],
    k, v [B, H_kv, d], caches [B, H_kv, cap, d] (bf16), updated in place."""
    _need_cuda(logits, q, k, v, k_cache, v_cache, cache_len, seq_pos, dev_status)
    B, Hq, d = q.shape
    Hkv = k.shape[1]
    if Hq % Hkv or k.shape != v.shape or k.shape[0] != B or k.shape[2] != d:
        raise ValueError("q [B, H_kv*g, d], k and v [B, H_kv, d]")
    g = Hq // Hkv
    cap = k_cache.shape[2]
    dev = q.device
    odt = q.dtype if out_dtype is None else out_dtype
    res = {"topk_idx": torch.empty(B, K_kv, dtype=torch.int32, device=dev),
           "gates": torch.empty(B, K_kv, dtype=torch.float32, device=dev),
           "out": torch.empty(B, d, dtype=odt, device=dev)}
    if ws is None:
        ws = workspace(int(lib().namoh_decode_grouped_workspace_size(B, Hkv, K_kv, g, d, cap)), dev)
    check(lib().namoh_decode_step_grouped(
        _ptr(logits), _ptr(q), _ptr(k), _ptr(v), dtype_code(q.dtype), _ptr(k_cache),
        _ptr(v_cache), _ptr(cache_len), _ptr(seq_pos), B, Hkv, K_kv, g, d, cap, float(rope_base),
        rope_mode, gate_mode, float(softmax_scale), _ptr(res["topk_idx"]), _ptr(res["gates"]),
        _ptr(res["out"]), dtype_code(odt), _ptr(dev_status), _ptr(ws), ws.numel(),
        _stream(dev)))
    return res


def qkv_proj(x: torch.Tensor, w_qkv: torch.Tensor, routing: dict, H: int, K: int,
             out: Optional[dict] = None) -> dict:
    """namoh_qkv_proj: q, k, v [B, H, T, d] (bf16) of the routed pairs from
    x [B, T, d_model] and w_qkv [H, 3, d, d_model] (bf16).  Rows of unrouted
    pairs are left as they are (uninitialised unless `out` is given)."""
    _need_cuda(x, w_qkv)
    if x.dtype != torch.bfloat16 or w_qkv.dtype != torch.bfloat16:
        raise ValueError("x and w_qkv must be bfloat16")
    B, T, dm = x.shape
    if w_qkv.dim() != 4 or w_qkv.shape[0] != H or w_qkv.shape[1] != 3 or w_qkv.shape[3] != dm:
        raise ValueError("w_qkv must be [H, 3, d, d_model]")
    d = w_qkv.shape[2]
    if out is None:
        out = {n: torch.empty(B, H, T, d, dtype=torch.bfloat16, device=x.device)
               for n in ("q", "k", "v")}
    for n in ("q", "k", "v"):
        _need_cuda(out[n])
        if out[n].dtype != torch.bfloat16 or tuple(out[n].shape) != (B, H, T, d):
            raise ValueError(f"out[{n!r}] must be bfloat16 [B, H, T, d]")
    check(lib().namoh_qkv_proj(_ptr(x), _ptr(w_qkv), B, T, H, K, d, dm,
                               _ptr(routing["seg_offsets"]), _ptr(routing["perm_token"]),
                               _ptr(out["q"]), _ptr(out["k"]), _ptr(out["v"]), _stream(x.device)))
    return out


def out_proj_workspace_size(B, T, H, K, d, d_model) -> int:
    return int(lib().namoh_out_proj_workspace_size(B, T, H, K, d, d_model))


def out_proj(head_out: torch.Tensor, w_o: torch.Tensor, routing: dict, B: int, T: int, H: int,
             K: int, out_dtype: torch.dtype = torch.float32, out: Optional[torch.Tensor] = None,
             ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """namoh_out_proj: o [B, T, d_model] = sum_k gate * (h W_O^(i)) from the
    packed head outputs head_out [B*T*K, d] (float32 or bf16) and
    w_o [H, d_model, d] (bf16)."""
    _need_cuda(head_out, w_o, out)
    if w_o.dtype != torch.bfloat16 or w_o.dim() != 3 or w_o.shape[0] != H:
        raise ValueError("w_o must be bfloat16 [H, d_model, d]")
    dm, d = w_o.shape[1], w_o.shape[2]
    if tuple(head_out.shape) != (B * T * K, d):
        raise ValueError("head_out must be [B*T*K, d]")
    if out is None:
        out = torch.empty(B, T, dm, dtype=out_dtype, device=w_o.device)
    if ws is None:
        ws = workspace(out_proj_workspace_size(B, T, H, K, d, dm), w_o.device)
    check(lib().namoh_out_proj(_ptr(head_out), dtype_code(head_out.dtype), _ptr(w_o),
                               _ptr(routing["gates"]), _ptr(routing["slot_pos"]),
                               _ptr(routing["seg_offsets"]), B, T, H, K, d, dm, _ptr(out),
                               dtype_code(out.dtype), _ptr(ws), ws.numel(), _stream(w_o.device)))
    return out


def decode_workspace_size(B, H, K, d, cap) -> int:
    return int(lib().namoh_decode_workspace_size(B, H, K, d, cap))


def decode_step(logits: torch.Tensor, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                k_cache: torch.Tensor, v_cache: torch.Tensor, cache_len: torch.Tensor,
                K: int, rope_base: float, rope_mode: int = ROPE_HEAD_RELATIVE,
                gate_mode: int = GATE_SOFTMAX_SELECTED, softmax_scale: float = 0.0,
                seq_pos: Optional[torch.Tensor] = None,
                out_dtype: Optional[torch.dtype] = None,
                dev_status: Optional[torch.Tensor] = None,
                out: Optional[dict] = None, ws: Optional[torch.Tensor] = None,
                bias: Optional[torch.Tensor] = None) -> dict:
    """namoh_decode_step; caches [B, H, cap, d] are updated in place.  With a
    float32 [H] `bias`, namoh_decode_step_biased (gate_mode is then ignored)."""
    _need_cuda(logits, q, k, v, k_cache, v_cache, cache_len, seq_pos, dev_status, bias)
    B, H, d = q.shape
    cap = k_cache.shape[2]
    dt = dtype_code(q.dtype)
    dev = q.device
    if out is None:
        out = {
            "topk_idx": torch.empty(B, K, dtype=torch.int32, device=dev),
            "gates": torch.empty(B, K, dtype=torch.float32, device=dev),
            "out": torch.empty(B, d, dtype=q.dtype if out_dtype is None else out_dtype, device=dev),
        }
    if ws is None:
        ws = workspace(decode_workspace_size(B, H, K, d, cap), dev)
    tail = (float(softmax_scale), _ptr(out["topk_idx"]), _ptr(out["gates"]), _ptr(out["out"]),
            dtype_code(out["out"].dtype), _ptr(dev_status), _ptr(ws), ws.numel(), _stream(dev))
    if bias is None:
        check(lib().namoh_decode_step(_ptr(logits), _ptr(q), _ptr(k), _ptr(v), dt,
                                      _ptr(k_cache), _ptr(v_cache), _ptr(cache_len),
                                      _ptr(seq_pos), B, H, K, d, cap, float(rope_base),
                                      rope_mode, gate_mode, *tail))
    else:
        if bias.dtype != torch.float32 or bias.shape != (H,):
            raise ValueError("bias must be float32 [H]")
        check(lib().namoh_decode_step_biased(_ptr(logits), _ptr(bias), _ptr(q), _ptr(k), _ptr(v),
                                             dt, _ptr(k_cache), _ptr(v_cache), _ptr(cache_len),
                                             _ptr(seq_pos), B, H, K, d, cap, float(rope_base),
                                             rope_mode, *tail))
    return out


def decode_step_noalloc(logits: torch.Tensor, q: torch.Tensor, k: torch.Tensor,
                        v: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                        cache_len: torch.Tensor, K: int, rope_base: float,
                        rope_mode: int = ROPE_HEAD_RELATIVE,
                        gate_mode: int = GATE_SOFTMAX_SELECTED, softmax_scale: float = 0.0,
                        seq_pos: Optional[torch.Tensor] = None,
                        dev_status: Optional[torch.Tensor] = None, out: dict = None) -> dict:
    """namoh_decode_step_noalloc: the decode step without a workspace (the
    library's fixed per-GPU scratch).  `out` holds caller-allocated
    topk_idx [B, K] int32, gates [B, K] float32 and out [B, d]."""
    _need_cuda(logits, q, k, v, k_cache, v_cache, cache_len, seq_pos, dev_status,
               out["topk_idx"], out["gates"], out["out"])
    B, H, d = q.shape
    cap = k_cache.shape[2]
    check(lib().namoh_decode_step_noalloc(
        _ptr(logits), _ptr(q), _ptr(k), _ptr(v), dtype_code(q.dtype), _ptr(k_cache),
        _ptr(v_cache), _ptr(cache_len), _ptr(seq_pos), B, H, K, d, cap, float(rope_base),
        rope_mode, gate_mode, float(softmax_scale), _ptr(out["topk_idx"]), _ptr(out["gates"]),
        _ptr(out["out"]), dtype_code(out["out"].dtype), _ptr(dev_status), _stream(q.device)))
    return out


# ----------------------------------------------------------------------------
def profile_enable(capacity: int) -> None:
    """Start (capacity > 0) or stop (0) event timing of the main kernels."""
    lib().namoh_profile_enable(int(capacity))


def profile_read(section: str):
    """(total milliseconds, launch count) of a timed section, or None."""
    ms = ctypes.c_double()
    n = ctypes.c_int()
    if lib().namoh_profile_read(section.encode(), ctypes.byref(ms), ctypes.byref(n)) != 0:
        return None
    return ms.value, n.value
