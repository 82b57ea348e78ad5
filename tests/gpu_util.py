"""Helpers shared by the GPU parity tests: device upload of the seeded
inputs, calls through the C-ABI binding, tolerance checks."""
import sys

import numpy as np
import torch

from paper_2609_38832_amd import _lib as L
from paper_2609_38832_amd import workloads as W

DEV = torch.device("cuda:0")

# Acceptance tolerances: fp32 max abs 1e-4; bf16 |got - ref| <= 2e-2 + 1e-2 |ref|
# against the float64 oracle; the relative L2 error gate 1e-2 is an extra
# internal check (bf16 rounding of rotated q/k and of the probabilities gives
# about 3e-3).
F32_ATOL = 1e-4
BF16_ATOL, BF16_RTOL, REL_L2 = 2e-2, 1e-2, 1e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def from_dev(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy()


def run_prefill(w: W.Workload, inp: dict, rope_mode=0, gate_mode=0, out_dtype=torch.float32,
                head_out=False):
    lg = torch.from_numpy(inp["logits"]).to(DEV)
    q, k, v = (to_dev(inp[n], w.dtype) for n in ("q", "k", "v"))
    r = L.route(lg, w.K, gate_mode)
    ho = None
    if head_out:
        ho = torch.empty(w.B * w.T * w.K, w.d, dtype=torch.float32, device=DEV)
    o = L.attn_fwd(q, k, v, r, w.K, w.rope_base, rope_mode, out_dtype=out_dtype, head_out=ho)
    torch.cuda.synchronize()
    res = {key: val.cpu().numpy() for key, val in r.items()}
    res["out"] = from_dev(o)
    if ho is not None:
        res["head_out"] = ho.cpu().numpy()
    return res


def assert_routing_exact(got: dict, ref: dict):
    for key in ("topk_idx", "head_len", "seg_offsets", "perm_token", "slot_pos"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)
    np.testing.assert_allclose(got["gates"], ref["gates"], rtol=2e-6, atol=1e-7)


def check_out(got: np.ndarray, ref: np.ndarray, dtype: str, what="out"):
    got = np.asarray(got, dtype=np.float64)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    diff = np.abs(got - ref)
    if dtype == "f32":
        assert diff.max() <= F32_ATOL, f"{what}: max abs err {diff.max():.3e}"
    else:
        bad = diff > BF16_ATOL + BF16_RTOL * np.abs(ref)
        assert not bad.any(), f"{what}: {bad.sum()} elements out of tolerance, max {diff.max():.3e}"
        rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
        assert rel <= REL_L2, f"{what}: relative L2 error {rel:.3e}"
    return float(diff.max())
