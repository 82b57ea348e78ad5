"""The bf16 gradient tolerance of the backward parity tests, checked on the CPU.

The MFMA backward rounds these operands to bf16 before their products and
accumulates in fp32 (Sec. 3.2 "Efficient execution": training runs the same
packed varlen attention): the scaled rotated queries, the rotated keys, the
values, the gated output gradients g*dout, the probabilities P (for dV) and
dS = P (dP - D) (for dQ and dK).  Here a float64 model of exactly those
rounding points is compared with the exact float64 gradients of one causal
head (the textbook softmax-attention backward, Eq. namoh-attention on one
segment), at the parity tests' shapes and scales:

* correct arithmetic with those roundings stays well inside the tolerance
  (the bound is not too tight), and
* a plausible mistake in the kernels (the -D term dropped, the row
  statistic taken as the maximum alone, the causal mask shifted by one, the
  ln 2 factor of dK missing) exceeds it (the bound is not too loose).
"""
import numpy as np
import pytest

from test_gpu_parity import GRAD_TOL_BF16

LOG2E = 1.4426950408889634


def bf16(x):
    """Round float64 values to bf16 (round to nearest even via float32)."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def exact_grads(q, k, v, do, scale):
    n = q.shape[0]
    s = (q @ k.T) * scale
    s[np.triu_indices(n, 1)] = -np.inf
    p = np.exp(s - s.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    o = p @ v
    dv = p.T @ do
    dp = do @ v.T
    ds = p * (dp - (do * o).sum(axis=1, keepdims=True))
    return ds @ k * scale, ds.T @ q * scale, dv


def kernel_model(q, k, v, do, scale, drop_d=False, max_only=False, mask_shift=0, ln2_dk=True):
    """The kernels' arithmetic: bf16 operands, float64 standing in for the
    fp32 accumulation, scores in log2 units."""
    n = q.shape[0]
    qs = bf16(q * scale * LOG2E)
    kb, vb, dob = bf16(k), bf16(v), bf16(do)
    s = qs @ kb.T
    s[np.triu_indices(n, 1 + mask_shift)] = -np.inf
    m = s.max(axis=1, keepdims=True)
    lse = m if max_only else m + np.log2(np.exp2(s - m).sum(axis=1, keepdims=True))
    p = np.exp2(s - lse)
    o = bf16(p) @ vb                       # the forward's head output (bf16 P . V)
    dd = 0.0 if drop_d else (dob * o).sum(axis=1, keepdims=True)
    dv = bf16(p).T @ dob
    dp = dob @ vb.T
    ds = bf16(p * (dp - dd))
    dq = (ds @ kb) * scale
    dk = (ds.T @ qs) * (np.log(2.0) if ln2_dk else 1.0)
    return dq, dk, dv


def within(got, ref, rel, rel_l2):
    scale = np.abs(ref).max()
    ok_max = np.all(np.abs(got - ref) <= rel * scale + rel * np.abs(ref))
    ok_l2 = np.linalg.norm(got - ref) / np.linalg.norm(ref) <= rel_l2
    return ok_max and ok_l2, float(np.abs(got - ref).max() / scale)


def case(n, d, seed):
    rng = np.random.default_rng(seed)
    # the parity workloads' draws: bf16 inputs, normal q/k/v, qkv scale d^-1/2
    q, k, v = (bf16(rng.standard_normal((n, d))) for _ in range(3))
    do = rng.standard_normal((n, d)) * 0.7    # g * dout with a gate below 1
    return q, k, v, do, 1.0 / np.sqrt(d)


@pytest.mark.parametrize("n,d,seed", [(300, 64, 1), (700, 64, 2), (500, 128, 3), (1200, 128, 4)])
def test_bf16_rounding_is_inside_the_tolerance(n, d, seed):
    q, k, v, do, scale = case(n, d, seed)
    ref = exact_grads(q, k, v, do, scale)
    got = kernel_model(q, k, v, do, scale)
    rel, rel_l2 = GRAD_TOL_BF16["rel"], GRAD_TOL_BF16["rel_l2"]
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        ok, err = within(g, r, rel, rel_l2)
        assert ok, f"{name}: rounding alone gives {err:.2e}"
        # with a margin: the observed GPU errors are 2e-3 .. 7e-3
        assert err < rel / 2, f"{name}: {err:.2e} leaves no margin under {rel}"


@pytest.mark.parametrize("mistake", ["drop_d", "mask_shift", "no_ln2", "max_only"])
def test_plausible_mistakes_exceed_the_tolerance(mistake):
    q, k, v, do, scale = case(500, 64, 5)
    ref = exact_grads(q, k, v, do, scale)
    kw = {"drop_d": dict(drop_d=True), "mask_shift": dict(mask_shift=1),
          "no_ln2": dict(ln2_dk=False), "max_only": dict(max_only=True)}[mistake]
    got = kernel_model(q, k, v, do, scale, **kw)
    rel, rel_l2 = GRAD_TOL_BF16["rel"], GRAD_TOL_BF16["rel_l2"]
    oks = [within(g, r, rel, rel_l2)[0] for g, r in zip(got, ref)]
    assert not all(oks), f"{mistake} passes the bf16 tolerance"
