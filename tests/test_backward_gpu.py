"""GPU parity of hybrid_attn_backward (the Stage-1 gradient of Section 3.2
with respect to W and alpha) against the fp64 oracle, through the C ABI.

Tolerances.  bf16 inputs: max |gpu - oracle| <= 2e-2 * rms(oracle) for dW,
and for dalpha and the loss (each compared as a vector over heads).  fp32
inputs: max |gpu - oracle| <= 1e-5 * max(1, max |oracle|): the gradients are
sums over every token of the sequence, so the fp32 bound is taken relative
to their scale (an absolute 1e-5 would ask for more than fp32 accumulation
of T terms can give once they reach order 10).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import act, announce, f32, host

pytestmark = pytest.mark.gpu


def _close(got, ref, dt, what):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite"
    err = float(np.abs(got - ref).max())
    amax = float(np.abs(ref).max())
    if dt == "f32":
        tol = 1e-5 * max(1.0, amax)
    else:
        tol = 2e-2 * float(np.sqrt(np.mean(ref ** 2)))
    print(f"[parity] {what}: max abs err {err:.3e} (tol {tol:.3e}, max |ref| {amax:.3e}"
          f"{', within the absolute 1e-5' if err <= 1e-5 else ''})")
    assert err <= tol, f"{what}: max abs err {err:.3e} > tol {tol:.3e}"


def _case(B, T, Hq, Hkv, d, L, F, dt, seed, w_std=None):
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=F, dtype=dt)
    q, k, v = synth.sequence_qkv(dims, T, seed, 1.0)
    Wt, alpha = synth.feature_weights(dims, seed + 1, seed + 2,
                                      w_std if w_std is not None else 1.0 / np.sqrt(d))
    g = synth.upstream(dims, T, seed + 3, 1.0)
    return dims, q, k, v, Wt, alpha, g


def _run(dims, q, k, v, Wt, alpha, L, dout=None, target=None):
    dt = dims.dtype
    dW, da, loss = hb.hybrid_attn_backward(
        act(q, dt), act(k, dt), act(v, dt), act(Wt, dt), f32(alpha), L,
        dout=act(dout, dt) if dout is not None else None,
        target=act(target, dt) if target is not None else None)
    torch.cuda.synchronize()
    return host(dW), host(da), (host(loss) if loss is not None else None)


SHAPES = [
    # (B, T, Hq, Hkv, d, L, F, dtype)
    (2, 96, 4, 2, 64, 32, 32, "f32"),
    (1, 64, 2, 1, 128, 32, 64, "f32"),
    (2, 80, 2, 2, 128, 16, 32, "f32"),
    (2, 128, 4, 2, 128, 32, 64, "bf16"),
    (2, 160, 4, 1, 64, 16, 64, "bf16"),
    (1, 40, 2, 2, 128, 8, 32, "bf16"),
    (1, 1024, 4, 2, 128, 32, 64, "bf16"),   # 8 sequence segments
    (3, 512, 8, 2, 64, 32, 32, "bf16"),
    (1, 32, 2, 1, 128, 32, 64, "bf16"),     # one block: both gradients vanish
    # 13 blocks: 3 segments of 5, increments in pieces of 3 blocks; the last
    # segment's second reverse piece is empty
    (1, 416, 2, 1, 64, 32, 32, "bf16"),
    (1, 416, 2, 1, 64, 32, 32, "f32"),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("mode", ["dout", "target"])
def test_backward_matches_oracle(shape, mode):
    B, T, Hq, Hkv, d, L, F, dt = shape
    announce(f"backward {shape} {mode}")
    dims, q, k, v, Wt, alpha, g = _case(B, T, Hq, Hkv, d, L, F, dt, seed=40)
    kw = dict(dout=g) if mode == "dout" else dict(target=g * 0.05)
    ref_W, ref_a, ref_l = oracle.backward(q, k, v, Wt, alpha, L, **kw)
    dW, da, loss = _run(dims, q, k, v, Wt, alpha, L, **kw)
    if T == L:
        # One block: dW is exactly zero (empty state, no later blocks); dalpha
        # is a sum of B*T terms g.acc_sm - (g.out) den that cancel exactly,
        # so only their fp32 rounding remains.
        assert np.abs(dW).max() == 0.0, "one block: dW must vanish"
        assert np.abs(da).max() <= 1e-5 * B * T
    else:
        _close(dW, ref_W, dt, f"dW {shape} {mode}")
        _close(da, ref_a, dt, f"dalpha {shape} {mode}")
    if mode == "target":
        _close(loss, ref_l, dt, f"loss {shape}")
    else:
        assert loss is None


def test_backward_peaky_and_deterministic():
    """Larger logits (sharper block softmax and feature map); two calls give
    the same bits."""
    dims, q, k, v, Wt, alpha, g = _case(2, 256, 4, 2, 128, 32, 64, "bf16", seed=41, w_std=0.15)
    q, k = q * 2.0, k * 2.0
    q, k = synth.to_dtype(q, "bf16"), synth.to_dtype(k, "bf16")
    announce("backward peaky")
    ref_W, ref_a, _ = oracle.backward(q, k, v, Wt, alpha, 32, dout=g)
    a = _run(dims, q, k, v, Wt, alpha, 32, dout=g)
    b = _run(dims, q, k, v, Wt, alpha, 32, dout=g)
    _close(a[0], ref_W, "bf16", "dW peaky")
    _close(a[1], ref_a, "bf16", "dalpha peaky")
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_backward_equal_values_vanish():
    """v_t equal for all t: out = v whatever W and alpha, so the gradients
    vanish (up to the rounding of the kernels' arithmetic)."""
    dims, q, k, v, Wt, alpha, g = _case(1, 128, 2, 1, 128, 32, 64, "f32", seed=42)
    v[:] = v[:, :1]
    dW, da, _ = _run(dims, q, k, v, Wt, alpha, 32, dout=g)
    ref_W, _, _ = oracle.backward(q, k, v, Wt, alpha, 32, dout=g)
    assert np.abs(ref_W).max() < 1e-12
    # scale of the terms that cancel: the same call with distinct values
    dims2, q2, k2, v2, _, _, _ = _case(1, 128, 2, 1, 128, 32, 64, "f32", seed=42)
    scale = np.abs(oracle.backward(q2, k2, v2, Wt, alpha, 32, dout=g)[0]).max()
    assert np.abs(dW).max() <= 1e-5 * max(1.0, scale)
    assert np.abs(da).max() <= 1e-5
