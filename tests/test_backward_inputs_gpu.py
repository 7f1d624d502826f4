"""GPU parity of hybrid_attn_backward_full: the gradients of the
block-causal hybrid layer with respect to its inputs q, k, v (end-to-end
training through the hybrid layers, Stage 2 of Section 3.2), and with them
dW, dalpha and the loss, against the fp64 oracle through the C ABI.

Tolerances as for hybrid_attn_backward: bf16 inputs, max |gpu - oracle|
<= 2e-2 * rms(oracle); fp32 inputs, max |gpu - oracle| <= 1e-5 * max(1,
max |oracle|) (each printed beside max |oracle|).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import act, announce, f32, host
from test_backward_gpu import _case, _close

pytestmark = pytest.mark.gpu


def _run_full(dims, q, k, v, Wt, alpha, L, dout=None, target=None):
    dt = dims.dtype
    res = hb.hybrid_attn_backward_full(
        act(q, dt), act(k, dt), act(v, dt), act(Wt, dt), f32(alpha), L,
        dout=act(dout, dt) if dout is not None else None,
        target=act(target, dt) if target is not None else None)
    torch.cuda.synchronize()
    return [host(x) if x is not None else None for x in res]


SHAPES = [
    # (B, T, Hq, Hkv, d, L, F, dtype)
    (2, 96, 4, 2, 64, 32, 32, "f32"),
    (1, 64, 2, 1, 128, 32, 64, "f32"),
    (2, 80, 2, 2, 128, 16, 32, "f32"),
    (2, 128, 4, 2, 128, 32, 64, "bf16"),
    (2, 160, 4, 1, 64, 16, 64, "bf16"),
    (1, 40, 2, 2, 128, 8, 32, "bf16"),
    (1, 1024, 4, 2, 128, 32, 64, "bf16"),   # 8 sequence segments
    (1, 35, 2, 1, 64, 5, 32, "bf16"),       # odd block length
    (1, 32, 2, 1, 128, 32, 64, "bf16"),     # one block: softmax attention only
    # 13 blocks: 3 segments of 5, increments in pieces of 3 blocks; the last
    # segment's second reverse piece is empty
    (1, 416, 2, 1, 64, 32, 32, "bf16"),
    (1, 416, 2, 1, 64, 32, 32, "f32"),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("mode", ["dout", "target"])
def test_input_gradients_match_oracle(shape, mode):
    B, T, Hq, Hkv, d, L, F, dt = shape
    announce(f"backward_full {shape} {mode}")
    dims, q, k, v, Wt, alpha, g = _case(B, T, Hq, Hkv, d, L, F, dt, seed=140)
    kw = dict(dout=g) if mode == "dout" else dict(target=g * 0.05)
    ref = oracle.backward(q, k, v, Wt, alpha, L, inputs=True, **kw)
    got = _run_full(dims, q, k, v, Wt, alpha, L, **kw)
    for x, r, what in zip((got[0], got[1], got[2]), ref[3:], ("dq", "dk", "dv")):
        _close(x, r, dt, f"{what} {shape} {mode}")
    if T > L:
        _close(got[3], ref[0], dt, f"dW (full call) {shape} {mode}")
        _close(got[4], ref[1], dt, f"dalpha (full call) {shape} {mode}")
    else:
        assert np.abs(got[3]).max() == 0.0
    if mode == "target":
        _close(got[5], ref[2], dt, f"loss (full call) {shape}")


def test_input_gradients_peaky_and_deterministic():
    dims, q, k, v, Wt, alpha, g = _case(2, 256, 4, 2, 128, 32, 64, "bf16", seed=141, w_std=0.15)
    q, k = synth.to_dtype(q * 2.0, "bf16"), synth.to_dtype(k * 2.0, "bf16")
    announce("backward_full peaky")
    ref = oracle.backward(q, k, v, Wt, alpha, 32, dout=g, inputs=True)
    a = _run_full(dims, q, k, v, Wt, alpha, 32, dout=g)
    b = _run_full(dims, q, k, v, Wt, alpha, 32, dout=g)
    for x, r, what in zip(a[:3], ref[3:], ("dq", "dk", "dv")):
        _close(x, r, "bf16", f"{what} peaky")
    for x, y in zip(a[:5], b[:5]):
        assert np.array_equal(x, y), "two calls differ"


def test_train8_input_gradients_full():
    """At the benchmark's training size (8 sequences of 2048 tokens, 16q/4kv,
    d=128, f=128, blocks of 32, attention-transfer mode): every element of dq,
    dk, dv against the oracle on the whole batch."""
    dims = synth.TRAIN8
    T = synth.TRAIN8_T
    q, k, v = synth.sequence_qkv(dims, T, 161, 1.0)
    Wt, alpha = synth.feature_weights(dims, 162, 163, 1.0 / math.sqrt(dims.d))
    tgt = synth.upstream(dims, T, 164, 0.05)
    announce("train8: backward_full B=8 x 2048 tokens")
    got = _run_full(dims, q, k, v, Wt, alpha, dims.L, target=tgt)
    ref = oracle.backward(q, k, v, Wt, alpha, dims.L, target=tgt, inputs=True)
    for x, r, what in zip(got[:3] + got[3:6], ref[3:] + ref[:3],
                          ("dq", "dk", "dv", "dW", "dalpha", "loss")):
        _close(x, r, "bf16", f"train8 {what}")
