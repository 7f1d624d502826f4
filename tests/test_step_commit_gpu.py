"""GPU parity of hybrid_attn_step_commit (the step fused with the commit of the
same block) against the fp64 oracle, through the C ABI.

The output is held to the step's rule on the state as it was, the state to
the commit's rule on the change it makes.  The output must also equal the
library's own hybrid_attn_step output bit for bit: the fused kernel computes
it with the same code before it touches the state.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import act, announce, assert_close, f32, host, i32, make_case, state_dev, state_host

pytestmark = pytest.mark.gpu


def _inputs(c, dt):
    return (act(c["q"], dt), act(c["k"], dt), act(c["v"], dt), act(c["Wt"], dt), f32(c["alpha"]))


def run_fused(c, dt, out_f32, slots=None):
    S, z = state_dev(c["S"]), f32(c["z"])
    out = hb.hybrid_attn_step_commit(*_inputs(c, dt), S, z, slots=slots, out_f32=out_f32)
    torch.cuda.synchronize()
    return out, S, z


def check_fused(c, dims, what):
    dt = dims.dtype
    ref_out, Sr, zr = oracle.step_commit(c["q"], c["k"], c["v"], c["Wt"], c["alpha"], c["S"], c["z"])
    o32, S1, z1 = run_fused(c, dt, out_f32=(dt == "bf16"))
    assert_close(host(o32), ref_out, dt, what + " out" + (" (fp32 out)" if dt == "bf16" else ""))
    assert_close(state_host(S1) - c["S"], Sr - c["S"], dt, what + " dS")
    assert_close(host(z1) - c["z"], zr - c["z"], dt, what + " dz")
    # the same output as the library's per-head step kernel (the fused
    # kernel is that kernel with the commit) on the untouched state
    step = hb.hybrid_attn_step(*_inputs(c, dt), state_dev(c["S"]), f32(c["z"]),
                               out_f32=(dt == "bf16"), kernel="whole")
    torch.cuda.synchronize()
    assert torch.equal(o32, step), f"{what}: fused output differs from the step's"
    if dt == "bf16":
        o16, S2, z2 = run_fused(c, dt, out_f32=False)
        assert torch.equal(o16.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16))
        assert torch.equal(S2, S1) and torch.equal(z2, z1), f"{what}: state not deterministic"


SHAPES = [
    # (B, Hq, Hkv, d, L, F, dtype, P)
    (2, 4, 2, 64, 8, 32, "f32", 24),
    (3, 4, 1, 64, 5, 32, "f32", 10),
    (2, 2, 2, 128, 32, 64, "f32", 64),
    (2, 8, 2, 128, 16, 128, "f32", 48),
    (2, 4, 4, 64, 32, 64, "bf16", 96),
    (3, 8, 1, 128, 1, 32, "bf16", 40),
    (2, 16, 4, 128, 32, 64, "bf16", 256),
    (2, 8, 8, 128, 32, 128, "bf16", 128),
    (2, 4, 2, 64, 17, 128, "bf16", 34),
    (2, 4, 2, 128, 7, 64, "bf16", 0),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("peaky", [False, True])
def test_step_commit_shapes(shape, peaky):
    B, Hq, Hkv, d, L, F, dt, P = shape
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=F, dtype=dt)
    announce(f"step_commit {shape} peaky={peaky}")
    c = make_case(dims, P, seed=15, peaky=peaky)
    check_fused(c, dims, f"step_commit {shape} peaky={peaky}")


def test_step_commit_slots_and_bad_slot():
    """Slot indirection; a request without a valid slot gets NaN outputs and
    leaves every state row untouched."""
    dims = synth.Dims(B=3, Hq=4, Hkv=2, d=128, L=32, F=64, dtype="bf16")
    slots = np.array([4, 0, 2], np.int32)
    announce("step_commit slots")
    c = make_case(dims, 64, seed=22, peaky=True, n_slots=5, slots=slots)
    bad = np.array([4, 7, 2], np.int32)
    out, S1, z1 = run_fused(c, "bf16", out_f32=True, slots=i32(bad))
    o = host(out)
    assert np.isnan(o[1]).all() and np.isfinite(o[[0, 2]]).all()
    good = np.array([4, 2], np.int32)
    sel = [0, 2]
    ref_out, Sr, zr = oracle.step_commit(c["q"][sel], c["k"][sel], c["v"][sel], c["Wt"], c["alpha"],
                                         c["S"], c["z"], slots=good)
    assert_close(o[sel], ref_out, "bf16", "step_commit slots out")
    assert_close(state_host(S1) - c["S"], Sr - c["S"], "bf16", "step_commit slots dS")
    assert_close(host(z1) - c["z"], zr - c["z"], "bf16", "step_commit slots dz")
    for s in (0, 1, 3):
        assert torch.equal(S1[s], state_dev(c["S"])[s])
        assert torch.equal(z1[s], f32(c["z"])[s])


def test_step_commit_walk_equals_prefill():
    """Serving 6 blocks with the fused call from a state equals the oracle's
    block-causal prefill of the same tokens (outputs and final state)."""
    dims = synth.Dims(B=2, Hq=8, Hkv=2, d=128, L=32, F=64, dtype="bf16")
    T = 6 * dims.L
    announce("step_commit walk")
    c = make_case(dims, 96, seed=23)
    q, k, v = synth.block_qkv(dims.with_(L=T), 24, 1.0 / np.sqrt(dims.d))
    S, z = state_dev(c["S"]), f32(c["z"])
    W, al = act(c["Wt"], "bf16"), f32(c["alpha"])
    outs = []
    for blk in range(T // dims.L):
        sl = slice(blk * dims.L, (blk + 1) * dims.L)
        outs.append(host(hb.hybrid_attn_step_commit(act(q[:, sl], "bf16"), act(k[:, sl], "bf16"),
                                                    act(v[:, sl], "bf16"), W, al, S, z,
                                                    out_f32=True)))
    torch.cuda.synchronize()
    o_r, Sr, zr = oracle.prefill(q, k, v, c["Wt"], c["alpha"], c["S"], c["z"], dims.L)
    assert_close(np.concatenate(outs, 1), o_r, "bf16", "step_commit walk outputs")
    assert_close(state_host(S) - c["S"], Sr - c["S"], "bf16", "step_commit walk dS")
    assert_close(host(z) - c["z"], zr - c["z"], "bf16", "step_commit walk dz")
