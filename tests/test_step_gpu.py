"""GPU parity of hybrid_attn_step against the fp64 oracle, through the C ABI."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import (act, announce, assert_close, check_outputs, f32, host, i32, make_case,
                      state_dev)

pytestmark = pytest.mark.gpu


# The step's three kernels: one wave per (request, head, 32-column slice),
# one workgroup per group of heads, and two workgroups per group of four
# heads each taking half of the columns.  Every parity case runs each one
# the shape supports (the column split: bf16, f <= 128, Hq / Hkv a multiple
# of 4).
KERNELS = ["split", "whole", "halves"]


def kernels_for(dims):
    ok = dims.dtype == "bf16" and dims.F <= 64 and (dims.Hq // dims.Hkv) % 4 == 0
    return [k for k in KERNELS if k != "halves" or ok]


def step_call(c, dims, slots=None, kernel=None):
    args = (act(c["q"], dims.dtype), act(c["k"], dims.dtype), act(c["v"], dims.dtype),
            act(c["Wt"], dims.dtype), f32(c["alpha"]), state_dev(c["S"]), f32(c["z"]))
    sl = None if slots is None else i32(slots)
    return lambda out_f32: hb.hybrid_attn_step(*args, slots=sl, out_f32=out_f32, kernel=kernel)


def run_step(c, dims, slots=None, kernel=None):
    out = step_call(c, dims, slots, kernel)(False)
    torch.cuda.synchronize()
    return host(out)


def check_step(c, dims, what, slots=None):
    ref = ref_step(c, slots)
    for kernel in kernels_for(dims):
        check_outputs(step_call(c, dims, slots, kernel), ref, dims.dtype, f"{what} [{kernel}]")


def ref_step(c, slots=None):
    return oracle.step(c["q"], c["k"], c["v"], c["Wt"], c["alpha"], c["S"], c["z"], slots)


def test_tiny_fp32_config():
    """Tiny fp32 hybrid step: 1 head, d=64, L=8, f=64, 4 committed blocks."""
    dims = synth.TINY
    announce("step tiny fp32")
    c = make_case(dims, synth.TINY_PREFIX, seed=0, scale=1.0, w_std=0.02)
    check_step(c, dims, "step tiny")


def test_decode1_bf16_config():
    """B=1, 16q/4kv, d=128, L=32, f=128, state of a 4096-token prefix."""
    dims = synth.DECODE1
    announce("step decode1 bf16")
    c = make_case(dims, synth.DECODE1_PREFIX, seed=20)
    check_step(c, dims, "step decode1")


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
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("peaky", [False, True])
def test_shapes(shape, peaky):
    B, Hq, Hkv, d, L, F, dt, P = shape
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=F, dtype=dt)
    announce(f"step {shape} peaky={peaky}")
    c = make_case(dims, P, seed=5, peaky=peaky)
    check_step(c, dims, f"step {shape} peaky={peaky}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("alpha", [-8.0, 0.0, 8.0])
def test_gate_extremes(dt, alpha):
    dims = synth.Dims(B=2, Hq=4, Hkv=2, d=128, L=32, F=64, dtype=dt)
    announce(f"step alpha={alpha} {dt}")
    c = make_case(dims, 64, seed=9, peaky=True)
    c["alpha"] = np.full(dims.Hq, alpha, np.float32)
    check_step(c, dims, f"step alpha={alpha}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_zero_state_and_zero_W(dt):
    dims = synth.Dims(B=2, Hq=4, Hkv=2, d=64, L=32, F=32, dtype=dt)
    announce(f"step empty state {dt}")
    c = make_case(dims, 0, seed=3, peaky=True)
    check_step(c, dims, "step empty state")
    announce(f"step W=0 {dt}")
    c = make_case(dims, 40, seed=4, peaky=True)
    c["Wt"] = np.zeros_like(c["Wt"])
    c["S"], c["z"] = [a.astype(np.float32) for a in oracle.state_from_prefix(c["kp"], c["vp"], c["Wt"])]
    check_step(c, dims, "step W=0")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_large_scores(dt):
    """Scores near 60 in magnitude: the merge must not overflow fp32."""
    dims = synth.Dims(B=1, Hq=2, Hkv=1, d=64, L=32, F=32, dtype=dt)
    announce(f"step large scores {dt}")
    c = make_case(dims, 32, seed=12, peaky=True)
    rng = np.random.default_rng(13)
    u = rng.standard_normal(dims.d)
    u /= np.linalg.norm(u)
    a = math.sqrt(60.0 * math.sqrt(dims.d))
    c["q"] = synth.to_dtype(a * u + 0.3 * rng.standard_normal(c["q"].shape), dt)
    c["k"] = synth.to_dtype(a * u + 0.3 * rng.standard_normal(c["k"].shape), dt)
    s = np.einsum("bld,bmd->blm", c["q"][:, :, 0].astype(np.float64),
                  c["k"][:, :, 0].astype(np.float64)) / math.sqrt(dims.d)
    assert 40 < np.abs(s).max() < 200
    check_step(c, dims, "step large scores")


@pytest.mark.parametrize("Hq", [4, 8])
def test_slots_and_bad_slot(Hq):
    dims = synth.Dims(B=3, Hq=Hq, Hkv=2, d=128, L=32, F=64, dtype="bf16")
    slots = np.array([4, 0, 2], np.int32)
    announce("step slots")
    c = make_case(dims, 64, seed=21, peaky=True, n_slots=5, slots=slots)
    check_step(c, dims, "step slots", slots)
    announce("step bad slot")
    bad = np.array([4, 7, -1], np.int32)
    good = ref_step(c, np.array([4, 0, 0], np.int32))[:1]
    for kernel in kernels_for(dims):
        out = host(step_call(c, dims, bad, kernel)(True))
        assert np.isnan(out[1:]).all()
        assert_close(out[:1], good, "bf16", f"step valid row next to bad slots [{kernel}]")
        assert np.isnan(run_step(c, dims, bad, kernel)[1:]).all()


@pytest.mark.parametrize("kernel", KERNELS)
def test_deterministic_and_guarded(kernel):
    """Bitwise identical across runs; bytes around the output stay untouched."""
    dims = synth.DECODE1.with_(B=4)
    announce(f"step determinism [{kernel}]")
    c = make_case(dims, 128, seed=30, peaky=True)
    q, k, v = (act(c[n], "bf16") for n in ("q", "k", "v"))
    W, al, S, z = act(c["Wt"], "bf16"), f32(c["alpha"]), state_dev(c["S"]), f32(c["z"])
    n = q.numel()
    guard = 4096
    buf = torch.full((n + 2 * guard,), float("nan"), dtype=torch.bfloat16, device="cuda")
    out = buf[guard:guard + n].view(q.shape)
    first = hb.hybrid_attn_step(q, k, v, W, al, S, z, kernel=kernel).clone()
    for _ in range(10):
        hb.hybrid_attn_step(q, k, v, W, al, S, z, out=out, kernel=kernel)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), first.view(torch.int16))
    assert torch.isnan(buf[:guard].float()).all() and torch.isnan(buf[guard + n:].float()).all()


def test_matches_commit_free_brute_force():
    """GPU step against the explicit prefix sum, independent of the state path."""
    from oracle import brute
    dims = synth.TINY
    announce("step vs brute")
    c = make_case(dims, synth.TINY_PREFIX, seed=0, scale=1.0, w_std=0.02)
    ref = brute.hybrid_block_brute(c["q"], c["k"], c["v"], c["kp"], c["vp"],
                                   np.array([synth.TINY_PREFIX]), c["Wt"], c["alpha"])
    check_outputs(step_call(c, dims), ref, "f32", "step tiny vs brute")


@pytest.mark.parametrize("B", [1, 8, 16, 20, 32, 48])
def test_small_batch_kernels(B):
    """Batch sizes of decode1 and the paper's Table 3 (B = 8, 32), serving
    shapes, peaky inputs, every kernel; the library's own choice is the
    column split while its 2 B Hq/4 workgroups fill 128 to 256 compute units,
    else the split kernel while its B * Hq * d/32 waves fit on the chip
    (1024), else the column split while its workgroups fit, else the per-head
    kernel."""
    dims = synth.DECODE1.with_(B=B)
    announce(f"step small batch B={B}")
    c = make_case(dims, 96, seed=40 + B, peaky=True)
    check_step(c, dims, f"step B={B}")
    auto = run_step(c, dims)
    groups2 = 2 * B * (dims.Hq // 4)
    want = ("halves" if 128 <= groups2 <= 256
            else "split" if B * dims.Hq * (dims.d // 32) <= 1024
            else "halves" if groups2 <= 256 else "whole")
    assert np.array_equal(auto, run_step(c, dims, kernel=want)), f"automatic choice is not {want}"
