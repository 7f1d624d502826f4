"""Shared helpers for the GPU parity tests: seeded cases, oracle states,
device transfer and the tolerance rule.

Tolerances: fp32 inputs -- max |gpu - oracle| <= 1e-5; bf16 inputs --
max |gpu - oracle| <= 2e-2 * rms(oracle), with the oracle run on the same
bf16-rounded inputs.  For bf16 inputs the bound is applied to the call's fp32
output (HYB_OUT_F32), and the bf16 output of the same call must then equal
that fp32 output rounded to bf16 bit for bit: the arithmetic is held to the
bound, and storing in bf16 adds only its own rounding.  States compare the
change a call makes, with the same rule applied to the oracle's change.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

import oracle
from paper_2608_06628_amd import synth

DEV = "cuda"


def announce(msg: str):
    """Name the case before its GPU step, flushed, so a crash names it."""
    print(f"[gpu case] {msg}", file=sys.stderr, flush=True)


def act(x, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(DEV)
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def f32(x) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(DEV)


def i32(x) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(DEV)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


# The oracle keeps each S_h as the f x d matrix of the paper; the library
# stores it transposed ([..][d][f], features contiguous).  These two convert
# between the layouts and do nothing else.
def state_dev(S) -> torch.Tensor:
    """Oracle-layout state [..][f][d] -> device tensor in the library layout."""
    return f32(np.swapaxes(np.asarray(S), -1, -2))


def state_host(S: torch.Tensor) -> np.ndarray:
    """Library-layout device state -> fp64 array in the oracle layout."""
    return np.ascontiguousarray(np.swapaxes(host(S), -1, -2))


def tol_for(ref: np.ndarray, dtype: str) -> float:
    if dtype == "f32":
        return 1e-5
    return 2e-2 * float(np.sqrt(np.mean(np.square(ref))))


def assert_close(got: np.ndarray, ref: np.ndarray, dtype: str, what: str):
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = float(np.abs(got - ref).max())
    tol = tol_for(ref, dtype)
    print(f"[parity] {what}: max abs err {err:.3e} (tol {tol:.3e})")
    assert err <= tol, f"{what}: max abs err {err:.3e} > tol {tol:.3e}"
    return err


def check_outputs(call, ref: np.ndarray, dtype: str, what: str):
    """call(out_f32) runs the GPU op and returns its output tensor."""
    if dtype == "f32":
        out = call(False)
        torch.cuda.synchronize()
        return assert_close(host(out), ref, "f32", what)
    o32 = call(True)
    o16 = call(False)
    torch.cuda.synchronize()
    assert o32.dtype == torch.float32 and o16.dtype == torch.bfloat16
    err = assert_close(host(o32), ref, "bf16", what + " (fp32 out)")
    same = torch.equal(o16.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16))
    assert same, f"{what}: bf16 output is not the rounded fp32 output"
    e16 = float(np.abs(host(o16) - ref).max())
    print(f"[parity] {what} (bf16 out): max abs err {e16:.3e} incl. output rounding")
    return err


def make_case(dims: synth.Dims, P: int, seed: int = 0, peaky: bool = False,
              scale: float | None = None, w_std: float | None = None,
              n_slots: int | None = None, slots=None):
    """Seeded block inputs, weights and an oracle-built fp32 state of a
    P-token prefix for every request (placed at slots[b] if given)."""
    if scale is None:
        scale = 1.0 if peaky else 1.0 / math.sqrt(dims.d)
    if w_std is None:
        w_std = 1.0 / math.sqrt(dims.d) if peaky else 0.02
    q, k, v = synth.block_qkv(dims, seed, scale)
    kp, vp = synth.prefix_kv(dims.B, P, dims.Hkv, dims.d, seed + 100, scale, dims.dtype)
    Wt, alpha = synth.feature_weights(dims, seed + 1, seed + 2, w_std)
    n_slots = n_slots or dims.B
    S, z = oracle.empty_state(n_slots, dims.Hq, dims.f, dims.d)
    if P > 0:
        S, z = oracle.commit(kp, vp, Wt, S, z, slots=slots)
    return dict(q=q, k=k, v=v, kp=kp, vp=vp, Wt=Wt, alpha=alpha,
                S=S.astype(np.float32), z=z.astype(np.float32), slots=slots)
