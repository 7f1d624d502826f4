"""Parity at the full sizes of the serving, prefill and softmax-prefix
workloads, in the launch configurations the bench times: the GPU runs the
whole batch, the fp64 oracle checks sampled requests (every head, every
query) on the same inputs.

Inputs too large to draw on the host come from synth.device_gaussian (a
seeded device generator); the rows a test checks are copied to the host for
the oracle.  States are built by the oracle from short synthetic prefixes,
so no oracle input comes from the library.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import act, announce, assert_close, f32, host, i32, state_dev, state_host

pytestmark = pytest.mark.gpu


def _bf16_host(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def _states(dims, n, P, seed):
    """Oracle-built states of n requests from P-token synthetic prefixes."""
    Wt, _ = synth.feature_weights(dims, seed + 1, seed + 2)
    kp, vp = synth.prefix_kv(n, P, dims.Hkv, dims.d, seed, 1.0 / math.sqrt(dims.d), "bf16")
    S, z = oracle.state_from_prefix(kp, vp, Wt)
    return S, z


def _step_sampled(dims, seed, sample, what):
    B = dims.B
    sc = 1.0 / math.sqrt(dims.d)
    q = synth.device_gaussian((B, dims.L, dims.Hq, dims.d), seed, sc)
    k = synth.device_gaussian((B, dims.L, dims.Hkv, dims.d), seed + 1, sc)
    v = synth.device_gaussian((B, dims.L, dims.Hkv, dims.d), seed + 2, sc)
    Wt, alpha = synth.feature_weights(dims, seed + 1, seed + 2)   # the states' W
    S, z = _states(dims, B, 64, seed)
    Sd, zd = state_dev(S), f32(z)
    W, al = act(Wt, "bf16"), f32(alpha)
    announce(f"{what}: step B={B}")
    o32 = hb.hybrid_attn_step(q, k, v, W, al, Sd, zd, out_f32=True)
    o16 = hb.hybrid_attn_step(q, k, v, W, al, Sd, zd)
    torch.cuda.synchronize()
    assert torch.isfinite(o32).all()
    assert torch.equal(o16.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16))
    s = np.array(sample)
    ref = oracle.step(_bf16_host(q[s]), _bf16_host(k[s]), _bf16_host(v[s]), Wt, alpha, S[s], z[s])
    assert_close(host(o32[s]), ref, "bf16", f"{what}: step, requests {sample}")
    return q, k, v, W, Wt, S, z, Sd, zd


def test_serve64_step_and_commit_sampled():
    """B=64 serving step and commit (the bench's launch configuration)."""
    dims = synth.SERVE64
    sample = [0, 21, 42, 63]
    q, k, v, W, Wt, S, z, Sd, zd = _step_sampled(dims, 401, sample, "serve64")
    announce("serve64: commit B=64")
    hb.hybrid_state_commit(k, v, W, Sd, zd)
    torch.cuda.synchronize()
    s = np.array(sample)
    Sr, zr = oracle.commit(_bf16_host(k[s]), _bf16_host(v[s]), Wt, S[s], z[s])
    S1, z1 = state_host(Sd)[s], host(zd)[s]
    assert_close(S1 - S[s], Sr - S[s], "bf16", f"serve64 commit dS, requests {sample}")
    assert_close(z1 - z[s], zr - z[s], "bf16", f"serve64 commit dz, requests {sample}")


def test_serve64_step_commit_sampled():
    """B=64 fused step+commit (the last denoising pass of a block in the
    bench's cycle): outputs on the old state, then the committed state."""
    dims = synth.SERVE64
    B = dims.B
    sc = 1.0 / math.sqrt(dims.d)
    q = synth.device_gaussian((B, dims.L, dims.Hq, dims.d), 441, sc)
    k = synth.device_gaussian((B, dims.L, dims.Hkv, dims.d), 442, sc)
    v = synth.device_gaussian((B, dims.L, dims.Hkv, dims.d), 443, sc)
    Wt, alpha = synth.feature_weights(dims, 442, 443)
    S, z = _states(dims, B, 64, 441)
    Sd, zd = state_dev(S), f32(z)
    announce("serve64: step_commit B=64")
    o32 = hb.hybrid_attn_step_commit(q, k, v, act(Wt, "bf16"), f32(alpha), Sd, zd, out_f32=True)
    torch.cuda.synchronize()
    assert torch.isfinite(o32).all()
    sample = [0, 31, 63]
    s = np.array(sample)
    ref_out, Sr, zr = oracle.step_commit(_bf16_host(q[s]), _bf16_host(k[s]), _bf16_host(v[s]),
                                         Wt, alpha, S[s], z[s])
    assert_close(host(o32[s]), ref_out, "bf16", f"serve64 step_commit out, requests {sample}")
    assert_close(state_host(Sd)[s] - S[s], Sr - S[s], "bf16", f"serve64 step_commit dS {sample}")
    assert_close(host(zd)[s] - z[s], zr - z[s], "bf16", f"serve64 step_commit dz {sample}")


def test_mix128_hybrid_step_sampled():
    """B=128 hybrid step (the hybrid side of the mix128 comparison)."""
    _step_sampled(synth.MIX128, 411, [0, 77, 127], "mix128")


def test_prefill8_sampled():
    """8 prompts x 8192 tokens from an empty state: outputs and final state of
    sampled prompts against the oracle's block-by-block prefill."""
    dims = synth.PREFILL8
    B, T, L = dims.B, synth.PREFILL8_T, dims.L
    sc = 1.0 / math.sqrt(dims.d)
    q = synth.device_gaussian((B, T, dims.Hq, dims.d), 421, sc)
    k = synth.device_gaussian((B, T, dims.Hkv, dims.d), 422, sc)
    v = synth.device_gaussian((B, T, dims.Hkv, dims.d), 423, sc)
    Wt, alpha = synth.feature_weights(dims, 424, 425)
    W, al = act(Wt, "bf16"), f32(alpha)
    Sd = torch.zeros((B, dims.Hq, dims.d, dims.f), device="cuda")
    zd = torch.zeros((B, dims.Hq, dims.f), device="cuda")
    announce("prefill8: B=8 x 8192 tokens")
    o32 = hb.hybrid_state_prefill(q, k, v, W, al, Sd, zd, L, out_f32=True)
    torch.cuda.synchronize()
    assert torch.isfinite(o32).all()
    s = np.array([0, 5])
    S0, z0 = oracle.empty_state(len(s), dims.Hq, dims.f, dims.d)
    o_r, Sr, zr = oracle.prefill(_bf16_host(q[s]), _bf16_host(k[s]), _bf16_host(v[s]), Wt, alpha,
                                 S0, z0, L)
    assert_close(host(o32[s]), o_r, "bf16", "prefill8 outputs, prompts [0, 5]")
    assert_close(state_host(Sd)[s], Sr, "bf16", "prefill8 final S, prompts [0, 5]")
    assert_close(host(zd)[s], zr, "bf16", "prefill8 final z, prompts [0, 5]")


def test_mix128_softmax_prefix_sampled():
    """B=128 exact softmax over a 32768-token bf16 KV cache plus the block."""
    dims = synth.MIX128
    B, P = dims.B, synth.MIX128_PREFIX
    sc = 1.0 / math.sqrt(dims.d)
    q = synth.device_gaussian((B, dims.L, dims.Hq, dims.d), 431, sc)
    k = synth.device_gaussian((B, dims.L, dims.Hkv, dims.d), 432, sc)
    v = synth.device_gaussian((B, dims.L, dims.Hkv, dims.d), 433, sc)
    kc = synth.device_gaussian((B, P, dims.Hkv, dims.d), 434, sc)
    vc = synth.device_gaussian((B, P, dims.Hkv, dims.d), 435, sc)
    plen = np.full(B, P, np.int32)
    announce("mix128: softmax prefix B=128, P=32768")
    o32 = hb.softmax_prefix_step(q, k, v, kc, vc, i32(plen), out_f32=True)
    torch.cuda.synchronize()
    assert torch.isfinite(o32).all()
    s = np.array([0, 127])
    ref = oracle.softmax_prefix(_bf16_host(q[s]), _bf16_host(k[s]), _bf16_host(v[s]),
                                _bf16_host(kc[s]), _bf16_host(vc[s]), plen[s])
    assert_close(host(o32[s]), ref, "bf16", "mix128 softmax prefix, requests [0, 127]")


def test_train8_backward_full():
    """The Stage-1 backward at the benchmark's training size (8 sequences of
    2048 tokens, 16q/4kv, d=128, f=128, blocks of 32, attention-transfer
    mode) in the bench's launch configuration, against the oracle on the
    whole batch: dW, dalpha and the loss (every element)."""
    dims = synth.TRAIN8
    T = synth.TRAIN8_T
    q, k, v = synth.sequence_qkv(dims, T, 61, 1.0)
    Wt, alpha = synth.feature_weights(dims, 62, 63, 1.0 / math.sqrt(dims.d))
    tgt = synth.upstream(dims, T, 64, 0.05)
    announce("train8: backward B=8 x 2048 tokens")
    dW, da, loss = hb.hybrid_attn_backward(act(q, "bf16"), act(k, "bf16"), act(v, "bf16"),
                                           act(Wt, "bf16"), f32(alpha), dims.L,
                                           target=act(tgt, "bf16"))
    torch.cuda.synchronize()
    ref_W, ref_a, ref_l = oracle.backward(q, k, v, Wt, alpha, dims.L, target=tgt)
    for got, ref, what in ((host(dW), ref_W, "dW"), (host(da), ref_a, "dalpha"),
                           (host(loss), ref_l, "loss")):
        err = float(np.abs(got - ref).max())
        tol = 2e-2 * float(np.sqrt(np.mean(ref ** 2)))
        print(f"[parity] train8 backward {what}: max abs err {err:.3e} (tol {tol:.3e})")
        assert np.isfinite(got).all() and err <= tol, what
