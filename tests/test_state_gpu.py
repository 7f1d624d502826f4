"""GPU parity of hybrid_state_commit and hybrid_state_prefill against the fp64
oracle, plus the state invariants across calls (incremental == one prefill,
checkpoint/resume, commit order)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import (act, announce, assert_close, check_outputs, f32, host, i32, make_case,
                      state_dev, state_host)

pytestmark = pytest.mark.gpu


def assert_state_delta(S1, z1, S0, z0, Sr, zr, dt, what):
    """Compare the change a GPU call made with the oracle's change."""
    assert_close(S1 - S0, Sr - S0, dt, what + " dS")
    assert_close(z1 - z0, zr - z0, dt, what + " dz")


SHAPES = [
    (1, 1, 1, 64, 8, 32, "f32", 32),
    (2, 4, 2, 64, 8, 32, "f32", 24),
    (2, 8, 2, 128, 32, 64, "f32", 64),
    (2, 4, 4, 128, 16, 128, "f32", 0),
    (2, 16, 4, 128, 32, 64, "bf16", 256),
    (3, 4, 1, 64, 5, 64, "bf16", 20),
    (2, 8, 8, 128, 32, 128, "bf16", 64),
    # the grouped commit kernel at its other shapes (bf16, four heads per KV
    # head, f <= d): d = 64 with f = 64, and f = 64 with a 7-token block
    (2, 8, 2, 64, 32, 32, "bf16", 48),
    (1, 4, 1, 128, 7, 32, "bf16", 16),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_commit(shape):
    B, Hq, Hkv, d, L, F, dt, P = shape
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=F, dtype=dt)
    announce(f"commit {shape}")
    c = make_case(dims, P, seed=7, peaky=True)
    S, z = state_dev(c["S"]), f32(c["z"])
    hb.hybrid_state_commit(act(c["k"], dt), act(c["v"], dt), act(c["Wt"], dt), S, z)
    torch.cuda.synchronize()
    Sr, zr = oracle.commit(c["k"], c["v"], c["Wt"], c["S"], c["z"])
    assert_state_delta(state_host(S), host(z), c["S"], c["z"], Sr, zr, dt, f"commit {shape}")


@pytest.mark.parametrize("Hq", [4, 8])
def test_commit_slots_and_bad_slot(Hq):
    """Hq = 4 over 2 KV heads takes the per-head kernel, Hq = 8 the grouped one."""
    dims = synth.Dims(B=3, Hq=Hq, Hkv=2, d=128, L=32, F=64, dtype="bf16")
    slots = np.array([3, 0, 5], np.int32)
    announce("commit slots")
    c = make_case(dims, 32, seed=8, peaky=True, n_slots=6, slots=slots)
    S, z = state_dev(c["S"]), f32(c["z"])
    bad = np.array([3, 9, 5], np.int32)   # request 1 has no valid slot
    hb.hybrid_state_commit(act(c["k"], "bf16"), act(c["v"], "bf16"), act(c["Wt"], "bf16"),
                           S, z, slots=i32(bad))
    torch.cuda.synchronize()
    k, v = c["k"][[0, 2]], c["v"][[0, 2]]
    Sr, zr = oracle.commit(k, v, c["Wt"], c["S"], c["z"], slots=np.array([3, 5], np.int32))
    assert_state_delta(state_host(S), host(z), c["S"], c["z"], Sr, zr, "bf16", "commit slots")
    # untouched slots are bit-identical
    for s in (0, 1, 2, 4):
        assert torch.equal(S[s].cpu(), state_dev(c["S"][s]).cpu())


PREFILL_SHAPES = [
    (1, 1, 1, 64, 8, 32, "f32", 64),
    (2, 4, 2, 64, 8, 32, "f32", 40),
    (2, 8, 2, 128, 32, 64, "f32", 128),
    (2, 16, 4, 128, 32, 64, "bf16", 256),
    (2, 4, 1, 64, 16, 128, "bf16", 96),
    (1, 8, 8, 128, 32, 128, "bf16", 96),
    (2, 4, 2, 128, 5, 64, "bf16", 35),
    # the pipelined walk and delta at d=64 with F=64, and at d=128 with F=32
    # (two segments of 5 blocks: an odd count for the delta's block pairs)
    (2, 8, 2, 64, 32, 64, "bf16", 256),
    (2, 8, 4, 128, 16, 32, "bf16", 160),
]


@pytest.mark.parametrize("shape", PREFILL_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_prefill(shape):
    B, Hq, Hkv, d, L, F, dt, T = shape
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=F, dtype=dt)
    announce(f"prefill {shape}")
    seq = dims.with_(L=T)
    q, k, v = synth.block_qkv(seq, 51, 1.0)
    Wt, alpha = synth.feature_weights(dims, 52, 53, 1.0 / np.sqrt(d))
    # start from a non-empty state so that continuation is exercised
    c0 = make_case(dims, 16, seed=54, peaky=True)
    o_r, Sr, zr = oracle.prefill(q, k, v, Wt, alpha, c0["S"], c0["z"], L)
    states = []

    def call(out_f32):
        S, z = state_dev(c0["S"]), f32(c0["z"])
        states.append((S, z))
        return hb.hybrid_state_prefill(act(q, dt), act(k, dt), act(v, dt), act(Wt, dt),
                                       f32(alpha), S, z, L, out_f32=out_f32)

    check_outputs(call, o_r, dt, f"prefill out {shape}")
    S, z = states[-1]
    assert_state_delta(state_host(S), host(z), c0["S"], c0["z"], Sr, zr, dt, f"prefill {shape}")
    # state only
    S2, z2 = state_dev(c0["S"]), f32(c0["z"])
    assert hb.hybrid_state_prefill(None, act(k, dt), act(v, dt), act(Wt, dt), None, S2, z2, L,
                                   want_out=False) is None
    torch.cuda.synchronize()
    assert_state_delta(state_host(S2), host(z2), c0["S"], c0["z"], Sr, zr, dt, f"prefill-state {shape}")


def test_prefill_equals_commits_and_resume():
    """256 commits == one prefill == oracle from scratch; a checkpointed state
    restored into a fresh buffer continues bit-identically."""
    dims = synth.Dims(B=2, Hq=16, Hkv=4, d=128, L=32, F=64, dtype="bf16")
    nblk = 256
    T = nblk * dims.L
    announce("prefill vs commits 8192 tokens")
    seq = dims.with_(L=T)
    _, k, v = synth.block_qkv(seq, 61, 1.0 / np.sqrt(dims.d))
    Wt, _ = synth.feature_weights(dims, 62, 63)
    kd, vd, Wd = act(k, "bf16"), act(v, "bf16"), act(Wt, "bf16")
    S1 = torch.zeros((2, 16, 128, 128), device="cuda")   # [B][Hq][d][f]
    z1 = torch.zeros((2, 16, 128), device="cuda")
    hb.hybrid_state_prefill(None, kd, vd, Wd, None, S1, z1, dims.L, want_out=False)
    S2, z2 = torch.zeros_like(S1), torch.zeros_like(z1)
    ck = None
    for blk in range(nblk):
        sl = slice(blk * dims.L, (blk + 1) * dims.L)
        hb.hybrid_state_commit(kd[:, sl].contiguous(), vd[:, sl].contiguous(), Wd, S2, z2)
        if blk == nblk // 2 - 1:
            ck = (S2.cpu().clone(), z2.cpu().clone())
    torch.cuda.synchronize()
    S0, z0 = oracle.empty_state(2, 16, 128, 128)
    Sr, zr = oracle.commit(k, v, Wt, S0, z0)
    assert_close(state_host(S1), Sr, "bf16", "prefill state 8192")
    assert_close(state_host(S2), Sr, "bf16", "256 commits state")
    assert_close(host(z1), zr, "bf16", "prefill z 8192")
    # resume from the checkpoint in fresh buffers
    S3, z3 = ck[0].cuda(), ck[1].cuda()
    for blk in range(nblk // 2, nblk):
        sl = slice(blk * dims.L, (blk + 1) * dims.L)
        hb.hybrid_state_commit(kd[:, sl].contiguous(), vd[:, sl].contiguous(), Wd, S3, z3)
    torch.cuda.synchronize()
    assert torch.equal(S3, S2) and torch.equal(z3, z2)
    # commit order: the same blocks in reverse give the same state up to rounding
    S4, z4 = torch.zeros_like(S1), torch.zeros_like(z1)
    for blk in reversed(range(nblk)):
        sl = slice(blk * dims.L, (blk + 1) * dims.L)
        hb.hybrid_state_commit(kd[:, sl].contiguous(), vd[:, sl].contiguous(), Wd, S4, z4)
    torch.cuda.synchronize()
    assert_close(state_host(S4), Sr, "bf16", "reverse-order commits state")


SEGMENT_CASES = [
    # (B, Hq, Hkv, d, L, F, dtype, nblk): few (request, head) units, so the
    # prompt is cut into several sequence segments; 37 blocks leave the last
    # segment short.
    (1, 4, 1, 64, 8, 32, "f32", 40),
    (1, 4, 2, 64, 8, 32, "bf16", 37),
    (2, 2, 1, 128, 32, 64, "bf16", 33),
]


@pytest.mark.parametrize("shape", SEGMENT_CASES, ids=lambda s: "x".join(map(str, s)))
def test_prefill_segments(shape):
    """Segmented prefill (state increments through the workspace) equals the
    oracle's block-by-block prefill, outputs and state, and the state-only
    call agrees with it."""
    B, Hq, Hkv, d, L, F, dt, nblk = shape
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=F, dtype=dt)
    T = nblk * L
    ws_need = hb.workspace_bytes(hb.make_dims(B, Hq, Hkv, d, L, 2 * F, hb.HYB_BF16 if dt == "bf16"
                                              else hb.HYB_F32, B), hb.OP_PREFILL, T)
    assert ws_need > 0, "case must exercise more than one segment"
    announce(f"prefill segments {shape}")
    seq = dims.with_(L=T)
    q, k, v = synth.block_qkv(seq, 91, 1.0)
    Wt, alpha = synth.feature_weights(dims, 92, 93, 1.0 / np.sqrt(d))
    c0 = make_case(dims, 16, seed=94, peaky=True)
    o_r, Sr, zr = oracle.prefill(q, k, v, Wt, alpha, c0["S"], c0["z"], L)
    states = []

    def call(out_f32):
        S, z = state_dev(c0["S"]), f32(c0["z"])
        states.append((S, z))
        # a workspace full of NaN bytes: every part the walk reads (the
        # increments and the snapshot of the incoming state) is written first
        ws = torch.full((ws_need,), 0xFF, dtype=torch.uint8, device="cuda")
        return hb.hybrid_state_prefill(act(q, dt), act(k, dt), act(v, dt), act(Wt, dt),
                                       f32(alpha), S, z, L, out_f32=out_f32, ws=ws)

    check_outputs(call, o_r, dt, f"prefill segments out {shape}")
    S, z = states[-1]
    assert_state_delta(state_host(S), host(z), c0["S"], c0["z"], Sr, zr, dt,
                       f"prefill segments {shape}")
    S2, z2 = state_dev(c0["S"]), f32(c0["z"])
    hb.hybrid_state_prefill(None, act(k, dt), act(v, dt), act(Wt, dt), None, S2, z2, L,
                            want_out=False)
    torch.cuda.synchronize()
    assert_state_delta(state_host(S2), host(z2), c0["S"], c0["z"], Sr, zr, dt,
                       f"prefill segments state-only {shape}")
