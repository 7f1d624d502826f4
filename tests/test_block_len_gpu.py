"""GPU parity of per-request block lengths (block_len) in the step, the fused
step+commit and the commit, against the fp64 oracle, through the C ABI.

A batch whose requests sit in blocks of different lengths (a prompt's last,
partial block beside full ones) is served in one call: request b acts as a
call with L = block_len[b] on its first block_len[b] rows.  The reference for
request b is therefore the oracle's plain call on those rows alone, at that
length, against b's own state slot.  The padding rows of q, k and v hold NaN,
so any read of them that reaches a result shows up; the padding rows of out
hold a sentinel that must survive.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import act, announce, assert_close, f32, host, i32, make_case, state_dev, state_host

pytestmark = pytest.mark.gpu

SENTINEL = 7.0

CASES = [
    # (B, Hq, Hkv, d, L, F, dtype, P, block_len, slots)
    (4, 4, 2, 128, 32, 64, "bf16", 64, [32, 17, 1, 0], None),
    (4, 4, 2, 64, 8, 32, "f32", 24, [8, 5, 1, 0], None),
    (4, 8, 8, 128, 32, 128, "bf16", 96, [31, 16, 2, 0], [3, 0, 5, 1]),
    (4, 4, 2, 64, 17, 128, "bf16", 34, [17, 9, 3, 0], None),
    (3, 4, 1, 128, 32, 32, "bf16", 40, [-3, 40, 13], [2, 1, 0]),
    (2, 2, 2, 128, 16, 64, "f32", 48, [15, 7], None),
    # four heads per KV head, f = 128: the grouped commit, the column-split
    # step and the fused kernel's early commit, with slots
    (4, 8, 2, 128, 32, 64, "bf16", 64, [32, 0, 19, 1], [1, 4, 0, 2]),
]


def _case(shape):
    B, Hq, Hkv, d, L, F, dt, P, bl, sl = shape
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=F, dtype=dt)
    slots = None if sl is None else np.asarray(sl, np.int32)
    n_slots = B if sl is None else max(sl) + 2
    c = make_case(dims, P, seed=31, peaky=True, n_slots=n_slots, slots=slots)
    lens = np.clip(np.asarray(bl), 0, L)
    # NaN in every padding row: a read of one that reaches a result shows up
    q, k, v = (np.array(c[n], np.float64) for n in ("q", "k", "v"))
    for b, n in enumerate(lens):
        q[b, n:] = np.nan
        k[b, n:] = np.nan
        v[b, n:] = np.nan
    return dims, c, slots, lens, (q, k, v), np.asarray(bl, np.int32)


def _slot(slots, b):
    return b if slots is None else int(slots[b])


def _reference(c, slots, lens, qkv):
    """Per request: the oracle's plain step at L = block_len[b] on b's rows,
    then its commit of those rows; requests with no rows are left out."""
    q, k, v = qkv
    outs = {}
    S, z = np.array(c["S"], np.float64), np.array(c["z"], np.float64)
    for b, n in enumerate(lens):
        if n == 0:
            continue
        s = np.array([_slot(slots, b)], np.int32)
        sl = (slice(b, b + 1), slice(0, n))
        outs[b] = oracle.step(q[sl], k[sl], v[sl], c["Wt"], c["alpha"], c["S"], c["z"], slots=s)[0]
        S, z = oracle.commit(k[sl], v[sl], c["Wt"], S, z, slots=s)
    return outs, S, z


def _dev_inputs(c, dt, qkv):
    q, k, v = qkv
    return act(q, dt), act(k, dt), act(v, dt), act(c["Wt"], dt), f32(c["alpha"])


def _check_out(out, outs, lens, dt, what):
    o = host(out)
    for b, n in enumerate(lens):
        if n > 0:
            assert_close(o[b, :n], outs[b], dt, f"{what} request {b} (len {n})")
        assert (o[b, n:] == SENTINEL).all(), f"{what}: padding rows of request {b} were written"


def _check_state(S1, z1, c, Sr, zr, dt, what):
    assert_close(state_host(S1) - c["S"], Sr - c["S"], dt, what + " dS")
    assert_close(host(z1) - c["z"], zr - c["z"], dt, what + " dz")


def _out_buf(q):
    return torch.full(q.shape, SENTINEL, dtype=torch.float32, device=q.device)


@pytest.mark.parametrize("shape", CASES, ids=lambda s: "x".join(map(str, s[:8])))
def test_block_len_step_fused_commit(shape):
    dims, c, slots, lens, qkv, bl = _case(shape)
    dt = dims.dtype
    announce(f"block_len {shape}")
    outs, Sr, zr = _reference(c, slots, lens, qkv)
    q, k, v, W, al = _dev_inputs(c, dt, qkv)
    sd = None if slots is None else i32(slots)
    bld = i32(bl)
    # the step (both kernels): reads the state, writes rows < block_len[b] only
    outs_split = _out_buf(q)
    hb.hybrid_attn_step(q, k, v, W, al, state_dev(c["S"]), f32(c["z"]), slots=sd, out=outs_split,
                        block_len=bld, kernel="split")
    torch.cuda.synchronize()
    _check_out(outs_split, outs, lens, dt, "step [split]")
    out = _out_buf(q)
    hb.hybrid_attn_step(q, k, v, W, al, state_dev(c["S"]), f32(c["z"]), slots=sd, out=out,
                        block_len=bld, kernel="whole")
    torch.cuda.synchronize()
    _check_out(out, outs, lens, dt, "step [whole]")
    if dt == "bf16" and dims.F <= 64 and (dims.Hq // dims.Hkv) % 4 == 0:
        outh = _out_buf(q)
        hb.hybrid_attn_step(q, k, v, W, al, state_dev(c["S"]), f32(c["z"]), slots=sd, out=outh,
                            block_len=bld, kernel="halves")
        torch.cuda.synchronize()
        _check_out(outh, outs, lens, dt, "step [halves]")
    # the fused step+commit: the same output, and the state as the commits
    S1, z1 = state_dev(c["S"]), f32(c["z"])
    outf = _out_buf(q)
    hb.hybrid_attn_step_commit(q, k, v, W, al, S1, z1, slots=sd, out=outf, block_len=bld)
    torch.cuda.synchronize()
    assert torch.equal(outf, out), "fused output differs from the step's"
    _check_state(S1, z1, c, Sr, zr, dt, "step_commit")
    # the commit alone
    S2, z2 = state_dev(c["S"]), f32(c["z"])
    hb.hybrid_state_commit(k, v, W, S2, z2, slots=sd, block_len=bld)
    torch.cuda.synchronize()
    _check_state(S2, z2, c, Sr, zr, dt, "commit")
    # slots that no request names, and requests with no rows, keep their state
    untouched = set(range(c["S"].shape[0])) - {_slot(slots, b) for b, n in enumerate(lens) if n}
    S0, z0 = state_dev(c["S"]), f32(c["z"])
    for s in untouched:
        for St, zt in ((S1, z1), (S2, z2)):
            assert torch.equal(St[s], S0[s]) and torch.equal(zt[s], z0[s]), f"slot {s} changed"


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_full_block_len_equals_null(dt):
    """block_len = L everywhere gives the call without block_len bit for bit."""
    dims = synth.Dims(B=3, Hq=8, Hkv=2, d=128, L=32 if dt == "bf16" else 16, F=64, dtype=dt)
    announce(f"block_len full {dt}")
    c = make_case(dims, 48, seed=33)
    q, k, v, W, al = _dev_inputs(c, dt, (c["q"], c["k"], c["v"]))
    full = i32(np.full(dims.B, dims.L, np.int32))
    a = hb.hybrid_attn_step(q, k, v, W, al, state_dev(c["S"]), f32(c["z"]), out_f32=True)
    b = hb.hybrid_attn_step(q, k, v, W, al, state_dev(c["S"]), f32(c["z"]), out_f32=True,
                            block_len=full)
    for kern in ("split", "whole") + (("halves",) if dt == "bf16" else ()):
        x = hb.hybrid_attn_step(q, k, v, W, al, state_dev(c["S"]), f32(c["z"]), out_f32=True,
                                kernel=kern)
        y = hb.hybrid_attn_step(q, k, v, W, al, state_dev(c["S"]), f32(c["z"]), out_f32=True,
                                block_len=full, kernel=kern)
        torch.cuda.synchronize()
        assert torch.equal(x, y), f"{kern}: block_len = L differs from no block_len"
    Sa, za, Sb, zb = state_dev(c["S"]), f32(c["z"]), state_dev(c["S"]), f32(c["z"])
    fa = hb.hybrid_attn_step_commit(q, k, v, W, al, Sa, za, out_f32=True)
    fb = hb.hybrid_attn_step_commit(q, k, v, W, al, Sb, zb, out_f32=True, block_len=full)
    Sc, zc, Sd, zd = state_dev(c["S"]), f32(c["z"]), state_dev(c["S"]), f32(c["z"])
    hb.hybrid_state_commit(k, v, W, Sc, zc)
    hb.hybrid_state_commit(k, v, W, Sd, zd, block_len=full)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(fa, fb)
    assert torch.equal(Sa, Sb) and torch.equal(za, zb)
    assert torch.equal(Sc, Sd) and torch.equal(zc, zd)


def test_partial_last_block_walk():
    """A prompt of 5 full blocks and one partial block of 11 tokens, served
    with the fused call (block_len on the last), equals the oracle's
    block-causal prefill of those 171 tokens."""
    dims = synth.Dims(B=2, Hq=8, Hkv=2, d=128, L=32, F=64, dtype="bf16")
    T = 6 * dims.L
    n_last = 11
    announce("block_len walk")
    c = make_case(dims, 64, seed=34)
    q, k, v = synth.block_qkv(dims.with_(L=T), 35, 1.0 / np.sqrt(dims.d))
    S, z = state_dev(c["S"]), f32(c["z"])
    W, al = act(c["Wt"], "bf16"), f32(c["alpha"])
    outs = []
    for blk in range(T // dims.L):
        sl = slice(blk * dims.L, (blk + 1) * dims.L)
        last = blk == T // dims.L - 1
        bl = i32(np.full(dims.B, n_last, np.int32)) if last else None
        o = hb.hybrid_attn_step_commit(act(q[:, sl], "bf16"), act(k[:, sl], "bf16"),
                                       act(v[:, sl], "bf16"), W, al, S, z, out_f32=True,
                                       block_len=bl)
        outs.append(host(o)[:, :n_last] if last else host(o))
    torch.cuda.synchronize()
    n = 5 * dims.L + n_last
    # the oracle's prefill in blocks of L over the first n tokens: its last
    # block is the partial one
    o_r, Sr, zr = _prefill_ragged(q[:, :n], k[:, :n], v[:, :n], c, dims.L)
    assert_close(np.concatenate(outs, 1), o_r, "bf16", "partial walk outputs")
    assert_close(state_host(S) - c["S"], Sr - c["S"], "bf16", "partial walk dS")
    assert_close(host(z) - c["z"], zr - c["z"], "bf16", "partial walk dz")


def _prefill_ragged(q, k, v, c, L):
    """Block-causal prefill whose last block may be short: the full blocks by
    the oracle's prefill, then the short block by its step and commit."""
    T = q.shape[1]
    nf = (T // L) * L
    o, S, z = oracle.prefill(q[:, :nf], k[:, :nf], v[:, :nf], c["Wt"], c["alpha"],
                             c["S"], c["z"], L)
    if nf == T:
        return o, S, z
    t = slice(nf, T)
    o2 = oracle.step(q[:, t], k[:, t], v[:, t], c["Wt"], c["alpha"], S, z)
    S, z = oracle.commit(k[:, t], v[:, t], c["Wt"], S, z)
    return np.concatenate([o, o2], 1), S, z
