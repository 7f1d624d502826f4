"""hybrid_state_prefill_noalloc (the prefill whose workspace is the
library-held scratch buffer) against hybrid_state_prefill on the same inputs,
through the C ABI.

Two calls in a row, the second with a smaller input, so the second runs on
the scratch contents the first left behind.  Both calls cut their prompts
into several sequence segments, so the scratch buffer is really used (segment
increments and the snapshot of the incoming state).  The two entry points run
the same kernels, so outputs and states must agree bit for bit; the outputs
are also held to the oracle at the usual bound.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth

from _helpers import act, announce, assert_close, f32, host, state_dev, state_host

pytestmark = pytest.mark.gpu

CALLS = [
    # (B, Hq, Hkv, d, L, F, dtype, nblk, seed): the second call is smaller
    (2, 4, 1, 128, 32, 64, "bf16", 40, 301),
    (1, 2, 1, 128, 32, 64, "bf16", 24, 302),
]


def _run(shape):
    B, Hq, Hkv, d, L, F, dt, nblk, seed = shape
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=F, dtype=dt)
    T = nblk * L
    hd = hb.make_dims(B, Hq, Hkv, d, L, 2 * F, hb.HYB_BF16 if dt == "bf16" else hb.HYB_F32, B)
    need = hb.workspace_bytes(hd, hb.OP_PREFILL, T)
    assert 0 < need <= hb.NOALLOC_SCRATCH_BYTES, "case must use the scratch buffer"
    q, k, v = synth.block_qkv(dims.with_(L=T), seed, 1.0)
    Wt, alpha = synth.feature_weights(dims, seed + 1, seed + 2, 1.0 / np.sqrt(d))
    S0 = np.zeros((B, Hq, 2 * F, d), np.float32)
    z0 = np.zeros((B, Hq, 2 * F), np.float32)
    # a non-empty incoming state: one oracle commit of a short prefix
    kp, vp = synth.prefix_kv(B, 16, Hkv, d, seed + 3, 1.0, dt)
    S0, z0 = oracle.commit(kp, vp, Wt, S0, z0)
    S0, z0 = S0.astype(np.float32), z0.astype(np.float32)
    ins = (act(q, dt), act(k, dt), act(v, dt), act(Wt, dt), f32(alpha))

    announce(f"prefill_noalloc {shape}")
    Sa, za = state_dev(S0), f32(z0)
    oa = hb.hybrid_state_prefill_noalloc(*ins, Sa, za, L, out_f32=True)
    Sb, zb = state_dev(S0), f32(z0)
    ob = hb.hybrid_state_prefill(*ins, Sb, zb, L, out_f32=True)
    torch.cuda.synchronize()
    assert torch.equal(oa, ob), f"{shape}: outputs differ from hybrid_state_prefill"
    assert torch.equal(Sa, Sb) and torch.equal(za, zb), f"{shape}: states differ"
    o_r, Sr, zr = oracle.prefill(q, k, v, Wt, alpha, S0, z0, L)
    assert_close(host(oa), o_r, dt, f"prefill_noalloc out {shape}")
    assert_close(state_host(Sa) - S0, Sr - S0, dt, f"prefill_noalloc dS {shape}")


def test_prefill_noalloc_two_calls():
    for shape in CALLS:
        _run(shape)
