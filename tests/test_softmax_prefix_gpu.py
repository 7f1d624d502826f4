"""GPU parity of softmax_prefix_step (exact softmax over a KV cache plus the
block) against the fp64 oracle, and its reduction to the hybrid step."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import act, announce, assert_close, check_outputs, f32, host, i32

pytestmark = pytest.mark.gpu

CASES = [
    # (B, Hq, Hkv, d, L, dtype, Pmax, plens)
    (1, 1, 1, 64, 8, "f32", 32, [32]),
    (2, 4, 2, 64, 8, "f32", 100, [100, 0]),
    (3, 8, 2, 128, 32, "f32", 300, [300, 17, 64]),
    (2, 16, 4, 128, 32, "bf16", 4096, [4096, 1000]),
    (3, 4, 4, 128, 16, "bf16", 777, [0, 777, 5]),
    (2, 8, 1, 64, 32, "bf16", 2048, [2048, 1536]),
    (2, 4, 2, 128, 7, "bf16", 96, [96, 200]),   # prefix_len above max is clamped
    # the copy-ring kernel at d=64 with 4 heads per KV head, and at d=128 with 8;
    # 3 heads per KV head take the register-staged kernel
    (2, 8, 2, 64, 16, "bf16", 500, [500, 260]),
    (1, 8, 1, 128, 32, "bf16", 5000, [4900]),
    (2, 6, 2, 64, 32, "bf16", 1000, [1000, 33]),
]


@pytest.mark.parametrize("case", CASES, ids=lambda s: "x".join(map(str, s[:7])))
def test_softmax_prefix(case):
    B, Hq, Hkv, d, L, dt, Pmax, plens = case
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=32, dtype=dt)
    announce(f"softmax_prefix {case}")
    q, k, v = synth.block_qkv(dims, 71, 1.0)
    kc, vc = synth.prefix_kv(B, Pmax, Hkv, d, 72, 1.0, dt)
    pl = np.array(plens, np.int32)
    args = (act(q, dt), act(k, dt), act(v, dt), act(kc, dt), act(vc, dt), i32(pl))
    ref = oracle.softmax_prefix(q, k, v, kc, vc, np.minimum(pl, Pmax))
    check_outputs(lambda o32: hb.softmax_prefix_step(*args, out_f32=o32), ref, dt,
                  f"softmax_prefix {case[:7]}")


def test_no_prefix_equals_hybrid_with_empty_state():
    dims = synth.Dims(B=2, Hq=16, Hkv=4, d=128, L=32, F=64, dtype="bf16")
    announce("softmax_prefix P=0 vs hybrid empty state")
    q, k, v = synth.block_qkv(dims, 81, 1.0)
    Wt, alpha = synth.feature_weights(dims, 82, 83)
    qd, kd, vd = act(q, "bf16"), act(k, "bf16"), act(v, "bf16")
    kc = torch.zeros((2, 0, 4, 128), dtype=torch.bfloat16, device="cuda")
    S = torch.zeros((2, 16, 128, 128), device="cuda")
    z = torch.zeros((2, 16, 128), device="cuda")
    ref = oracle.softmax_prefix(q, k, v, np.zeros((2, 0, 4, 128)), np.zeros((2, 0, 4, 128)),
                                np.zeros(2, np.int32))
    check_outputs(lambda o32: hb.softmax_prefix_step(qd, kd, vd, kc, kc, i32([0, 0]),
                                                     out_f32=o32), ref, "bf16", "softmax P=0")
    check_outputs(lambda o32: hb.hybrid_attn_step(qd, kd, vd, act(Wt, "bf16"), f32(alpha), S, z,
                                                  out_f32=o32), ref, "bf16", "hybrid empty state")
