"""GPU parity of softmax_prefix_step_paged (exact softmax over a paged KV
cache plus the block) against the fp64 oracle, and bit-for-bit agreement
with softmax_prefix_step on the same cache gathered into contiguous rows.

The oracle computes on the logical sequence of each request; the test turns
the paged layout into that sequence by plain indexing (which page holds
which tokens).  Pages are scattered in a random order, shared between two
requests where the case says so, and every page no request uses is filled
with NaN, so reading a wrong page cannot go unnoticed.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_06628_amd import binding as hb
from paper_2608_06628_amd import synth
from _helpers import act, announce, check_outputs, i32

pytestmark = pytest.mark.gpu

CASES = [
    # (B, Hq, Hkv, d, L, dtype, page_size, max_pages, plens, share)
    (2, 16, 4, 128, 32, "bf16", 32, 40, [1250, 31], False),
    (3, 8, 2, 64, 16, "bf16", 64, 12, [700, 0, 64], True),
    (2, 8, 1, 128, 32, "bf16", 128, 40, [5000, 4097], True),       # several splits
    (2, 4, 2, 128, 7, "bf16", 32, 3, [96, 500], False),             # prefix clamped
    (2, 6, 2, 64, 32, "bf16", 32, 20, [600, 33], False),            # register-staged kernel
    (2, 4, 2, 64, 8, "f32", 64, 6, [300, 64], True),
    (1, 4, 4, 128, 32, "f32", 256, 2, [511], False),
]


def paged_cache(B, plens, ps, max_pages, Hkv, d, dt, seed, share):
    """Logical caches [B][max_pages*ps][Hkv][d], their page pools with the
    pages in a random order (NaN in pages nobody reads), and the table."""
    Pmax = max_pages * ps
    kc, vc = synth.prefix_kv(B, Pmax, Hkv, d, seed, 1.0, dt)
    rng = np.random.default_rng(seed + 1)
    used = [-(-min(p, Pmax) // ps) for p in plens]
    if share and B > 1 and used[0] > 0 and used[1] > 0:
        # request 1 starts with request 0's first page (a shared prompt prefix)
        kc[1, :ps], vc[1, :ps] = kc[0, :ps], vc[0, :ps]
    n_pages = sum(used) + 5
    order = rng.permutation(n_pages)
    kp = np.full((n_pages, ps, Hkv, d), np.nan, np.float32)
    vp = np.full_like(kp, np.nan)
    table = np.full((B, max_pages), -7, np.int32)       # unread entries hold junk
    nxt = 0
    for b in range(B):
        for i in range(used[b]):
            if share and b == 1 and i == 0:
                table[b, i] = table[0, 0]
                continue
            pg = order[nxt]
            nxt += 1
            table[b, i] = pg
            kp[pg] = kc[b, i * ps:(i + 1) * ps]
            vp[pg] = vc[b, i * ps:(i + 1) * ps]
    return kc, vc, kp, vp, table


@pytest.mark.parametrize("case", CASES, ids=lambda s: "x".join(map(str, s[:8])))
def test_softmax_prefix_paged(case):
    B, Hq, Hkv, d, L, dt, ps, max_pages, plens, share = case
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=32, dtype=dt)
    announce(f"softmax_prefix_paged {case}")
    q, k, v = synth.block_qkv(dims, 171, 1.0)
    kc, vc, kp, vp, table = paged_cache(B, plens, ps, max_pages, Hkv, d, dt, 172, share)
    Pmax = max_pages * ps
    pl = np.array(plens, np.int32)
    ref = oracle.softmax_prefix(q, k, v, kc, vc, np.minimum(pl, Pmax))
    blk = (act(q, dt), act(k, dt), act(v, dt))
    pages = (act(kp, dt), act(vp, dt), i32(table), i32(pl))
    check_outputs(lambda o32: hb.softmax_prefix_step_paged(*blk, *pages, out_f32=o32), ref, dt,
                  f"softmax_prefix_paged {case[:8]}")
    # the contiguous entry point on the gathered cache gives the same bits
    got = hb.softmax_prefix_step_paged(*blk, *pages, out_f32=True)
    cont = hb.softmax_prefix_step(*blk, act(kc, dt), act(vc, dt), i32(pl), out_f32=True)
    torch.cuda.synchronize()
    assert torch.equal(got, cont), "paged and contiguous caches differ"


def test_softmax_prefix_paged_page_clamp():
    """A page number outside the pool is clamped to its last page."""
    B, Hq, Hkv, d, L, dt, ps = 1, 4, 1, 128, 32, "bf16", 32
    dims = synth.Dims(B=B, Hq=Hq, Hkv=Hkv, d=d, L=L, F=32, dtype=dt)
    announce("softmax_prefix_paged page clamp")
    q, k, v = synth.block_qkv(dims, 181, 1.0)
    kp, vp = synth.prefix_kv(3, ps, Hkv, d, 182, 1.0, dt)     # 3 pages of ps rows
    kp, vp = kp[:, :, :, :], vp[:, :, :, :]
    table = np.array([[2, 99, -4]], np.int32)                # -> pages 2, 2, 0
    pl = np.array([3 * ps], np.int32)
    kc = np.concatenate([kp[2], kp[2], kp[0]])[None]
    vc = np.concatenate([vp[2], vp[2], vp[0]])[None]
    ref = oracle.softmax_prefix(q, k, v, kc, vc, pl)
    check_outputs(lambda o32: hb.softmax_prefix_step_paged(
        act(q, dt), act(k, dt), act(v, dt), act(kp, dt), act(vp, dt), i32(table), i32(pl),
        out_f32=o32), ref, dt, "softmax_prefix_paged clamp")
