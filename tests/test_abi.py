"""The C ABI on the CPU: the library loads, exports every symbol the header
declares, and rejects bad arguments before any HIP call.

Every call here is built to fail validation, so nothing is ever launched:
the pointers are small fake addresses that no kernel may see.
"""
import ctypes
import os
import re

import pytest

from paper_2608_06628_amd import binding as hb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hybrid_attn.h")

FAKE = ctypes.c_void_p(0x1000)      # aligned, never dereferenced
MISALIGNED = ctypes.c_void_p(0x1008)


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|size_t|const char\*)\s+(\w+)\s*\(", text, re.M)))


def test_exports_match_header():
    lib = hb.load()
    names = _declared()
    assert set(names) == set(hb.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def _dims(**kw):
    base = dict(batch=2, n_q_heads=16, n_kv_heads=4, head_dim=128, block=32,
                feat_dim=128, dtype=hb.HYB_BF16, n_slots=2, flags=0)
    base.update(kw)
    return hb.Dims(*[base[n] for n, _ in hb.Dims._fields_])


def _step(dims, ptrs=None):
    lib = hb.load()
    p = ptrs or [FAKE] * 10
    return lib.hybrid_attn_step(ctypes.byref(dims) if dims is not None else None, *p, None)


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96), 5), (dict(feat_dim=96), 5), (dict(block=33), 5),
    (dict(block=0), 2), (dict(n_kv_heads=3), 2), (dict(batch=-1), 2),
    (dict(dtype=7), 4), (dict(n_slots=0), 2), (dict(n_q_heads=0), 2),
    (dict(flags=2), 2), (dict(flags=-1), 2),
])
def test_step_rejects_bad_dims(kw, code):
    assert _step(_dims(**kw)) == code
    assert hb.last_error()


def test_null_and_alignment():
    assert _step(None) == 1
    for i in range(10):
        if i in (7, 8):   # slots and block_len may be NULL; misaligned is still rejected
            p = [FAKE] * 10
            p[i] = MISALIGNED
            assert _step(_dims(), p) == 3
            continue
        p = [FAKE] * 10
        p[i] = None
        assert _step(_dims(), p) == 1, i
        p[i] = MISALIGNED
        assert _step(_dims(), p) == 3, i


def test_out_aliasing_rejected():
    p = [FAKE] * 10
    p[9] = p[0]     # out == q
    assert _step(_dims(), p) == 2
    assert "overlap" in hb.last_error()
    p = [_addr(i) for i in range(10)]
    p[9] = p[8]     # out == block_len
    assert _step(_dims(), p) == 2
    assert "overlap" in hb.last_error()


def test_zero_batch_is_a_noop():
    assert _step(_dims(batch=0), [None] * 10) == 0
    assert hb.last_error() == ""


def _addr(i):
    return ctypes.c_void_p(0x1000000 * (i + 1))   # 16 MiB apart: disjoint, aligned, never dereferenced


def test_step_commit_validation():
    """The fused step+commit: null, alignment and every written/read overlap."""
    lib = hb.load()
    d = _dims()
    call = lambda p, dims=d: lib.hybrid_attn_step_commit(ctypes.byref(dims), *p, None)
    ok = [_addr(i) for i in range(10)]
    ok[7] = None                                    # slots may be NULL
    for i in range(10):
        if i in (7, 8):                             # slots, block_len may be NULL
            continue
        p = list(ok)
        p[i] = None
        assert call(p) == 1, i
        p[i] = MISALIGNED
        assert call(p) == 3, i
    assert call(list(ok), _dims(head_dim=96)) == 5
    # written buffers: out (9), S (5), z (6); read: q k v W alpha (0-4),
    # block_len (8); slots (7) is NULL here and checked below
    for w_i in (5, 6, 9):
        for r_i in (0, 1, 2, 3, 4, 5, 6, 8, 9):
            if r_i == w_i:
                continue
            p = list(ok)
            p[w_i] = p[r_i]
            assert call(p) == 2, (w_i, r_i)
            assert "overlap" in hb.last_error()
    for w_i in (5, 6, 9):
        p = list(ok)
        p[7] = _addr(12)
        p[w_i] = p[7]
        assert call(p) == 2, ("slots", w_i)
    p = list(ok)
    p[8] = MISALIGNED
    assert call(p) == 3
    assert lib.hybrid_attn_step_commit(ctypes.byref(_dims(batch=0)), *([None] * 10), None) == 0


def test_commit_prefill_softmax_validation():
    lib = hb.load()
    d = _dims()
    assert lib.hybrid_state_commit(ctypes.byref(d), FAKE, FAKE, FAKE, None, FAKE, None, None,
                                   None) == 1
    assert lib.hybrid_state_commit(ctypes.byref(_dims(feat_dim=48)), FAKE, FAKE, FAKE, FAKE,
                                   FAKE, None, None, None) == 5
    # S and z overlapping
    assert lib.hybrid_state_commit(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, None, None,
                                   None) == 2
    # block_len misaligned
    assert lib.hybrid_state_commit(ctypes.byref(d), _addr(0), _addr(1), _addr(2), _addr(3),
                                   _addr(4), None, MISALIGNED, None) == 3
    # prefill: seq_len not a multiple of the block
    assert lib.hybrid_state_prefill(ctypes.byref(d), 40, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                    FAKE, None, None, None, 0, None) == 2
    assert lib.hybrid_state_prefill(ctypes.byref(d), 0, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                    FAKE, None, None, None, 0, None) == 2
    # prefill over many blocks for few (request, head) units needs a workspace
    dp = _dims(batch=1, n_q_heads=4, n_kv_heads=1, n_slots=1)
    need_p = lib.hybrid_workspace_bytes(ctypes.byref(dp), hb.OP_PREFILL, 32 * 64)
    assert need_p > 0
    assert lib.hybrid_state_prefill(ctypes.byref(dp), 32 * 64, FAKE, FAKE, FAKE, FAKE, FAKE,
                                    ctypes.c_void_p(0x100000), ctypes.c_void_p(0x200000),
                                    None, None, None, 0, None) == 6
    assert lib.hybrid_state_prefill(ctypes.byref(dp), 32 * 64, FAKE, FAKE, FAKE, FAKE, FAKE,
                                    ctypes.c_void_p(0x100000), ctypes.c_void_p(0x200000),
                                    None, None, ctypes.c_void_p(0x300000), need_p - 1,
                                    None) == 6
    # softmax prefix: missing workspace
    need = lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_SOFTMAX_PREFIX, 4096)
    assert need > 0
    assert lib.softmax_prefix_step(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4096,
                                   FAKE, None, 0, None) == 6
    assert lib.softmax_prefix_step(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4096,
                                   ctypes.c_void_p(0x100000), FAKE, need - 1, None) == 6
    assert lib.softmax_prefix_step(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, -1,
                                   FAKE, FAKE, need, None) == 2
    # more than 8 query heads per KV head
    assert lib.softmax_prefix_step(ctypes.byref(_dims(n_kv_heads=1)), FAKE, FAKE, FAKE, FAKE,
                                   FAKE, FAKE, 64, FAKE, FAKE, need, None) == 5


def test_workspace_query():
    lib = hb.load()
    d = _dims(batch=128)
    assert lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_STEP, 0) == 0
    assert lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_COMMIT, 0) == 0
    ws = lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_SOFTMAX_PREFIX, 32768)
    # n_split partial rows of (d + 2) floats per (request, head, query)
    assert ws % (128 * 16 * 32 * 130 * 4) == 0 and ws > 0
    assert lib.hybrid_workspace_bytes(ctypes.byref(_dims(head_dim=5)), hb.OP_STEP, 0) == 0
    assert lib.hybrid_workspace_bytes(None, hb.OP_STEP, 0) == 0
    # a short prefix is not split: the kernel writes out directly, no workspace
    assert lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_SOFTMAX_PREFIX, 64) == 0


def test_softmax_prefix_workspace_overlap():
    lib = hb.load()
    d = _dims(batch=2)
    need = lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_SOFTMAX_PREFIX, 4096)
    assert need > 0
    # q k v k_cache v_cache prefix_len | out ws
    ptrs = [_addr(i) for i in range(8)]
    call = lambda p: lib.softmax_prefix_step(ctypes.byref(d), *p[:6], 4096, p[6], p[7], need, None)
    for r_i in range(6):
        p = list(ptrs)
        p[7] = p[r_i]
        assert call(p) == 2, r_i
        assert "overlap" in hb.last_error()


def test_prefill_workspace_holds_the_snapshot():
    # the increments of the pieces of segments 0 .. nseg-2 (at most 7
    # segments of at most 16 pieces here: 64 blocks, pieces of 2 or more),
    # then a snapshot of the incoming state
    lib = hb.load()
    d = _dims(batch=1, n_q_heads=4, n_kv_heads=1, n_slots=1)
    T = 32 * 64
    need = lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_PREFILL, T)
    f, D, units = 128, 128, 4
    per = (D * f + f) * 4
    assert need % (units * per) == 0
    pieces = need // (units * per) - 1
    assert 1 <= pieces <= 7 * 16


def test_backward_validation():
    lib = hb.load()
    d = _dims(feat_dim=128)
    T = 64
    need = lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_BACKWARD, T)
    assert need > 0
    assert lib.hybrid_workspace_bytes(ctypes.byref(_dims(feat_dim=256)), hb.OP_BACKWARD, T) == 0
    assert lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_BACKWARD, 40) == 0
    # q k v W alpha dout target dW dalpha loss ws
    ok = [_addr(i) for i in range(11)]
    ok[6] = None   # dout mode
    ok[9] = None   # no loss without a target
    call = lambda p, dims=d, t=T, n=need: lib.hybrid_attn_backward(
        ctypes.byref(dims), t, *p[:10], p[10], n, None)
    for i in (0, 1, 2, 3, 4, 7, 8, 10):
        p = list(ok)
        p[i] = None
        assert call(p) == (6 if i == 10 else 1), i
        p[i] = MISALIGNED
        assert call(p) == 3, i
    p = list(ok)
    p[6] = _addr(6)                          # dout and target
    assert call(p) == 2 and "exactly one" in hb.last_error()
    p = list(ok)
    p[5] = None                              # neither
    assert call(p) == 2
    p = list(ok)
    p[9] = _addr(9)                          # loss without a target
    assert call(p) == 2
    assert call(list(ok), _dims(feat_dim=256)) == 5
    assert call(list(ok), _dims(feat_dim=128, flags=1)) == 2
    assert call(list(ok), d, 48) == 2        # not a multiple of the block
    assert call(list(ok), d, T, need - 1) == 6
    # written buffers dW (7), dalpha (8), ws (10) against the inputs and each other
    for w_i in (7, 8, 10):
        for r_i in (0, 1, 2, 3, 4, 5, 7, 8, 10):
            if r_i == w_i:
                continue
            p = list(ok)
            p[w_i] = p[r_i]
            assert call(p) == 2, (w_i, r_i)
            assert "overlap" in hb.last_error()
    assert lib.hybrid_attn_backward(ctypes.byref(_dims(batch=0, feat_dim=128)), T,
                                    *([None] * 11), 0, None) == 0


def test_prefill_noalloc_rejects_beyond_scratch():
    """The entry point that allocates nothing refuses a call whose workspace
    exceeds the library-held scratch buffer, before any HIP call."""
    lib = hb.load()
    # (48 units: 6 segments, their increments in 10 pieces, f = 256)
    d = _dims(batch=3, n_q_heads=16, n_kv_heads=4, feat_dim=256, n_slots=3)
    T = 32 * 64
    need = lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_PREFILL, T)
    assert need > hb.NOALLOC_SCRATCH_BYTES
    p = [_addr(i) for i in range(10)]
    rc = lib.hybrid_state_prefill_noalloc(ctypes.byref(d), T, p[0], p[1], p[2], p[3], p[4],
                                          p[5], p[6], None, p[7], None)
    assert rc == 6
    assert "scratch" in hb.last_error() and str(hb.NOALLOC_SCRATCH_BYTES) in hb.last_error()
    # the same validation as hybrid_state_prefill
    assert lib.hybrid_state_prefill_noalloc(ctypes.byref(d), 40, *p[:7], None, p[7], None) == 2
    assert lib.hybrid_state_prefill_noalloc(ctypes.byref(d), T, None, p[1], *p[2:7], None,
                                            p[7], None) == 1
    assert lib.hybrid_state_prefill_noalloc(ctypes.byref(_dims(batch=0)), T,
                                            *([None] * 10)) == 0


def test_softmax_prefix_paged_validation():
    lib = hb.load()
    d = _dims(batch=2)
    # q k v k_pages v_pages | page_table prefix_len out ws
    p = [_addr(i) for i in range(9)]
    need = lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_SOFTMAX_PREFIX, 64 * 32)

    def call(n_pages=10, ps=32, max_pages=64, ptrs=p, ws_bytes=None, dims=d):
        return lib.softmax_prefix_step_paged(
            ctypes.byref(dims), *ptrs[:5], n_pages, ps, ptrs[5], max_pages, ptrs[6], ptrs[7],
            ptrs[8], need if ws_bytes is None else ws_bytes, None)

    for ps in (0, 16, 48, 1 << 17):
        assert call(ps=ps) == 5, ps
        assert "page_size" in hb.last_error()
    assert call(max_pages=-1) == 2
    assert call(n_pages=0) == 2
    for i in (0, 1, 2, 3, 4, 5, 6, 7):
        q = list(p)
        q[i] = None
        assert call(ptrs=q) == 1, i
        q[i] = MISALIGNED
        assert call(ptrs=q) == 3, i
    assert call(ws_bytes=need - 1) == 6
    # out and the workspace against every input
    for w_i in (7, 8):
        for r_i in range(7):
            q = list(p)
            q[w_i] = q[r_i]
            assert call(ptrs=q) == 2, (w_i, r_i)
            assert "overlap" in hb.last_error()
    assert call(dims=_dims(batch=0)) == 0
    # the workspace is sized by max_pages * page_size
    assert need == lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_SOFTMAX_PREFIX, 2048)


def test_backward_full_validation():
    lib = hb.load()
    d = _dims(feat_dim=128)
    T = 64
    need = lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_BACKWARD_FULL, T)
    assert need > lib.hybrid_workspace_bytes(ctypes.byref(d), hb.OP_BACKWARD, T)
    # q k v W alpha dout target dq dk dv dW dalpha loss ws
    ok = [_addr(i) for i in range(14)]
    ok[6] = None   # dout mode
    ok[12] = None  # no loss without a target
    call = lambda p, n=need: lib.hybrid_attn_backward_full(ctypes.byref(d), T, *p[:13], p[13], n,
                                                           None)
    for i in (7, 8, 9):
        p = list(ok)
        p[i] = None
        assert call(p) == 1, i
        p[i] = MISALIGNED
        assert call(p) == 3, i
    assert call(ok, need - 1) == 6
    # dq, dk, dv against the inputs, each other and the workspace
    for w_i in (7, 8, 9):
        for r_i in (0, 1, 2, 3, 4, 5, 7, 8, 9, 10, 11, 13):
            if r_i == w_i:
                continue
            p = list(ok)
            p[w_i] = p[r_i]
            assert call(p) == 2, (w_i, r_i)
            assert "overlap" in hb.last_error()


def test_step_kernel_flags():
    lib = hb.load()
    p = [_addr(i) for i in range(11)]
    step = lambda dims: lib.hybrid_attn_step(ctypes.byref(dims), *p[:7], None, None, p[10], None)
    assert step(_dims(flags=hb.HYB_STEP_SPLIT | hb.HYB_STEP_WHOLE)) == 2
    assert "more than one" in hb.last_error()
    assert step(_dims(flags=hb.HYB_STEP_WHOLE | hb.HYB_STEP_HALVES)) == 2
    assert step(_dims(flags=16)) == 2
    # the column-split kernel: bf16, feat_dim <= 128, Hq / Hkv a multiple of 4
    for kw in (dict(dtype=hb.HYB_F32), dict(feat_dim=256), dict(n_kv_heads=8)):
        assert step(_dims(flags=hb.HYB_STEP_HALVES, **kw)) == 5, kw
        assert "HYB_STEP_HALVES" in hb.last_error()
    d = _dims(flags=hb.HYB_STEP_HALVES)
    assert lib.hybrid_state_commit(ctypes.byref(d), *p[:5], None, None, None) == 2
    assert "hybrid_attn_step only" in hb.last_error()
    # the other entry points reject them
    d = _dims(flags=hb.HYB_STEP_SPLIT)
    assert lib.hybrid_state_commit(ctypes.byref(d), *p[:5], None, None, None) == 2
    assert "hybrid_attn_step only" in hb.last_error()
    assert lib.hybrid_attn_step_commit(ctypes.byref(d), *p[:7], None, None, p[10], None) == 2
    assert lib.softmax_prefix_step(ctypes.byref(d), *p[:6], 64, p[6], p[7], 1 << 30, None) == 2
