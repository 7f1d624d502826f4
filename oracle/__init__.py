"""fp64 CPU oracle for the block-hybrid attention layer (test infrastructure).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use this package; the library path
never does.  It shares no code with the HIP library.

``oracle.c`` evaluates the paper's definitions literally in double precision
(Section 3.1 for the hybrid step, the state and its update; Section 2.2 for
softmax attention; Figure 2 for the block-causal prefill pattern), and the
exact reverse-mode gradient of that prefill with respect to the Stage-1
parameters {W, alpha} of Section 3.2.  This module
compiles it with gcc and wraps it with NumPy arrays.  ``brute.py`` holds
independent dense formulations used to pin it.

All arrays follow the documented layouts:
  q, out [B][L][Hq][d]; k, v [B][L][Hkv][d]; Wt [Hq][F][d] (W_h transposed);
  alpha [Hq]; S [n_slots][Hq][2F][d]; z [n_slots][Hq][2F]; slots [B] int32;
  k_cache, v_cache [B][Pmax][Hkv][d]; plen [B] int32.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)


def build() -> str:
    """Compile oracle.c into liboracle.so next to it (plain -O2, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC", _SRC,
           "-o", _LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    i = ctypes.c_int
    lib.oracle_step.argtypes = [i] * 6 + [_dp] * 7 + [_ip, _dp]
    lib.oracle_commit.argtypes = [i] * 6 + [_dp] * 5 + [_ip]
    lib.oracle_prefill.argtypes = [i] * 7 + [_dp] * 7 + [_ip, _dp]
    lib.oracle_softmax_prefix.argtypes = [i] * 6 + [_dp] * 5 + [_ip, _dp]
    lib.oracle_feature_map.argtypes = [i] * 3 + [_dp] * 3
    lib.oracle_backward.argtypes = [i] * 7 + [_dp] * 13
    lib.oracle_set_threads.argtypes = [i]
    lib.oracle_max_threads.restype = i
    for fn in (lib.oracle_step, lib.oracle_commit, lib.oracle_prefill,
               lib.oracle_softmax_prefix, lib.oracle_feature_map, lib.oracle_backward):
        fn.restype = ctypes.c_int
    _lib = lib
    return lib


def _d(a):
    a = np.ascontiguousarray(a, dtype=np.float64)
    return a, a.ctypes.data_as(_dp)


def _slots(slots, B):
    if slots is None:
        return None, None
    s = np.ascontiguousarray(slots, dtype=np.int32)
    assert s.shape == (B,)
    return s, s.ctypes.data_as(_ip)


def _check(rc, what):
    if rc == 1:
        raise FloatingPointError(f"{what}: an exponent reached |x| >= 700")
    if rc != 0:
        raise ValueError(f"{what}: invalid arguments (rc={rc})")


def feature_map(X, Wt):
    """phi(x) = [softmax(xW), softmax(-xW)] for every row of X [n][d]."""
    lib = _load()
    X, pX = _d(X)
    Wt, pW = _d(Wt)
    n, d = X.shape
    F = Wt.shape[0]
    assert Wt.shape == (F, d)
    out = np.zeros((n, 2 * F))
    _check(lib.oracle_feature_map(n, d, F, pX, pW, out.ctypes.data_as(_dp)),
           "feature_map")
    return out


def step(q, k, v, Wt, alpha, S, z, slots=None):
    """Hybrid output of every active-block query; returns out [B][L][Hq][d]."""
    lib = _load()
    q, pq = _d(q)
    k, pk = _d(k)
    v, pv = _d(v)
    Wt, pW = _d(Wt)
    alpha, pa = _d(alpha)
    S, pS = _d(S)
    z, pz = _d(z)
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    F = Wt.shape[1]
    assert k.shape == (B, L, Hkv, d) and v.shape == k.shape
    assert Wt.shape == (Hq, F, d) and S.shape[1:] == (Hq, 2 * F, d)
    assert z.shape == S.shape[:3] and Hq % Hkv == 0
    s, ps = _slots(slots, B)
    out = np.zeros_like(q)
    _check(lib.oracle_step(B, Hq, Hkv, d, L, F, pq, pk, pv, pW, pa, pS, pz, ps,
                           out.ctypes.data_as(_dp)), "step")
    return out


def commit(k, v, Wt, S, z, slots=None):
    """Returns (S', z') = state with the block's tokens folded in (copies)."""
    lib = _load()
    k, pk = _d(k)
    v, pv = _d(v)
    Wt, pW = _d(Wt)
    S = np.array(S, dtype=np.float64, copy=True, order="C")
    z = np.array(z, dtype=np.float64, copy=True, order="C")
    B, L, Hkv, d = k.shape
    Hq, F = Wt.shape[0], Wt.shape[1]
    assert S.shape[1:] == (Hq, 2 * F, d) and z.shape == S.shape[:3]
    s, ps = _slots(slots, B)
    _check(lib.oracle_commit(B, Hq, Hkv, d, L, F, pk, pv, pW,
                             S.ctypes.data_as(_dp), z.ctypes.data_as(_dp), ps),
           "commit")
    return S, z


def step_commit(q, k, v, Wt, alpha, S, z, slots=None):
    """The last denoising step of a block fused with its commit (Section 3.3:
    one pass computes the within-block softmax, the readout, the gated merge
    and the causal state update).  By definition: the step's output on the
    state as it was, then the commit of the same block's keys and values.
    Returns (out, S', z') (copies)."""
    out = step(q, k, v, Wt, alpha, S, z, slots)
    S1, z1 = commit(k, v, Wt, S, z, slots)
    return out, S1, z1


def prefill(q, k, v, Wt, alpha, S, z, L, slots=None, want_out=True):
    """Block-causal prefill of T tokens in blocks of L.

    Returns (out or None, S', z'); the state arrays are copies.
    """
    lib = _load()
    k, pk = _d(k)
    v, pv = _d(v)
    Wt, pW = _d(Wt)
    alpha, pa = _d(alpha)
    S = np.array(S, dtype=np.float64, copy=True, order="C")
    z = np.array(z, dtype=np.float64, copy=True, order="C")
    B, T, Hkv, d = k.shape
    Hq, F = Wt.shape[0], Wt.shape[1]
    s, ps = _slots(slots, B)
    if want_out:
        q, pq = _d(q)
        assert q.shape == (B, T, Hq, d)
        out = np.zeros_like(q)
        pout = out.ctypes.data_as(_dp)
    else:
        pq, out, pout = None, None, None
    _check(lib.oracle_prefill(B, T, Hq, Hkv, d, L, F, pq, pk, pv, pW, pa,
                              S.ctypes.data_as(_dp), z.ctypes.data_as(_dp), ps,
                              pout), "prefill")
    return out, S, z


def softmax_prefix(q, k, v, k_cache, v_cache, plen):
    """Exact softmax of each block query over its cached prefix plus the block."""
    lib = _load()
    q, pq = _d(q)
    k, pk = _d(k)
    v, pv = _d(v)
    kc, pkc = _d(k_cache)
    vc, pvc = _d(v_cache)
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    Pmax = kc.shape[1]
    assert kc.shape == (B, Pmax, Hkv, d) and vc.shape == kc.shape
    pl = np.ascontiguousarray(plen, dtype=np.int32)
    assert pl.shape == (B,) and (pl >= 0).all() and (pl <= Pmax).all()
    out = np.zeros_like(q)
    _check(lib.oracle_softmax_prefix(B, Hq, Hkv, d, L, Pmax, pq, pk, pv, pkc,
                                     pvc, pl.ctypes.data_as(_ip),
                                     out.ctypes.data_as(_dp)), "softmax_prefix")
    return out


def backward(q, k, v, Wt, alpha, L, dout=None, target=None, inputs=False):
    """Gradient of the block-causal hybrid layer over a training sequence
    (empty starting state, blocks of L) with respect to W and alpha, the
    parameters Stage 1 of Section 3.2 trains, and (inputs=True) with respect
    to the layer's inputs q, k, v, which end-to-end training through the
    layer (Stage 2) needs.

    Exactly one of dout (upstream gradient, objective sum <dout, out>) and
    target (the softmax teacher's output; objective sum |out - target|^2,
    the attention-transfer loss) is given.  Returns (dWt [Hq][F][d],
    dalpha [Hq], loss [Hq] or None), then with inputs=True also (dq, dk, dv)
    in the layouts of q, k, v; dW and dalpha are summed over the batch, dk
    and dv over the query heads that share a KV head.
    """
    assert (dout is None) != (target is None)
    lib = _load()
    q, pq = _d(q)
    k, pk = _d(k)
    v, pv = _d(v)
    Wt, pW = _d(Wt)
    alpha, pa = _d(alpha)
    B, T, Hq, d = q.shape
    Hkv = k.shape[2]
    F = Wt.shape[1]
    if dout is not None:
        g, pg = _d(dout)
        assert g.shape == q.shape
        pt = None
    else:
        t, pt = _d(target)
        assert t.shape == q.shape
        pg = None
    dW = np.zeros((Hq, F, d))
    da = np.zeros(Hq)
    loss = np.zeros(Hq) if target is not None else None
    dq = np.zeros(q.shape) if inputs else None
    dk = np.zeros(k.shape) if inputs else None
    dv = np.zeros(v.shape) if inputs else None
    ptr = lambda a: a.ctypes.data_as(_dp) if a is not None else None
    _check(lib.oracle_backward(B, T, Hq, Hkv, d, L, F, pq, pk, pv, pW, pa, pg, pt,
                               ptr(dW), ptr(da), ptr(loss), ptr(dq), ptr(dk), ptr(dv)),
           "backward")
    if inputs:
        return dW, da, loss, dq, dk, dv
    return dW, da, loss


def set_threads(n: int) -> None:
    """Host threads the oracle's loops use from now on."""
    _load().oracle_set_threads(int(n))


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def empty_state(n_slots, Hq, f, d):
    return np.zeros((n_slots, Hq, f, d)), np.zeros((n_slots, Hq, f))


def state_from_prefix(kp, vp, Wt, n_slots=None, slots=None):
    """State of a prefix kp/vp [B][P][Hkv][d] built token by token (commit)."""
    B, P, Hkv, d = kp.shape
    Hq, F = Wt.shape[0], Wt.shape[1]
    S, z = empty_state(n_slots or B, Hq, 2 * F, d)
    if P == 0:
        return S, z
    return commit(kp, vp, Wt, S, z, slots=slots)
