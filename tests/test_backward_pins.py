"""Pins of the oracle's backward (the Stage-1 gradient of Section 3.2) on
the CPU: against things other than its own reverse-mode code.

* Central finite differences of the oracle's forward (the block-causal
  prefill) in fp64, for every entry of W and alpha.
* torch.autograd in fp64 through a dense formulation of the Figure 2
  pattern written here (no recurrent state, no hand-written derivative).
* Closed forms: a single block makes the output independent of W and alpha
  (w cancels in the shared normaliser, the state is empty), so both
  gradients vanish; equal values v_t make every output equal that value,
  so both gradients vanish for any upstream gradient.
* Structure: linear in the upstream gradient; the attention-transfer mode
  equals the plain mode with dout = 2 (out - target), and its loss is the
  squared error of the forward's output.
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _case(B=2, T=12, Hq=2, Hkv=1, d=8, F=4, L=4, seed=0, wscale=0.5):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(B, T, Hq, d))
    k = rng.normal(size=(B, T, Hkv, d))
    v = rng.normal(size=(B, T, Hkv, d))
    Wt = rng.normal(size=(Hq, F, d)) * wscale
    alpha = rng.normal(size=Hq)
    g = rng.normal(size=(B, T, Hq, d))
    return q, k, v, Wt, alpha, g, L


def _forward(q, k, v, Wt, alpha, L):
    B, T, Hq, d = q.shape
    S, z = oracle.empty_state(B, Hq, 2 * Wt.shape[1], d)
    out, _, _ = oracle.prefill(q, k, v, Wt, alpha, S, z, L)
    return out


def test_backward_matches_finite_differences():
    q, k, v, Wt, alpha, g, L = _case()
    dW, da, loss = oracle.backward(q, k, v, Wt, alpha, L, dout=g)
    assert loss is None
    eps = 1e-6
    obj = lambda W_, a_: float((_forward(q, k, v, W_, a_, L) * g).sum())
    fd = np.zeros_like(Wt)
    for idx in np.ndindex(*Wt.shape):
        Wp, Wm = Wt.copy(), Wt.copy()
        Wp[idx] += eps
        Wm[idx] -= eps
        fd[idx] = (obj(Wp, alpha) - obj(Wm, alpha)) / (2 * eps)
    fda = np.zeros_like(alpha)
    for h in range(alpha.size):
        ap, am = alpha.copy(), alpha.copy()
        ap[h] += eps
        am[h] -= eps
        fda[h] = (obj(Wt, ap) - obj(Wt, am)) / (2 * eps)
    scale = np.abs(fd).max()
    assert scale > 1e-2
    np.testing.assert_allclose(dW, fd, rtol=0, atol=1e-7 * max(1.0, scale))
    np.testing.assert_allclose(da, fda, rtol=0, atol=1e-7 * max(1.0, np.abs(fda).max()))


def _dense_torch(q, k, v, Wt, alpha, L):
    """Figure 2 as one dense weight matrix per (request, head), in torch fp64:
    w exp(q.k/sqrt(d)) inside the block, phi(q).phi(k) for earlier blocks,
    zero after, rows normalised (the shared normaliser of Section 3.1)."""
    B, T, Hq, d = q.shape
    Hkv = k.shape[2]
    blk = torch.arange(T) // L
    same = blk[:, None] == blk[None, :]
    before = blk[None, :] < blk[:, None]

    def phi(X, Wh):
        U = X @ Wh.T
        return torch.cat([torch.softmax(U, -1), torch.softmax(-U, -1)], -1)

    outs = []
    for b in range(B):
        per_head = []
        for h in range(Hq):
            gk = h // (Hq // Hkv)
            Q, K, V = q[b, :, h], k[b, :, gk], v[b, :, gk]
            w = torch.sigmoid(alpha[h])
            A = torch.where(same, w * torch.exp(Q @ K.T / d ** 0.5), torch.zeros(()))
            A = A + torch.where(before, phi(Q, Wt[h]) @ phi(K, Wt[h]).T, torch.zeros(()))
            per_head.append((A @ V) / A.sum(1, keepdim=True))
        outs.append(torch.stack(per_head, 1))
    return torch.stack(outs, 0)


@pytest.mark.parametrize("seed,Hq,Hkv", [(1, 2, 1), (2, 4, 2)])
def test_backward_matches_autograd_of_dense_form(seed, Hq, Hkv):
    q, k, v, Wt, alpha, g, L = _case(B=2, T=16, Hq=Hq, Hkv=Hkv, d=8, F=4, L=4, seed=seed)
    for mode in ("dout", "target"):
        tq = [torch.tensor(x) for x in (q, k, v)]
        tW = torch.tensor(Wt, requires_grad=True)
        ta = torch.tensor(alpha, requires_grad=True)
        out = _dense_torch(*tq, tW, ta, L)
        if mode == "dout":
            obj = (out * torch.tensor(g)).sum()
            dW, da, _ = oracle.backward(q, k, v, Wt, alpha, L, dout=g)
        else:
            tgt = g * 0.3
            obj = ((out - torch.tensor(tgt)) ** 2).sum()
            dW, da, loss = oracle.backward(q, k, v, Wt, alpha, L, target=tgt)
            np.testing.assert_allclose(loss.sum(), obj.item(), rtol=1e-12)
        obj.backward()
        np.testing.assert_allclose(dW, tW.grad.numpy(), rtol=0, atol=1e-10)
        np.testing.assert_allclose(da, ta.grad.numpy(), rtol=0, atol=1e-10)


def test_single_block_gradients_vanish():
    """T = L: the state is empty, lin = 0, and out = sm_num / sm_den does not
    depend on W or on w."""
    q, k, v, Wt, alpha, g, L = _case(T=8, L=8, seed=3)
    dW, da, _ = oracle.backward(q, k, v, Wt, alpha, L, dout=g)
    assert np.abs(dW).max() == 0.0
    assert np.abs(da).max() < 1e-12


def test_equal_values_gradients_vanish():
    """v_t = v for all t: both branches are convex combinations of v, so
    out = v everywhere, whatever W and alpha."""
    q, k, v, Wt, alpha, g, L = _case(seed=4)
    v[:] = v[:, :1]
    dW, da, _ = oracle.backward(q, k, v, Wt, alpha, L, dout=g)
    assert np.abs(dW).max() < 1e-12
    assert np.abs(da).max() < 1e-12
    out = _forward(q, k, v, Wt, alpha, L)
    np.testing.assert_allclose(out, np.broadcast_to(v[:, :1].repeat(q.shape[2], 2), out.shape),
                               atol=1e-12)


def test_linear_in_dout_and_transfer_mode():
    q, k, v, Wt, alpha, g, L = _case(seed=5)
    g2 = np.random.default_rng(6).normal(size=g.shape)
    a = oracle.backward(q, k, v, Wt, alpha, L, dout=g)
    b = oracle.backward(q, k, v, Wt, alpha, L, dout=g2)
    c = oracle.backward(q, k, v, Wt, alpha, L, dout=g + 2.0 * g2)
    np.testing.assert_allclose(c[0], a[0] + 2.0 * b[0], atol=1e-12)
    np.testing.assert_allclose(c[1], a[1] + 2.0 * b[1], atol=1e-12)
    target = np.random.default_rng(7).normal(size=g.shape) * 0.2
    out = _forward(q, k, v, Wt, alpha, L)
    dW, da, loss = oracle.backward(q, k, v, Wt, alpha, L, target=target)
    dW2, da2, _ = oracle.backward(q, k, v, Wt, alpha, L, dout=2.0 * (out - target))
    np.testing.assert_allclose(dW, dW2, atol=1e-12)
    np.testing.assert_allclose(da, da2, atol=1e-12)
    np.testing.assert_allclose(loss, ((out - target) ** 2).sum(axis=(0, 1, 3)), rtol=1e-12)


def test_batch_sums_and_gqa_heads():
    """Gradients are sums over requests; a query head uses its own W_h but the
    KV head h / (Hq / Hkv)."""
    q, k, v, Wt, alpha, g, L = _case(B=3, Hq=4, Hkv=2, seed=8)
    dW, da, _ = oracle.backward(q, k, v, Wt, alpha, L, dout=g)
    acc_W, acc_a = np.zeros_like(dW), np.zeros_like(da)
    for b in range(3):
        sl = slice(b, b + 1)
        x = oracle.backward(q[sl], k[sl], v[sl], Wt, alpha, L, dout=g[sl])
        acc_W += x[0]
        acc_a += x[1]
    np.testing.assert_allclose(dW, acc_W, atol=1e-12)
    np.testing.assert_allclose(da, acc_a, atol=1e-12)
    # heads 0 and 1 share KV head 0: swapping their W and alpha swaps their gradients
    Wsw, asw = Wt.copy(), alpha.copy()
    Wsw[[0, 1]], asw[[0, 1]] = Wt[[1, 0]], alpha[[1, 0]]
    qsw, gsw = q.copy(), g.copy()
    qsw[:, :, [0, 1]], gsw[:, :, [0, 1]] = q[:, :, [1, 0]], g[:, :, [1, 0]]
    y = oracle.backward(qsw, k, v, Wsw, asw, L, dout=gsw)
    perm = [1, 0, 2, 3]
    np.testing.assert_allclose(y[0][perm], dW, atol=1e-12)
    np.testing.assert_allclose(y[1][perm], da, atol=1e-12)


def test_backward_rejects_bad_arguments():
    q, k, v, Wt, alpha, g, L = _case()
    with pytest.raises(AssertionError):
        oracle.backward(q, k, v, Wt, alpha, L)
    with pytest.raises(ValueError):
        oracle.backward(q, k, v, Wt, alpha, 5, dout=g)


# ---------------------------------------------------------------------------
# Gradients with respect to the inputs q, k, v (end-to-end training through
# the hybrid layers, Stage 2 of Section 3.2).
# ---------------------------------------------------------------------------


def test_input_gradients_match_finite_differences():
    """Central differences of the oracle's forward for every entry of q, k
    and v; two query heads share one KV head, so dk and dv sum over them."""
    q, k, v, Wt, alpha, g, L = _case(B=1, T=12, Hq=2, Hkv=1, d=6, F=4, L=4, seed=11)
    _, _, _, dq, dk, dv = oracle.backward(q, k, v, Wt, alpha, L, dout=g, inputs=True)
    eps = 1e-6
    obj = lambda q_, k_, v_: float((_forward(q_, k_, v_, Wt, alpha, L) * g).sum())
    for name, x, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        fd = np.zeros_like(x)
        for idx in np.ndindex(*x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            args_p = {"q": q, "k": k, "v": v}
            args_m = dict(args_p)
            args_p[name], args_m[name] = xp, xm
            fd[idx] = (obj(**{n + "_": a for n, a in args_p.items()}) -
                       obj(**{n + "_": a for n, a in args_m.items()})) / (2 * eps)
        scale = np.abs(fd).max()
        assert scale > 1e-2, name
        np.testing.assert_allclose(grad, fd, rtol=0, atol=1e-7 * max(1.0, scale), err_msg=name)


@pytest.mark.parametrize("seed,Hq,Hkv", [(12, 2, 1), (13, 4, 2)])
def test_input_gradients_match_autograd_of_dense_form(seed, Hq, Hkv):
    q, k, v, Wt, alpha, g, L = _case(B=2, T=16, Hq=Hq, Hkv=Hkv, d=8, F=4, L=4, seed=seed)
    for mode in ("dout", "target"):
        tq = [torch.tensor(x, requires_grad=True) for x in (q, k, v)]
        out = _dense_torch(*tq, torch.tensor(Wt), torch.tensor(alpha), L)
        if mode == "dout":
            obj = (out * torch.tensor(g)).sum()
            res = oracle.backward(q, k, v, Wt, alpha, L, dout=g, inputs=True)
        else:
            tgt = g * 0.3
            obj = ((out - torch.tensor(tgt)) ** 2).sum()
            res = oracle.backward(q, k, v, Wt, alpha, L, target=tgt, inputs=True)
        obj.backward()
        for got, t in zip(res[3:], tq):
            np.testing.assert_allclose(got, t.grad.numpy(), rtol=0, atol=1e-10)


def test_single_block_input_gradients_are_softmax_attention_gradients():
    """T = L: the layer is plain bidirectional softmax attention over the
    block (the state is empty), so its input gradients are those of torch's
    scaled_dot_product_attention, with each KV head repeated for its query
    heads."""
    q, k, v, Wt, alpha, g, L = _case(B=2, T=8, Hq=4, Hkv=2, d=8, F=4, L=8, seed=14)
    _, _, _, dq, dk, dv = oracle.backward(q, k, v, Wt, alpha, L, dout=g, inputs=True)
    tq, tk, tv = (torch.tensor(x, requires_grad=True) for x in (q, k, v))
    G = q.shape[2] // k.shape[2]
    out = torch.nn.functional.scaled_dot_product_attention(
        tq.transpose(1, 2), tk.repeat_interleave(G, 2).transpose(1, 2),
        tv.repeat_interleave(G, 2).transpose(1, 2)).transpose(1, 2)
    (out * torch.tensor(g)).sum().backward()
    np.testing.assert_allclose(dq, tq.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dk, tk.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dv, tv.grad.numpy(), rtol=0, atol=1e-12)


def test_input_gradient_invariants():
    """Every output is a convex combination of values, so with v_t = v for
    all t the output is v whatever q and k are (dq = dk = 0); and with a
    constant upstream gradient c, the value gradients of a KV head sum to
    (queries reading it) x c."""
    q, k, v, Wt, alpha, g, L = _case(B=2, T=12, Hq=4, Hkv=2, seed=15)
    ve = v.copy()
    ve[:] = ve[:, :1]
    _, _, _, dq, dk, _ = oracle.backward(q, k, ve, Wt, alpha, L, dout=g, inputs=True)
    assert np.abs(dq).max() < 1e-12 and np.abs(dk).max() < 1e-12
    c = np.random.default_rng(16).normal(size=q.shape[3])
    gc = np.broadcast_to(c, g.shape).copy()
    _, _, _, _, _, dv = oracle.backward(q, k, v, Wt, alpha, L, dout=gc, inputs=True)
    B, T, Hq, d = q.shape
    G = Hq // k.shape[2]
    np.testing.assert_allclose(dv.sum(axis=1), np.broadcast_to(T * G * c, dv.sum(axis=1).shape),
                               atol=1e-10)
