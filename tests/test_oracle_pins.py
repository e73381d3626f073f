"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

None of these re-types the oracle's own formula: each compares it with an
independent route (autograd, finite differences, SVD, a library SwiGLU, a
per-token loop, brute-force invariants) so that a dropped term, a wrong sign,
a wrong index or a transposed operand in the oracle fails at least one test.
"""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import lact_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
torch.set_default_dtype(torch.float64)


def _rng(seed):
    return np.random.default_rng(seed)


def _weights(rng, h, d, unit=False, scale=1.0):
    W1 = rng.standard_normal((h, d)) * scale
    W2 = rng.standard_normal((d, h)) * scale
    W3 = rng.standard_normal((h, d)) * scale
    if unit:
        W1, W2, W3 = (w / np.linalg.norm(w, axis=1, keepdims=True) for w in (W1, W2, W3))
    return W1, W2, W3


def _tokens(rng, n, d):
    x = rng.standard_normal((n, d))
    return x / np.linalg.norm(x, axis=1, keepdims=True)


def _torch_swiglu(W1, W2, W3, X):
    """Library SwiGLU MLP without biases: F.linear + F.silu (independent of the oracle)."""
    t = lambda a: torch.as_tensor(np.asarray(a, dtype=np.float64))
    x = t(X)
    return F.linear(F.silu(F.linear(x, t(W1))) * F.linear(x, t(W3)), t(W2))


def _torch_loss(W1, W2, W3, K, V, eta):
    """sum_i eta_i * (-f_W(k_i)^T v_i), built from library ops."""
    f = _torch_swiglu(W1, W2, W3, K) if not isinstance(W1, torch.Tensor) else \
        F.linear(F.silu(F.linear(K, W1)) * F.linear(K, W3), W2)
    Vt = V if isinstance(V, torch.Tensor) else torch.as_tensor(V)
    et = eta if isinstance(eta, torch.Tensor) else torch.as_tensor(eta)
    return -(et * (f * Vt).sum(-1)).sum()


# ----------------------------------------------------------------------------- apply


def test_swiglu_apply_matches_library_mlp():
    rng = _rng(1)
    h, d = 7, 5                                   # non-square catches transposes
    W1, W2, W3 = _weights(rng, h, d)
    X = rng.standard_normal((9, d))
    ref = _torch_swiglu(W1, W2, W3, X).numpy()
    np.testing.assert_allclose(O.swiglu_apply(W1, W2, W3, X), ref, rtol=1e-13, atol=1e-13)


def test_sigmoid_silu_extremes():
    z = np.array([-800.0, -30.0, -1.0, 0.0, 1.0, 30.0, 800.0])
    np.testing.assert_allclose(O.sigmoid(z), torch.sigmoid(torch.as_tensor(z)).numpy(), rtol=1e-15)
    np.testing.assert_allclose(O.silu(z), F.silu(torch.as_tensor(z)).numpy(), rtol=1e-15, atol=1e-300)


def test_silu_derivative_against_autograd():
    # includes the saturated ends (derivative 0 and 1) and the minimum of SiLU
    # near z = -1.2785 (derivative 0)
    z = np.concatenate([np.linspace(-40.0, 40.0, 401), [-800.0, -1.2784645427610738, 800.0]])
    tz = torch.as_tensor(z).requires_grad_(True)
    F.silu(tz).sum().backward()
    np.testing.assert_allclose(O.silu_derivative(z), tz.grad.numpy(), rtol=1e-13, atol=1e-15)


# ----------------------------------------------------------------------------- gradient


@pytest.mark.parametrize("h,d,n", [(3, 5, 7), (8, 3, 4), (5, 5, 8)])
def test_chunk_gradient_autograd(h, d, n):
    rng = _rng(10 + h + d + n)
    W = _weights(rng, h, d)
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    eta = rng.uniform(0.1, 2.0, n)
    tw = [torch.tensor(w, requires_grad=True) for w in W]
    _torch_loss(*tw, torch.as_tensor(K), torch.as_tensor(V), torch.as_tensor(eta)).backward()
    g = O.chunk_gradient(*W, K, V, eta)
    for gi, twi in zip(g, tw):
        np.testing.assert_allclose(gi, twi.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("h,d,n", [(3, 5, 7), (8, 3, 4)])
def test_chunk_gradient_finite_differences(h, d, n):
    rng = _rng(20 + h + d + n)
    W = list(_weights(rng, h, d))
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    eta = rng.uniform(0.1, 2.0, n)
    loss = lambda ws: float(_torch_loss(*ws, K, V, eta))
    g = O.chunk_gradient(*W, K, V, eta)
    step = 1e-6
    for j in range(3):
        fd = np.zeros_like(W[j])
        for idx in np.ndindex(*W[j].shape):
            wp = [w.copy() for w in W]; wm = [w.copy() for w in W]
            wp[j][idx] += step; wm[j][idx] -= step
            fd[idx] = (loss(wp) - loss(wm)) / (2 * step)
        err = np.max(np.abs(fd - g[j])) / np.max(np.abs(g[j]))
        assert err < 1e-7, (j, err)


def test_gradient_is_additive_over_token_shards():
    """§3.4: the chunk gradient is a sum over its tokens, so shards add up."""
    rng = _rng(3)
    h, d, n = 6, 4, 23
    W = _weights(rng, h, d)
    K, V, eta = _tokens(rng, n, d), _tokens(rng, n, d), rng.uniform(0, 0.1, n)
    full = O.chunk_gradient(*W, K, V, eta)
    cuts = [0, 5, 6, 17, n]
    parts = [O.chunk_gradient(*W, K[a:b], V[a:b], eta[a:b]) for a, b in zip(cuts[:-1], cuts[1:])]
    for j in range(3):
        np.testing.assert_allclose(sum(p[j] for p in parts), full[j], rtol=1e-12, atol=1e-15)
    blocked = O.chunk_gradient(*W, K, V, eta, token_block=4)   # reading R7
    for j in range(3):
        np.testing.assert_allclose(blocked[j], full[j], rtol=1e-12, atol=1e-15)


def test_gradient_token_permutation_invariance():
    """A chunk is a set of tokens: permuting (k, v, eta) leaves the gradient unchanged."""
    rng = _rng(4)
    W = _weights(rng, 5, 6)
    K, V, eta = _tokens(rng, 11, 6), _tokens(rng, 11, 6), rng.uniform(0, 0.1, 11)
    p = rng.permutation(11)
    a = O.chunk_gradient(*W, K, V, eta)
    b = O.chunk_gradient(*W, K[p], V[p], eta[p])
    for j in range(3):
        np.testing.assert_allclose(a[j], b[j], rtol=1e-12, atol=1e-16)


# ----------------------------------------------------------------------------- Newton-Schulz


def _golden_ns():
    vals = {}
    with open(os.path.join(GOLDEN, "ns_coefficients.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, v = line.split()
                vals[k] = float(v)
    return vals


def test_ns_coefficients_match_paper():
    g = _golden_ns()
    assert O.NS_COEFFS == (g["a"], g["b"], g["c"])
    assert O.NS_STEPS_DEFAULT == int(g["steps"])


def _scalar_quintic(s, steps):
    g = _golden_ns()
    for _ in range(steps):
        s = g["a"] * s + g["b"] * s ** 3 + g["c"] * s ** 5
    return s


@pytest.mark.parametrize("shape", [(5, 8), (8, 5), (6, 6), (1, 4)])
@pytest.mark.parametrize("steps", [0, 1, 5])
def test_ns_commutes_with_svd(shape, steps):
    """NS acts on singular values only: NS(G) = U p^T(S / (||G||_F + eps)) V^T."""
    rng = _rng(5 + shape[0] * 10 + shape[1])
    G = rng.standard_normal(shape)
    U, S, Vt = np.linalg.svd(G, full_matrices=False)
    s = _scalar_quintic(S / (np.linalg.norm(G) + O.NS_EPS), steps)
    ref = (U * s) @ Vt
    np.testing.assert_allclose(O.newton_schulz(G, steps), ref, rtol=1e-10, atol=1e-12)


def test_ns_rank_one_closed_form():
    rng = _rng(6)
    u = rng.standard_normal(7); u /= np.linalg.norm(u)
    v = rng.standard_normal(3); v /= np.linalg.norm(v)
    G = 2.5 * np.outer(u, v)
    p5 = _scalar_quintic(2.5 / (2.5 + O.NS_EPS), 5)
    np.testing.assert_allclose(O.newton_schulz(G, 5), p5 * np.outer(u, v), rtol=1e-12, atol=1e-14)
    assert abs(p5 - 0.6964) < 1e-3


@pytest.mark.parametrize("shape", [(16, 32), (32, 16), (24, 64)])
def test_ns_spectrum_near_one(shape):
    """Muon(g) ~ U V^T: the singular values of the 5-step output sit near 1."""
    rng = _rng(7 + shape[0])
    G = rng.standard_normal(shape)
    s = np.linalg.svd(O.newton_schulz(G, 5), compute_uv=False)
    assert s.min() > 0.6 and s.max() < 1.2, s


def test_ns_zero_gradient_is_zero():
    assert np.all(O.newton_schulz(np.zeros((4, 6)), 5) == 0.0)   # reading R3


# ----------------------------------------------------------------------------- weight update


def test_weight_update_preserves_row_norms_nonsquare():
    rng = _rng(8)
    W = rng.standard_normal((7, 4)) * 3.0
    g = rng.standard_normal((7, 4))
    Wn = O.weight_update(W, g)
    np.testing.assert_allclose(np.linalg.norm(Wn, axis=1), np.linalg.norm(W, axis=1), rtol=1e-13)
    # direction of every row is that of W - g
    U = W - g
    cos = np.sum(Wn * U, axis=1) / (np.linalg.norm(Wn, axis=1) * np.linalg.norm(U, axis=1))
    np.testing.assert_allclose(cos, 1.0, rtol=1e-13)


# ----------------------------------------------------------------------------- layer


def _layer_inputs(seed, n_q, n_kv, d, h, unit=True, eta_scale=0.05):
    rng = _rng(seed)
    W = _weights(rng, h, d, unit=unit, scale=1 / np.sqrt(d))
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = eta_scale * np.log1p(np.exp(rng.standard_normal(n_kv)))
    return q, k, v, eta, W


@pytest.mark.parametrize("order", [0, 1])
@pytest.mark.parametrize("muon", [0, 1])
def test_eta_zero_layer_is_plain_swiglu_mlp(order, muon):
    q, k, v, eta, W = _layer_inputs(9, 40, 33, 6, 10)
    o, Wf = O.lact_forward_instance(q, k, v, np.zeros_like(eta), *W, chunk=8, order=order,
                                    use_muon=bool(muon), ns_steps=5)
    np.testing.assert_allclose(o, _torch_swiglu(*W, q).numpy(), rtol=1e-13, atol=1e-14)
    for a, b in zip(Wf, W):
        np.testing.assert_allclose(a, b, rtol=1e-14, atol=1e-16)


@pytest.mark.parametrize("muon", [0, 1])
def test_row_norms_after_every_update(muon):
    q, k, v, eta, W = _layer_inputs(10, 30, 30, 5, 9, unit=False, eta_scale=0.5)
    W = tuple(w * np.arange(1, w.shape[0] + 1)[:, None] for w in W)   # distinct norms
    trace = []
    _, Wf = O.lact_forward_instance(q, k, v, eta, *W, chunk=7, order=0, use_muon=bool(muon),
                                    trace=trace)
    for Ws in trace[1:] + [Wf]:
        for a, b in zip(Ws, W):
            np.testing.assert_allclose(np.linalg.norm(a, axis=1), np.linalg.norm(b, axis=1),
                                       rtol=1e-12)
    q, k, v, eta, Wu = _layer_inputs(11, 30, 30, 5, 9, unit=True, eta_scale=0.5)
    _, Wf = O.lact_forward_instance(q, k, v, eta, *Wu, chunk=7, order=1, use_muon=bool(muon))
    for a in Wf:
        np.testing.assert_allclose(np.linalg.norm(a, axis=1), 1.0, rtol=1e-12)


@pytest.mark.parametrize("order", [0, 1])
def test_dependency_mask(order):
    """Apply-then-update is shifted block-causal, update-then-apply block-causal;
    the tail sees every key (§3.1, execution orders)."""
    C, n_kv, n_q = 4, 12, 15
    q, k, v, eta, W = _layer_inputs(12, n_q, n_kv, 4, 6, eta_scale=0.5)
    o0, _ = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=order)
    for j in range(n_kv):
        k2 = k.copy(); k2[j] += 0.3
        o1, _ = O.lact_forward_instance(q, k2, v, eta, *W, chunk=C, order=order)
        changed = np.any(np.abs(o1 - o0) > 1e-13, axis=1)
        for i in range(n_q):
            if i >= n_kv:
                expect = True
            elif order == 0:
                expect = j // C < i // C
            else:
                expect = j // C <= i // C
            assert changed[i] == expect, (order, i, j)


def test_single_chunk_orders():
    q, k, v, eta, W = _layer_inputs(13, 10, 10, 4, 8, eta_scale=0.5)
    o0, W0f = O.lact_forward_instance(q, k, v, eta, *W, chunk=10, order=0)
    o1, W1f = O.lact_forward_instance(q, k, v, eta, *W, chunk=10, order=1)
    np.testing.assert_allclose(o0, _torch_swiglu(*W, q).numpy(), rtol=1e-13)
    np.testing.assert_allclose(o1, _torch_swiglu(*W1f, q).numpy(), rtol=1e-13)
    for a, b in zip(W0f, W1f):
        np.testing.assert_allclose(a, b, rtol=1e-14)


def test_query_permutation_within_chunk_permutes_output():
    q, k, v, eta, W = _layer_inputs(14, 16, 16, 4, 6, eta_scale=0.5)
    p = np.concatenate([np.arange(8), 8 + _rng(0).permutation(8)])
    o, _ = O.lact_forward_instance(q, k, v, eta, *W, chunk=8, order=0)
    op, _ = O.lact_forward_instance(q[p], k, v, eta, *W, chunk=8, order=0)
    np.testing.assert_allclose(op, o[p], rtol=1e-13)


@pytest.mark.parametrize("muon", [0, 1])
def test_resume_from_returned_state(muon):
    """The fast weight is the only state carried between chunks (§3, Fig. 2)."""
    q, k, v, eta, W = _layer_inputs(15, 24, 24, 5, 7, eta_scale=0.3)
    o, Wf = O.lact_forward_instance(q, k, v, eta, *W, chunk=6, order=0, use_muon=bool(muon))
    oa, Wa = O.lact_forward_instance(q[:12], k[:12], v[:12], eta[:12], *W, chunk=6, order=0,
                                     use_muon=bool(muon))
    ob, Wb = O.lact_forward_instance(q[12:], k[12:], v[12:], eta[12:], *Wa, chunk=6, order=0,
                                     use_muon=bool(muon))
    np.testing.assert_allclose(np.concatenate([oa, ob]), o, rtol=1e-12, atol=1e-15)
    for a, b in zip(Wb, Wf):
        np.testing.assert_allclose(a, b, rtol=1e-12)


def test_ns_is_scale_free():
    """Muon normalises the absolute scale of the gradient (§3.2): without the
    reading-R3 epsilon NS(alpha G) == NS(G) exactly up to rounding."""
    rng = _rng(16)
    G = rng.standard_normal((6, 9))
    for alpha in (1e-3, 0.5, 40.0):
        np.testing.assert_allclose(O.newton_schulz(alpha * G, 5, eps=0.0),
                                   O.newton_schulz(G, 5, eps=0.0), rtol=1e-12, atol=1e-14)


def test_muon_makes_lr_scale_irrelevant():
    """With Muon, eta only sets the relative weight of tokens in a chunk (§3.2);
    the only scale left is the 1e-7 of reading R3, amplified at most a^5 ~ 484x."""
    q, k, v, eta, W = _layer_inputs(16, 20, 20, 6, 6, eta_scale=5.0)
    _, Wa = O.lact_forward_instance(q, k, v, eta, *W, chunk=10, order=0, use_muon=True)
    for alpha in (0.5, 4.0):
        _, Wb = O.lact_forward_instance(q, k, v, alpha * eta, *W, chunk=10, order=0, use_muon=True)
        for a, b in zip(Wa, Wb):
            np.testing.assert_allclose(a, b, rtol=1e-3, atol=1e-4)


@pytest.mark.parametrize("order", [0, 1])
def test_chunk_one_is_per_token_ttt(order):
    """Chunk size 1 is the per-token TTT layer of §2.1 (update eq. per token, then
    the normalised step), computed here with autograd in a separate loop."""
    n, d, h = 9, 4, 5
    q, k, v, eta, W = _layer_inputs(17, n, n, d, h, eta_scale=0.7)
    o_ref = np.zeros((n, d))
    tw = [torch.tensor(w) for w in W]
    for i in range(n):
        if order == 0:
            o_ref[i] = F.linear(F.silu(F.linear(torch.as_tensor(q[i]), tw[0])) *
                                F.linear(torch.as_tensor(q[i]), tw[2]), tw[1]).numpy()
        req = [w.clone().requires_grad_(True) for w in tw]
        _torch_loss(*req, torch.as_tensor(k[i:i + 1]), torch.as_tensor(v[i:i + 1]),
                    torch.as_tensor(eta[i:i + 1])).backward()
        new = []
        for w, r in zip(tw, req):
            u = w - r.grad
            new.append(u / u.norm(dim=1, keepdim=True) * w.norm(dim=1, keepdim=True))
        tw = new
        if order == 1:
            o_ref[i] = F.linear(F.silu(F.linear(torch.as_tensor(q[i]), tw[0])) *
                                F.linear(torch.as_tensor(q[i]), tw[2]), tw[1]).numpy()
    o, Wf = O.lact_forward_instance(q, k, v, eta, *W, chunk=1, order=order)
    np.testing.assert_allclose(o, o_ref, rtol=1e-11, atol=1e-14)
    for a, b in zip(Wf, tw):
        np.testing.assert_allclose(a, b.numpy(), rtol=1e-11)


def test_partial_last_chunk_and_tail():
    q, k, v, eta, W = _layer_inputs(18, 19, 13, 4, 6, eta_scale=0.4)
    o, Wf = O.lact_forward_instance(q, k, v, eta, *W, chunk=5, order=0)
    # chunks [0,5) [5,10) [10,13): the last partial chunk still updates W
    Wm = tuple(W)
    for s, e in ((0, 5), (5, 10), (10, 13)):
        Wm = O.update(Wm, k[s:e], v[s:e], eta[s:e])
    for a, b in zip(Wf, Wm):
        np.testing.assert_allclose(a, b, rtol=1e-13)
    np.testing.assert_allclose(o[13:], _torch_swiglu(*Wm, q[13:]).numpy(), rtol=1e-13)


# ----------------------------------------------------------------------------- flops


def test_layer_flops_match_paper_counts():
    vals = {}
    with open(os.path.join(GOLDEN, "flops_per_token.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                a, b = line.split()
                vals[a] = float(b)
    d, h = 64, 64
    assert O.layer_flops(1, d, h, 1, 1, 1) == vals["total"] * d * h
    assert O.layer_flops(1, d, h, 0, 1, 1) == vals["query_apply"] * d * h
    assert O.layer_flops(1, d, h, 1, 0, 1) == (vals["key_forward"] + vals["gradients"]) * d * h
    for r in (1, 2):
        m = 32
        mu = O.layer_flops(1, m, r * m, 0, 0, 1, use_muon=True, ns_steps=1)
        assert mu == 3 * vals[f"muon_r{r}_per_iter_over_m3"] * m ** 3


# ----------------------------------------------------------------------------- momentum
# App. A (implementing momentum for test-time optimizers) and Table 3:
#   M <- M * mean_chunk(beta) + g,  W <- L2norm(W - M)  or  L2norm(W - Muon(M)).


def _beta(seed, n, lo=0.05, hi=0.95):
    return _rng(seed).uniform(lo, hi, n)


@pytest.mark.parametrize("order", [0, 1])
@pytest.mark.parametrize("muon", [0, 1])
def test_momentum_beta_zero_is_gradient_descent(order, muon):
    """beta = 0 keeps no memory: M is the chunk's own gradient and the layer is
    the plain update (a sign error or a beta on the wrong term fails here)."""
    q, k, v, eta, W = _layer_inputs(30, 27, 24, 5, 7, eta_scale=0.4)
    o, Wf = O.lact_forward_instance(q, k, v, eta, *W, chunk=8, order=order, use_muon=bool(muon))
    trace = []
    om, Wm, M = O.lact_forward_instance(q, k, v, eta, *W, chunk=8, order=order, use_muon=bool(muon),
                                        beta=np.zeros(24), trace=trace)
    np.testing.assert_array_equal(om, o)
    for a, b in zip(Wm, Wf):
        np.testing.assert_array_equal(a, b)
    g = O.chunk_gradient(*trace[-1], k[16:], v[16:], eta[16:])
    for a, b in zip(M, g):
        np.testing.assert_allclose(a, b, rtol=1e-14, atol=1e-16)


def test_momentum_single_chunk_is_gradient_descent():
    q, k, v, eta, W = _layer_inputs(31, 12, 12, 4, 6, eta_scale=0.4)
    o, Wf = O.lact_forward_instance(q, k, v, eta, *W, chunk=12, order=1)
    om, Wm, _ = O.lact_forward_instance(q, k, v, eta, *W, chunk=12, order=1, beta=_beta(0, 12))
    np.testing.assert_allclose(om, o, rtol=1e-14)
    for a, b in zip(Wm, Wf):
        np.testing.assert_allclose(a, b, rtol=1e-14)


def test_momentum_factor_is_the_current_chunks_mean():
    """The factor of chunk c is the mean of chunk c's own beta: zero beta in the
    second chunk gives two plain updates whatever the first chunk's beta; any
    beta with the same per-chunk means (or permuted in a chunk) gives the same
    layer."""
    C = 8
    q, k, v, eta, W = _layer_inputs(32, 16, 16, 5, 6, eta_scale=0.4)
    beta = np.concatenate([_beta(1, C), np.zeros(C)])
    o, Wf = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=0)
    om, Wm, _ = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=0, beta=beta)
    np.testing.assert_allclose(om, o, rtol=1e-14)
    for a, b in zip(Wm, Wf):
        np.testing.assert_allclose(a, b, rtol=1e-14)
    q, k, v, eta, W = _layer_inputs(33, 24, 24, 5, 6, eta_scale=0.4)
    b1 = _beta(2, 24)
    b2 = b1.copy()
    for s in range(0, 24, C):                     # same means, different tokens
        seg = b2[s:s + C]
        seg[:] = seg.mean() + 0.5 * (_rng(s).uniform(-1, 1, C) * min(seg.mean(), 1 - seg.mean()))
        seg += b1[s:s + C].mean() - seg.mean()
    b3 = np.concatenate([_rng(7).permutation(b1[s:s + C]) for s in range(0, 24, C)])
    ref = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=1, beta=b1)
    for bb in (b2, b3):
        got = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=1, beta=bb)
        np.testing.assert_allclose(got[0], ref[0], rtol=1e-12)
        for a, b in zip(got[1] + got[2], ref[1] + ref[2]):
            np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-15)
    bad = b1.copy(); bad[C] += 0.3               # a different mean (after M0 = 0) changes it
    got = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=1, beta=bad)
    assert np.max(np.abs(got[1][0] - ref[1][0])) > 1e-8


def _torch_ns(G, steps):
    a, b, c = 3.4445, -4.7750, 2.0315
    X = G.T if G.shape[0] > G.shape[1] else G
    X = X / (torch.linalg.matrix_norm(X) + 1e-7)
    for _ in range(steps):
        A = X @ X.T
        X = a * X + (b * A + c * A @ A) @ X
    return X.T if G.shape[0] > G.shape[1] else X


@pytest.mark.parametrize("muon", [0, 1])
def test_momentum_matches_autograd_loop(muon):
    """An independent loop: torch autograd for each chunk's gradient, the
    recurrence of Table 3 and the row normalisation in torch ops."""
    C, n = 6, 18
    q, k, v, eta, W = _layer_inputs(34, n, n, 4, 7, unit=False, eta_scale=0.6)
    beta = _beta(3, n)
    o, Wf, Mf = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=0, use_muon=bool(muon), beta=beta)
    Wt = [torch.as_tensor(w.copy()) for w in W]
    Mt = [torch.zeros_like(w) for w in Wt]
    outs = []
    for s in range(0, n, C):
        Kc, Vc, ec = (torch.as_tensor(a[s:s + C]) for a in (k, v, eta))
        outs.append(_torch_swiglu(*[w.numpy() for w in Wt], q[s:s + C]).numpy())
        Wg = [w.clone().requires_grad_(True) for w in Wt]
        _torch_loss(*Wg, Kc, Vc, ec).backward()
        bbar = float(np.mean(beta[s:s + C]))
        Mt = [bbar * m + w.grad for m, w in zip(Mt, Wg)]
        new = []
        for w, m in zip(Wt, Mt):
            st = _torch_ns(m, 5) if muon else m
            u = w - st
            new.append(u * (w.norm(dim=1, keepdim=True) / u.norm(dim=1, keepdim=True)))
        Wt = new
    np.testing.assert_allclose(o, np.concatenate(outs), rtol=1e-11, atol=1e-13)
    for a, b in zip(Wf, Wt):
        np.testing.assert_allclose(a, b.numpy(), rtol=1e-11, atol=1e-13)
    for a, b in zip(Mf, Mt):
        np.testing.assert_allclose(a, b.detach().numpy(), rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("muon", [0, 1])
def test_momentum_resume_from_returned_state(muon):
    """With momentum the carried state is (W, M)."""
    q, k, v, eta, W = _layer_inputs(35, 24, 24, 5, 7, eta_scale=0.3)
    beta = _beta(4, 24)
    o, Wf, Mf = O.lact_forward_instance(q, k, v, eta, *W, chunk=6, order=0, use_muon=bool(muon), beta=beta)
    oa, Wa, Ma = O.lact_forward_instance(q[:12], k[:12], v[:12], eta[:12], *W, chunk=6, order=0,
                                         use_muon=bool(muon), beta=beta[:12])
    ob, Wb, Mb = O.lact_forward_instance(q[12:], k[12:], v[12:], eta[12:], *Wa, chunk=6, order=0,
                                         use_muon=bool(muon), beta=beta[12:], M=Ma)
    np.testing.assert_allclose(np.concatenate([oa, ob]), o, rtol=1e-12, atol=1e-15)
    for a, b in zip(Wb + Mb, Wf + Mf):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-15)


def test_momentum_muon_acts_on_the_accumulated_state():
    """Muon(M) rather than M + Muon(g): a global eta scale scales every M and
    leaves W unchanged (up to the 1e-7 of reading R3), while scaling only the
    second chunk's eta changes the mix inside M and so the update."""
    C = 8
    q, k, v, eta, W = _layer_inputs(36, 16, 16, 6, 6, eta_scale=5.0)
    beta = np.full(16, 0.9)
    _, Wa, _ = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=0, use_muon=True, beta=beta)
    _, Wb, _ = O.lact_forward_instance(q, k, v, 3.0 * eta, *W, chunk=C, order=0, use_muon=True, beta=beta)
    for a, b in zip(Wa, Wb):
        np.testing.assert_allclose(a, b, rtol=1e-3, atol=1e-4)
    e2 = eta.copy(); e2[C:] *= 3.0
    _, Wc, _ = O.lact_forward_instance(q, k, v, e2, *W, chunk=C, order=0, use_muon=True, beta=beta)
    assert max(np.max(np.abs(a - c)) for a, c in zip(Wa, Wc)) > 1e-3


# ----------------------------------------------------------------------------- per-matrix rates
# Alg. 1 (update): lr [b, l, 3] = (lr1, lr2, lr3) weights the W1, W2, W3 gradients.


def _lr3(seed, n, scale=0.3):
    return scale * np.log1p(np.exp(_rng(seed).standard_normal((n, 3))))


def test_per_matrix_rates_with_equal_columns_are_the_single_rate():
    q, k, v, eta, W = _layer_inputs(40, 20, 20, 5, 7, eta_scale=0.3)
    g = O.chunk_gradient(*W, k, v, eta)
    g3 = O.chunk_gradient(*W, k, v, np.stack([eta] * 3, axis=1))
    for a, b in zip(g, g3):
        np.testing.assert_array_equal(a, b)


def test_per_matrix_rates_match_three_autograd_losses():
    """g_j is the gradient w.r.t. W_j of the loss weighted by column j alone."""
    rng = _rng(41)
    d, h, n = 5, 7, 13
    W = _weights(rng, h, d)
    k, v = _tokens(rng, n, d), _tokens(rng, n, d)
    lr = _lr3(42, n)
    got = O.chunk_gradient(*W, k, v, lr)
    for j in range(3):
        Wt = [torch.as_tensor(w.copy()).requires_grad_(True) for w in W]
        _torch_loss(*Wt, torch.as_tensor(k), torch.as_tensor(v), torch.as_tensor(lr[:, j])).backward()
        np.testing.assert_allclose(got[j], Wt[j].grad.numpy(), rtol=1e-12, atol=1e-14)


def test_zero_rate_column_leaves_that_matrix():
    q, k, v, eta, W = _layer_inputs(43, 16, 16, 5, 7)
    lr = _lr3(44, 16)
    lr[:, 1] = 0.0
    _, Wf = O.lact_forward_instance(q, k, v, lr, *W, chunk=8, order=0)
    np.testing.assert_array_equal(Wf[1], W[1])
    assert np.max(np.abs(Wf[0] - W[0])) > 1e-6 and np.max(np.abs(Wf[2] - W[2])) > 1e-6


# ----------------------------------------------------------------------------- schedule
# The ttt_config loop of Alg. 1: (mode, begin, end) segments in list order.


@pytest.mark.parametrize("order", [0, 1])
@pytest.mark.parametrize("muon", [0, 1])
def test_uniform_schedule_is_the_chunk_loop(order, muon):
    q, k, v, eta, W = _layer_inputs(45, 29, 22, 5, 6, eta_scale=0.3)
    C = 8
    sched = [(order, s, min(22, s + C)) for s in range(0, 22, C)] + [("apply_only", 22, 29)]
    a = O.lact_forward_instance(q, k, v, eta, *W, chunk=C, order=order, use_muon=bool(muon))
    b = O.lact_forward_schedule_instance(q, k, v, eta, *W, sched, use_muon=bool(muon))
    np.testing.assert_array_equal(a[0], b[0])
    for x, y in zip(a[1], b[1]):
        np.testing.assert_array_equal(x, y)


def test_split_modes_compose_into_the_fused_modes():
    q, k, v, eta, W = _layer_inputs(46, 24, 24, 5, 6, eta_scale=0.3)
    pairs = [([("update_only", 3, 17), ("apply_only", 3, 17)], [("update_then_apply", 3, 17)]),
             ([("apply_only", 3, 17), ("update_only", 3, 17)], [("apply_then_update", 3, 17)])]
    for split, fused in pairs:
        a = O.lact_forward_schedule_instance(q, k, v, eta, *W, split)
        b = O.lact_forward_schedule_instance(q, k, v, eta, *W, fused)
        np.testing.assert_array_equal(a[0], b[0])
        for x, y in zip(a[1], b[1]):
            np.testing.assert_array_equal(x, y)


def test_uncovered_rows_are_zero_and_later_applies_win():
    q, k, v, eta, W = _layer_inputs(47, 30, 20, 5, 6, eta_scale=0.3)
    o, _ = O.lact_forward_schedule_instance(q, k, v, eta, *W, [("update_only", 0, 20)])
    assert not o.any()
    sched = [("apply_only", 0, 30), ("update_only", 0, 12), ("apply_only", 5, 18)]
    o, Wf = O.lact_forward_schedule_instance(q, k, v, eta, *W, sched)
    W1 = O.update(tuple(np.asarray(w) for w in W), k[:12], v[:12], eta[:12])
    np.testing.assert_allclose(o[5:18], _torch_swiglu(*W1, q[5:18]).numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(np.concatenate([o[:5], o[18:]]),
                               _torch_swiglu(*W, np.concatenate([q[:5], q[18:]])).numpy(), rtol=1e-12, atol=1e-14)


def _video_schedule(C, n_clean):
    """Teacher forcing of §4.3: [X1_noise, X1, X2_noise, X2, ..., XN_noise];
    noisy chunks are applied only, clean chunks update then apply."""
    sched, t = [], 0
    for i in range(n_clean + 1):
        sched.append(("apply_only", t, t + C))
        t += C
        if i < n_clean:
            sched.append(("update_then_apply", t, t + C))
            t += C
    return sched, t


def test_video_strided_mask_updates_on_clean_chunks_only():
    C, N = 6, 3
    sched, n = _video_schedule(C, N)
    q, k, v, eta, W = _layer_inputs(48, n, n, 5, 6, eta_scale=0.4)
    o, Wf = O.lact_forward_schedule_instance(q, k, v, eta, *W, sched)
    noisy = np.concatenate([np.arange(s, e) for m, s, e in sched if m == "apply_only"])
    clean = np.concatenate([np.arange(s, e) for m, s, e in sched if m != "apply_only"])
    # noisy keys, values and rates never reach the fast weights
    k2, v2, e2 = k.copy(), v.copy(), eta.copy()
    k2[noisy] = _tokens(_rng(49), len(noisy), 5)
    v2[noisy] *= -1.0
    e2[noisy] *= 7.0
    o2, W2 = O.lact_forward_schedule_instance(q, k2, v2, e2, *W, sched)
    np.testing.assert_array_equal(o2, o)
    for a, b in zip(W2, Wf):
        np.testing.assert_array_equal(a, b)
    # the clean chunks alone run an ordinary update-then-apply chunk loop, and
    # each noisy chunk sees the weights after the clean chunks before it
    oc, Wc = O.lact_forward_instance(q[clean], k[clean], v[clean], eta[clean], *W, chunk=C, order=1)
    np.testing.assert_array_equal(o[clean], oc)
    for a, b in zip(Wc, Wf):
        np.testing.assert_array_equal(a, b)
    Wi = tuple(np.asarray(w, dtype=np.float64) for w in W)
    for i, (m, s, e) in enumerate(x for x in sched if x[0] == "apply_only"):
        np.testing.assert_allclose(o[s:e], _torch_swiglu(*Wi, q[s:e]).numpy(), rtol=1e-12, atol=1e-14)
        if i < N:
            cs = s + C
            Wi = O.update(Wi, k[cs:cs + C], v[cs:cs + C], eta[cs:cs + C])


def test_schedule_with_momentum_and_per_matrix_rates():
    q, k, v, _, W = _layer_inputs(50, 24, 24, 5, 6)
    lr = _lr3(51, 24)
    beta = _beta(52, 24)
    sched = [("update_only", 0, 8), ("apply_then_update", 8, 16), ("update_then_apply", 16, 24)]
    o, Wf, M = O.lact_forward_schedule_instance(q, k, v, lr, *W, sched, beta=beta)
    Wr, Mr = tuple(np.asarray(w, dtype=np.float64) for w in W), tuple(np.zeros_like(w) for w in W)
    for s in (0, 8, 16):
        Wr, Mr = O.momentum_update(Wr, Mr, k[s:s + 8], v[s:s + 8], lr[s:s + 8], beta[s:s + 8])
    for a, b in zip(Wf + M, Wr + Mr):
        np.testing.assert_array_equal(a, b)
    assert not o[:8].any()


# ----------------------------------------------------------------------------- prologue / output norm
# The steps around the path in Alg. 1 (layer): silu(qkv), q/||q||, k/||k||,
# softplus(lr + bias), per-head RMSNorm of o.


def _raw(seed, B, L, H, hd, R):
    rng = _rng(seed)
    return (rng.standard_normal((B, L, 3, H, hd)), rng.standard_normal((B, L, H, R)),
            rng.standard_normal((B, L, H)))


@pytest.mark.parametrize("R", [1, 3])
def test_prologue_matches_library_ops(R):
    from einops import rearrange
    B, L, H, hd = 2, 7, 3, 10
    qkv, lr, br = _raw(60, B, L, H, hd, R)
    q, k, v, eta, beta = O.qkv_prologue(qkv, lr, -1.5, br)
    t = torch.as_tensor(qkv)
    act = F.silu(t)
    for j, (got, unit) in enumerate(((q, True), (k, True), (v, False))):
        ref = rearrange(act[:, :, j], "b l h d -> (b h) l d")
        if unit:
            ref = F.normalize(ref, dim=-1, eps=0.0)
        np.testing.assert_allclose(got, ref.numpy(), rtol=1e-13, atol=1e-15)
    ref_eta = rearrange(F.softplus(torch.as_tensor(lr) - 1.5), "b l h r -> (b h) l r")
    np.testing.assert_allclose(eta, ref_eta.numpy()[..., 0] if R == 1 else ref_eta.numpy(), rtol=1e-13)
    np.testing.assert_allclose(beta, rearrange(torch.sigmoid(torch.as_tensor(br)), "b l h -> (b h) l").numpy(),
                               rtol=1e-13)
    np.testing.assert_allclose(np.linalg.norm(q, axis=-1), 1.0, rtol=1e-13)


def test_prologue_zero_vector_and_softplus_range():
    qkv, lr, _ = _raw(61, 1, 3, 1, 4, 1)
    qkv[0, 1, 0] = 0.0                                   # q of token 1 is zero after SiLU
    q, *_ = O.qkv_prologue(qkv, lr, 0.0)
    assert not q[0, 1].any() and np.all(np.isfinite(q))
    x = np.array([-800.0, -30.0, 0.0, 30.0, 800.0])
    sp = O.softplus(x)
    np.testing.assert_allclose(sp, F.softplus(torch.as_tensor(x)).numpy(), rtol=1e-14)
    assert sp[-1] == 800.0 and sp[0] >= 0.0


def test_output_rmsnorm_matches_library():
    from einops import rearrange
    B, H, L, hd = 2, 3, 5, 8
    o = _rng(62).standard_normal((B * H, L, hd))
    w = _rng(63).standard_normal((H, hd))
    y = O.rmsnorm_out(o, B, H, w, eps=1e-5)
    t = rearrange(torch.as_tensor(o), "(b h) l d -> b l h d", b=B)
    ref = F.rms_norm(t, (hd,), eps=1e-5) * torch.as_tensor(w)
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-13, atol=1e-15)
    y0 = O.rmsnorm_out(o, B, H, None, eps=1e-5)
    np.testing.assert_allclose(np.sqrt(np.mean(y0 ** 2, axis=-1)),
                               np.sqrt(np.mean(o ** 2, -1) / (np.mean(o ** 2, -1) + 1e-5)).reshape(B, H, L)
                               .transpose(0, 2, 1), rtol=1e-12)


# ----------------------------------------------------------------------------- linear fast weight
# §5.4: f_W(x) = W x with the same dot-product loss and update rules.


def test_linear_gradient_matches_autograd():
    rng = _rng(90)
    d, n = 6, 11
    W = rng.standard_normal((d, d))
    k, v = _tokens(rng, n, d), _tokens(rng, n, d)
    eta = 0.3 * np.log1p(np.exp(rng.standard_normal(n)))
    Wt = torch.as_tensor(W.copy()).requires_grad_(True)
    loss = -(torch.as_tensor(eta) * (F.linear(torch.as_tensor(k), Wt) * torch.as_tensor(v)).sum(-1)).sum()
    loss.backward()
    np.testing.assert_allclose(O.linear_gradient(W, k, v, eta), Wt.grad.numpy(), rtol=1e-13, atol=1e-15)


def test_linear_one_token_chunk_is_a_rank_one_step():
    """A one-token chunk moves W by eta v k^T before the row rescaling."""
    rng = _rng(91)
    d = 5
    W = _weights(rng, d, d, unit=True)[0]
    q, k, v = _tokens(rng, 1, d), _tokens(rng, 1, d), _tokens(rng, 1, d)
    eta = np.array([0.2])
    o, Wf = O.lact_forward_linear_instance(q, k, v, eta, W, chunk=1, order=1)
    U = W + 0.2 * np.outer(v[0], k[0])
    ref = U * (np.linalg.norm(W, axis=1) / np.linalg.norm(U, axis=1))[:, None]
    np.testing.assert_allclose(Wf, ref, rtol=1e-14)
    np.testing.assert_allclose(o[0], ref @ q[0], rtol=1e-14)


@pytest.mark.parametrize("muon", [0, 1])
def test_linear_layer_eta_zero_and_autograd_loop(muon):
    rng = _rng(92)
    d, n, C = 6, 20, 7
    W = _weights(rng, d, d, unit=True)[0]
    q, k, v = _tokens(rng, n, d), _tokens(rng, n, d), _tokens(rng, n, d)
    o0, W0 = O.lact_forward_linear_instance(q, k, v, np.zeros(n), W, chunk=C, order=0, use_muon=bool(muon))
    np.testing.assert_array_equal(W0, W)
    np.testing.assert_allclose(o0, q @ W.T, rtol=1e-14)
    eta = 0.5 * np.log1p(np.exp(rng.standard_normal(n)))
    o, Wf = O.lact_forward_linear_instance(q, k, v, eta, W, chunk=C, order=0, use_muon=bool(muon))
    Wt = torch.as_tensor(W.copy())
    outs = []
    for s in range(0, n, C):
        e = min(n, s + C)
        outs.append((torch.as_tensor(q[s:e]) @ Wt.T).numpy())
        Wg = Wt.clone().requires_grad_(True)
        loss = -(torch.as_tensor(eta[s:e]) * (F.linear(torch.as_tensor(k[s:e]), Wg) *
                                             torch.as_tensor(v[s:e])).sum(-1)).sum()
        loss.backward()
        g = _torch_ns(Wg.grad, 5) if muon else Wg.grad
        u = Wt - g
        Wt = u * (Wt.norm(dim=1, keepdim=True) / u.norm(dim=1, keepdim=True))
    np.testing.assert_allclose(o, np.concatenate(outs), rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(Wf, Wt.numpy(), rtol=1e-11, atol=1e-13)


def test_linear_flops():
    assert O.linear_flops(2, 8, 10, 12, 3) == 2 * 2 * 64 * 22
    assert O.linear_flops(1, 4, 4, 4, 2, True, 5) == 2 * 16 * 8 + 2 * 5 * 6 * 64


# ----------------------------------------------------------------------------- batched drivers


def test_batched_drivers_stack_their_instances():
    # every batched driver is its per-instance function over the selected
    # instances, stacked in the selection's order (instances are independent)
    rng = _rng(91)
    BH, d, h, n, C = 3, 8, 12, 40, 16
    q, k, v = (np.stack([_tokens(rng, n, d) for _ in range(BH)]) for _ in range(3))
    eta = 0.05 * rng.random((BH, n))
    beta = rng.random((BH, n))
    W = [np.stack(ws) for ws in zip(*[_weights(rng, h, d) for _ in range(BH)])]
    Wl = np.stack([rng.standard_normal((d, d)) for _ in range(BH)])
    pick = [2, 0]
    sched = [("apply_then_update", 0, 16), ("update_only", 16, 40), ("apply_only", 16, 40)]
    one = lambda i: O.lact_forward_instance(q[i], k[i], v[i], eta[i], W[0][i], W[1][i], W[2][i], C, 0, True, 3)
    got = O.lact_forward(q, k, v, eta, *W, chunk=C, order=0, use_muon=True, ns_steps=3, instances=pick)
    for s, i in enumerate(pick):
        o, Wi = one(i)
        assert np.array_equal(got[0][s], o) and all(np.array_equal(got[1 + j][s], Wi[j]) for j in range(3))
    got = O.lact_forward_momentum(q, k, v, eta, beta, *W, chunk=C, order=1, instances=pick)
    for s, i in enumerate(pick):
        o, Wi, Mi = O.lact_forward_instance(q[i], k[i], v[i], eta[i], W[0][i], W[1][i], W[2][i], C, 1,
                                            beta=beta[i])
        ref = (o, *Wi, *Mi)
        assert all(np.array_equal(got[j][s], ref[j]) for j in range(7))
    got = O.lact_forward_linear(q, k, v, eta, Wl, chunk=C, order=0, instances=pick)
    for s, i in enumerate(pick):
        o, Wi = O.lact_forward_linear_instance(q[i], k[i], v[i], eta[i], Wl[i], C, 0)
        assert np.array_equal(got[0][s], o) and np.array_equal(got[1][s], Wi)
    got = O.lact_forward_schedule(q, k, v, eta, *W, sched, instances=pick)
    for s, i in enumerate(pick):
        o, Wi = O.lact_forward_schedule_instance(q[i], k[i], v[i], eta[i], W[0][i], W[1][i], W[2][i], sched)
        assert np.array_equal(got[0][s], o) and all(np.array_equal(got[1 + j][s], Wi[j]) for j in range(3))


# ----------------------------------------------------------------------------- backward (linear fast weight)


def _torch_linear_layer(q, k, v, eta, W, chunk, order):
    """The linear fast weight's chunk loop from library ops (torch autograd
    sees every step): o_t = W q_t, W <- rownorm-preserving (W - g) with
    g = -sum_t eta_t v_t k_t^T."""
    n_q, n_kv = q.shape[0], k.shape[0]
    outs = []
    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        if order == 0:
            outs.append(q[s:e] @ W.T)
        g = -(v[s:e] * eta[s:e, None]).T @ k[s:e]
        U = W - g
        W = U * (torch.linalg.vector_norm(W, dim=1, keepdim=True) / torch.linalg.vector_norm(U, dim=1, keepdim=True))
        if order == 1:
            outs.append(q[s:e] @ W.T)
    if n_q > n_kv:
        outs.append(q[n_kv:] @ W.T)
    return torch.cat(outs), W


def test_weight_update_vjp_matches_autograd():
    rng = _rng(101)
    W, step, dWn = (rng.standard_normal((6, 5)) for _ in range(3))
    t = lambda a: torch.tensor(a, requires_grad=True)
    Wt, St = t(W), t(step)
    U = Wt - St
    Wn = U * (torch.linalg.vector_norm(Wt, dim=1, keepdim=True) / torch.linalg.vector_norm(U, dim=1, keepdim=True))
    (Wn * torch.tensor(dWn)).sum().backward()
    dW, dstep = O.weight_update_vjp(W, step, dWn)
    assert np.allclose(dW, Wt.grad.numpy(), rtol=1e-11, atol=1e-12)
    assert np.allclose(dstep, St.grad.numpy(), rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("order,final", [(0, False), (1, False), (0, True), (1, True)])
def test_linear_backward_matches_autograd(order, final):
    # several chunks, the last one ragged, and an apply-only tail
    rng = _rng(102 + order + 2 * final)
    d, n_kv, n_q, C = 6, 23, 29, 7
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.05 + 0.2 * rng.random(n_kv)
    W0 = rng.standard_normal((d, d))
    do = rng.standard_normal((n_q, d))
    dWf = rng.standard_normal((d, d)) if final else None
    t = lambda a: torch.tensor(a, requires_grad=True)
    qt, kt, vt, et, Wt = t(q), t(k), t(v), t(eta), t(W0)
    o, Wfin = _torch_linear_layer(qt, kt, vt, et, Wt, C, order)
    loss = (o * torch.tensor(do)).sum() + ((Wfin * torch.tensor(dWf)).sum() if final else 0.0)
    loss.backward()
    got = O.lact_backward_linear_instance(q, k, v, eta, W0, do, C, order, dWf)
    for name, g, ref in zip(("dq", "dk", "dv", "deta", "dW0"), got, (qt, kt, vt, et, Wt)):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-9, atol=1e-11), name
    # the forward the backward replays is the oracle's own forward
    o_ref, W_ref = O.lact_forward_linear_instance(q, k, v, eta, W0, C, order)
    assert np.allclose(o.detach().numpy(), o_ref, rtol=1e-12, atol=1e-13)
    assert np.allclose(Wfin.detach().numpy(), W_ref, rtol=1e-12, atol=1e-13)


def test_linear_backward_finite_differences():
    # central differences of the NumPy forward oracle on a scalar read-out
    rng = _rng(107)
    d, n_kv, n_q, C = 4, 9, 11, 4
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.3 * rng.random(n_kv)
    W0 = rng.standard_normal((d, d))
    do, dWf = rng.standard_normal((n_q, d)), rng.standard_normal((d, d))
    for order in (0, 1):
        def readout(q_, k_, v_, eta_, W_):
            o, W = O.lact_forward_linear_instance(q_, k_, v_, eta_, W_, C, order)
            return float(np.sum(o * do) + np.sum(W * dWf))
        grads = O.lact_backward_linear_instance(q, k, v, eta, W0, do, C, order, dWf)
        args = [q, k, v, eta, W0]
        for which, idx in ((0, (3, 1)), (0, (10, 2)), (1, (2, 0)), (1, (8, 3)), (2, (5, 1)), (3, (6,)), (4, (1, 2))):
            h = 1e-6
            plus = [a.copy() for a in args]
            minus = [a.copy() for a in args]
            plus[which][idx] += h
            minus[which][idx] -= h
            fd = (readout(*plus) - readout(*minus)) / (2 * h)
            assert abs(fd - grads[which][idx]) <= 1e-6 * max(1.0, abs(fd)), (order, which, idx, fd, grads[which][idx])


# ----------------------------------------------------------------------------- SwiGLU backward


def _torch_swiglu_t(W1, W2, W3, X):
    """Library SwiGLU MLP on tensors (autograd sees it): F.linear + F.silu."""
    return F.linear(F.silu(F.linear(X, W1)) * F.linear(X, W3), W2)


def test_silu_second_derivative_matches_autograd():
    z = torch.linspace(-30.0, 30.0, 241, requires_grad=True)
    (g,) = torch.autograd.grad(F.silu(z).sum(), z, create_graph=True)
    (gg,) = torch.autograd.grad(g.sum(), z)
    assert np.allclose(O.silu_second_derivative(z.detach().numpy()), gg.numpy(), rtol=1e-12, atol=1e-14)


def test_swiglu_apply_vjp_matches_autograd():
    rng = _rng(111)
    h, d, n = 7, 5, 9
    W1, W2, W3 = _weights(rng, h, d)
    X, dO = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    t = lambda a: torch.tensor(a, requires_grad=True)
    W1t, W2t, W3t, Xt = t(W1), t(W2), t(W3), t(X)
    (_torch_swiglu_t(W1t, W2t, W3t, Xt) * torch.tensor(dO)).sum().backward()
    got = O.swiglu_apply_vjp(W1, W2, W3, X, dO)
    for g, ref in zip(got, (Xt, W1t, W2t, W3t)):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-11, atol=1e-12)


def _torch_chunk_gradient(W1, W2, W3, K, V, eta):
    """The chunk gradient by torch autograd of the chunk loss, kept in the
    graph (create_graph) so that it can be differentiated again. With
    per-matrix rates (eta [n, 3]) the gradient of W_j is that of the loss
    weighted by column j."""
    f = _torch_swiglu_t(W1, W2, W3, K)
    if eta.dim() == 2:
        return tuple(torch.autograd.grad(-(eta[:, j:j + 1] * f * V).sum(), W, create_graph=True)[0]
                     for j, W in enumerate((W1, W2, W3)))
    loss = -(eta[:, None] * f * V).sum()
    return torch.autograd.grad(loss, (W1, W2, W3), create_graph=True)


def test_chunk_gradient_vjp_matches_double_backward():
    rng = _rng(112)
    h, d, n = 6, 4, 11
    W1, W2, W3 = _weights(rng, h, d)
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    eta = 0.1 + rng.random(n)
    G = (rng.standard_normal((h, d)), rng.standard_normal((d, h)), rng.standard_normal((h, d)))
    t = lambda a: torch.tensor(a, requires_grad=True)
    ins = [t(a) for a in (W1, W2, W3, K, V, eta)]
    g = _torch_chunk_gradient(*ins)
    # the oracle's forward closed form is the autograd gradient
    for a, b in zip(g, O.chunk_gradient(W1, W2, W3, K, V, eta)):
        assert np.allclose(a.detach().numpy(), b, rtol=1e-11, atol=1e-12)
    sum(((gj * torch.tensor(Gj)).sum() for gj, Gj in zip(g, G))).backward()
    got = O.chunk_gradient_vjp(W1, W2, W3, K, V, eta, *G)
    for name, a, ref in zip(("dW1", "dW2", "dW3", "dK", "dV", "deta"), got, ins):
        assert np.allclose(a, ref.grad.numpy(), rtol=1e-10, atol=1e-12), name


def _torch_swiglu_layer(q, k, v, eta, W, chunk, order):
    """The SwiGLU fast weight's chunk loop in torch: the chunk gradient by
    autograd (create_graph), the row-norm-preserving update, both orders and
    an apply-only tail; autograd sees every step."""
    n_q, n_kv = q.shape[0], k.shape[0]
    outs = []
    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        if order == 0:
            outs.append(_torch_swiglu_t(*W, q[s:e]))
        g = _torch_chunk_gradient(*W, k[s:e], v[s:e], eta[s:e])
        new = []
        for w, gj in zip(W, g):
            U = w - gj
            new.append(U * (torch.linalg.vector_norm(w, dim=1, keepdim=True)
                            / torch.linalg.vector_norm(U, dim=1, keepdim=True)))
        W = tuple(new)
        if order == 1:
            outs.append(_torch_swiglu_t(*W, q[s:e]))
    if n_q > n_kv:
        outs.append(_torch_swiglu_t(*W, q[n_kv:]))
    return torch.cat(outs), W


@pytest.mark.parametrize("order,final", [(0, False), (1, False), (0, True), (1, True)])
def test_swiglu_backward_matches_autograd(order, final):
    # several chunks, the last one ragged, an apply-only tail, non-square h x d
    rng = _rng(113 + order + 2 * final)
    d, h, n_kv, n_q, C = 5, 7, 17, 21, 6
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random(n_kv)
    W0 = _weights(rng, h, d, unit=True)
    do = rng.standard_normal((n_q, d))
    dWf = tuple(rng.standard_normal(w.shape) for w in W0) if final else None
    t = lambda a: torch.tensor(a, requires_grad=True)
    qt, kt, vt, et = t(q), t(k), t(v), t(eta)
    Wt = tuple(t(w) for w in W0)
    o, Wfin = _torch_swiglu_layer(qt, kt, vt, et, Wt, C, order)
    loss = (o * torch.tensor(do)).sum()
    if final:
        loss = loss + sum((w * torch.tensor(x)).sum() for w, x in zip(Wfin, dWf))
    loss.backward()
    dq, dk, dv, deta, dW = O.lact_backward_instance(q, k, v, eta, *W0, do, C, order, dWf)
    for name, g, ref in zip(("dq", "dk", "dv", "deta", "dW1", "dW2", "dW3"), (dq, dk, dv, deta, *dW),
                            (qt, kt, vt, et, *Wt)):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-9, atol=1e-11), name
    # the forward the backward replays is the oracle's own forward
    o_ref, W_ref = O.lact_forward_instance(q, k, v, eta, *W0, C, order)
    assert np.allclose(o.detach().numpy(), o_ref, rtol=1e-12, atol=1e-13)
    for a, b in zip(Wfin, W_ref):
        assert np.allclose(a.detach().numpy(), b, rtol=1e-12, atol=1e-13)


def test_swiglu_backward_finite_differences():
    # central differences of the NumPy forward oracle on a scalar read-out
    rng = _rng(118)
    d, h, n_kv, n_q, C = 4, 6, 9, 11, 4
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.3 * rng.random(n_kv)
    W0 = _weights(rng, h, d, unit=True)
    do = rng.standard_normal((n_q, d))
    dWf = tuple(rng.standard_normal(w.shape) for w in W0)
    for order in (0, 1):
        def readout(q_, k_, v_, eta_, W1_, W2_, W3_):
            o, W = O.lact_forward_instance(q_, k_, v_, eta_, W1_, W2_, W3_, C, order)
            return float(np.sum(o * do) + sum(np.sum(a * b) for a, b in zip(W, dWf)))
        dq, dk, dv, deta, dW = O.lact_backward_instance(q, k, v, eta, *W0, do, C, order, dWf)
        grads = (dq, dk, dv, deta, *dW)
        args = [q, k, v, eta, *W0]
        for which, idx in ((0, (3, 1)), (0, (10, 2)), (1, (2, 0)), (1, (8, 3)), (2, (5, 1)), (3, (6,)),
                           (4, (1, 2)), (5, (3, 4)), (6, (5, 0))):
            eps = 1e-6
            plus = [a.copy() for a in args]
            minus = [a.copy() for a in args]
            plus[which][idx] += eps
            minus[which][idx] -= eps
            fd = (readout(*plus) - readout(*minus)) / (2 * eps)
            assert abs(fd - grads[which][idx]) <= 2e-6 * max(1.0, abs(fd)), (order, which, idx, fd, grads[which][idx])


def test_swiglu_backward_at_eta_zero_is_the_apply_chain():
    # eta = 0: the gradient is zero for every W, so each update is the
    # identity map and passes the weights' cotangent through unchanged; k and
    # v get none, and dW0 is the apply's reverse over all tokens at once
    rng = _rng(119)
    d, h, n, C = 4, 6, 10, 4
    q, k, v = _tokens(rng, n, d), _tokens(rng, n, d), _tokens(rng, n, d)
    W0 = _weights(rng, h, d, unit=True)
    do = rng.standard_normal((n, d))
    for order in (0, 1):
        dq, dk, dv, deta, dW = O.lact_backward_instance(q, k, v, np.zeros(n), *W0, do, C, order)
        dx, a1, a2, a3 = O.swiglu_apply_vjp(*W0, q, do)
        assert np.allclose(dq, dx, rtol=1e-12, atol=1e-13)
        assert np.array_equal(dk, np.zeros_like(dk)) and np.array_equal(dv, np.zeros_like(dv))
        for g, a in zip(dW, (a1, a2, a3)):
            assert np.allclose(g, a, rtol=1e-11, atol=1e-12)


def test_swiglu_backward_batched_driver_stacks_instances():
    rng = _rng(120)
    BH, d, h, n, C = 3, 4, 6, 9, 4
    q, k, v = (np.stack([_tokens(rng, n, d) for _ in range(BH)]) for _ in range(3))
    eta = 0.1 + 0.3 * rng.random((BH, n))
    Ws = [_weights(rng, h, d, unit=True) for _ in range(BH)]
    W1, W2, W3 = (np.stack([w[j] for w in Ws]) for j in range(3))
    do = rng.standard_normal((BH, n, d))
    got = O.lact_backward(q, k, v, eta, W1, W2, W3, do, C, 1, instances=[2, 0])
    for pos, i in enumerate((2, 0)):
        dq, dk, dv, deta, dW = O.lact_backward_instance(q[i], k[i], v[i], eta[i], W1[i], W2[i], W3[i], do[i], C, 1)
        for a, b in zip(got, (dq, dk, dv, deta, *dW)):
            assert np.array_equal(a[pos], b)


# ----------------------------------------------------------------------------- Muon backward


def _torch_newton_schulz(G, steps=5):
    """Muon's quintic iteration in torch (wide orientation, G / (||G|| + 1e-7))."""
    a, b, c = 3.4445, -4.7750, 2.0315
    tall = G.shape[0] > G.shape[1]
    X = G.T if tall else G
    X = X / (torch.linalg.matrix_norm(X) + 1e-7)
    for _ in range(steps):
        A = X @ X.T
        X = a * X + (b * A + c * A @ A) @ X
    return X.T if tall else X


@pytest.mark.parametrize("shape", [(6, 9), (9, 6), (7, 7)])
def test_newton_schulz_vjp_matches_autograd(shape):
    rng = _rng(121 + shape[0])
    G, dX = rng.standard_normal(shape), rng.standard_normal(shape)
    Gt = torch.tensor(G, requires_grad=True)
    (_torch_newton_schulz(Gt) * torch.tensor(dX)).sum().backward()
    assert np.allclose(O.newton_schulz(G), _torch_newton_schulz(torch.tensor(G)).numpy(), rtol=1e-12, atol=1e-13)
    assert np.allclose(O.newton_schulz_vjp(G, dX), Gt.grad.numpy(), rtol=1e-9, atol=1e-11)


def test_newton_schulz_vjp_finite_differences():
    rng = _rng(124)
    G, dX = rng.standard_normal((5, 8)), rng.standard_normal((5, 8))
    got = O.newton_schulz_vjp(G, dX)
    for idx in ((0, 0), (2, 5), (4, 7), (3, 1)):
        eps = 1e-6
        P, M = G.copy(), G.copy()
        P[idx] += eps
        M[idx] -= eps
        fd = (np.sum(O.newton_schulz(P) * dX) - np.sum(O.newton_schulz(M) * dX)) / (2 * eps)
        assert abs(fd - got[idx]) <= 1e-6 * max(1.0, abs(fd))


def _torch_swiglu_layer_muon(q, k, v, eta, W, chunk, order):
    n_q, n_kv = q.shape[0], k.shape[0]
    outs = []
    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        if order == 0:
            outs.append(_torch_swiglu_t(*W, q[s:e]))
        g = _torch_chunk_gradient(*W, k[s:e], v[s:e], eta[s:e])
        new = []
        for w, gj in zip(W, g):
            U = w - _torch_newton_schulz(gj)
            new.append(U * (torch.linalg.vector_norm(w, dim=1, keepdim=True)
                            / torch.linalg.vector_norm(U, dim=1, keepdim=True)))
        W = tuple(new)
        if order == 1:
            outs.append(_torch_swiglu_t(*W, q[s:e]))
    if n_q > n_kv:
        outs.append(_torch_swiglu_t(*W, q[n_kv:]))
    return torch.cat(outs), W


@pytest.mark.parametrize("order", [0, 1])
def test_swiglu_muon_backward_matches_autograd(order):
    # three chunks (the last ragged), a tail, h != d (W1, W3 tall, W2 wide)
    rng = _rng(125 + order)
    d, h, n_kv, n_q, C = 5, 7, 15, 19, 6
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random(n_kv)
    W0 = _weights(rng, h, d, unit=True)
    do = rng.standard_normal((n_q, d))
    dWf = tuple(rng.standard_normal(w.shape) for w in W0)
    t = lambda a: torch.tensor(a, requires_grad=True)
    qt, kt, vt, et = t(q), t(k), t(v), t(eta)
    Wt = tuple(t(w) for w in W0)
    o, Wfin = _torch_swiglu_layer_muon(qt, kt, vt, et, Wt, C, order)
    loss = (o * torch.tensor(do)).sum() + sum((w * torch.tensor(x)).sum() for w, x in zip(Wfin, dWf))
    loss.backward()
    dq, dk, dv, deta, dW = O.lact_backward_instance(q, k, v, eta, *W0, do, C, order, dWf, use_muon=True)
    for name, g, ref in zip(("dq", "dk", "dv", "deta", "dW1", "dW2", "dW3"), (dq, dk, dv, deta, *dW),
                            (qt, kt, vt, et, *Wt)):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-8, atol=1e-10), name
    o_ref, W_ref = O.lact_forward_instance(q, k, v, eta, *W0, C, order, use_muon=True)
    assert np.allclose(o.detach().numpy(), o_ref, rtol=1e-11, atol=1e-12)


def test_linear_muon_backward_matches_autograd():
    rng = _rng(127)
    d, n_kv, n_q, C = 6, 17, 20, 6
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random(n_kv)
    W0 = rng.standard_normal((d, d))
    do, dWf = rng.standard_normal((n_q, d)), rng.standard_normal((d, d))
    for order in (0, 1):
        t = lambda a: torch.tensor(a, requires_grad=True)
        qt, kt, vt, et, Wt = t(q), t(k), t(v), t(eta), t(W0)
        W = Wt
        outs = []
        for s in range(0, n_kv, C):
            e = min(n_kv, s + C)
            if order == 0:
                outs.append(qt[s:e] @ W.T)
            g = -(vt[s:e] * et[s:e, None]).T @ kt[s:e]
            U = W - _torch_newton_schulz(g)
            W = U * (torch.linalg.vector_norm(W, dim=1, keepdim=True) / torch.linalg.vector_norm(U, dim=1, keepdim=True))
            if order == 1:
                outs.append(qt[s:e] @ W.T)
        outs.append(qt[n_kv:] @ W.T)
        loss = (torch.cat(outs) * torch.tensor(do)).sum() + (W * torch.tensor(dWf)).sum()
        loss.backward()
        got = O.lact_backward_linear_instance(q, k, v, eta, W0, do, C, order, dWf, use_muon=True)
        for name, g, ref in zip(("dq", "dk", "dv", "deta", "dW0"), got, (qt, kt, vt, et, Wt)):
            assert np.allclose(g, ref.grad.numpy(), rtol=1e-8, atol=1e-10), (order, name)


def test_newton_schulz_vjp_amplifies_the_null_space_by_a_per_step():
    # G = s u w^T (rank one): a cotangent y z^T with y orthogonal to u and z
    # orthogonal to w leaves A = X X^T unchanged and is annihilated by B, so
    # each step multiplies it by a; through five steps and the scaling the
    # reverse returns a^5 y z^T / (s + eps) (the amplification that makes the
    # reverse ill-conditioned when a chunk gradient is rank-deficient)
    rng = _rng(128)
    m, n, s = 4, 6, 0.37
    u = rng.standard_normal(m); u /= np.linalg.norm(u)
    w = rng.standard_normal(n); w /= np.linalg.norm(w)
    y = rng.standard_normal(m); y -= (y @ u) * u
    z = rng.standard_normal(n); z -= (z @ w) * w
    G, dX = s * np.outer(u, w), np.outer(y, z)
    a = O.NS_COEFFS[0]
    assert np.allclose(O.newton_schulz_vjp(G, dX, 5), a ** 5 * dX / (s + O.NS_EPS), rtol=1e-10, atol=1e-12)
    assert np.allclose(O.newton_schulz_vjp(G, dX, 2), a ** 2 * dX / (s + O.NS_EPS), rtol=1e-10, atol=1e-12)


# ----------------------------------------------------------------------------- momentum backward


def _torch_momentum_layer(q, k, v, eta, beta, W, M, chunk, order, muon, linear):
    """The chunk loop with the momentum optimizer in torch (chunk gradient by
    autograd, bbar the chunk's mean of beta), SwiGLU or linear."""
    n_q, n_kv = q.shape[0], k.shape[0]
    f = (lambda W_, X: X @ W_[0].T) if linear else (lambda W_, X: _torch_swiglu_t(*W_, X))
    outs = []
    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        if order == 0:
            outs.append(f(W, q[s:e]))
        if linear:
            g = (-(v[s:e] * eta[s:e, None]).T @ k[s:e],)
        else:
            g = _torch_chunk_gradient(*W, k[s:e], v[s:e], eta[s:e])
        bbar = beta[s:e].mean()
        M = tuple(bbar * m + gj for m, gj in zip(M, g))
        new = []
        for w, m in zip(W, M):
            U = w - (_torch_newton_schulz(m) if muon else m)
            new.append(U * (torch.linalg.vector_norm(w, dim=1, keepdim=True)
                            / torch.linalg.vector_norm(U, dim=1, keepdim=True)))
        W = tuple(new)
        if order == 1:
            outs.append(f(W, q[s:e]))
    if n_q > n_kv:
        outs.append(f(W, q[n_kv:]))
    return torch.cat(outs), W, M


@pytest.mark.parametrize("linear,muon,order", [(False, False, 0), (False, True, 1), (True, False, 1), (True, True, 0)])
def test_momentum_backward_matches_autograd(linear, muon, order):
    rng = _rng(131 + 2 * linear + muon)
    d, h, n_kv, n_q, C = 5, (5 if linear else 7), 15, 19, 6
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random(n_kv)
    beta = rng.random(n_kv)
    if linear:
        W0 = (rng.standard_normal((d, d)),)
        M0 = (0.1 * rng.standard_normal((d, d)),)
    else:
        W0 = _weights(rng, h, d, unit=True)
        M0 = tuple(0.1 * rng.standard_normal(w.shape) for w in W0)
    do = rng.standard_normal((n_q, d))
    dWf = tuple(rng.standard_normal(w.shape) for w in W0)
    dMf = tuple(rng.standard_normal(w.shape) for w in W0)
    t = lambda a: torch.tensor(a, requires_grad=True)
    qt, kt, vt, et, bt = t(q), t(k), t(v), t(eta), t(beta)
    Wt, Mt = tuple(t(w) for w in W0), tuple(t(m) for m in M0)
    o, Wfin, Mfin = _torch_momentum_layer(qt, kt, vt, et, bt, Wt, Mt, C, order, muon, linear)
    loss = (o * torch.tensor(do)).sum() + sum((w * torch.tensor(x)).sum() for w, x in zip(Wfin, dWf)) \
        + sum((m * torch.tensor(x)).sum() for m, x in zip(Mfin, dMf))
    loss.backward()
    one = (lambda a: a[0]) if linear else (lambda a: a)
    r = O.lact_backward_momentum_instance(q, k, v, eta, beta, one(W0), one(M0), do, C, order, one(dWf), one(dMf),
                                          use_muon=muon)
    for name, g, ref in zip(("dq", "dk", "dv", "deta", "dbeta"), r[:5], (qt, kt, vt, et, bt)):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-8, atol=1e-10), name
    dW, dM = ((r[5],), (r[6],)) if linear else (r[5], r[6])
    for a, ref in zip(dW, Wt):
        assert np.allclose(a, ref.grad.numpy(), rtol=1e-8, atol=1e-10)
    for a, ref in zip(dM, Mt):
        assert np.allclose(a, ref.grad.numpy(), rtol=1e-8, atol=1e-10)


def test_momentum_backward_at_beta_zero_is_the_plain_backward():
    # beta = 0 and M0 = 0: every chunk's state is its own gradient, so the
    # reverse is the plain one (dbeta is not zero: the factor still matters)
    rng = _rng(135)
    d, h, n, C = 4, 6, 13, 5
    q, k, v = _tokens(rng, n, d), _tokens(rng, n, d), _tokens(rng, n, d)
    eta = 0.1 + 0.3 * rng.random(n)
    W0 = _weights(rng, h, d, unit=True)
    M0 = tuple(np.zeros_like(w) for w in W0)
    do = rng.standard_normal((n, d))
    for muon in (False, True):
        r = O.lact_backward_momentum_instance(q, k, v, eta, np.zeros(n), W0, M0, do, C, 1, use_muon=muon)
        dq, dk, dv, deta, dW = O.lact_backward_instance(q, k, v, eta, *W0, do, C, 1, use_muon=muon)
        for a, b in zip(r[:4] + tuple(r[5]), (dq, dk, dv, deta) + tuple(dW)):
            assert np.allclose(a, b, rtol=1e-11, atol=1e-12)


def test_momentum_backward_batched_driver_stacks_instances():
    rng = _rng(136)
    BH, d, h, n, C = 3, 4, 6, 9, 4
    q, k, v = (np.stack([_tokens(rng, n, d) for _ in range(BH)]) for _ in range(3))
    eta, beta = 0.1 + 0.3 * rng.random((BH, n)), rng.random((BH, n))
    Ws = [_weights(rng, h, d, unit=True) for _ in range(BH)]
    W = tuple(np.stack([w[j] for w in Ws]) for j in range(3))
    M = tuple(0.1 * rng.standard_normal(w.shape) for w in W)
    do = rng.standard_normal((BH, n, d))
    got = O.lact_backward_momentum(q, k, v, eta, beta, W, M, do, C, 0, instances=[2, 0])
    for pos, i in enumerate((2, 0)):
        r = O.lact_backward_momentum_instance(q[i], k[i], v[i], eta[i], beta[i], tuple(w[i] for w in W),
                                              tuple(m[i] for m in M), do[i], C, 0)
        for a, b in zip(got[:5], r[:5]):
            assert np.array_equal(a[pos], b)
        for a, b in zip(got[5] + got[6], r[5] + r[6]):
            assert np.array_equal(a[pos], b)
    lin = O.lact_backward_momentum(q, k, v, eta, beta, W[0][:, :d, :], M[0][:, :d, :], do, C, 1, instances=[1])
    r = O.lact_backward_momentum_instance(q[1], k[1], v[1], eta[1], beta[1], W[0][1, :d, :], M[0][1, :d, :], do[1], C, 1)
    for a, b in zip(lin, r):
        assert np.array_equal(a[0], b)


def test_momentum_backward_dbeta_scale():
    # one chunk, no cotangent of o or of the final weights: dM' is the final
    # state's cotangent; with dM_final = M0 the inner product <dM', M0> meets
    # its Cauchy-Schwarz bound, so dbeta equals the scale ||M0||^2 / n
    rng = _rng(137)
    d, h, n = 4, 6, 7
    q, k, v = _tokens(rng, n, d), _tokens(rng, n, d), _tokens(rng, n, d)
    eta, beta = 0.1 + 0.3 * rng.random(n), rng.random(n)
    W0 = _weights(rng, h, d, unit=True)
    M0 = tuple(0.1 * rng.standard_normal(w.shape) for w in W0)
    r = O.lact_backward_momentum_instance(q, k, v, eta, beta, W0, M0, np.zeros((n, d)), n, 0, dM_final=M0,
                                          dbeta_scale=True)
    m2 = sum(float(np.sum(m * m)) for m in M0)
    assert np.allclose(r[4], m2 / n, rtol=1e-13)
    assert np.allclose(r[7], m2 / n, rtol=1e-13)
    # in general |dbeta| stays within the scale, over chunks, orders and Muon
    for order, muon in ((0, False), (1, True)):
        do = rng.standard_normal((n, d))
        dMf = tuple(rng.standard_normal(w.shape) for w in W0)
        r = O.lact_backward_momentum_instance(q, k, v, eta, beta, W0, M0, do, 3, order, dM_final=dMf, use_muon=muon,
                                              dbeta_scale=True)
        plain = O.lact_backward_momentum_instance(q, k, v, eta, beta, W0, M0, do, 3, order, dM_final=dMf,
                                                  use_muon=muon)
        assert len(r) == 8 and len(plain) == 7
        assert np.all(np.abs(r[4]) <= r[7] * (1 + 1e-12)) and np.all(r[7] > 0)
        for a, b in zip(r[:5], plain[:5]):
            assert np.array_equal(a, b)


# ----------------------------------------------------------------------------- per-matrix rates, backward


def test_chunk_gradient_vjp_per_matrix_rates_matches_double_backward():
    rng = _rng(140)
    h, d, n = 6, 4, 11
    W1, W2, W3 = _weights(rng, h, d)
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    eta = 0.1 + rng.random((n, 3))
    G = (rng.standard_normal((h, d)), rng.standard_normal((d, h)), rng.standard_normal((h, d)))
    t = lambda a: torch.tensor(a, requires_grad=True)
    ins = [t(a) for a in (W1, W2, W3, K, V, eta)]
    g = _torch_chunk_gradient(*ins)
    for a, b in zip(g, O.chunk_gradient(W1, W2, W3, K, V, eta)):
        assert np.allclose(a.detach().numpy(), b, rtol=1e-11, atol=1e-12)
    sum(((gj * torch.tensor(Gj)).sum() for gj, Gj in zip(g, G))).backward()
    got = O.chunk_gradient_vjp(W1, W2, W3, K, V, eta, *G)
    assert got[5].shape == (n, 3)
    for name, a, ref in zip(("dW1", "dW2", "dW3", "dK", "dV", "deta"), got, ins):
        assert np.allclose(a, ref.grad.numpy(), rtol=1e-10, atol=1e-12), name


def test_chunk_gradient_vjp_equal_rate_columns_reduce_to_one_rate():
    # three equal columns: every cotangent but deta is the one-rate result,
    # and deta's columns sum to the one-rate deta
    rng = _rng(141)
    h, d, n = 7, 5, 9
    W = _weights(rng, h, d)
    K, V = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    eta = 0.1 + rng.random(n)
    G = (rng.standard_normal((h, d)), rng.standard_normal((d, h)), rng.standard_normal((h, d)))
    one = O.chunk_gradient_vjp(*W, K, V, eta, *G)
    three = O.chunk_gradient_vjp(*W, K, V, np.repeat(eta[:, None], 3, axis=1), *G)
    for a, b in zip(one[:5], three[:5]):
        assert np.allclose(a, b, rtol=1e-13, atol=1e-15)
    assert np.allclose(three[5].sum(axis=1), one[5], rtol=1e-12, atol=1e-14)
    # a rate that is zero for one matrix: that matrix's gradient, and its
    # cotangents through it, vanish (W2: no dV through e2 A, no e2 column)
    eta3 = np.repeat(eta[:, None], 3, axis=1)
    eta3[:, 1] = 0.0
    G2only = (np.zeros((h, d)), G[1], np.zeros((h, d)))
    r = O.chunk_gradient_vjp(*W, K, V, eta3, *G2only)
    assert np.allclose(r[0], 0) and np.allclose(r[2], 0) and np.allclose(r[1], 0) and np.allclose(r[3], 0)
    assert np.allclose(r[5][:, 0], 0) and np.allclose(r[5][:, 2], 0)


@pytest.mark.parametrize("order", [0, 1])
def test_swiglu_backward_per_matrix_rates_matches_autograd(order):
    rng = _rng(142 + order)
    d, h, n_kv, n_q, C = 5, 7, 17, 21, 6
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random((n_kv, 3))
    W0 = _weights(rng, h, d, unit=True)
    do = rng.standard_normal((n_q, d))
    dWf = tuple(rng.standard_normal(w.shape) for w in W0)
    t = lambda a: torch.tensor(a, requires_grad=True)
    qt, kt, vt, et = t(q), t(k), t(v), t(eta)
    Wt = tuple(t(w) for w in W0)
    o, Wfin = _torch_swiglu_layer(qt, kt, vt, et, Wt, C, order)
    loss = (o * torch.tensor(do)).sum() + sum((w * torch.tensor(x)).sum() for w, x in zip(Wfin, dWf))
    loss.backward()
    dq, dk, dv, deta, dW = O.lact_backward_instance(q, k, v, eta, *W0, do, C, order, dWf)
    assert deta.shape == (n_kv, 3)
    for name, g, ref in zip(("dq", "dk", "dv", "deta", "dW1", "dW2", "dW3"), (dq, dk, dv, deta, *dW),
                            (qt, kt, vt, et, *Wt)):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-9, atol=1e-11), name
    # with Muon and with momentum too (the same per-matrix chunk gradient)
    beta = rng.random(n_kv)
    M0 = tuple(0.05 * rng.standard_normal(w.shape) for w in W0)
    bt, Mt = t(beta), tuple(t(m) for m in M0)
    qt, kt, vt, et = t(q), t(k), t(v), t(eta)
    Wt = tuple(t(w) for w in W0)
    o, Wfin, Mfin = _torch_momentum_layer(qt, kt, vt, et, bt, Wt, Mt, C, order, True, False)
    ((o * torch.tensor(do)).sum() + sum((w * torch.tensor(x)).sum() for w, x in zip(Wfin, dWf))).backward()
    r = O.lact_backward_momentum_instance(q, k, v, eta, beta, W0, M0, do, C, order, dWf, use_muon=True)
    for name, g, ref in zip(("dq", "dk", "dv", "deta", "dbeta"), r[:5], (qt, kt, vt, et, bt)):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-8, atol=1e-10), name
    for a, ref in zip(r[5] + r[6], Wt + Mt):
        assert np.allclose(a, ref.grad.numpy(), rtol=1e-8, atol=1e-10)


# ----------------------------------------------------------------------------- backward of a general schedule


def _torch_schedule_layer(q, k, v, eta, W, schedule, beta=None, M=None, muon=False):
    """The schedule's segments in torch (autograd sees every step): an apply
    overwrites its rows of o (rows applied twice keep the later value), an
    update takes the chunk gradient by autograd, the momentum recurrence with
    the segment's mean of beta, Muon, and the row-norm-preserving update."""
    o = torch.zeros(q.shape, dtype=q.dtype)
    parts = {"update_then_apply": ("update", "apply"), "apply_then_update": ("apply", "update"),
             "update_only": ("update",), "apply_only": ("apply",)}
    for mode, b, e in schedule:
        for kind in parts[mode]:
            if kind == "apply":
                rows = torch.zeros(q.shape[0], 1, dtype=q.dtype)
                rows[b:e] = 1.0
                full = torch.zeros(q.shape, dtype=q.dtype)
                full = torch.cat([full[:b], _torch_swiglu_t(*W, q[b:e]), full[e:]])
                o = o * (1 - rows) + full
                continue
            g = _torch_chunk_gradient(*W, k[b:e], v[b:e], eta[b:e])
            if beta is not None:
                M = tuple(beta[b:e].mean() * m + gj for m, gj in zip(M, g))
                g = M
            new = []
            for w, x in zip(W, g):
                U = w - (_torch_newton_schulz(x) if muon else x)
                new.append(U * (torch.linalg.vector_norm(w, dim=1, keepdim=True)
                                / torch.linalg.vector_norm(U, dim=1, keepdim=True)))
            W = tuple(new)
    return o, W, M


@pytest.mark.parametrize("mom,muon", [(False, False), (True, False), (True, True)])
def test_schedule_backward_matches_autograd(mom, muon):
    # every mode, an apply-only stretch between updates, rows applied twice
    # (the later apply keeps them), key rows updated twice, an unapplied row
    # range and unused key rows
    rng = _rng(150 + 2 * mom + muon)
    d, h, n_kv, n_q = 4, 6, 20, 26
    schedule = [("apply_then_update", 0, 5), ("apply_only", 5, 9), ("update_then_apply", 5, 9),
                ("update_only", 9, 14), ("apply_then_update", 3, 8), ("apply_only", 14, 20), ("apply_only", 22, 26)]
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random(n_kv)
    beta = rng.random(n_kv) if mom else None
    W0 = _weights(rng, h, d, unit=True)
    M0 = tuple(0.05 * rng.standard_normal(w.shape) for w in W0) if mom else None
    do = rng.standard_normal((n_q, d))
    dWf = tuple(rng.standard_normal(w.shape) for w in W0)
    dMf = tuple(rng.standard_normal(w.shape) for w in W0) if mom else None
    t = lambda a: torch.tensor(a, requires_grad=True)
    qt, kt, vt, et = t(q), t(k), t(v), t(eta)
    Wt = tuple(t(w) for w in W0)
    bt = t(beta) if mom else None
    Mt = tuple(t(m) for m in M0) if mom else None
    o, Wfin, Mfin = _torch_schedule_layer(qt, kt, vt, et, Wt, schedule, bt, Mt, muon)
    loss = (o * torch.tensor(do)).sum() + sum((w * torch.tensor(x)).sum() for w, x in zip(Wfin, dWf))
    if mom:
        loss = loss + sum((m * torch.tensor(x)).sum() for m, x in zip(Mfin, dMf))
    loss.backward()
    r = O.lact_backward_schedule_instance(q, k, v, eta, *W0, do, schedule, dWf, use_muon=muon, beta=beta, M=M0,
                                          dM_final=dMf)
    refs = (qt, kt, vt, et) + ((bt,) if mom else ())
    for name, g, ref in zip(("dq", "dk", "dv", "deta", "dbeta"), r, refs):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-8, atol=1e-10), name
    dW = r[5] if mom else r[4]
    for a, ref in zip(dW, Wt):
        assert np.allclose(a, ref.grad.numpy(), rtol=1e-8, atol=1e-10)
    if mom:
        for a, ref in zip(r[6], Mt):
            assert np.allclose(a, ref.grad.numpy(), rtol=1e-8, atol=1e-10)
    # rows no apply covers get no cotangent, nor key rows no update uses
    assert not np.any(r[0][20:22]) and not np.any(r[1][14:]) and not np.any(r[3][14:])
    # the forward the backward replays is the oracle's own forward
    fw = O.lact_forward_schedule_instance(q, k, v, eta, *W0, schedule, use_muon=muon, beta=beta, M=M0)
    assert np.allclose(o.detach().numpy(), fw[0], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("order,muon", [(0, False), (1, False), (0, True)])
def test_schedule_backward_of_uniform_chunks_is_the_chunk_loop_backward(order, muon):
    rng = _rng(155 + order + 2 * muon)
    d, h, n_kv, n_q, C = 4, 6, 13, 17, 5
    mode = "apply_then_update" if order == 0 else "update_then_apply"
    schedule = [(mode, s, min(n_kv, s + C)) for s in range(0, n_kv, C)] + [("apply_only", n_kv, n_q)]
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random((n_kv, 3))
    W0 = _weights(rng, h, d, unit=True)
    do = rng.standard_normal((n_q, d))
    dWf = tuple(rng.standard_normal(w.shape) for w in W0)
    got = O.lact_backward_schedule_instance(q, k, v, eta, *W0, do, schedule, dWf, use_muon=muon)
    ref = O.lact_backward_instance(q, k, v, eta, *W0, do, C, order, dWf, use_muon=muon)
    for a, b in zip(got[:4] + got[4], ref[:4] + ref[4]):
        assert np.allclose(a, b, rtol=1e-13, atol=1e-15)
    beta = rng.random(n_kv)
    M0 = tuple(0.05 * rng.standard_normal(w.shape) for w in W0)
    dMf = tuple(rng.standard_normal(w.shape) for w in W0)
    got = O.lact_backward_schedule_instance(q, k, v, eta, *W0, do, schedule, dWf, use_muon=muon, beta=beta, M=M0,
                                            dM_final=dMf)
    ref = O.lact_backward_momentum_instance(q, k, v, eta, beta, W0, M0, do, C, order, dWf, dMf, use_muon=muon)
    for a, b in zip(got[:5] + got[5] + got[6], ref[:5] + ref[5] + ref[6]):
        assert np.allclose(a, b, rtol=1e-13, atol=1e-15)


def test_schedule_backward_batched_driver_stacks_instances():
    rng = _rng(160)
    BH, d, h, n = 3, 4, 6, 12
    schedule = [("apply_only", 0, 4), ("update_then_apply", 4, 8), ("apply_only", 8, 12)]
    q, k, v = (np.stack([_tokens(rng, n, d) for _ in range(BH)]) for _ in range(3))
    eta, beta = 0.1 + 0.3 * rng.random((BH, n)), rng.random((BH, n))
    Ws = [_weights(rng, h, d, unit=True) for _ in range(BH)]
    W = tuple(np.stack([w[j] for w in Ws]) for j in range(3))
    M = tuple(0.1 * rng.standard_normal(w.shape) for w in W)
    do = rng.standard_normal((BH, n, d))
    got = O.lact_backward_schedule(q, k, v, eta, *W, do, schedule, beta=beta, M=M, instances=[2, 0])
    assert len(got) == 11
    for pos, i in enumerate((2, 0)):
        r = O.lact_backward_schedule_instance(q[i], k[i], v[i], eta[i], *(w[i] for w in W), do[i], schedule,
                                              beta=beta[i], M=tuple(m[i] for m in M))
        for a, b in zip(got, r[:5] + r[5] + r[6]):
            assert np.array_equal(a[pos], b)



def _torch_linear_schedule_layer(q, k, v, eta, W, schedule, beta=None, M=None, muon=False):
    """The schedule's segments with the linear fast weight in torch: an apply
    overwrites its rows of o with W q, an update takes the gradient of the
    chunk loss -sum eta (W k) . v by autograd (kept in the graph), then the
    momentum recurrence, Muon and the row-norm-preserving update."""
    o = torch.zeros(q.shape, dtype=q.dtype)
    parts = {"update_then_apply": ("update", "apply"), "apply_then_update": ("apply", "update"),
             "update_only": ("update",), "apply_only": ("apply",)}
    for mode, b, e in schedule:
        for kind in parts[mode]:
            if kind == "apply":
                rows = torch.zeros(q.shape[0], 1, dtype=q.dtype)
                rows[b:e] = 1.0
                full = torch.zeros(q.shape, dtype=q.dtype)
                full = torch.cat([full[:b], F.linear(q[b:e], W), full[e:]])
                o = o * (1 - rows) + full
                continue
            loss = -(eta[b:e] * (F.linear(k[b:e], W) * v[b:e]).sum(-1)).sum()
            g = torch.autograd.grad(loss, W, create_graph=True)[0]
            if beta is not None:
                M = beta[b:e].mean() * M + g
                g = M
            U = W - (_torch_newton_schulz(g) if muon else g)
            W = U * (torch.linalg.vector_norm(W, dim=1, keepdim=True) / torch.linalg.vector_norm(U, dim=1, keepdim=True))
    return o, W, M


@pytest.mark.parametrize("mom,muon", [(False, False), (True, False), (False, True), (True, True)])
def test_linear_schedule_backward_matches_autograd(mom, muon):
    # the schedule of the SwiGLU test: every mode, rows applied twice, key
    # rows updated twice, an unapplied row range and unused key rows
    rng = _rng(170 + 2 * mom + muon)
    d, n_kv, n_q = 5, 20, 26
    schedule = [("apply_then_update", 0, 5), ("apply_only", 5, 9), ("update_then_apply", 5, 9),
                ("update_only", 9, 14), ("apply_then_update", 3, 8), ("apply_only", 14, 20), ("apply_only", 22, 26)]
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random(n_kv)
    beta = rng.random(n_kv) if mom else None
    W0 = rng.standard_normal((d, d)) / np.sqrt(d)
    M0 = 0.05 * rng.standard_normal((d, d)) if mom else None
    do = rng.standard_normal((n_q, d))
    dWf = rng.standard_normal((d, d))
    dMf = rng.standard_normal((d, d)) if mom else None
    t = lambda a: torch.tensor(a, requires_grad=True)
    qt, kt, vt, et, Wt = t(q), t(k), t(v), t(eta), t(W0)
    bt = t(beta) if mom else None
    Mt = t(M0) if mom else None
    o, Wfin, Mfin = _torch_linear_schedule_layer(qt, kt, vt, et, Wt, schedule, bt, Mt, muon)
    loss = (o * torch.tensor(do)).sum() + (Wfin * torch.tensor(dWf)).sum()
    if mom:
        loss = loss + (Mfin * torch.tensor(dMf)).sum()
    loss.backward()
    r = O.lact_backward_schedule_instance(q, k, v, eta, W0, None, None, do, schedule, dWf, use_muon=muon,
                                          beta=beta, M=M0, dM_final=dMf)
    refs = (qt, kt, vt, et) + ((bt, Wt, Mt) if mom else (Wt,))
    for name, g, ref in zip(("dq", "dk", "dv", "deta") + (("dbeta", "dW", "dM") if mom else ("dW",)), r, refs):
        assert np.allclose(g, ref.grad.numpy(), rtol=1e-8, atol=1e-10), name
    assert not np.any(r[0][20:22]) and not np.any(r[1][14:]) and not np.any(r[3][14:])
    # the forward the backward replays is the oracle's own linear forward
    fw = O.lact_forward_schedule_instance(q, k, v, eta, W0, None, None, schedule, use_muon=muon, beta=beta, M=M0)
    assert np.allclose(o.detach().numpy(), fw[0], rtol=1e-12, atol=1e-13)
    assert np.allclose(Wfin.detach().numpy(), fw[1], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("order,muon", [(0, False), (1, False), (1, True)])
def test_linear_schedule_of_uniform_chunks_is_the_linear_chunk_loop(order, muon):
    rng = _rng(180 + order + 2 * muon)
    d, n_kv, n_q, C = 4, 13, 17, 5
    mode = "apply_then_update" if order == 0 else "update_then_apply"
    schedule = [(mode, s, min(n_kv, s + C)) for s in range(0, n_kv, C)] + [("apply_only", n_kv, n_q)]
    q, k, v = _tokens(rng, n_q, d), _tokens(rng, n_kv, d), _tokens(rng, n_kv, d)
    eta = 0.1 + 0.4 * rng.random(n_kv)
    W0 = rng.standard_normal((d, d)) / 2
    do = rng.standard_normal((n_q, d))
    dWf = rng.standard_normal((d, d))
    fw = O.lact_forward_schedule_instance(q, k, v, eta, W0, None, None, schedule, use_muon=muon)
    ref = O.lact_forward_linear_instance(q, k, v, eta, W0, C, order, use_muon=muon)
    for a, b in zip(fw, ref):
        assert np.allclose(a, b, rtol=1e-13, atol=1e-15)
    got = O.lact_backward_schedule_instance(q, k, v, eta, W0, None, None, do, schedule, dWf, use_muon=muon)
    ref = O.lact_backward_linear_instance(q, k, v, eta, W0, do, C, order, dWf, use_muon=muon)
    for a, b in zip(got, ref):
        assert np.allclose(a, b, rtol=1e-13, atol=1e-15)
    beta = rng.random(n_kv)
    M0 = 0.05 * rng.standard_normal((d, d))
    dMf = rng.standard_normal((d, d))
    got = O.lact_backward_schedule_instance(q, k, v, eta, W0, None, None, do, schedule, dWf, use_muon=muon,
                                            beta=beta, M=M0, dM_final=dMf)
    ref = O.lact_backward_momentum_instance(q, k, v, eta, beta, W0, M0, do, C, order, dWf, dMf, use_muon=muon)
    for a, b in zip(got, ref):
        assert np.allclose(a, b, rtol=1e-13, atol=1e-15)


def test_linear_schedule_backward_batched_driver():
    rng = _rng(185)
    BH, d, n = 3, 4, 12
    schedule = [("apply_only", 0, 4), ("update_then_apply", 4, 8), ("update_only", 0, 4)]
    q, k, v = (np.stack([_tokens(rng, n, d) for _ in range(BH)]) for _ in range(3))
    eta, beta = 0.1 + 0.3 * rng.random((BH, n)), rng.random((BH, n))
    W = rng.standard_normal((BH, d, d))
    M = 0.1 * rng.standard_normal((BH, d, d))
    do = rng.standard_normal((BH, n, d))
    got = O.lact_backward_schedule(q, k, v, eta, W, None, None, do, schedule, beta=beta, M=M, instances=[2, 0])
    assert len(got) == 7
    for pos, i in enumerate((2, 0)):
        r = O.lact_backward_schedule_instance(q[i], k[i], v[i], eta[i], W[i], None, None, do[i], schedule,
                                              beta=beta[i], M=M[i])
        for a, b in zip(got, r):
            assert np.array_equal(a[pos], b)


# ----------------------------------------------------------------------------- backward of the prologue and output norm


def _torch_prologue(qkv, lr_raw, lr_bias, beta_raw, n_kv):
    """The prologue in torch (autograd sees it): F.silu, a per-vector norm,
    softplus and sigmoid, k, v and the rates for the first n_kv tokens."""
    B, L, _, H, hd = qkv.shape
    act = F.silu(qkv)
    heads = lambda t: t.permute(0, 2, 1, 3).reshape(B * H, L, hd)
    q, k, v = (heads(act[:, :, j]) for j in range(3))
    q = q / torch.linalg.vector_norm(q, dim=-1, keepdim=True)
    k = k / torch.linalg.vector_norm(k, dim=-1, keepdim=True)
    R = lr_raw.shape[-1]
    eta = F.softplus(lr_raw + lr_bias).permute(0, 2, 1, 3).reshape(B * H, L, R)
    beta = torch.sigmoid(beta_raw).permute(0, 2, 1).reshape(B * H, L)
    return q, k[:, :n_kv], v[:, :n_kv], eta[:, :n_kv], beta[:, :n_kv]


@pytest.mark.parametrize("R", [1, 3])
def test_prologue_vjp_matches_autograd(R):
    rng = _rng(170 + R)
    B, L, H, hd, n_kv = 2, 7, 3, 5, 4
    qkv = rng.standard_normal((B, L, 3, H, hd))
    lr_raw, beta_raw = rng.standard_normal((B, L, H, R)), rng.standard_normal((B, L, H))
    t = lambda a: torch.tensor(a, requires_grad=True)
    xt, lt, bt = t(qkv), t(lr_raw), t(beta_raw)
    outs = _torch_prologue(xt, lt, -1.3, bt, n_kv)
    cts = [rng.standard_normal(tuple(o.shape)) for o in outs]
    sum((o * torch.tensor(c)).sum() for o, c in zip(outs, cts)).backward()
    deta = cts[3] if R == 3 else cts[3][..., 0]
    dqkv, dlr, dbr = O.qkv_prologue_vjp(qkv, lr_raw, -1.3, beta_raw, cts[0], cts[1], cts[2], deta, cts[4])
    assert np.allclose(dqkv, xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.allclose(dlr, lt.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.allclose(dbr, bt.grad.numpy(), rtol=1e-10, atol=1e-12)
    # tokens past n_kv: nothing through k, v, the rates and beta
    assert not np.any(dqkv[:, n_kv:, 1:]) and not np.any(dlr[:, n_kv:]) and not np.any(dbr[:, n_kv:])
    # the forward this reverses is the oracle's own prologue
    q, k, v, eta, beta = O.qkv_prologue(qkv, lr_raw, -1.3, beta_raw)
    assert np.allclose(outs[0].detach().numpy(), q, rtol=1e-12) and np.allclose(outs[2].detach().numpy(), v[:, :n_kv])


def test_prologue_vjp_zero_vector_and_scale_invariance():
    # a q vector that SiLU maps to zero has no cotangent; the unit-norm map
    # is blind to scaling u, so a cotangent along y itself has none either
    rng = _rng(175)
    B, L, H, hd = 1, 3, 1, 4
    qkv = rng.standard_normal((B, L, 3, H, hd))
    qkv[0, 1, 0, 0] = 0.0
    lr = rng.standard_normal((B, L, H, 1))
    q = O.qkv_prologue(qkv, lr, 0.0)[0]
    qkv_z = qkv.copy()
    qkv_z[0, 1, 0, 0] = np.zeros(hd)
    dq = rng.standard_normal((H * B, L, hd))
    dq_along = q * 2.5                                   # cotangent parallel to y
    z = np.zeros((1, L, hd))
    r = O.qkv_prologue_vjp(qkv_z, lr, 0.0, None, dq, z, z, np.zeros((1, L)))
    assert not np.any(r[0][0, 1, 0, 0])
    r = O.qkv_prologue_vjp(qkv, lr, 0.0, None, dq_along, z, z, np.zeros((1, L)))
    assert np.allclose(r[0][:, :, 0], 0.0, atol=1e-13)


@pytest.mark.parametrize("weighted", [False, True])
def test_rmsnorm_out_vjp_matches_autograd(weighted):
    rng = _rng(176 + weighted)
    B, H, L, hd = 2, 3, 5, 6
    o = rng.standard_normal((B * H, L, hd))
    w = rng.standard_normal((H, hd)) if weighted else None
    dy = rng.standard_normal((B, L, H, hd))
    ot = torch.tensor(o, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True) if weighted else None
    y = F.rms_norm(ot, (hd,), eps=1e-6).reshape(B, H, L, hd)
    if weighted:
        y = y * wt[None, :, None, :]
    (y.permute(0, 2, 1, 3) * torch.tensor(dy)).sum().backward()
    do, dw = O.rmsnorm_out_vjp(o, B, H, dy, w, 1e-6)
    assert np.allclose(do, ot.grad.numpy(), rtol=1e-10, atol=1e-12)
    if weighted:
        assert np.allclose(dw, wt.grad.numpy(), rtol=1e-10, atol=1e-12)
    else:
        assert dw is None
