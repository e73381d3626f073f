"""Oracle for the LaCT fast-weight layer forward: plain, slow, fp64, CPU.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module. The product (the HIP library and its
Python binding) never calls it and shares no code with it.

It follows "Test-Time Training Done Right" (LaCT) step by step, per
(batch, head) instance, in float64 NumPy:

* fast weight      f_W(x) = W2 [SiLU(W1 x) o (W3 x)]           (§3.1, SwiGLU eq.)
* loss             L(f_W(k), v) = -f_W(k)^T v                   (§3.1, loss eq.)
* chunk gradient   g = grad_W sum_i eta_i L(f_W(k_i), v_i)      (§3.1, chunk-gradient eq.)
* weight update    W <- L2-Normalize(W - g)  or  W - Muon(g)    (§3.2, both update eqs.)
                   normalisation per row along the input dimension, rescaled
                   to the row norm W had before the update (Alg. 1, update)
* Muon(g)          Newton-Schulz quintic iteration on g/||g||_F  (App. A, Details of Muon)
* chunk schedule   apply-then-update / update-then-apply         (§3.1 orders; Alg. 1)
* momentum         M <- M * mean_i(beta_i) + g, then the update with M in
                   place of g: W - M, or W - Muon(M)                (App. A, implementing
                   momentum for test-time optimizers; Table 3, Momentum and Muon rows)
* per-matrix rates one learning rate per token for each of W1, W2, W3 (the
                   lr of shape [b, l, 3] in the update of Alg. 1)
* linear weight    f_W(x) = W x with W in R^{d x d}, the same loss and update
                   rules (gradient -sum_i eta_i v_i k_i^T)          (§5.4 linear vs.
                   nonlinear fast weight; §3.1 loss eq.)
* prologue         per token and head: q, k, v = SiLU of the projections,
                   q and k divided by their L2 norm, lr = softplus(raw + bias),
                   beta = sigmoid(raw); heads moved next to the batch  (Alg. 1, layer)
* output norm      per-head RMSNorm of o, heads moved back next to the
                   channels                                          (Alg. 1, layer)
* backward (linear) the reverse of the linear fast weight's chunk loop: from the
                   cotangents of o (and of the final W) to those of q, k, v,
                   eta and the initial W, through the apply (o = W q), the
                   chunk gradient and the norm-preserving update of every
                   chunk (§3.1 loss and update; §5.4; reverse mode written out
                   by hand: the chunk gradient -sum eta v k^T does not depend
                   on W, so no second derivative enters)
* backward (SwiGLU) the reverse of the SwiGLU fast weight's chunk loop, the same
                   cotangents in and out (W0 = (W1, W2, W3)); the chunk
                   gradient depends on W, so its reverse carries the second
                   derivative of SiLU (reverse mode written out by hand,
                   step by step against the forward's closed form); with
                   Muon, the reverse of every Newton-Schulz step between
                   the gradient and the update (both fast weights); with
                   momentum, the state's cotangent carried from chunk to
                   chunk and the factor's cotangent spread over the chunk's
                   tokens
* schedule         a list of (mode, begin, end) segments, each one of
                   update-then-apply, apply-then-update, update-only or
                   apply-only on its token range (the ttt_config loop of Alg. 1;
                   §3.1 masks, including the strided video mask of §4.3)

Math layout (one instance): W1, W3 in R^{h x d}, W2 in R^{d x h}; a "row" is
the input dimension of the matrix (d for W1 and W3, h for W2). Tokens are rows
of q, k, v in R^{n x d}.

Readings taken where the paper is silent or ambiguous (each one is also a
test):
  R1 norm target: the pseudocode rescales W - g to the row norms of the
     pre-update W; this oracle does that (it coincides with unit rows when the
     initial rows are unit-norm).
  R2 one learning rate eta_i per token scales the loss of token i; the three
     per-matrix rates of the pseudocode are the same number here.
  R3 Newton-Schulz divides by ||G||_F + 1e-7 (the paper writes ||G||_F), so a
     zero gradient gives a zero update instead of 0/0.
  R4 Newton-Schulz works on the wide orientation (transpose when rows > cols,
     transpose back); the iteration is identical in exact arithmetic either way.
  R5 (G G^T)^2 G is evaluated as (b A + c A A) X with A = X X^T.
  R6 the last chunk may be partial; the final update is always performed, so
     the returned fast weights include it; query tokens past the last key
     token (a "tail") are applied with the final fast weights.
  R7 a chunk's gradient is summed over token blocks of at most ``token_block``
     tokens; the gradient is a sum over tokens (the linearity that §3.4 uses
     to shard a chunk over devices), so this only bounds host memory.
  R8 momentum: beta_i in (0, 1) is an input per token (its projection and
     sigmoid are outside the fast-weight path, like eta); a chunk's factor is
     the mean of its own tokens' beta_i; M starts at zero unless given, and
     the returned M is the state after the last update.
  R9 per-matrix rates: eta of shape [n, 3] holds (lr1, lr2, lr3) per token and
     weights the W1, W2 and W3 gradients respectively; with equal columns it
     is the single-rate gradient of the chunk-gradient eq.
  R11 prologue/epilogue layouts: the projections arrive as [B, L, 3, H, hd]
     (q, k, v blocks of heads, the split of Alg. 1), raw rates as
     [B, L, H, R] (R = 1 or 3), raw momentum logits as [B, L, H]; outputs are
     [B*H, L, hd] and [B*H, L(, R)]. A zero vector normalises to zero (Alg. 1
     divides by the norm without an epsilon). The RMSNorm weight is [H, hd]
     (or none); y = x / sqrt(mean(x^2) + eps) * w, returned as [B, L, H, hd].
  R10 schedule: segments run in list order and each is one update (one
     chunk) over its whole range; output rows of tokens that no apply
     segment covers are zero (Alg. 1 starts o at zero); a token applied by
     two segments keeps the later value; a segment is never empty.

parity: pinned (see tests/test_oracle_pins.py for each pin).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "NS_COEFFS", "NS_EPS", "sigmoid", "silu", "silu_derivative", "swiglu_apply", "chunk_gradient",
    "newton_schulz", "weight_update", "update", "momentum_update", "lact_forward_instance",
    "lact_forward", "lact_forward_momentum", "SCHEDULE_MODES", "lact_forward_schedule_instance",
    "lact_forward_schedule", "softplus", "qkv_prologue", "rmsnorm_out", "linear_gradient",
    "lact_forward_linear_instance", "lact_forward_linear", "linear_flops", "layer_flops",
    "weight_update_vjp", "lact_backward_linear_instance", "lact_backward_linear",
    "silu_second_derivative", "swiglu_apply_vjp", "chunk_gradient_vjp", "lact_backward_instance",
    "lact_backward", "newton_schulz_vjp", "lact_backward_momentum_instance", "lact_backward_momentum",
]

# Newton-Schulz quintic coefficients and iteration count (App. A, Details of Muon).
NS_COEFFS = (3.4445, -4.7750, 2.0315)
NS_STEPS_DEFAULT = 5
NS_EPS = 1e-7  # reading R3


def sigmoid(z: np.ndarray) -> np.ndarray:
    # Written in the two stable branches so large |z| does not overflow exp.
    out = np.empty_like(z, dtype=np.float64)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z * sigmoid(z) (the activation of the SwiGLU fast weight)."""
    return z * sigmoid(z)


def swiglu_apply(W1, W2, W3, X):
    """Apply operation o = f_W(x) for every row x of X (§2.1 apply eq.; §3.1 SwiGLU eq.).

    W1, W3: [h, d]; W2: [d, h]; X: [n, d] -> [n, d].
    """
    X = np.asarray(X, dtype=np.float64)
    Z1 = X @ W1.T             # W1 x for every token, [n, h]
    Z3 = X @ W3.T             # W3 x, [n, h]
    H = silu(Z1) * Z3         # SiLU(W1 x) o (W3 x)
    return H @ W2.T           # W2 [ ... ], [n, d]


def silu_derivative(z: np.ndarray) -> np.ndarray:
    """dSiLU/dz: with s = sigmoid(z), d(z s)/dz = s + z s (1 - s) (ds/dz = s (1 - s))."""
    s = sigmoid(z)
    return s + z * s * (1.0 - s)


def chunk_gradient(W1, W2, W3, K, V, eta, token_block: int = 65536):
    """Gradient of sum_i eta_i * (-f_W(k_i)^T v_i) w.r.t. (W1, W2, W3)
    (§3.1 chunk-gradient and loss eqs.), in closed form.

    For one token, f_W(k)^T v = c^T (SiLU(z1) o z3) with z1 = W1 k, z3 = W3 k
    and c = W2^T v (W2 only enters through c), so the product and chain rules
    give
        d/dW2 [f^T v] = v (SiLU(z1) o z3)^T
        d/dW3 [f^T v] = (c o SiLU(z1)) k^T
        d/dW1 [f^T v] = (c o z3 o SiLU'(z1)) k^T
    and the loss carries -eta_i. Over a block of tokens stacked as rows
    (K, V: [b, d]; Z1 = K W1^T, Z3 = K W3^T, C = V W2: [b, h]) each sum of
    outer products is one matrix product. eta is [n] (one rate) or [n, 3]:
    column j weights the gradient of W_{j+1} only (per-matrix rates of
    Alg. 1, reading R9).

    Returns (g1 [h, d], g2 [d, h], g3 [h, d]) in float64.
    """
    h, d = W1.shape
    g1 = np.zeros((h, d))
    g2 = np.zeros((d, h))
    g3 = np.zeros((h, d))
    n = K.shape[0]
    for s in range(0, n, token_block):   # reading R7
        e = min(n, s + token_block)
        Kb = np.asarray(K[s:e], dtype=np.float64)
        Vb = np.asarray(V[s:e], dtype=np.float64)
        lr = np.asarray(eta[s:e], dtype=np.float64)
        r1, r2, r3 = (lr[:, j:j + 1] for j in range(3)) if lr.ndim == 2 else (lr[:, None],) * 3
        Z1, Z3, C = Kb @ W1.T, Kb @ W3.T, Vb @ W2
        g2 -= (r2 * Vb).T @ (silu(Z1) * Z3)
        g3 -= (r3 * C * silu(Z1)).T @ Kb
        g1 -= (r1 * C * Z3 * silu_derivative(Z1)).T @ Kb
    return g1, g2, g3


def newton_schulz(G, steps: int = NS_STEPS_DEFAULT, coeffs=NS_COEFFS, eps: float = NS_EPS):
    """Muon's orthogonalisation of a matrix gradient (App. A, Details of Muon; §3.2).

    X_0 = G / (||G||_F + eps);  X_k = a X + b (X X^T) X + c (X X^T)^2 X.
    Readings R3 (eps), R4 (orientation) and R5 (evaluation order).
    """
    a, b, c = coeffs
    X = np.asarray(G, dtype=np.float64)
    transposed = X.shape[0] > X.shape[1]
    if transposed:
        X = X.T
    X = X / (np.linalg.norm(X) + eps)
    for _ in range(steps):
        A = X @ X.T
        Bm = b * A + c * (A @ A)
        X = a * X + Bm @ X
    return X.T if transposed else X


def weight_update(W, step):
    """W <- L2-Normalize(W - step), per row along the input dimension (§3.2).

    Rows are rescaled to the norm they had before the update (reading R1).
    """
    U = W - step
    n_old = np.sqrt(np.sum(W * W, axis=1, keepdims=True))
    n_new = np.sqrt(np.sum(U * U, axis=1, keepdims=True))
    return U * (n_old / n_new)


def update(W, K, V, eta, use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT,
           token_block: int = 65536):
    """Update operation on one chunk: gradient, optional Muon, normalised step."""
    W1, W2, W3 = W
    g1, g2, g3 = chunk_gradient(W1, W2, W3, K, V, eta, token_block)
    if use_muon:
        g1, g2, g3 = (newton_schulz(g, ns_steps) for g in (g1, g2, g3))
    return weight_update(W1, g1), weight_update(W2, g2), weight_update(W3, g3)


def momentum_update(W, M, K, V, eta, beta, use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT,
                    token_block: int = 65536):
    """Update with momentum on one chunk (App. A, implementing momentum; Table 3):

    g = grad_W sum_i eta_i L_i;  M <- M * (sum_i beta_i / b) + g;
    W <- weight-update(W, M), or weight-update(W, Muon(M)).
    Returns (W, M) (reading R8).
    """
    W1, W2, W3 = W
    g = chunk_gradient(W1, W2, W3, K, V, eta, token_block)
    bbar = float(np.mean(np.asarray(beta, dtype=np.float64)))
    M = tuple(bbar * np.asarray(m, dtype=np.float64) + gj for m, gj in zip(M, g))
    steps = tuple(newton_schulz(m, ns_steps) for m in M) if use_muon else M
    return tuple(weight_update(w, st) for w, st in zip(W, steps)), M


def lact_forward_instance(q, k, v, eta, W1, W2, W3, chunk: int, order: int,
                          use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT,
                          token_block: int = 65536, trace: list | None = None,
                          beta=None, M=None):
    """One (batch, head) instance of the layer's fast-weight path.

    q [n_q, d], k, v [n_kv, d], eta [n_kv]; W1, W3 [h, d], W2 [d, h].
    order 0 = apply-then-update (shifted block-causal), 1 = update-then-apply
    (§3.1, execution orders; Alg. 1). Returns (o [n_q, d], (W1, W2, W3)).
    With ``beta`` [n_kv] the updates use momentum (``M`` = initial
    (M1, M2, M3), zeros if omitted) and the return is (o, W, M).
    If ``trace`` is a list, the fast weights entering every chunk are appended.
    """
    W = tuple(np.asarray(w, dtype=np.float64).copy() for w in (W1, W2, W3))
    mom = beta is not None
    if mom:
        M = tuple(np.zeros_like(w) for w in W) if M is None else tuple(
            np.asarray(m, dtype=np.float64).copy() for m in M)
    n_q, n_kv = q.shape[0], k.shape[0]
    assert n_q >= n_kv and chunk > 0

    def step(W, M, s, e):
        if mom:
            return momentum_update(W, M, k[s:e], v[s:e], eta[s:e], beta[s:e], use_muon, ns_steps, token_block)
        return update(W, k[s:e], v[s:e], eta[s:e], use_muon, ns_steps, token_block), M

    o = np.zeros((n_q, q.shape[1]))
    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        if trace is not None:
            trace.append(W)
        if order == 0:
            o[s:e] = swiglu_apply(*W, q[s:e])
            W, M = step(W, M, s, e)
        else:
            W, M = step(W, M, s, e)
            o[s:e] = swiglu_apply(*W, q[s:e])
    if n_q > n_kv:                       # reading R6: apply-only tail
        o[n_kv:] = swiglu_apply(*W, q[n_kv:])
    return (o, W, M) if mom else (o, W)


def lact_forward(q, k, v, eta, W1, W2, W3, chunk: int, order: int, use_muon: bool = False,
                 ns_steps: int = NS_STEPS_DEFAULT, instances=None, token_block: int = 65536):
    """Batched driver over the (batch*head) instances (Alg. 1 merges heads into batch).

    Arrays carry a leading instance axis. ``instances`` optionally selects a
    subset. Returns (o, W1, W2, W3) stacked over the selected instances.
    """
    idx = range(q.shape[0]) if instances is None else instances
    outs, w1s, w2s, w3s = [], [], [], []
    for i in idx:
        o, (a, b, c) = lact_forward_instance(q[i], k[i], v[i], eta[i], W1[i], W2[i], W3[i],
                                             chunk, order, use_muon, ns_steps, token_block)
        outs.append(o); w1s.append(a); w2s.append(b); w3s.append(c)
    return np.stack(outs), np.stack(w1s), np.stack(w2s), np.stack(w3s)


def lact_forward_momentum(q, k, v, eta, beta, W1, W2, W3, M1=None, M2=None, M3=None, *, chunk: int,
                          order: int, use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT, instances=None,
                          token_block: int = 65536):
    """Batched driver with momentum: returns (o, W1, W2, W3, M1, M2, M3) stacked
    over the selected instances; M1..M3 default to zeros."""
    idx = range(q.shape[0]) if instances is None else instances
    res = [[] for _ in range(7)]
    for i in idx:
        M = None if M1 is None else (M1[i], M2[i], M3[i])
        o, W, Mo = lact_forward_instance(q[i], k[i], v[i], eta[i], W1[i], W2[i], W3[i], chunk, order, use_muon,
                                         ns_steps, token_block, beta=beta[i], M=M)
        for j, x in enumerate((o, *W, *Mo)):
            res[j].append(x)
    return tuple(np.stack(r) for r in res)


def softplus(x):
    """log(1 + exp(x)), in the overflow-free form max(x, 0) + log1p(exp(-|x|))."""
    x = np.asarray(x, dtype=np.float64)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def qkv_prologue(qkv, lr_raw, lr_bias: float, beta_raw=None):
    """The steps of the layer before the fast-weight path (Alg. 1, layer; R11).

    qkv [B, L, 3, H, hd]: projections; lr_raw [B, L, H, R]; beta_raw [B, L, H]
    or None. Returns (q, k, v [B*H, L, hd], eta [B*H, L, R] (R = 3) or
    [B*H, L] (R = 1), beta [B*H, L] or None), float64.
    """
    qkv = np.asarray(qkv, dtype=np.float64)
    B, L, _, H, hd = qkv.shape
    act = silu(qkv)                                    # qkv = silu(LinearQKV(x))
    heads = lambda t: np.ascontiguousarray(t.transpose(0, 2, 1, 3).reshape(B * H, L, hd))
    q, k, v = (heads(act[:, :, j]) for j in range(3))

    def unit(x):
        n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
        return np.divide(x, n, out=np.zeros_like(x), where=n > 0)

    q, k = unit(q), unit(k)                            # q / ||q||, k / ||k||
    lr = softplus(np.asarray(lr_raw, dtype=np.float64) + lr_bias)   # [B, L, H, R]
    R = lr.shape[-1]
    eta = np.ascontiguousarray(lr.transpose(0, 2, 1, 3).reshape(B * H, L, R))
    if R == 1:
        eta = eta[..., 0]
    beta = None
    if beta_raw is not None:
        beta = sigmoid(np.asarray(beta_raw, dtype=np.float64).transpose(0, 2, 1).reshape(B * H, L))
    return q, k, v, eta, beta


def rmsnorm_out(o, B: int, H: int, weight=None, eps: float = 1e-6):
    """Per-head RMSNorm of the path's output (Alg. 1, layer; R11).

    o [B*H, L, hd] -> y [B, L, H, hd], y = o / sqrt(mean_hd(o^2) + eps) * w[h].
    """
    o = np.asarray(o, dtype=np.float64)
    BH, L, hd = o.shape
    y = o / np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + eps)
    y = y.reshape(B, H, L, hd)
    if weight is not None:
        y = y * np.asarray(weight, dtype=np.float64)[None, :, None, :]
    return np.ascontiguousarray(y.transpose(0, 2, 1, 3))


def qkv_prologue_vjp(qkv, lr_raw, lr_bias: float, beta_raw, dq, dk, dv, deta, dbeta=None):
    """Reverse of qkv_prologue (Alg. 1, layer; R11) for the path's inputs as
    the path takes them: q for all L tokens, k, v, eta (and beta) for the
    first n_kv = dk.shape[1] tokens. Given their cotangents (dq [B*H, L, hd],
    dk, dv [B*H, n_kv, hd], deta [B*H, n_kv(, R)], dbeta [B*H, n_kv] or None),
    returns (dqkv [B, L, 3, H, hd], dlr_raw [B, L, H, R], dbeta_raw [B, L, H]
    or None); tokens past n_kv get no cotangent through k, v, eta, beta.

    With u = SiLU(x) and y = u / |u| (q, k):  du = (dy - y (y . dy)) / |u|
    (zero where u = 0, whose forward value is the constant 0); dx = du SiLU'(x).
    v = SiLU(x): dx = dv SiLU'(x). eta = softplus(r + bias): dr = deta
    sigmoid(r + bias). beta = sigmoid(z): dz = dbeta beta (1 - beta).
    """
    qkv = np.asarray(qkv, dtype=np.float64)
    B, L, _, H, hd = qkv.shape
    n_kv = np.asarray(dk).shape[1]
    heads = lambda t: t.transpose(0, 2, 1, 3).reshape(B * H, L, hd)          # [B, L, H, hd] -> [BH, L, hd]
    back = lambda t: t.reshape(B, H, L, hd).transpose(0, 2, 1, 3)             # the inverse
    dqkv = np.zeros_like(qkv)

    def unit_vjp(x, dy):
        u = silu(x)
        n = np.sqrt(np.sum(u * u, axis=-1, keepdims=True))
        y = np.divide(u, n, out=np.zeros_like(u), where=n > 0)
        du = np.divide(dy - y * np.sum(y * dy, axis=-1, keepdims=True), n, out=np.zeros_like(u), where=n > 0)
        return du * silu_derivative(x)

    dqkv[:, :, 0] = back(unit_vjp(heads(qkv[:, :, 0]), np.asarray(dq, dtype=np.float64)))
    kx, vx = heads(qkv[:, :, 1])[:, :n_kv], heads(qkv[:, :, 2])[:, :n_kv]
    dkx = np.zeros((B * H, L, hd))
    dvx = np.zeros((B * H, L, hd))
    dkx[:, :n_kv] = unit_vjp(kx, np.asarray(dk, dtype=np.float64))
    dvx[:, :n_kv] = np.asarray(dv, dtype=np.float64) * silu_derivative(vx)
    dqkv[:, :, 1] = back(dkx)
    dqkv[:, :, 2] = back(dvx)
    lr = np.asarray(lr_raw, dtype=np.float64)
    R = lr.shape[-1]
    de = np.asarray(deta, dtype=np.float64).reshape(B * H, n_kv, R)
    dlr = np.zeros_like(lr)
    dlr_kv = de * sigmoid(lr.transpose(0, 2, 1, 3).reshape(B * H, L, R)[:, :n_kv] + lr_bias)
    dlr[:, :n_kv] = dlr_kv.reshape(B, H, n_kv, R).transpose(0, 2, 1, 3)
    dbeta_raw = None
    if beta_raw is not None:
        z = np.asarray(beta_raw, dtype=np.float64)
        dbeta_raw = np.zeros_like(z)
        if dbeta is not None:
            b = sigmoid(z.transpose(0, 2, 1).reshape(B * H, L)[:, :n_kv])
            g = np.asarray(dbeta, dtype=np.float64) * b * (1.0 - b)
            dbeta_raw[:, :n_kv] = g.reshape(B, H, n_kv).transpose(0, 2, 1)
    return dqkv, dlr, dbeta_raw


def rmsnorm_out_vjp(o, B: int, H: int, dy, weight=None, eps: float = 1e-6):
    """Reverse of rmsnorm_out: from dy [B, L, H, hd], (do [B*H, L, hd],
    dweight [H, hd] or None). Per vector, with r = 1 / sqrt(mean(o^2) + eps)
    and g = w o dy (g = dy without a weight):
        do = r g - (r^3 / hd) o (g . o),   dw = sum over (b, l) of dy o r o.
    """
    o = np.asarray(o, dtype=np.float64)
    BH, L, hd = o.shape
    d = np.asarray(dy, dtype=np.float64).transpose(0, 2, 1, 3).reshape(BH, L, hd)
    r = 1.0 / np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + eps)
    w = None if weight is None else np.asarray(weight, dtype=np.float64)
    g = d if w is None else d * np.tile(w, (B, 1))[:, None, :]   # instance b * H + h takes w[h]
    do = r * g - (r ** 3 / hd) * o * np.sum(g * o, axis=-1, keepdims=True)
    dw = None
    if w is not None:
        dw = (d * o * r).reshape(B, H, L, hd).sum(axis=(0, 2))
    return do, dw


def linear_gradient(W, K, V, eta):
    """Gradient of sum_i eta_i * (-(W k_i)^T v_i) w.r.t. W for the linear fast
    weight f_W(x) = W x (§5.4; §3.1 loss eq.): -sum_i eta_i v_i k_i^T, [d, d]."""
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    lr = np.asarray(eta, dtype=np.float64)[:, None]
    return -(V * lr).T @ K


def lact_forward_linear_instance(q, k, v, eta, W, chunk: int, order: int, use_muon: bool = False,
                                 ns_steps: int = NS_STEPS_DEFAULT, beta=None, M=None):
    """One instance with the linear fast weight: the chunk loop of
    lact_forward_instance with o = W q, g = linear_gradient, the same
    normalised (optionally Muon, optionally momentum) update. Returns
    (o, W) or, with beta, (o, W, M)."""
    W = np.asarray(W, dtype=np.float64).copy()
    mom = beta is not None
    if mom:
        M = np.zeros_like(W) if M is None else np.asarray(M, dtype=np.float64).copy()
    n_q, n_kv = q.shape[0], k.shape[0]
    o = np.zeros((n_q, q.shape[1]))
    apply = lambda W, X: np.asarray(X, dtype=np.float64) @ W.T

    def upd(W, M, s, e):
        g = linear_gradient(W, k[s:e], v[s:e], eta[s:e])
        if mom:
            M = float(np.mean(np.asarray(beta[s:e], dtype=np.float64))) * M + g
            g = M
        return weight_update(W, newton_schulz(g, ns_steps) if use_muon else g), M

    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        if order == 0:
            o[s:e] = apply(W, q[s:e])
            W, M = upd(W, M, s, e)
        else:
            W, M = upd(W, M, s, e)
            o[s:e] = apply(W, q[s:e])
    if n_q > n_kv:
        o[n_kv:] = apply(W, q[n_kv:])
    return (o, W, M) if mom else (o, W)


def weight_update_vjp(W, step, dWn):
    """Reverse of weight_update (W' = (n / u) U with U = W - step, n and u the
    row norms of W and U): from the cotangent dWn of W', the cotangents of W
    and of step. Per row, with a = dWn . U:
        dU    = (n / u) dWn - (n a / u^3) U
        dW    = dU + (a / (u n)) W        (W enters through U and through n)
        dstep = -dU
    """
    W = np.asarray(W, dtype=np.float64)
    U = W - np.asarray(step, dtype=np.float64)
    dWn = np.asarray(dWn, dtype=np.float64)
    n = np.sqrt(np.sum(W * W, axis=1, keepdims=True))
    u = np.sqrt(np.sum(U * U, axis=1, keepdims=True))
    a = np.sum(dWn * U, axis=1, keepdims=True)
    dU = (n / u) * dWn - (n * a / u ** 3) * U
    return dU + (a / (u * n)) * W, -dU


def newton_schulz_vjp(G, dX, steps: int = NS_STEPS_DEFAULT, coeffs=NS_COEFFS, eps: float = NS_EPS):
    """Reverse of newton_schulz: from the cotangent dX of its result, the
    cotangent of G. The iterates are replayed in the wide orientation; one
    step X' = a X + B X with B = b A + c A A and A = X X^T (A and B
    symmetric) goes back as
        dB = dX' X^T,  dA = b dB + c (dB A + A dB),
        dX = a dX' + B dX' + (dA + dA^T) X,
    and the scaling X_0 = G / (s + eps), s = ||G||_F, as
        dG = dX_0 / (s + eps) - <dX_0, G> G / ((s + eps)^2 s).
    """
    a, b, c = coeffs
    G = np.asarray(G, dtype=np.float64)
    dX = np.asarray(dX, dtype=np.float64)
    transposed = G.shape[0] > G.shape[1]
    if transposed:
        G, dX = G.T, dX.T
    s = np.linalg.norm(G)
    X = G / (s + eps)
    Xs = []
    for _ in range(steps):
        Xs.append(X)
        A = X @ X.T
        X = a * X + (b * A + c * (A @ A)) @ X
    for X in reversed(Xs):
        A = X @ X.T
        Bm = b * A + c * (A @ A)
        dB = dX @ X.T
        dA = b * dB + c * (dB @ A + A @ dB)
        dX = a * dX + Bm.T @ dX + (dA + dA.T) @ X
    dG = dX / (s + eps) - (np.sum(dX * G) / ((s + eps) ** 2 * s)) * G
    return dG.T if transposed else dG


def lact_backward_linear_instance(q, k, v, eta, W0, do, chunk: int, order: int, dW_final=None,
                                  use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT):
    """Reverse of lact_forward_linear_instance (no momentum; Muon optional): given the
    cotangent ``do`` [n_q, d] of the outputs and optionally ``dW_final`` of the
    returned fast weight, the cotangents (dq, dk, dv, deta, dW0) of the inputs.

    The forward chunk loop is replayed to recover the fast weight entering
    every chunk; the chunks are then reversed. With o_t = W q_t the apply
    gives dW += do^T q and dq = do W; the chunk gradient g = -sum_t eta_t v_t
    k_t^T, with dg its cotangent (weight_update_vjp), gives
        dv_t = -eta_t dg k_t,  dk_t = -eta_t dg^T v_t,  deta_t = -v_t^T dg k_t.
    Apply-then-update applies the weights entering the chunk, update-then-apply
    those leaving it; the tail is applied with the final weights. With Muon
    the update's step is newton_schulz(g) and its cotangent goes back through
    newton_schulz_vjp before it reaches g.
    """
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    eta = np.asarray(eta, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    n_q, n_kv = q.shape[0], k.shape[0]
    step_of = (lambda g: newton_schulz(g, ns_steps)) if use_muon else (lambda g: g)
    Ws = [np.asarray(W0, dtype=np.float64).copy()]
    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        Ws.append(weight_update(Ws[-1], step_of(linear_gradient(Ws[-1], k[s:e], v[s:e], eta[s:e]))))
    dW = np.zeros_like(Ws[0]) if dW_final is None else np.asarray(dW_final, dtype=np.float64).copy()
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    deta = np.zeros(n_kv)
    if n_q > n_kv:
        dW += do[n_kv:].T @ q[n_kv:]
        dq[n_kv:] = do[n_kv:] @ Ws[-1]
    starts = list(range(0, n_kv, chunk))
    for c in reversed(range(len(starts))):
        s, e = starts[c], min(n_kv, starts[c] + chunk)
        if order == 1:                      # applied with the weights leaving the chunk
            dW += do[s:e].T @ q[s:e]
            dq[s:e] = do[s:e] @ Ws[c + 1]
        g = linear_gradient(Ws[c], k[s:e], v[s:e], eta[s:e])
        dW, dg = weight_update_vjp(Ws[c], step_of(g), dW)
        if use_muon:
            dg = newton_schulz_vjp(g, dg, ns_steps)
        kg = k[s:e] @ dg.T                  # rows dg k_t
        dv[s:e] = -eta[s:e, None] * kg
        dk[s:e] = -eta[s:e, None] * (v[s:e] @ dg)
        deta[s:e] = -np.sum(v[s:e] * kg, axis=1)
        if order == 0:                      # applied with the weights entering the chunk
            dW += do[s:e].T @ q[s:e]
            dq[s:e] = do[s:e] @ Ws[c]
    return dq, dk, dv, deta, dW


def lact_backward_linear(q, k, v, eta, W0, do, chunk: int, order: int, dW_final=None, instances=None,
                         use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT):
    """Batched driver of lact_backward_linear_instance: (dq, dk, dv, deta, dW0)
    stacked over the selected instances."""
    idx = range(q.shape[0]) if instances is None else instances
    res = [lact_backward_linear_instance(q[i], k[i], v[i], eta[i], W0[i], do[i], chunk, order,
                                         None if dW_final is None else dW_final[i], use_muon, ns_steps)
           for i in idx]
    return tuple(np.stack(col) for col in zip(*res))


def silu_second_derivative(z: np.ndarray) -> np.ndarray:
    """d^2 SiLU / dz^2: differentiating s + z s (1 - s) once more with
    ds/dz = s (1 - s) gives s (1 - s) (2 + z (1 - 2 s))."""
    s = sigmoid(z)
    return s * (1.0 - s) * (2.0 + z * (1.0 - 2.0 * s))


def swiglu_apply_vjp(W1, W2, W3, X, dO):
    """Reverse of swiglu_apply: from the cotangent dO [n, d] of O = f_W(X),
    the cotangents (dX [n, d], dW1 [h, d], dW2 [d, h], dW3 [h, d]).

    With Z1 = X W1^T, Z3 = X W3^T, H = SiLU(Z1) o Z3 and O = H W2^T:
    dW2 = dO^T H, dH = dO W2, dZ3 = dH o SiLU(Z1), dZ1 = dH o Z3 o SiLU'(Z1),
    dW1 = dZ1^T X, dW3 = dZ3^T X, dX = dZ1 W1 + dZ3 W3.
    """
    X = np.asarray(X, dtype=np.float64)
    dO = np.asarray(dO, dtype=np.float64)
    Z1, Z3 = X @ W1.T, X @ W3.T
    H = silu(Z1) * Z3
    dH = dO @ W2
    dZ3 = dH * silu(Z1)
    dZ1 = dH * Z3 * silu_derivative(Z1)
    return dZ1 @ W1 + dZ3 @ W3, dZ1.T @ X, dO.T @ H, dZ3.T @ X


def chunk_gradient_vjp(W1, W2, W3, K, V, eta, G1, G2, G3):
    """Reverse of chunk_gradient: from the cotangents (G1, G2, G3) of the
    gradients (g1, g2, g3), the cotangents (dW1, dW2, dW3, dK, dV, deta) of
    its inputs; eta (and deta) [n] for one rate per token or [n, 3] for
    per-matrix rates (column j that of W_{j+1}).

    The forward in the notation of chunk_gradient, with rates e1, e2, e3 of
    W1, W2, W3 (all equal to eta with one rate):
        Z1 = K W1^T, Z3 = K W3^T, C = V W2, S = SiLU(Z1), S1 = SiLU'(Z1)
        A  = S o Z3,  R3 = e3 C o S,  R1 = e1 C o Z3 o S1
        g2 = -(e2 V)^T A,  g3 = -R3^T K,  g1 = -R1^T K
    and its reverse, one step at a time from the last:
        dA  = -e2 (V G2),  dV = -e2 (A G2^T),  de2 = -rowsum(V o (A G2^T))
        dR3 = -K G3^T,     dK = -R3 G3
        dR1 = -K G1^T,     dK -= R1 G1
        R3:  dC = e3 dR3 o S,  dS = e3 dR3 o C,  de3 = rowsum(dR3 o C o S)
        R1:  dC += e1 dR1 o Z3 o S1,  dZ3 = e1 dR1 o C o S1,
             dS1 = e1 dR1 o C o Z3,   de1 = rowsum(dR1 o C o Z3 o S1)
        A:   dS += dA o Z3,  dZ3 += dA o S
        S, S1 (both of Z1):  dZ1 = dS o S1 + dS1 o SiLU''(Z1)
        C = V W2:   dV += dC W2^T,  dW2 = V^T dC
        Z1, Z3:     dK += dZ1 W1 + dZ3 W3,  dW1 = dZ1^T K,  dW3 = dZ3^T K
    With one rate, deta = de1 + de2 + de3.
    """
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    eta = np.asarray(eta, dtype=np.float64)
    per_matrix = eta.ndim == 2
    e1, e2, e3 = (eta[:, j:j + 1] for j in range(3)) if per_matrix else (eta[:, None],) * 3
    G1, G2, G3 = (np.asarray(g, dtype=np.float64) for g in (G1, G2, G3))
    Z1, Z3, C = K @ W1.T, K @ W3.T, V @ W2
    S, S1 = silu(Z1), silu_derivative(Z1)
    A = S * Z3
    R3, R1 = e3 * C * S, e1 * C * Z3 * S1
    AG2 = A @ G2.T
    dA = -e2 * (V @ G2)
    dV = -e2 * AG2
    de2 = -np.sum(V * AG2, axis=1)
    dR3 = -K @ G3.T
    dR1 = -K @ G1.T
    dK = -R3 @ G3 - R1 @ G1
    dC = e3 * dR3 * S + e1 * dR1 * Z3 * S1
    dS = e3 * dR3 * C + dA * Z3
    dZ3 = e1 * dR1 * C * S1 + dA * S
    dS1 = e1 * dR1 * C * Z3
    de3 = np.sum(dR3 * C * S, axis=1)
    de1 = np.sum(dR1 * C * Z3 * S1, axis=1)
    deta = np.stack([de1, de2, de3], axis=1) if per_matrix else de2 + de3 + de1
    dZ1 = dS * S1 + dS1 * silu_second_derivative(Z1)
    dV = dV + dC @ W2.T
    dK = dK + dZ1 @ W1 + dZ3 @ W3
    return dZ1.T @ K, V.T @ dC, dZ3.T @ K, dK, dV, deta


def lact_backward_instance(q, k, v, eta, W1, W2, W3, do, chunk: int, order: int, dW_final=None,
                           use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT):
    """Reverse of lact_forward_instance for the SwiGLU fast weight (Muon
    optional, no momentum; eta [n_kv] or per-matrix [n_kv, 3], deta shaped
    like it): given the cotangent ``do`` [n_q, d] of
    the outputs and optionally ``dW_final`` = (dW1, dW2, dW3) of the returned
    fast weights, the cotangents (dq, dk, dv, deta, (dW1, dW2, dW3)) of the
    inputs, the last three those of the initial fast weights.

    The chunk loop is replayed to recover the fast weights entering every
    chunk; the chunks are then reversed. A chunk's update W' = (n / u)(W - g)
    per matrix goes back through weight_update_vjp (the cotangent of g is
    minus that of U) and then through chunk_gradient_vjp (g depends on W, k,
    v and eta); its apply goes back through swiglu_apply_vjp with the weights
    it used (entering the chunk with apply-then-update, leaving it with
    update-then-apply; the tail uses the final weights). With Muon the
    update's steps are newton_schulz(g_j), and their cotangents go back
    through newton_schulz_vjp before they reach the gradients.
    """
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    eta = np.asarray(eta, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    n_q, n_kv = q.shape[0], k.shape[0]
    step_of = (lambda g: newton_schulz(g, ns_steps)) if use_muon else (lambda g: g)
    Ws = [tuple(np.asarray(w, dtype=np.float64).copy() for w in (W1, W2, W3))]
    gs = []
    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        g = chunk_gradient(*Ws[-1], k[s:e], v[s:e], eta[s:e])
        gs.append(g)
        Ws.append(tuple(weight_update(w, step_of(gj)) for w, gj in zip(Ws[-1], g)))
    dW = [np.zeros_like(w) for w in Ws[0]] if dW_final is None else [
        np.asarray(w, dtype=np.float64).copy() for w in dW_final]
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    deta = np.zeros(eta.shape)

    def apply_back(W, s, e):
        dx, a1, a2, a3 = swiglu_apply_vjp(*W, q[s:e], do[s:e])
        dq[s:e] = dx
        for j, a in enumerate((a1, a2, a3)):
            dW[j] += a

    if n_q > n_kv:
        apply_back(Ws[-1], n_kv, n_q)
    starts = list(range(0, n_kv, chunk))
    for c in reversed(range(len(starts))):
        s, e = starts[c], min(n_kv, starts[c] + chunk)
        if order == 1:                      # applied with the weights leaving the chunk
            apply_back(Ws[c + 1], s, e)
        dg = []
        for j in range(3):
            dW[j], dgj = weight_update_vjp(Ws[c][j], step_of(gs[c][j]), dW[j])
            dg.append(newton_schulz_vjp(gs[c][j], dgj, ns_steps) if use_muon else dgj)
        b1, b2, b3, dkc, dvc, detac = chunk_gradient_vjp(*Ws[c], k[s:e], v[s:e], eta[s:e], *dg)
        dW[0] += b1
        dW[1] += b2
        dW[2] += b3
        dk[s:e], dv[s:e], deta[s:e] = dkc, dvc, detac
        if order == 0:                      # applied with the weights entering the chunk
            apply_back(Ws[c], s, e)
    return dq, dk, dv, deta, tuple(dW)


def lact_backward(q, k, v, eta, W1, W2, W3, do, chunk: int, order: int, dW_final=None, instances=None,
                  use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT):
    """Batched driver of lact_backward_instance: (dq, dk, dv, deta, dW1, dW2,
    dW3) stacked over the selected instances; dW_final is None or a triple
    of [BH, ...] arrays."""
    idx = range(q.shape[0]) if instances is None else instances
    res = []
    for i in idx:
        dq, dk, dv, deta, dW = lact_backward_instance(
            q[i], k[i], v[i], eta[i], W1[i], W2[i], W3[i], do[i], chunk, order,
            None if dW_final is None else tuple(w[i] for w in dW_final), use_muon, ns_steps)
        res.append((dq, dk, dv, deta, *dW))
    return tuple(np.stack(col) for col in zip(*res))


def lact_backward_momentum_instance(q, k, v, eta, beta, W0, M0, do, chunk: int, order: int, dW_final=None,
                                    dM_final=None, use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT,
                                    dbeta_scale: bool = False):
    """Reverse of the chunk loop with the momentum optimizer (momentum_update;
    App. A), SwiGLU (W0, M0 triples) or linear (W0, M0 single [d, d] arrays)
    fast weight, Muon optional. Per chunk c with M' = bbar_c M + g_c and
    W' = weight_update(W, step(M')), step = Muon or the identity:
        dM'   = (cotangent carried from M') + step^T(d step)
        g_c's cotangent = dM';  carried to M: bbar_c dM'
        d bbar_c = <dM', M>, shared equally by the chunk's tokens (bbar is
        their mean of beta).
    Returns (dq, dk, dv, deta, dbeta, dW0, dM0), dW0 and dM0 triples for
    SwiGLU, single arrays for the linear fast weight; with dbeta_scale also,
    per token, |dM'| |M| / (chunk length) of its chunk (norms over the
    matrices together): by Cauchy-Schwarz the largest |dbeta| that vectors
    of those norms give, the scale of dbeta's rounding error.
    """
    linear = not isinstance(W0, (tuple, list))
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    eta = np.asarray(eta, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    tup = (lambda a: (a,)) if linear else (lambda a: tuple(a))
    W = tuple(np.asarray(w, dtype=np.float64).copy() for w in tup(W0))
    M = tuple(np.asarray(m, dtype=np.float64).copy() for m in tup(M0))
    n_q, n_kv = q.shape[0], k.shape[0]
    step_of = (lambda g: newton_schulz(g, ns_steps)) if use_muon else (lambda g: g)
    grad = (lambda Wc, s, e: (linear_gradient(Wc[0], k[s:e], v[s:e], eta[s:e]),)) if linear else \
        (lambda Wc, s, e: chunk_gradient(*Wc, k[s:e], v[s:e], eta[s:e]))
    apply_vjp = (lambda Wc, X, dO: (dO @ Wc[0], dO.T @ X)) if linear else \
        (lambda Wc, X, dO: (lambda r: (r[0], r[1], r[2], r[3]))(swiglu_apply_vjp(*Wc, X, dO)))
    Ws, Ms, bbars = [W], [M], []
    for s in range(0, n_kv, chunk):
        e = min(n_kv, s + chunk)
        g = grad(Ws[-1], s, e)
        bbar = float(np.mean(beta[s:e]))
        Mn = tuple(bbar * m + gj for m, gj in zip(Ms[-1], g))
        Ws.append(tuple(weight_update(w, step_of(m)) for w, m in zip(Ws[-1], Mn)))
        Ms.append(Mn)
        bbars.append(bbar)
    nm = len(W)
    dW = [np.zeros_like(w) for w in W] if dW_final is None else [
        np.asarray(x, dtype=np.float64).copy() for x in tup(dW_final)]
    dM = [np.zeros_like(m) for m in M] if dM_final is None else [
        np.asarray(x, dtype=np.float64).copy() for x in tup(dM_final)]
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    deta, dbeta, bscale = np.zeros(eta.shape), np.zeros(n_kv), np.zeros(n_kv)

    def apply_back(Wc, s, e):
        r = apply_vjp(Wc, q[s:e], do[s:e])
        dq[s:e] = r[0]
        for j in range(nm):
            dW[j] += r[1 + j]

    if n_q > n_kv:
        apply_back(Ws[-1], n_kv, n_q)
    starts = list(range(0, n_kv, chunk))
    for c in reversed(range(len(starts))):
        s, e = starts[c], min(n_kv, starts[c] + chunk)
        if order == 1:
            apply_back(Ws[c + 1], s, e)
        dMt = []
        for j in range(nm):
            dW[j], dst = weight_update_vjp(Ws[c][j], step_of(Ms[c + 1][j]), dW[j])
            dMt.append(dM[j] + (newton_schulz_vjp(Ms[c + 1][j], dst, ns_steps) if use_muon else dst))
        if linear:
            kg = k[s:e] @ dMt[0].T
            dv[s:e] = -eta[s:e, None] * kg
            dk[s:e] = -eta[s:e, None] * (v[s:e] @ dMt[0])
            deta[s:e] = -np.sum(v[s:e] * kg, axis=1)
        else:
            b1, b2, b3, dk[s:e], dv[s:e], deta[s:e] = chunk_gradient_vjp(*Ws[c], k[s:e], v[s:e], eta[s:e], *dMt)
            for j, b in enumerate((b1, b2, b3)):
                dW[j] += b
        dbeta[s:e] = sum(float(np.sum(a * m)) for a, m in zip(dMt, Ms[c])) / (e - s)
        bscale[s:e] = np.sqrt(sum(float(np.sum(a * a)) for a in dMt) *
                              sum(float(np.sum(m * m)) for m in Ms[c])) / (e - s)
        dM = [bbars[c] * a for a in dMt]
        if order == 0:
            apply_back(Ws[c], s, e)
    out = (lambda t: t[0]) if linear else tuple
    res = (dq, dk, dv, deta, dbeta, out(dW), out(dM))
    return res + (bscale,) if dbeta_scale else res


def lact_backward_momentum(q, k, v, eta, beta, W0, M0, do, chunk: int, order: int, dW_final=None, dM_final=None,
                           use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT, instances=None,
                           dbeta_scale: bool = False):
    """Batched driver of lact_backward_momentum_instance: W0, M0 (and the
    final cotangents) are triples of [BH, ...] arrays (SwiGLU) or single
    [BH, d, d] arrays (linear); returns (dq, dk, dv, deta, dbeta) stacked and
    dW0, dM0 stacked the same way (and the stacked dbeta scales with
    dbeta_scale)."""
    linear = not isinstance(W0, (tuple, list))
    idx = range(q.shape[0]) if instances is None else instances
    pick = (lambda a, i: a[i]) if linear else (lambda a, i: tuple(x[i] for x in a))
    res = [lact_backward_momentum_instance(q[i], k[i], v[i], eta[i], beta[i], pick(W0, i), pick(M0, i), do[i], chunk,
                                           order, None if dW_final is None else pick(dW_final, i),
                                           None if dM_final is None else pick(dM_final, i), use_muon, ns_steps,
                                           dbeta_scale)
           for i in idx]
    cols = list(zip(*res))
    head = tuple(np.stack(c) for c in cols[:5])
    tail = (np.stack(cols[7]),) if dbeta_scale else ()
    if linear:
        return head + (np.stack(cols[5]), np.stack(cols[6])) + tail
    return head + (tuple(np.stack([r[j] for r in cols[5]]) for j in range(3)),
                   tuple(np.stack([r[j] for r in cols[6]]) for j in range(3))) + tail


def lact_forward_linear(q, k, v, eta, W, chunk: int, order: int, use_muon: bool = False,
                        ns_steps: int = NS_STEPS_DEFAULT, instances=None, beta=None, M=None):
    """Batched driver of the linear fast weight: (o, W) stacked (and M with beta)."""
    idx = range(q.shape[0]) if instances is None else instances
    res = [lact_forward_linear_instance(q[i], k[i], v[i], eta[i], W[i], chunk, order, use_muon, ns_steps,
                                        None if beta is None else beta[i],
                                        None if (beta is None or M is None) else M[i]) for i in idx]
    return tuple(np.stack(col) for col in zip(*res))


def linear_flops(BH: int, d: int, n_kv: int, n_q: int, n_chunks: int, use_muon: bool = False,
                 ns_steps: int = NS_STEPS_DEFAULT) -> float:
    """FLOPs of the linear fast weight: the gradient V^T (eta K) costs 2 d^2 per
    updated token and the apply W q 2 d^2 per applied token (the loss needs no
    forward on the keys); Muon as in layer_flops with m = n = d, one matrix."""
    f = BH * 2.0 * d * d * (n_kv + n_q)
    if use_muon:
        f += BH * n_chunks * ns_steps * 6.0 * d ** 3
    return f


SCHEDULE_MODES = ("apply_then_update", "update_then_apply", "update_only", "apply_only")


def lact_forward_schedule_instance(q, k, v, eta, W1, W2, W3, schedule, use_muon: bool = False,
                                   ns_steps: int = NS_STEPS_DEFAULT, beta=None, M=None,
                                   token_block: int = 65536):
    """One instance under a general schedule (the ttt_config loop of Alg. 1).

    schedule: sequence of (mode, begin, end), mode one of SCHEDULE_MODES (or its
    index), each segment a single update and/or apply over tokens [begin, end)
    (reading R10). q [n_q, d]; k, v [n_kv, d]; eta [n_kv] or [n_kv, 3]; with
    ``beta`` the updates use momentum (state ``M``, zeros if omitted).
    With W2 and W3 None the fast weight is the linear one of §5.4 (W1 [d, d],
    o = W1 q, g = linear_gradient, M a single [d, d] array).
    Returns (o [n_q, d], (W1, W2, W3)) or, with beta, (o, W, M); W and M
    single arrays for the linear fast weight.
    """
    linear = W2 is None and W3 is None
    W = tuple(np.asarray(w, dtype=np.float64).copy() for w in ((W1,) if linear else (W1, W2, W3)))
    mom = beta is not None
    if mom:
        M = tuple(np.zeros_like(w) for w in W) if M is None else tuple(
            np.asarray(m, dtype=np.float64).copy() for m in ((M,) if linear else M))
    o = np.zeros((q.shape[0], q.shape[1]))

    def upd(W, M, b, e):
        assert e <= k.shape[0]
        if linear:
            g = linear_gradient(W[0], k[b:e], v[b:e], eta[b:e])
            if mom:
                M = (float(np.mean(np.asarray(beta[b:e], dtype=np.float64))) * M[0] + g,)
                g = M[0]
            return (weight_update(W[0], newton_schulz(g, ns_steps) if use_muon else g),), M
        if mom:
            return momentum_update(W, M, k[b:e], v[b:e], eta[b:e], beta[b:e], use_muon, ns_steps, token_block)
        return update(W, k[b:e], v[b:e], eta[b:e], use_muon, ns_steps, token_block), M

    apply_fw = (lambda Wl, X: np.asarray(X, dtype=np.float64) @ Wl.T) if linear else swiglu_apply

    for mode, b, e in schedule:
        mode = SCHEDULE_MODES[mode] if not isinstance(mode, str) else mode
        assert 0 <= b < e, "segments are non-empty"
        if mode == "update_then_apply":
            W, M = upd(W, M, b, e)
            o[b:e] = apply_fw(*W, q[b:e])
        elif mode == "apply_then_update":
            o[b:e] = apply_fw(*W, q[b:e])
            W, M = upd(W, M, b, e)
        elif mode == "update_only":
            W, M = upd(W, M, b, e)
        elif mode == "apply_only":
            o[b:e] = apply_fw(*W, q[b:e])
        else:
            raise ValueError(mode)
    if linear:
        W, M = W[0], (M[0] if mom else M)
    return (o, W, M) if mom else (o, W)


def lact_forward_schedule(q, k, v, eta, W1, W2, W3, schedule, use_muon: bool = False,
                          ns_steps: int = NS_STEPS_DEFAULT, beta=None, M1=None, M2=None, M3=None,
                          instances=None, token_block: int = 65536):
    """Batched driver of lact_forward_schedule_instance (one schedule for every
    instance): returns (o, W1, W2, W3) stacked, plus (M1, M2, M3) with beta;
    with W2 and W3 None (the linear fast weight) (o, W) and (o, W, M)."""
    linear = W2 is None and W3 is None
    idx = range(q.shape[0]) if instances is None else instances
    res = []
    for i in idx:
        kw = {}
        if beta is not None:
            if linear:
                kw = dict(beta=beta[i], M=None if M1 is None else M1[i])
            else:
                kw = dict(beta=beta[i], M=None if M1 is None else (M1[i], M2[i], M3[i]))
        r = lact_forward_schedule_instance(q[i], k[i], v[i], eta[i], W1[i], None if linear else W2[i],
                                           None if linear else W3[i], schedule, use_muon, ns_steps,
                                           token_block=token_block, **kw)
        if linear:
            res.append(tuple(r))
        else:
            res.append((r[0], *r[1]) + (tuple(r[2]) if beta is not None else ()))
    return tuple(np.stack(col) for col in zip(*res))


def lact_backward_schedule_instance(q, k, v, eta, W1, W2, W3, do, schedule, dW_final=None,
                                    use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT, beta=None, M=None,
                                    dM_final=None):
    """Reverse of lact_forward_schedule_instance (the ttt_config loop of
    Alg. 1; reading R10): the cotangents of q, k, v, eta (and beta with
    momentum) and of the initial fast weights (and state) given ``do`` and,
    optionally, those of the final weights (and state).

    The schedule's events (an apply or an update over its segment's tokens,
    in the segment's order) are replayed to recover the weights (and state)
    that each event used, then reversed: an apply goes back through
    swiglu_apply_vjp with its weights; an update through weight_update_vjp,
    Muon and the momentum recurrence as in lact_backward_momentum_instance,
    then chunk_gradient_vjp over its tokens. An output row written by more
    than one apply keeps the last value, so only the last apply of a row
    receives that row's cotangent; key rows used by more than one update
    collect every update's share. With W2 and W3 None the fast weight is the
    linear one (W1 [d, d]; M, dW_final, dM_final single arrays): an apply
    gives dq = dO W and dW += dO^T q, an update's gradient cotangent dg
    gives dv, dk, deta as in lact_backward_linear_instance.
    Returns (dq, dk, dv, deta, (dW1, dW2, dW3)) or, with beta,
    (dq, dk, dv, deta, dbeta, (dW1, dW2, dW3), (dM1, dM2, dM3)); dW and dM
    single arrays for the linear fast weight.
    """
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    eta = np.asarray(eta, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    mom = beta is not None
    linear = W2 is None and W3 is None
    tup = (lambda a: (a,)) if linear else tuple
    step_of = (lambda g: newton_schulz(g, ns_steps)) if use_muon else (lambda g: g)
    grad = (lambda Wc, b, e: (linear_gradient(Wc[0], k[b:e], v[b:e], eta[b:e]),)) if linear else \
        (lambda Wc, b, e: chunk_gradient(*Wc, k[b:e], v[b:e], eta[b:e]))
    W = tuple(np.asarray(w, dtype=np.float64).copy() for w in ((W1,) if linear else (W1, W2, W3)))
    Mc = tuple(np.zeros_like(w) for w in W) if M is None else tuple(np.asarray(m, dtype=np.float64).copy()
                                                                    for m in tup(M))
    nm = len(W)
    parts = {"update_then_apply": ("update", "apply"), "apply_then_update": ("apply", "update"),
             "update_only": ("update",), "apply_only": ("apply",)}
    Ws, Ms, steps, bbars, events = [W], [Mc], [], [], []
    for mode, b, e in schedule:
        mode = SCHEDULE_MODES[mode] if not isinstance(mode, str) else mode
        for kind in parts[mode]:
            events.append((kind, b, e, len(Ws) - 1))
            if kind == "update":
                g = grad(Ws[-1], b, e)
                if mom:
                    bbar = float(np.mean(np.asarray(beta, dtype=np.float64)[b:e]))
                    src = tuple(bbar * m + gj for m, gj in zip(Ms[-1], g))
                    Ms.append(src)
                    bbars.append(bbar)
                else:
                    src = g
                steps.append(src)
                Ws.append(tuple(weight_update(w, step_of(x)) for w, x in zip(Ws[-1], src)))
    dW = [np.zeros_like(w) for w in W] if dW_final is None else [
        np.asarray(x, dtype=np.float64).copy() for x in tup(dW_final)]
    dM = [np.zeros_like(w) for w in W] if dM_final is None else [
        np.asarray(x, dtype=np.float64).copy() for x in tup(dM_final)]
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    deta, dbeta = np.zeros(eta.shape), np.zeros(k.shape[0])
    claimed = np.zeros(q.shape[0], dtype=bool)
    for kind, b, e, wi in reversed(events):
        if kind == "apply":
            dO = np.where(claimed[b:e, None], 0.0, do[b:e])
            claimed[b:e] = True
            if linear:
                dq[b:e] += dO @ Ws[wi][0]
                dW[0] += dO.T @ q[b:e]
                continue
            dx, a1, a2, a3 = swiglu_apply_vjp(*Ws[wi], q[b:e], dO)
            dq[b:e] += dx
            for j, a in enumerate((a1, a2, a3)):
                dW[j] += a
            continue
        dg = []
        for j in range(nm):
            dW[j], dst = weight_update_vjp(Ws[wi][j], step_of(steps[wi][j]), dW[j])
            dg.append(newton_schulz_vjp(steps[wi][j], dst, ns_steps) if use_muon else dst)
        if mom:
            dg = [a + x for a, x in zip(dM, dg)]
        if linear:                          # g = -sum eta v k^T does not depend on W
            kg = k[b:e] @ dg[0].T
            dv[b:e] += -eta[b:e, None] * kg
            dk[b:e] += -eta[b:e, None] * (v[b:e] @ dg[0])
            deta[b:e] += -np.sum(v[b:e] * kg, axis=1)
        else:
            b1, b2, b3, dkc, dvc, detac = chunk_gradient_vjp(*Ws[wi], k[b:e], v[b:e], eta[b:e], *dg)
            for j, x in enumerate((b1, b2, b3)):
                dW[j] += x
            dk[b:e] += dkc
            dv[b:e] += dvc
            deta[b:e] += detac
        if mom:
            dbeta[b:e] += sum(float(np.sum(a * m)) for a, m in zip(dg, Ms[wi])) / (e - b)
            dM = [bbars[wi] * a for a in dg]
    out = (lambda t: t[0]) if linear else tuple
    if mom:
        return dq, dk, dv, deta, dbeta, out(dW), out(dM)
    return dq, dk, dv, deta, out(dW)


def lact_backward_schedule(q, k, v, eta, W1, W2, W3, do, schedule, dW_final=None, use_muon: bool = False,
                           ns_steps: int = NS_STEPS_DEFAULT, beta=None, M=None, dM_final=None, instances=None):
    """Batched driver of lact_backward_schedule_instance (one schedule for
    every instance): (dq, dk, dv, deta, dW1, dW2, dW3) stacked, and with beta
    (dq, dk, dv, deta, dbeta, dW1, dW2, dW3, dM1, dM2, dM3); W, M and the
    final cotangents are triples of [BH, ...] arrays (or None). With W2 and
    W3 None (the linear fast weight) they are single [BH, d, d] arrays and
    dW (dM) one stacked array each."""
    linear = W2 is None and W3 is None
    idx = range(q.shape[0]) if instances is None else instances
    if linear:
        pick = lambda t, i: None if t is None else t[i]
        lst = lambda a: (a,)
    else:
        pick = lambda t, i: None if t is None else tuple(x[i] for x in t)
        lst = tuple
    res = []
    for i in idx:
        r = lact_backward_schedule_instance(q[i], k[i], v[i], eta[i], W1[i], None if linear else W2[i],
                                            None if linear else W3[i], do[i], schedule,
                                            pick(dW_final, i), use_muon, ns_steps,
                                            None if beta is None else beta[i], pick(M, i), pick(dM_final, i))
        flat = r[:4] + lst(r[4]) if beta is None else r[:5] + lst(r[5]) + lst(r[6])
        res.append(flat)
    return tuple(np.stack(col) for col in zip(*res))


def layer_flops(BH: int, d: int, h: int, n_kv: int, n_q: int, n_chunks: int,
                use_muon: bool = False, ns_steps: int = NS_STEPS_DEFAULT) -> float:
    """Algorithmic FLOPs of the path (App. A, FLOPs calculation).

    Per head: an updated token costs 2 forward matmuls on the key (4dh),
    4 gradient matmuls including the hidden gradient (8dh); an applied token
    costs 3 matmuls (6dh), so a token that is both updated and applied costs
    18dh. Muon adds per matrix and iteration 3 matmuls on the m x n matrix
    (m <= n): X X^T (2 m^2 n), A A (2 m^3), B X (2 m^2 n).
    """
    f = BH * (12.0 * d * h * n_kv + 6.0 * d * h * n_q)
    if use_muon:
        m, n = min(d, h), max(d, h)
        f += BH * n_chunks * 3 * ns_steps * (4.0 * m * m * n + 2.0 * m ** 3)
    return f
