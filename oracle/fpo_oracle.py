"""Plain float64 CPU oracle of the FPO output-projected pseudogradient hot path.

TEST INFRASTRUCTURE ONLY. Only tests/, the smoke check and the benchmark's
CPU-baseline leg may import or call this module. It shares no code with the
HIP path (no kernels, headers, helpers or constants) and imports nothing from
it. Inputs arrive as storage arrays (float32, or bfloat16 bit patterns in
uint16) and are upcast exactly to float64; every step below is then the plain
definition, written in the order of the paper's method section (Sec. 3.1),
the final-norm Jacobian (Sec. 3.2 and App. E, eq. rmsnorm-vjp), the W3 update
(eq. w3update with the 1/(B*L) divisor of the App. A pseudocode), the W1/W2
feedback path (eq. errh), the relative clip and fp32 masters (App. A), the
optimizers named at the end of Sec. 3.1, and the diagnostic cosine
(eq. cosine, Sec. 2.2-2.3).

Vocabulary chunking (`vocab_chunk`) only bounds host memory: each chunk's
logits are formed, reduced and dropped, and the result is the same plain
definition evaluated in a fixed order.

Readings of points the paper leaves open (each listed in the design notes):
  * the min-RMS clamp replaces rho everywhere inside the VJP, including in
    x_hat = x / rho (App. E "Min-RMS clamp"), and is not applied in the forward;
  * eps sits inside rho in both forward and VJP;
  * dW is divided by the token count T; e, g and g~ stay per token;
  * the 1% clip applies to the gradient before the optimizer (App. A
    pseudocode), against the Frobenius norm of the fp32 master;
    s = 1 when ||dW|| = 0; the other reading (App. A prose: the weight update
    itself is clipped) is the *_update_clip pair;
  * a target outside [0, V) zeroes that token's error row, gives loss 0 and
    is counted;
  * argmax takes the lowest index among equal maxima;
  * SGD uses momentum 0.9 without dampening or Nesterov (first step stores the
    gradient); AdamW uses betas (0.9, 0.999), eps 1e-8, decoupled weight decay
    0.01 and bias correction;
  * a cosine with a zero-norm side is 0; the model summary averages the last
    round(N/4) layers;
  * the post-FFN composition uses the fp32 g~ (before any bf16 rounding) and
    the same eps and min-RMS clamp as the final norm;
  * the pre-MLP composition (layer_signal) is the same VJP at the pre-MLP
    norm's input and gain, after the post-FFN one when both apply.
Parity status: every function below is pinned by tests/test_oracle_pins.py
(layer_signal's arithmetic by autograd; its placement on the W3 path is a
reading of the paper, "parity unpinned"),
the clamp branch of rmsnorm_vjp (rho < min_rms, shared by post_ffn_signal)
included: it equals the autograd VJP of a plain RMSNorm whose epsilon is
raised, per row, so that the row's RMS is exactly the floor.
"""
from __future__ import annotations

import math

import numpy as np


def _f64(a) -> np.ndarray:
    """Exact upcast of a storage array (float32/float64, or bf16 bits in uint16)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# --------------------------------------------------------------------------
# Final RMSNorm forward (Sec. 3.2: y = gamma * x / sqrt(mean(x^2) + eps)).
def rmsnorm_forward(x, gamma, eps):
    """Return (rho [T], y [T, d]) with rho = sqrt(mean_k x_k^2 + eps), no clamp."""
    x = _f64(x)
    g = _f64(gamma)
    rho = np.sqrt(np.mean(x * x, axis=1) + eps)
    return rho, g[None, :] * x / rho[:, None]


# --------------------------------------------------------------------------
# Output-layer error and its projection through the unembedding
# (Sec. 3.1 steps 2-3, eq. gproj; App. A pseudocode).
def output_error(x, gamma, W_U, targets, eps=1e-6, min_rms=0.5, vocab_chunk=8192):
    """Full per-token output error path for the rows of x.

    Returns a dict with
      g_pre   [T, d]  g_t = sum_v (softmax(z_t)_v - [v == y_t]) W_U[v]  (eq. gproj)
      g_tilde [T, d]  rmsnorm_vjp(g, x, gamma) with the min-RMS clamp
      lse, loss [T]   log-sum-exp of z_t and lse_t - z_{t, y_t}
      zmax [T], argmax [T] (lowest index among equal maxima)
      rho [T]         forward RMS
      bad             number of targets outside [0, V)
    """
    Wf = W_U  # upcast chunk by chunk below
    V = Wf.shape[0]
    rho, y = rmsnorm_forward(x, gamma, eps)
    T, d = y.shape
    tg = np.asarray(targets, dtype=np.int64)
    valid = (tg >= 0) & (tg < V)

    # pass 1: row maxima and first arg-max
    zmax = np.full(T, -np.inf)
    amax = np.zeros(T, dtype=np.int64)
    ztgt = np.zeros(T)
    for v0 in range(0, V, vocab_chunk):
        Wc = _f64(Wf[v0:v0 + vocab_chunk])
        z = y @ Wc.T
        cm = z.max(axis=1)
        ca = z.argmax(axis=1) + v0          # numpy argmax: first occurrence
        better = cm > zmax                  # strict: earlier chunk keeps ties
        amax[better] = ca[better]
        zmax = np.maximum(zmax, cm)
        inside = valid & (tg >= v0) & (tg < v0 + Wc.shape[0])
        rows = np.nonzero(inside)[0]
        ztgt[rows] = z[rows, tg[rows] - v0]

    # pass 2: partition function
    S = np.zeros(T)
    for v0 in range(0, V, vocab_chunk):
        Wc = _f64(Wf[v0:v0 + vocab_chunk])
        S += np.exp(y @ Wc.T - zmax[:, None]).sum(axis=1)
    lse = zmax + np.log(S)

    # pass 3: g = e W_U with e = softmax(z) - onehot(y)
    g = np.zeros((T, d))
    for v0 in range(0, V, vocab_chunk):
        Wc = _f64(Wf[v0:v0 + vocab_chunk])
        p = np.exp(y @ Wc.T - lse[:, None])
        g += p @ Wc
    rows = np.nonzero(valid)[0]
    g[rows] -= _f64(Wf[tg[rows]])
    g[~valid] = 0.0
    loss = np.where(valid, lse - ztgt, 0.0)

    g_tilde = rmsnorm_vjp(g, x, gamma, eps, min_rms)
    return dict(g_pre=g, g_tilde=g_tilde, lse=lse, loss=loss, zmax=zmax, argmax=amax,
                rho=rho, bad=int((~valid).sum()))


def error_rows(x, gamma, W_U, targets, eps=1e-6):
    """Dense output error e [T, V] = softmax(z) - onehot(y) (Sec. 3.1 step 2).
    Small inputs only (materialises T x V)."""
    _, y = rmsnorm_forward(x, gamma, eps)
    z = y @ _f64(W_U).T
    z = z - z.max(axis=1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=1, keepdims=True)
    tg = np.asarray(targets, dtype=np.int64)
    p[np.arange(len(tg)), tg] -= 1.0
    return p


def logit(x, gamma, W_U, t, v, eps=1e-6):
    """Single logit z_{t,v} of the unclamped forward."""
    _, y = rmsnorm_forward(np.asarray(x)[t:t + 1], gamma, eps)
    return float(y[0] @ _f64(np.asarray(W_U)[v]))


# --------------------------------------------------------------------------
# Closed-form RMSNorm VJP with the min-RMS clamp (App. E eq. rmsnorm-vjp and
# "Min-RMS clamp"; Sec. 3.2).
def rmsnorm_vjp(g, x, gamma, eps=1e-6, min_rms=0.5):
    """(1/rho~) (gamma*g - x_hat * (1/d) <x_hat, gamma*g>), rho~ = max(rho, min_rms),
    x_hat = x / rho~, rho = sqrt(mean x^2 + eps)."""
    g = _f64(g)
    x = _f64(x)
    gam = _f64(gamma)
    d = x.shape[1]
    rho = np.sqrt(np.mean(x * x, axis=1) + eps)
    rt = np.maximum(rho, min_rms)
    xh = x / rt[:, None]
    gg = gam[None, :] * g
    c = np.sum(xh * gg, axis=1) / d
    return (gg - xh * c[:, None]) / rt[:, None]


# --------------------------------------------------------------------------
# Per-layer down-projection pseudogradient (eq. w3update; App. A divisor).
def pseudograd(g_tilde, a, scale=None):
    """D[i, j] = scale * sum_t g~[t, i] a[t, j]; scale defaults to 1/T. [d, d_ff]."""
    g = _f64(g_tilde)
    af = _f64(a)
    s = 1.0 / g.shape[0] if scale is None else scale
    return s * (g.T @ af)


# --------------------------------------------------------------------------
# Post-feedforward RMSNorm composition (Sec. 3.2 "Post-feedforward RMSNorm";
# the App. A pseudocode's per-layer rmsnorm_vjp on the cached MLP output;
# the per-architecture composition appendix): architectures that normalize
# the MLP output before the residual add (OLMo-2, Gemma 3) pass g~ through
# that norm's closed-form VJP, with the same min-RMS clamp, before the
# layer's outer product.
def post_ffn_signal(g_tilde, mlp_out, gamma_pffn, eps=1e-6, min_rms=0.5):
    """g_l = rmsnorm_vjp(g~, mlp_out_l, gamma_pffn_l) [T, d]: the layer's left
    operand (for the W3 outer product and, in full-MLP mode, E = g_l W3_init)."""
    return rmsnorm_vjp(g_tilde, mlp_out, gamma_pffn, eps, min_rms)


# --------------------------------------------------------------------------
# Pre-MLP RMSNorm composition (Sec. 3.2 "Pre-MLP RMSNorm (Qwen3, Gemma 3)";
# the per-architecture composition appendix and its summary table): the
# families that apply it also pass each target layer's signal through the
# closed-form VJP of that layer's pre-MLP RMSNorm. The paper does not say
# where on the W3 path it enters; the reading taken here applies it the way
# the App. A pseudocode applies the post-FFN norm's: rmsnorm_vjp at the norm's
# cached input (the residual stream entering the MLP sub-block) with its gain
# and the same eps and min-RMS clamp, after the post-FFN composition when a
# family has both (Gemma 3), i.e. in the order the chain of norms from the
# output meets them. Each factor is an exact RMSNorm VJP (pinned by autograd);
# the placement itself has no value or identity in the paper to pin it
# ("parity unpinned" for the placement).
def layer_signal(g_tilde, mlp_out=None, gamma_pffn=None, pre_in=None, gamma_pre=None, eps=1e-6,
                 min_rms=0.5):
    """Left operand of a target layer's outer product (and of E = g W3_init):
    g~, then the post-FFN VJP when mlp_out is given, then the pre-MLP VJP when
    pre_in is given. [T, d]"""
    g = _f64(g_tilde)
    if mlp_out is not None:
        g = rmsnorm_vjp(g, mlp_out, gamma_pffn, eps, min_rms)
    if pre_in is not None:
        g = rmsnorm_vjp(g, pre_in, gamma_pre, eps, min_rms)
    return g


# --------------------------------------------------------------------------
# Full-MLP mode: W1 (gate) and W2 (up) through the fixed feedback W3_init
# (eq. errh), with exact SwiGLU derivatives.
def silu(z):
    return z / (1.0 + np.exp(-z))


def silu_prime(z):
    s = 1.0 / (1.0 + np.exp(-z))
    return s * (1.0 + z * (1.0 - s))


def full_mlp_grads(g_tilde, W3_init, q, u, x_in, scale=None):
    """Return (D1, D2) [d_ff, d]:
    E = g~ W3_init [T, d_ff]; delta_up = E * SiLU(q); delta_gate = E * u * SiLU'(q);
    D1 = scale * delta_gate^T x_in (gate), D2 = scale * delta_up^T x_in (up)."""
    g = _f64(g_tilde)
    E = g @ _f64(W3_init)
    qf, uf, xf = _f64(q), _f64(u), _f64(x_in)
    s = 1.0 / g.shape[0] if scale is None else scale
    d_up = E * silu(qf)
    d_gate = E * uf * silu_prime(qf)
    return s * (d_gate.T @ xf), s * (d_up.T @ xf)


# --------------------------------------------------------------------------
# Relative clip (App. A: ||dW||_F <= 0.01 ||W||_F, applied before the step).
def clip_scale(d_sumsq, w_sumsq, frac=0.01):
    if frac <= 0:
        return 1.0
    if d_sumsq == 0.0:
        return 1.0
    return min(1.0, frac * math.sqrt(w_sumsq) / math.sqrt(d_sumsq))


# --------------------------------------------------------------------------
# Optimizers on the fp32 master (Sec. 3.1 end; App. A).
def sgd_momentum(W, buf, G, lr, momentum=0.9, step=1):
    """Return (W', buf'). buf' = G at step 1, else momentum*buf + G; W' = W - lr*buf'."""
    G = _f64(G)
    b = G.copy() if step == 1 else momentum * _f64(buf) + G
    return _f64(W) - lr * b, b


def adamw(W, m, v, G, lr, step, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01):
    """Return (W', m', v') with decoupled weight decay and bias correction."""
    G = _f64(G)
    m2 = beta1 * _f64(m) + (1.0 - beta1) * G
    v2 = beta2 * _f64(v) + (1.0 - beta2) * G * G
    mh = m2 / (1.0 - beta1 ** step)
    vh = v2 / (1.0 - beta2 ** step)
    W2 = _f64(W) * (1.0 - lr * weight_decay) - lr * mh / (np.sqrt(vh) + eps)
    return W2, m2, v2


# --------------------------------------------------------------------------
# The other reading of the 1% clip (App. A prose: each step's weight update is
# clipped, ||W' - W||_F <= frac ||W||_F): the optimizer runs on the unclipped
# gradient, its state advances unclipped, and only the step applied to W is
# scaled.
def sgd_momentum_update_clip(W, buf, G, lr, momentum=0.9, step=1, frac=0.01):
    """Return (W', buf', s): buf' as in sgd_momentum, delta = -lr * buf',
    s = clip_scale(||delta||^2, ||W||^2, frac), W' = W + s * delta."""
    G = _f64(G)
    b = G.copy() if step == 1 else momentum * _f64(buf) + G
    W = _f64(W)
    delta = -lr * b
    s = clip_scale(float(np.sum(delta * delta)), float(np.sum(W * W)), frac)
    return W + s * delta, b, s


def adamw_update_clip(W, m, v, G, lr, step, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, frac=0.01):
    """Return (W', m', v', s): moments as in adamw, delta = -lr * wd * W -
    lr * m_hat / (sqrt(v_hat) + eps) (the whole AdamW step, decay included),
    s = clip_scale(||delta||^2, ||W||^2, frac), W' = W + s * delta."""
    G = _f64(G)
    m2 = beta1 * _f64(m) + (1.0 - beta1) * G
    v2 = beta2 * _f64(v) + (1.0 - beta2) * G * G
    mh = m2 / (1.0 - beta1 ** step)
    vh = v2 / (1.0 - beta2 ** step)
    W = _f64(W)
    delta = -lr * weight_decay * W - lr * mh / (np.sqrt(vh) + eps)
    s = clip_scale(float(np.sum(delta * delta)), float(np.sum(W * W)), frac)
    return W + s * delta, m2, v2, s


# --------------------------------------------------------------------------
# Diagnostic cosine (eq. cosine) and the model-level summary (Sec. 2.3).
def cosine(A, B):
    """Return (dot, |A|^2, |B|^2, cos); cos = 0 when either norm is zero."""
    a = _f64(A).ravel()
    b = _f64(B).ravel()
    dot = float(a @ b)
    na = float(a @ a)
    nb = float(b @ b)
    c = 0.0 if na == 0.0 or nb == 0.0 else dot / math.sqrt(na * nb)
    return dot, na, nb, c


def layer_summary(cos_per_layer):
    """Mean cosine over the last round(N/4) layers."""
    c = list(cos_per_layer)
    k = int(round(len(c) / 4))
    k = max(k, 1)
    return float(np.mean(c[-k:]))
