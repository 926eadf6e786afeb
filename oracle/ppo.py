"""PPO learner update, plain CPU definition (numpy, fp64).

TEST INFRASTRUCTURE ONLY: the oracle is the plain CPU definition the HIP
path is checked against.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import this module.  It shares no code
with the HIP library and never imports it.

What is computed (PPO is the DRL algorithm of the reported results,
Section 5.2; its hyper-parameters are Table 2: Adam, learning rate 2^-14,
batch 2^10, repeat 2^3, ratio clip 0.25, entropy coefficient 0.02; the
learner of a pod trains the networks on the stored transitions, Section
4.3).  For a minibatch of B stored transitions (x_i, a_i, logp_old_i, A_i,
R_i) and the flat parameter vector of one agent:

  actor   mu = W3 tanh(W2 tanh(W1 x + b1) + b2) + b3,  sigma = exp(log_std)
  logp_i  = sum_k [ -(a_ik - mu_ik)^2 / (2 sigma_k^2) - log_std_k ] - (n/2) ln(2 pi)
  rho_i   = exp(logp_i - logp_old_i)
  L_clip  = -(1/B) sum_i min(rho_i A_i, clip(rho_i, 1 - eps, 1 + eps) A_i)
  H       = sum_k (log_std_k + (1 + ln(2 pi)) / 2)      (Gaussian entropy)
  L_actor = L_clip - c_ent H
  critic  V = w3 . tanh(Wc2 tanh(Wc1 x + bc1) + bc2) + bc3
  L_critic = (1/B) sum_i (V_i - R_i)^2

and the gradient of L_actor + L_critic (the two networks share no
parameter, so this is each network's own loss gradient), then one Adam step
(Kingma and Ba, Algorithm 1) over the whole vector:

  m = b1 m + (1 - b1) g;  v = b2 v + (1 - b2) g^2;
  theta -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps_adam).

Readings where the paper is silent (each listed in the design notes): the
PPO objective is the clipped surrogate of Schulman et al. without advantage
normalisation; the entropy bonus is the closed-form entropy of the diagonal
Gaussian policy; the critic loss is the mean squared error to the GAE
return, with no coefficient (the networks have separate losses); Adam uses
b1 = 0.9, b2 = 0.999, eps_adam = 1e-8; no gradient clipping.  Forward
precision follows the actor oracle: products accumulated in fp64, rounded
to fp32; tanh in fp32; bf16 configs use bf16-rounded weights and round the
hidden activations to bf16.  The backward pass is fp64 and treats these
roundings as the identity (straight-through); exact=True drops the
roundings altogether (a smooth function, for finite-difference pins).

Flat parameter layout of one agent (fp32 [P]; dims S, H1, H2, n of the
actor, C1, C2 of the critic):
  W1 [H1][S], b1 [H1], W2 [H2][H1], b2 [H2], W3 [n][H2], b3 [n], log_std [n],
  Wc1 [C1][S], bc1 [C1], Wc2 [C2][C1], bc2 [C2], wc3 [C2], bc3 [1].
"""

from __future__ import annotations

import math

import numpy as np

LN_2PI = math.log(2.0 * math.pi)


def layout(S, H1, H2, n, C1, C2):
    """(name, shape) of each segment of the flat vector, in order."""
    return [("W1", (H1, S)), ("b1", (H1,)), ("W2", (H2, H1)), ("b2", (H2,)),
            ("W3", (n, H2)), ("b3", (n,)), ("log_std", (n,)),
            ("Wc1", (C1, S)), ("bc1", (C1,)), ("Wc2", (C2, C1)), ("bc2", (C2,)),
            ("wc3", (C2,)), ("bc3", (1,))]


def param_count(S, H1, H2, n, C1, C2):
    return sum(int(np.prod(s)) for _, s in layout(S, H1, H2, n, C1, C2))


def unflatten(flat, dims):
    """Views of the segments of a flat vector (dims = S, H1, H2, n, C1, C2)."""
    out, off = {}, 0
    for name, shape in layout(*dims):
        size = int(np.prod(shape))
        out[name] = flat[off:off + size].reshape(shape)
        off += size
    assert off == flat.shape[0]
    return out


def flatten(parts, dims):
    return np.concatenate([np.asarray(parts[name], np.float64).reshape(-1)
                           for name, _ in layout(*dims)])


def bf16_round(x):
    """fp32 -> nearest bf16 value (ties to even), returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    return np.where(np.isnan(x), x, out)


class _Prec:
    """The forward's roundings: identity when exact."""

    def __init__(self, bf16, exact):
        self.bf16, self.exact = bf16, exact

    def weight(self, w):
        if self.exact:
            return np.asarray(w, np.float64)
        w = np.asarray(w, np.float32)
        return np.asarray(bf16_round(w) if self.bf16 else w, np.float64)

    def pre(self, z64):
        """a product accumulated in fp64, rounded to fp32"""
        return z64 if self.exact else z64.astype(np.float32).astype(np.float64)

    def tanh(self, z):
        if self.exact:
            t = np.tanh(z)
            return t, t
        t = np.tanh(z.astype(np.float32)).astype(np.float32)
        h = bf16_round(t) if self.bf16 else t
        return t.astype(np.float64), h.astype(np.float64)


def forward(p, x, bf16, exact=False):
    """Both networks on rows x [B][S] (fp64 values; bf16-exact for bf16
    configs).  Returns a dict of the intermediate values the gradient uses."""
    pr = _Prec(bf16, exact)
    x = np.asarray(x, np.float64)
    f = {"x": x}
    # actor
    W1, W2, W3 = pr.weight(p["W1"]), pr.weight(p["W2"]), pr.weight(p["W3"])
    t1, h1 = pr.tanh(pr.pre(x @ W1.T + np.asarray(p["b1"], np.float64)))
    t2, h2 = pr.tanh(pr.pre(h1 @ W2.T + np.asarray(p["b2"], np.float64)))
    mu = pr.pre(h2 @ W3.T + np.asarray(p["b3"], np.float64))
    f.update(W1=W1, W2=W2, W3=W3, t1=t1, h1=h1, t2=t2, h2=h2, mu=mu)
    # critic
    Wc1, Wc2, wc3 = pr.weight(p["Wc1"]), pr.weight(p["Wc2"]), pr.weight(p["wc3"])
    tc1, hc1 = pr.tanh(pr.pre(x @ Wc1.T + np.asarray(p["bc1"], np.float64)))
    tc2, hc2 = pr.tanh(pr.pre(hc1 @ Wc2.T + np.asarray(p["bc2"], np.float64)))
    v = pr.pre(hc2 @ wc3 + float(p["bc3"][0]))
    f.update(Wc1=Wc1, Wc2=Wc2, wc3=wc3, tc1=tc1, hc1=hc1, tc2=tc2, hc2=hc2, v=v)
    return f


def log_prob(a, mu, log_std):
    """Diagonal Gaussian log-density of rows a [B][n] (fp64)."""
    log_std = np.asarray(log_std, np.float64)
    var = np.exp(2.0 * log_std)
    d = np.asarray(a, np.float64) - mu
    return (-(d * d) / (2.0 * var) - log_std).sum(axis=1) - 0.5 * mu.shape[1] * LN_2PI


def entropy(log_std):
    """Entropy of the diagonal Gaussian policy (the same for every state)."""
    log_std = np.asarray(log_std, np.float64)
    return float((log_std + 0.5 * (1.0 + LN_2PI)).sum())


def loss_and_grad(flat, dims, x, a, logp_old, adv, ret, clip=0.25, ent_coef=0.02,
                  bf16=False, exact=False):
    """Returns (stats, grad): stats = [L_clip, H, L_critic, clip fraction]
    (fp64) and the gradient of L_actor + L_critic as a flat fp64 vector."""
    flat = np.asarray(flat)
    p = unflatten(flat, dims)
    f = forward(p, x, bf16, exact)
    B = f["x"].shape[0]
    log_std = np.asarray(p["log_std"], np.float64)
    var = np.exp(2.0 * log_std)
    a = np.asarray(a, np.float64)
    adv = np.asarray(adv, np.float64)
    ret = np.asarray(ret, np.float64)
    mu = f["mu"]
    lp = log_prob(a, mu, log_std)
    rho = np.exp(lp - np.asarray(logp_old, np.float64))
    rho_c = np.minimum(np.maximum(rho, 1.0 - clip), 1.0 + clip)
    unclipped = rho * adv <= rho_c * adv          # the min picks rho * A
    surr = np.where(unclipped, rho * adv, rho_c * adv)
    H = entropy(log_std)
    stats = [-surr.mean(), H, float(((f["v"] - ret) ** 2).mean()),
             float(np.mean(np.abs(rho - 1.0) > clip))]
    # d L / d logp_i: the clipped branch has zero derivative in rho
    g_lp = np.where(unclipped, -adv * rho / B, 0.0)
    d = a - mu
    g_mu = g_lp[:, None] * d / var                              # [B][n]
    g_ls = (g_lp[:, None] * (d * d / var - 1.0)).sum(axis=0) - ent_coef
    g = {}
    g["W3"] = g_mu.T @ f["h2"]
    g["b3"] = g_mu.sum(axis=0)
    g["log_std"] = g_ls
    g_z2 = (g_mu @ f["W3"]) * (1.0 - f["t2"] ** 2)
    g["W2"] = g_z2.T @ f["h1"]
    g["b2"] = g_z2.sum(axis=0)
    g_z1 = (g_z2 @ f["W2"]) * (1.0 - f["t1"] ** 2)
    g["W1"] = g_z1.T @ f["x"]
    g["b1"] = g_z1.sum(axis=0)
    # critic
    g_v = 2.0 * (f["v"] - ret) / B
    g["wc3"] = g_v @ f["hc2"]
    g["bc3"] = np.array([g_v.sum()])
    g_zc2 = (g_v[:, None] * f["wc3"][None, :]) * (1.0 - f["tc2"] ** 2)
    g["Wc2"] = g_zc2.T @ f["hc1"]
    g["bc2"] = g_zc2.sum(axis=0)
    g_zc1 = (g_zc2 @ f["Wc2"]) * (1.0 - f["tc1"] ** 2)
    g["Wc1"] = g_zc1.T @ f["x"]
    g["bc1"] = g_zc1.sum(axis=0)
    return np.array(stats), flatten(g, dims)


def loss(flat, dims, x, a, logp_old, adv, ret, clip=0.25, ent_coef=0.02, bf16=False,
         exact=False):
    """L_actor + L_critic (the scalar the gradient above differentiates)."""
    s, _ = loss_and_grad(flat, dims, x, a, logp_old, adv, ret, clip, ent_coef, bf16, exact)
    return s[0] - ent_coef * s[1] + s[2]


def adam(theta, m, v, g, step, lr=2.0 ** -14, b1=0.9, b2=0.999, eps=1e-8):
    """One Adam step (fp64) at step number `step` >= 1; returns new copies."""
    g = np.asarray(g, np.float64)
    m = b1 * np.asarray(m, np.float64) + (1.0 - b1) * g
    v = b2 * np.asarray(v, np.float64) + (1.0 - b2) * g * g
    mhat = m / (1.0 - b1 ** step)
    vhat = v / (1.0 - b2 ** step)
    theta = np.asarray(theta, np.float64) - lr * mhat / (np.sqrt(vhat) + eps)
    return theta, m, v


def gather(obs, action, logp, adv, ret, idx, S):
    """Rows idx of a time-major trajectory ([L][E][...] flattened to rows
    r = j E + e): observation columns 0..S-1 as fp64, raw actions, old
    log-probabilities, advantages and returns."""
    o = np.asarray(obs).reshape(-1, np.asarray(obs).shape[-1])
    x = np.asarray(o[idx, :S], np.float64)
    n = np.asarray(action).shape[-1]
    a = np.asarray(action, np.float64).reshape(-1, n)[idx]
    return (x, a, np.asarray(logp, np.float64).reshape(-1)[idx],
            np.asarray(adv, np.float64).reshape(-1)[idx],
            np.asarray(ret, np.float64).reshape(-1)[idx])


def update(flat, m, v, step, dims, batch, clip=0.25, ent_coef=0.02, lr=2.0 ** -14,
           bf16=False):
    """One learner update on a gathered minibatch (x, a, logp_old, adv, ret):
    the gradient above, then Adam.  Returns (theta, m, v, stats, grad); theta
    is rounded to fp32 (the masters are fp32)."""
    stats, g = loss_and_grad(flat, dims, *batch, clip=clip, ent_coef=ent_coef, bf16=bf16)
    theta, m, v = adam(flat, m, v, g, step, lr)
    return theta.astype(np.float32), m, v, stats, g
