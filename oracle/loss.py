"""Oracle log-prob and clipped policy-ratio loss, with gradients.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Follows Eq. (loss) of App. E ("RL objective"): for every trained action token
t with importance ratio rho_t = pi_theta(a_t | x_<t) / pi_rollout(a_t | x_<t)
and the advantage A of its rollout (shared by all segments of the rollout),
the objective is  min(rho A, clip(rho, 1 - eps_l, 1 + eps_h) A),  summed over
trained tokens and negated.

Readings taken where the paper is silent:
* logits are logit_scale * (h W^T) over the full vocabulary;
* the loss reduction is a caller-given loss_scale times the sum over rows;
* optional ratio cap c > 0 (the paper's "clip ratio cap"): for A < 0 the
  objective is max(objective, c A) (dual clip);
* at exact ties with a clip bound the unclipped branch is taken (strict
  inequalities decide clipping);
* the KL penalty lambda * D_KL(pi_theta || pi_ref) of the same equation is
  applied per trained token with the estimator GRPO (the paper's base
  algorithm) uses, kl = exp(ref - logp) - (ref - logp) - 1; the paper names
  no estimator.  Its expectation under pi_theta is the exact KL divergence.
"""
from __future__ import annotations

import numpy as np


def logprob(h, w, target, logit_scale=1.0):
    """h [r, H], w [V, H], target [r] -> (logp [r], lse [r], z [r, V]) in float64."""
    z = logit_scale * (h @ w.T)
    m = z.max(axis=1, keepdims=True)
    lse = (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]
    logp = z[np.arange(len(target)), target] - lse
    return logp, lse, z


def clipped_objective(logp, old_logp, adv_rows, eps_low, eps_high, dual_clip_c=0.0):
    """Per-row objective, loss (= -objective), ratio and the clipped flag."""
    rho = np.exp(logp - old_logp)
    unclipped = rho * adv_rows
    clipped_val = np.clip(rho, 1.0 - eps_low, 1.0 + eps_high) * adv_rows
    obj = np.minimum(unclipped, clipped_val)
    if dual_clip_c > 0:
        obj = np.where(adv_rows < 0, np.maximum(obj, dual_clip_c * adv_rows), obj)
    # which branch is constant in rho (strict inequalities)
    clipped = ((adv_rows > 0) & (rho > 1.0 + eps_high)) | \
              ((adv_rows < 0) & (rho < 1.0 - eps_low))
    if dual_clip_c > 0:
        clipped |= (adv_rows < 0) & (rho > dual_clip_c)
    return obj, -obj, rho, clipped


def kl_estimate(logp, ref_logp):
    """Per-token estimate of KL(pi_theta || pi_ref) at a token drawn from
    pi_theta: r - log r - 1 with r = pi_ref / pi_theta (>= 0)."""
    r = np.exp(ref_logp - logp)
    return r - np.log(r) - 1.0


def loss_and_grads(h, w, target, old_logp, adv_rows, eps_low, eps_high,
                   loss_scale=1.0, logit_scale=1.0, dual_clip_c=0.0, want_grad=True,
                   ref_logp=None, kl_coef=0.0):
    """Everything the fused kernel returns, from the definitions.

    Returns dict(logp, loss_tok, clipped, kl_tok, loss_sum, dh, dw, g).
    """
    logp, lse, z = logprob(h, w, target, logit_scale)
    obj, loss_tok, rho, clipped = clipped_objective(logp, old_logp, adv_rows, eps_low,
                                                    eps_high, dual_clip_c)
    kl = np.zeros_like(logp) if ref_logp is None else kl_estimate(logp, ref_logp)
    loss_tok = loss_tok + kl_coef * kl
    out = dict(logp=logp, loss_tok=loss_tok, clipped=clipped, kl_tok=kl,
               loss_sum=loss_scale * loss_tok.sum(), lse=lse)
    if not want_grad:
        return out
    # d(loss_scale * sum(-obj + kl_coef * kl)) / d logp: -loss_scale * rho * A
    # on the branch that depends on rho, 0 on a constant (clipped) branch;
    # the KL term adds loss_scale * kl_coef * (1 - pi_ref / pi_theta).
    g = np.where(clipped, 0.0, -loss_scale * rho * adv_rows)
    if ref_logp is not None:
        g = g + loss_scale * kl_coef * (1.0 - np.exp(ref_logp - logp))
    soft = np.exp(z - lse[:, None])
    onehot = np.zeros_like(z)
    onehot[np.arange(len(target)), target] = 1.0
    dz = g[:, None] * (onehot - soft)
    out["g"] = g
    out["dh"] = logit_scale * (dz @ w)
    out["dw"] = logit_scale * (dz.T @ h)
    return out
