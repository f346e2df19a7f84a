"""Coupling-routed loss and its gradient, in float64.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

SAKI, Sec. 3.4 and App. H:
  accepted row (C = 0):  L_RKL = -A * log pi_theta(y),
                         A = -sg[log p(y) - log pi_T(y)]  (Eq. k1_advantage_token)
  corrected row (C = 1): L_TM  = -log pi_theta(v*),  v* = argmax_v pi_T(v)
                         (Eq. teacher_mode_loss); no RKL term at that row.
  L = (1 / N_valid) * sum_t M_t [ (1 - C_t) L_RKL,t + C_t L_TM,t ]
                                               (Eq. general_objective)
The trainable student pi_theta and the behaviour student p share the same
logits here, so log pi_theta = log_softmax(s); gradients flow only through
log pi_theta and A is a constant (App. B: the policy-gradient loss -A log p(y)
has gradient k1(y) * grad log p(y)).  With d/ds_j log softmax(s)_y =
1[j = y] - p_j the gradient of one row is
  g_j = scale * M * [ (1 - C) * (-A) * (1[j = y] - p_j) + C * (p_j - 1[j = v*]) ].
The caller supplies scale = 1 / N_valid for the whole batch; row losses are
returned unscaled and the loss sum is scaled.
"""
import numpy as np

from .bridge import log_softmax


def route_rows(s, token, corrected, teacher_argmax, advantage, valid_mask=None,
               grad_scale=1.0, want_grad=True):
    """Row losses, scaled loss sum and (optionally) the gradient w.r.t. s.

    advantage[r] = log pi_T(y_r) - log p(y_r) (the A of Eq. k1_advantage_token).
    Returns (row_loss [n], loss_sum, grad [n, V] or None).
    """
    s = np.atleast_2d(np.asarray(s, np.float64))
    n, V = s.shape
    token = np.asarray(token, np.int64)
    C = np.asarray(corrected, np.float64)
    vstar = np.asarray(teacher_argmax, np.int64)
    A = np.asarray(advantage, np.float64)
    M = np.ones(n) if valid_mask is None else np.asarray(valid_mask, np.float64)
    logp = log_softmax(s)
    idx = np.arange(n)
    l_rkl = -A * logp[idx, token]
    l_tm = -logp[idx, vstar]
    row_loss = M * ((1.0 - C) * l_rkl + C * l_tm)
    # masked rows contribute exactly zero (also when a logit is extreme)
    row_loss = np.where(M > 0, row_loss, 0.0)
    loss_sum = float(grad_scale * row_loss.sum())
    grad = None
    if want_grad:
        p = np.exp(logp)
        onehot_y = np.zeros_like(p)
        onehot_y[idx, token] = 1.0
        onehot_v = np.zeros_like(p)
        onehot_v[idx, vstar] = 1.0
        grad = ((1.0 - C)[:, None] * (-A)[:, None] * (onehot_y - p)
                + C[:, None] * (p - onehot_v))
        grad = grad_scale * M[:, None] * grad
        grad[M == 0] = 0.0
    return row_loss, loss_sum, grad


def couple_and_route(coupled, s, valid_mask=None, grad_scale=1.0, want_grad=True):
    """Route the events of oracle.coupling.couple_rows through route_rows."""
    adv = coupled["logt_token"] - coupled["logp_token"]
    return route_rows(s, coupled["token"], coupled["corrected"], coupled["teacher_argmax"],
                      adv, valid_mask, grad_scale, want_grad)
