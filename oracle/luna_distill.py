"""Stage-1 attention distillation, plain float64 CPU oracle.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import or
run this module; the GPU library never does and shares no code with it.

The conversion recipe of the Implementation Details appendix (BERT on GLUE, ViT-B/16
on ImageNet-1K) starts with an attention-distillation stage: every pretrained weight
is frozen and only the feature-map parameters are trained, so that the attention
distribution LUNA induces matches the teacher's softmax attention (eq. (1) of
Section 2).  The paper names the objective but not its divergence; the readings
(listed in the design notes):

* teacher  A_ts = softmax over s of q_t . k_s / sqrt(d), over s <= t when causal;
* student  Ahat_ts = (P_ts + eps / n_t) / (den_t + eps) with P = phi(Q) phi(K)^T,
  den_t = sum_s P_ts and n_t the number of keys row t sees (n, or t + 1 when causal):
  an exact distribution that is LUNA's attention weights P_ts / den_t (eq. (9) of
  Section 3.1) as eps -> 0, and stays positive where ReLU features give P_ts = 0;
* loss of row t  CE_t = -sum_s A_ts log Ahat_ts, the soft cross-entropy (KL(A_t ||
  Ahat_t) plus the teacher's entropy, which does not depend on phi); the objective is
  its mean over every (batch, head, row).

Since sum_s A_ts = 1,  CE_t = -sum_s A_ts log(P_ts + eps / n_t) + log(den_t + eps),
and with N rows in all the gradient of the mean with respect to P is
  G_ts = (1/N) (1 / (den_t + eps) - A_ts / (P_ts + eps / n_t))   (s visible to t),
so dphi(q_t) = sum_s G_ts phi(k_s) and dphi(k_s) = sum_t G_ts phi(q_t); the feature-map
parameters follow through the map's own backward (featuremap_backward).
"""

from __future__ import annotations

import math

import numpy as np

from .luna_oracle import PARAM_NAMES, _f64, featuremap, featuremap_backward


def _visible(n, causal):
    """[n, n] mask of the keys s each query t sees."""
    if causal:
        return np.tril(np.ones((n, n), dtype=bool))
    return np.ones((n, n), dtype=bool)


def teacher(Q, K, causal=False):
    """Softmax attention weights A [..., n, n] of eq. (1) (rows sum to 1 over the
    visible keys, 0 elsewhere)."""
    Q, K = _f64(Q), _f64(K)
    n, d = Q.shape[-2], Q.shape[-1]
    logits = (Q @ np.swapaxes(K, -1, -2)) / math.sqrt(d)
    vis = _visible(n, causal)
    logits = np.where(vis, logits, -np.inf)
    m = logits.max(axis=-1, keepdims=True)
    e = np.where(vis, np.exp(logits - m), 0.0)
    return e / e.sum(axis=-1, keepdims=True)


def student(phiQ, phiK, causal=False, eps=1e-6):
    """Ahat [..., n, n] = (P + eps / n_t) / (den + eps) over the visible keys."""
    phiQ, phiK = _f64(phiQ), _f64(phiK)
    n = phiQ.shape[-2]
    vis = _visible(n, causal)
    P = np.where(vis, phiQ @ np.swapaxes(phiK, -1, -2), 0.0)
    den = P.sum(axis=-1, keepdims=True)
    nt = vis.sum(axis=-1, keepdims=True).astype(np.float64)
    return np.where(vis, (P + eps / nt) / (den + eps), 0.0)


def distill_rows_features(Q, K, phiQ, phiK, causal=False, eps=1e-6):
    """CE_t for every row [..., n], for given student features."""
    A = teacher(Q, K, causal)
    Ah = student(phiQ, phiK, causal, eps)
    vis = _visible(A.shape[-1], causal)
    return -np.where(vis, A * np.log(np.where(vis, Ah, 1.0)), 0.0).sum(axis=-1)


def distill_rows(Q, K, p, causal=False, eps=1e-6):
    """CE_t for every row, the student features from the map of p."""
    return distill_rows_features(Q, K, featuremap(Q, p), featuremap(K, p), causal, eps)


def distill_feature_grads(Q, K, phiQ, phiK, causal=False, eps=1e-6):
    """Gradients of mean(CE) with respect to phi(Q) and phi(K) (same shapes)."""
    phiQ, phiK = _f64(phiQ), _f64(phiK)
    A = teacher(Q, K, causal)
    n = A.shape[-1]
    vis = _visible(n, causal)
    P = np.where(vis, phiQ @ np.swapaxes(phiK, -1, -2), 0.0)
    den = P.sum(axis=-1, keepdims=True)
    nt = vis.sum(axis=-1, keepdims=True).astype(np.float64)
    rows = float(np.prod(A.shape[:-1]))
    G = np.where(vis, (1.0 / (den + eps) - A / (P + eps / nt)) / rows, 0.0)
    return G @ phiK, np.swapaxes(G, -1, -2) @ phiQ


def distill_backward(Q, K, p, causal=False, eps=1e-6):
    """(CE rows, gradients of mean(CE) with respect to the feature-map parameters): the
    feature gradients through the map's backward for the queries and for the keys."""
    phiQ, phiK = featuremap(Q, p), featuremap(K, p)
    rows = distill_rows_features(Q, K, phiQ, phiK, causal, eps)
    dphiQ, dphiK = distill_feature_grads(Q, K, phiQ, phiK, causal, eps)
    _, gq = featuremap_backward(Q, p, dphiQ)
    _, gk = featuremap_backward(K, p, dphiK)
    return rows, {k: gq[k] + gk[k] for k in PARAM_NAMES}


def distill_rows_at(Q, K, phiQ, phiK, rows, causal=False, eps=1e-6):
    """CE_t for the listed rows t of one head (Q, K [n, d], features [n, D]), each from
    its own teacher and student rows: O(n) per row, for sampled rows of long sequences."""
    Q, K, phiQ, phiK = _f64(Q), _f64(K), _f64(phiQ), _f64(phiK)
    n, d = Q.shape
    out = np.empty(len(rows))
    for i, t in enumerate(rows):
        nt = t + 1 if causal else n
        logits = K[:nt] @ Q[t] / math.sqrt(d)
        A = np.exp(logits - logits.max())
        A /= A.sum()
        P = phiK[:nt] @ phiQ[t]
        out[i] = -(A * np.log((P + eps / nt) / (P.sum() + eps))).sum()
    return out
