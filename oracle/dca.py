"""Depth-coupled acceptance loss with verify-gated masking (test infrastructure;
see the package docstring).

Sec. "The Depth-Coupled Acceptance Loss" and "Learning up to the First
Rejection", App. "DCA" (Eqs. alpha, chain, dca, vgm, weight, dca-partial,
dca-tail, dca-coeff, dca-identity), with the sparse overlap of App.
"Implementing Draft-Path Reconstruction in verl": the head distribution q_k is
normalised over the whole vocabulary and gathered at the recorded target's
top-64 ids; the mass of each distribution outside those ids forms one residual
bin.  Per cycle:

    alpha_k = sum_{d in S_k} min(p_k(d), q_k(d)) + min(p_k(R), q_k(R)),
    M       = sum_{l=1}^{L} prod_{i<=l} alpha_i,   L = min(j, K) (VGM) or K,
    loss    = -log M,

with j = n_accept + 1 the first rejected position (j = K + 1 when every draft is
accepted, so L = K).  The gradient with respect to the head logits z_k is

    d loss / d alpha_k = -(prod_{i<k} alpha_i) D_k / M  for k <= L (else 0),
    D_k = sum_{l=k}^{L} prod_{i=k+1}^{l} alpha_i                      (Eq. dca-tail)
    d alpha_k / d z_k = q_k * (g_k - sum_x q_k(x) g_k(x)),             (softmax Jacobian)

where g_k(x) = [q_k(x) < p_k(x)] for x in S_k and g_k(x) = [q_k(R) < p_k(R)]
otherwise (the subgradient of min taken as 0 where the two are equal).

Readings: p_k(d) = exp of the recorded bf16 log-probability; p_k(R) =
max(0, 1 - sum_S p_k); q_k = softmax(z_k) at temperature one.
"""
import numpy as np

from .numerics import softmax


def dca_loss(head_logits, rec_ids, rec_logp, n_accept, vgm: bool = True):
    """head_logits [N, K, V]; rec_ids [N, K, W] int; rec_logp [N, K, W] (bf16 values);
    n_accept [N] in 0..K.  Returns (loss [N], alpha [N, K], grad [N, K, V]) in float64,
    grad = d loss_n / d head_logits[n]."""
    z = np.asarray(head_logits, dtype=np.float64)
    N, K, V = z.shape
    q = softmax(z)                                              # full-vocabulary normalisation
    rows = np.arange(N)[:, None, None], np.arange(K)[None, :, None]
    qS = q[rows[0], rows[1], rec_ids]                           # gathered at the target's top ids
    pS = np.exp(np.asarray(rec_logp, dtype=np.float64))
    pR = np.maximum(0.0, 1.0 - pS.sum(-1))
    qR = 1.0 - qS.sum(-1)
    alpha = np.minimum(pS, qS).sum(-1) + np.minimum(pR, qR)     # Eq. alpha on the sparse support
    loss = np.zeros(N)
    grad = np.zeros((N, K, V))
    for n in range(N):
        L = min(int(n_accept[n]) + 1, K) if vgm else K          # Eq. vgm: through the first rejection
        prefix = np.cumprod(alpha[n, :L])
        M = prefix.sum()                                         # Eq. chain: -L_TV
        loss[n] = -np.log(M)                                     # Eq. dca / vgm
        for k in range(L):
            D = sum(np.prod(alpha[n, k + 1:l + 1]) for l in range(k, L))          # Eq. dca-tail
            before = np.prod(alpha[n, :k])
            dl_dalpha = -before * D / M                                          # Eq. dca-coeff
            g = np.full(V, 1.0 if qR[n, k] < pR[n, k] else 0.0)
            g[rec_ids[n, k]] = (qS[n, k] < pS[n, k]).astype(np.float64)
            gbar = np.dot(q[n, k], g)
            grad[n, k] = dl_dalpha * q[n, k] * (g - gbar)
    return loss, alpha, grad
