"""CPU oracle of DGAP's runtime path over one logit row (fp64, NumPy).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product library.  It shares no
code with the HIP path.

What the paper fixes (Methodology):
- "DGAP Overview", online restoration framework: at each step the detector
  scores the quantized logits z^ from features phi = Phi(z^); when the risk
  r exceeds tau the corrector updates only S = TopK(z^, K_b) and the slice
  is merged back; otherwise z^ is used unchanged.
- "Distribution-Risk Detector": r = sigmoid(f_theta(phi)); the features are
  entropy, top-K_b probability mass, local gap statistics, probability-mass
  concentration and dispersion among high-probability candidates, all from
  z^ alone.
- "Selective Top-K Distribution Corrector": candidate features from local
  logits, ranks, margins and probabilities; Delta = g_psi(xi_S, phi); sparse
  merge z~_j = z^_j + Delta_j for j in S when r > tau, z^_j otherwise.
- Ablation, "Effect of risk threshold": tau = 0.60; "Detector-corrector
  architecture": MLP detector and corrector.

Readings where the paper is silent:
- TopK orders by logit, descending, ties by lower vocabulary index.
- phi has 12 entries (see ``features``); xi has 5 per candidate.
- f_theta and g_psi are one-hidden-layer ReLU MLPs; g_psi is shared by all
  candidates and sees [xi_k, phi].
- K_b per precision: K1V1 128, K2V2 64, K4V4 32, K8V8 16 (the paper
  calibrates them from traces that are not available; lower bits, larger
  windows, as it states).
- Logarithms are natural; probabilities are softmax(z^) over the whole
  vocabulary.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

TAU = 0.60
K_BY_BITS = {1: 128, 2: 64, 4: 32, 8: 16}
N_FEATURES = 12
N_CAND = 5


def log_softmax_terms(z: np.ndarray):
    """Maximum M, log-sum-exp lse and probabilities p of a logit row."""
    z = np.asarray(z, dtype=np.float64)
    M = z.max()
    lse = M + np.log(np.exp(z - M).sum())
    return M, lse, np.exp(z - lse)


def topk(z: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest logits, largest first, equal logits by lower index."""
    z = np.asarray(z, dtype=np.float64)
    order = np.lexsort((np.arange(z.size), -z))
    return order[:k]


def features(z: np.ndarray, k: int) -> np.ndarray:
    """phi: the 12 distribution-shape statistics of a logit row (Distribution-Risk
    Detector, runtime features), with v_1 >= ... >= v_k the top-k logits and
    P_i = softmax(z)_i:
      0 entropy H = -sum_i p_i log p_i       6 gap v_1 - v_2
      1 H / log V                             7 gap v_2 - v_3
      2 log P_1 (top-1 log probability)      8 mean gap (v_1 - v_k) / (k - 1)
      3 top-k mass sum_{j<=k} P_j            9 smallest gap among v_1..v_8
      4 top-8 mass                           10 standard deviation of v_1..v_k
      5 concentration sum_i p_i^2            11 entropy of the top-k mass renormalized
    (terms with probability 0 add 0 to either entropy)."""
    z = np.asarray(z, dtype=np.float64)
    if k < 8 or k > z.size:
        raise ValueError("features need 8 <= k <= V")
    _, lse, p = log_softmax_terms(z)
    v = z[topk(z, k)]
    P = np.exp(v - lse)
    mass = P.sum()
    q = P / mass
    nz, qz = p > 0, q > 0  # 0 log 0 = 0
    H = -(p[nz] * np.log(p[nz])).sum()
    return np.array([
        H,
        H / np.log(z.size),
        v[0] - lse,
        mass,
        P[:8].sum(),
        (p * p).sum(),
        v[0] - v[1],
        v[1] - v[2],
        (v[0] - v[k - 1]) / (k - 1),
        np.min(v[:7] - v[1:8]),
        v.std(),
        -(q[qz] * np.log(q[qz])).sum(),
    ])


def candidate_features(z: np.ndarray, k: int) -> np.ndarray:
    """xi [k][5] for the top-k candidates in order: logit relative to the top
    one, log probability, rank (k - 1 scaled to [0, 1]), margin to the
    candidate above (0 for the first) and to the one below (0 for the last)."""
    z = np.asarray(z, dtype=np.float64)
    _, lse, _ = log_softmax_terms(z)
    v = z[topk(z, k)]
    above = np.concatenate([[0.0], v[:-1] - v[1:]])
    below = np.concatenate([v[:-1] - v[1:], [0.0]])
    return np.stack([v - v[0], v - lse, np.arange(k) / (k - 1), above, below], axis=1)


def detector(phi: np.ndarray, w) -> float:
    """r = sigmoid(f(phi)), f(phi) = w2 . relu(W1^T phi + b1) + b2."""
    h = np.maximum(phi @ w.w1.astype(np.float64) + w.b1.astype(np.float64), 0.0)
    s = h @ w.w2.astype(np.float64) + float(w.b2)
    return 1.0 / (1.0 + np.exp(-s))


def corrector(xi: np.ndarray, phi: np.ndarray, w) -> np.ndarray:
    """Delta_k = c2 . relu(C1^T [xi_k, phi] + cb1) + cb2 for every candidate."""
    x = np.concatenate([xi, np.broadcast_to(phi, (xi.shape[0], phi.size))], axis=1)
    h = np.maximum(x @ w.c1.astype(np.float64) + w.cb1.astype(np.float64), 0.0)
    return h @ w.c2.astype(np.float64) + float(w.cb2)


@dataclass
class Restored:
    logits: np.ndarray   # z~ (fp64)
    risk: float
    corrected: bool
    idx: np.ndarray      # S in TopK order
    delta: np.ndarray    # Delta over S (zeros when not corrected)
    phi: np.ndarray


def restore(z: np.ndarray, k: int, w, tau: float = TAU) -> Restored:
    """One DGAP step on one logit row (online restoration framework)."""
    z = np.asarray(z, dtype=np.float64)
    phi = features(z, k)
    r = detector(phi, w)
    idx = topk(z, k)
    out = z.copy()
    if r > tau:
        delta = corrector(candidate_features(z, k), phi, w)
        out[idx] += delta
        return Restored(out, r, True, idx, delta, phi)
    return Restored(out, r, False, idx, np.zeros(k), phi)
