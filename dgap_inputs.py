"""Seeded synthetic inputs for DGAP's logit-side runtime path.

This module draws random numbers and nothing else: it holds none of DGAP's
arithmetic (features, detector, top-K, corrector, merge), so both the CPU
oracle and the HIP path consume its outputs without sharing any of the
method.

The paper runs DGAP on the vocabulary logits of Llama-3.1-8B, Mistral-7B and
Qwen2.5-14B (Experimental Setup) with a detector and corrector trained on
PG-19 traces (Methodology, "Offline supervision").  Neither the models nor
the trained weights are available, so the logits are synthetic rows of the
models' vocabulary sizes, and the detector / corrector weights are random
draws of the MLP shapes this repository fixes (the paper gives only "MLP"
and the total size).

Logit rows: a broad N(0, 2.5^2) background over the vocabulary plus a few
"candidate" tokens lifted by U(4, 12) above it (the local top-K region the
paper restores); ``kind="flat"`` lifts them less (a high-entropy step),
``kind="ties"`` rounds logits to a coarse grid so that exact ties occur
inside and at the edge of the top-K.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

MAGIC = 0x444741  # "DGA"

VOCAB = {"llama3_8b": 128256, "mistral_7b": 32768, "qwen2_5_14b": 152064}

N_FEATURES = 12   # runtime features of a logit row
N_CAND = 5        # per-candidate inputs of the corrector (before the row features)


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng([MAGIC, *key])


def gen_logits(vocab: int, batch: int = 1, seed: int = 0, kind: str = "peaked") -> np.ndarray:
    """fp32 logits [batch][vocab]."""
    r = _rng(1, vocab, seed, {"peaked": 0, "flat": 1, "ties": 2}[kind])
    z = (2.5 * r.standard_normal((batch, vocab))).astype(np.float64)
    lift_lo, lift_hi = (4.0, 12.0) if kind != "flat" else (1.0, 3.0)
    for b in range(batch):
        cand = r.choice(vocab, size=24, replace=False)
        z[b, cand] += r.uniform(lift_lo, lift_hi, size=cand.size)
    if kind == "ties":
        z = np.round(z * 4.0) / 4.0
    return z.astype(np.float32)


@dataclass(frozen=True)
class DgapWeights:
    """Detector f(phi) = w2 . relu(W1^T phi + b1) + b2 and corrector
    g(xi, phi) = c2 . relu(C1^T [xi, phi] + cb1) + cb2 (fp32)."""

    w1: np.ndarray   # [N_FEATURES][hd]
    b1: np.ndarray   # [hd]
    w2: np.ndarray   # [hd]
    b2: float
    c1: np.ndarray   # [N_CAND + N_FEATURES][hc]
    cb1: np.ndarray  # [hc]
    c2: np.ndarray   # [hc]
    cb2: float


def gen_weights(seed: int = 0, hidden_det: int = 32, hidden_corr: int = 32, det_bias: float = 0.0,
                scale: float = 1.0) -> DgapWeights:
    """Random MLP weights, N(0, scale^2 / fan_in); the detector's output bias is
    ``det_bias`` (large positive: every step is corrected; large negative: none)."""
    r = _rng(2, seed, hidden_det, hidden_corr)
    f, c = N_FEATURES, N_CAND + N_FEATURES
    w1 = (r.standard_normal((f, hidden_det)) * scale / np.sqrt(f)).astype(np.float32)
    b1 = (r.standard_normal(hidden_det) * 0.1).astype(np.float32)
    w2 = (r.standard_normal(hidden_det) * scale / np.sqrt(hidden_det)).astype(np.float32)
    c1 = (r.standard_normal((c, hidden_corr)) * scale / np.sqrt(c)).astype(np.float32)
    cb1 = (r.standard_normal(hidden_corr) * 0.1).astype(np.float32)
    c2 = (r.standard_normal(hidden_corr) * 0.5 / np.sqrt(hidden_corr)).astype(np.float32)
    return DgapWeights(w1, b1, w2, float(np.float32(det_bias)), c1, cb1, c2, float(np.float32(0.05)))
