"""Latency model of the attention term of the DiT cost model, fitted on one MI355X.

The paper's DiT latency model (Section IV-B, Eq. (9)) charges linear work alpha_1 (B S) and
self-attention alpha_2 (B S^2) for a bucket of B sequences of length S, divided by the
parallel degree k, plus communication. For one GPU (k = 1) and the attention operator only,
this module fits

    t(pack, H, D) = beta_2 * H * D * sum_s L_s^2 + beta_1 * H * D * sum_s L_s + c_0

to measured fwd+bwd times of libt2vattn. For a bucket of B clips of length S the sums are
B S^2 and B S, so alpha_2 = beta_2 H D and alpha_1 = beta_1 H D in the paper's notation; a
packed mix of clips of different lengths is the same expression summed clip by clip (the
operator is block-diagonal over clips). beta_1 covers the per-token work (the Delta pass,
epilogues, tile edges), c_0 the launch overhead of the four kernels.

Host-only numpy code: the measurements come from ``bench.py --cost-model``.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class AttentionCostModel:
    """t_ms = beta2 * H * D * sum(L^2) + beta1 * H * D * sum(L) + c0 (milliseconds)."""
    beta2: float   # ms per (head * dim * token^2)
    beta1: float   # ms per (head * dim * token)
    c0: float      # ms

    def alpha2(self, heads: int, head_dim: int) -> float:
        """The paper's alpha_2 for a model shape: ms per (B * S^2)."""
        return self.beta2 * heads * head_dim

    def alpha1(self, heads: int, head_dim: int) -> float:
        """The linear (per-token) part of the attention operator: ms per (B * S)."""
        return self.beta1 * heads * head_dim

    def predict_lengths(self, lengths, heads: int, head_dim: int) -> float:
        """Predicted fwd+bwd milliseconds for a pack of clips with these token counts."""
        L = np.asarray(lengths, dtype=np.float64)
        L = L[L > 0]
        hd = float(heads * head_dim)
        return self.beta2 * hd * float(np.sum(L * L)) + self.beta1 * hd * float(np.sum(L)) + self.c0

    def predict_bucket(self, batch: int, seq: int, heads: int, head_dim: int, k: int = 1) -> float:
        """Eq. (9)'s computation term for B clips of length S at parallel degree k (no communication)."""
        hd = float(heads * head_dim)
        return (self.beta2 * hd * batch * float(seq) ** 2 + self.beta1 * hd * batch * seq) / k + self.c0


def design_row(lengths, heads: int, head_dim: int) -> np.ndarray:
    L = np.asarray(lengths, dtype=np.float64)
    L = L[L > 0]
    hd = float(heads * head_dim)
    return np.array([hd * float(np.sum(L * L)), hd * float(np.sum(L)), 1.0])


def fit(samples) -> tuple[AttentionCostModel, dict]:
    """Least-squares fit on samples [(lengths, heads, head_dim, t_ms), ...].

    The rows are weighted by 1 / t so that the fit minimises relative error (the samples span
    three orders of magnitude in time). Returns the model and fit statistics (max and rms
    relative error over the samples).
    """
    if len(samples) < 3:
        raise ValueError("need at least three samples to fit three coefficients")
    X = np.stack([design_row(l, h, d) for l, h, d, _ in samples])
    t = np.array([s[3] for s in samples], dtype=np.float64)
    if np.any(t <= 0):
        raise ValueError("sample times must be positive")
    w = 1.0 / t
    coef, *_ = np.linalg.lstsq(X * w[:, None], t * w, rcond=None)
    model = AttentionCostModel(beta2=float(coef[0]), beta1=float(coef[1]), c0=float(coef[2]))
    rel = (X @ coef - t) / t
    return model, {"max_rel_err": float(np.max(np.abs(rel))), "rms_rel_err": float(np.sqrt(np.mean(rel ** 2))),
                   "n": int(len(samples))}


def relative_errors(model: AttentionCostModel, samples) -> np.ndarray:
    """(predicted - measured) / measured for samples [(lengths, heads, head_dim, t_ms), ...]."""
    return np.array([(model.predict_lengths(l, h, d) - t) / t for l, h, d, t in samples])
