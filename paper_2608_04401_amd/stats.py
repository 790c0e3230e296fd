"""Host-side load-balance statistics of a routing (Section 2.4 and Appendix A.3).

These work on per-expert assignment counts (what the dispatch step produces on the GPU)
and are used to report mean k, utilisation and its coefficient of variation next to the
fixed top-K baseline.  They are not on the GPU hot path.

Definitions:
  utilisation   q_i = L_i / sum_j L_j, L_i = share of tokens routed to expert i
                (Appendix A.3, Notation);
  pruning rate  delta = 1 - E[k] / K (Section 2.4);
  CV            CV^2(q) = N ||q||_2^2 - 1 (Appendix A.3, Corollary 2);
  Theorem 1     ||q_elb - q_top||_1 <= 2 delta / (1 - delta);
  Corollary 1   | ||q_elb||_inf - ||q_top||_inf | <= 2 delta / (1 - delta);
  Corollary 2   | CV^2(q_elb) - CV^2(q_top) | <= 2 N delta / (1 - delta)^2;
  Table 1       % change in top-1 share = (max q_top - max q_elb) / max q_top * 100,
                % change in CV          = (CV_top - CV_elb) / CV_top * 100
                (a negative value means the elbow routing increased it).
"""
from __future__ import annotations

import math

import numpy as np


def utilization(counts) -> np.ndarray:
    c = np.asarray(counts, dtype=np.float64)
    s = c.sum()
    if s <= 0:
        raise ValueError("no assignments")
    return c / s


def cv2(q) -> float:
    q = np.asarray(q, dtype=np.float64)
    return float(q.size * np.dot(q, q) - 1.0)


def cv(q) -> float:
    return math.sqrt(max(cv2(q), 0.0))


def pruning_rate(mean_k: float, K: int) -> float:
    return 1.0 - float(mean_k) / float(K)


def theorem1_bound(delta: float) -> float:
    return 2.0 * delta / (1.0 - delta)


def corollary2_bound(N: int, delta: float) -> float:
    return 2.0 * N * delta / (1.0 - delta) ** 2


def load_balance_report(counts_elb, counts_top, K: int, T: int) -> dict:
    """Compare an elbow routing with the top-K routing of the same tokens."""
    counts_elb = np.asarray(counts_elb, dtype=np.float64)
    counts_top = np.asarray(counts_top, dtype=np.float64)
    N = counts_elb.size
    q_e, q_t = utilization(counts_elb), utilization(counts_top)
    mean_k = counts_elb.sum() / T
    delta = pruning_rate(mean_k, K)
    l1 = float(np.abs(q_e - q_t).sum())
    top1_t, top1_e = float(q_t.max()), float(q_e.max())
    cv_t, cv_e = cv(q_t), cv(q_e)
    return {
        "mean_k": float(mean_k),
        "delta": float(delta),
        "l1": l1,
        "l1_bound": theorem1_bound(delta),
        "top1_share_change_pct": (top1_t - top1_e) / top1_t * 100.0,
        "top1_bound": theorem1_bound(delta),
        "top1_abs_change": abs(top1_e - top1_t),
        "cv_top": cv_t,
        "cv_elbow": cv_e,
        "cv_change_pct": (cv_t - cv_e) / cv_t * 100.0 if cv_t > 0 else 0.0,
        "cv2_abs_change": abs(cv2(q_e) - cv2(q_t)),
        "cv2_bound": corollary2_bound(N, delta),
    }
