"""CPU oracle for the teacher-forced training forward and its loss.

TEST INFRASTRUCTURE ONLY (same rules as domino_oracle).  Float64.

What it follows (Sec. 4.2, Training):
* Teacher-forced causal encoding: the GRU consumes the ground-truth token
  embeddings of the block (the anchor, then label_1 .. label_{B-2}), so the
  forward is domino_oracle.draft_step with forced = labels.
* Base-anchored curriculum: L = (1 - lambda) L_final + lambda L_base, with
  L_final and L_base cross-entropies of the final logits L_i and the base
  logits L_i^base against the labels.
* Position weights w_k = exp(-k / gamma) over the draft positions.
Readings (the paper fixes neither): k = 0 .. B-2 is the draft position's
index within the block (the first draft position has weight 1), and each loss
is the weighted mean sum_{b,k} w_k CE_{b,k} / (bs * sum_k w_k).
"""
from __future__ import annotations

import numpy as np

from . import domino_oracle as _do

F64 = np.float64


def cross_entropy(logits, label):
    """-log softmax(logits)[label] for one row (NaN as -inf)."""
    z = _do.order_key(logits)
    m = np.max(z)
    return float(m + np.log(np.sum(np.exp(z - m))) - z[int(label)])


def position_weights(depth, gamma):
    return np.exp(-np.arange(depth, dtype=F64) / F64(gamma))


def curriculum_loss(base_logits, final_logits, labels, lam, gamma):
    """Returns (total, base, final, ce_base [bs, B-1], ce_final [bs, B-1])."""
    base_logits = np.asarray(base_logits)
    bs, depth = labels.shape
    ce_b = np.empty((bs, depth))
    ce_f = np.empty((bs, depth))
    for b in range(bs):
        for k in range(depth):
            ce_b[b, k] = cross_entropy(base_logits[b, k], labels[b, k])
            ce_f[b, k] = cross_entropy(final_logits[b, k], labels[b, k])
    w = position_weights(depth, gamma)
    lb = float(np.sum(ce_b * w) / (bs * np.sum(w)))
    lf = float(np.sum(ce_f * w) / (bs * np.sum(w)))
    return (1.0 - lam) * lf + lam * lb, lb, lf, ce_b, ce_f


def train_forward(cfg, w, anchor, ctx_lens, ctx_k, ctx_v, labels, lam, gamma, ctx_hidden=None):
    """Teacher-forced forward of one block per batch row and its curriculum loss."""
    ref = _do.draft_step(cfg, w, anchor, ctx_lens, ctx_k, ctx_v, 1, forced=labels, ctx_hidden=ctx_hidden)
    total, lb, lf, ce_b, ce_f = curriculum_loss(ref["base_logits"], ref["final_logits"], np.asarray(labels), lam,
                                                gamma)
    ref.update({"loss": total, "loss_base": lb, "loss_final": lf, "ce_base": ce_b, "ce_final": ce_f})
    return ref
