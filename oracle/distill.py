"""The adaptation objective of Sec. 3.2 on given logits (oracle; test infrastructure only).

Plain float64 numpy, written from the definitions: student logits cover the
extended vocabulary (the teacher's V tokens plus the added side-channel
tokens); the teacher's distribution over V is extended with zero probability
on the added tokens.  Rows are prediction positions:

* kind 1 -- a transcription token or delimiter: masked cross-entropy against
  its target (L_ASR is the mean over these rows);
* kind 2 -- a native prediction position aligned with the teacher: the
  divergence T^2 KL(P_T || P_S) at temperature T (L_native is its mean over
  these rows);
* kind 0 -- neither (no loss).

L_dec groups the native rows that are a unit's first decision by the token fed
(listen / speak / other; ``dec_group`` 0 / 1 / 2, -1 for the rest), L_turn the
native non-decision rows by whether the fed token ends the turn (``turn_group``
1 / 0, -1 for the rest); each averages the same per-row divergences within a
group and then over the groups present.  L is the sum of the four terms (unit
weights).  The gradient with respect to the student logits is given for the
fused kernel's second output.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict

import numpy as np

KIND_NONE, KIND_ASR, KIND_NATIVE = 0, 1, 2
N_DEC_GROUPS, N_TURN_GROUPS = 3, 2


def log_softmax(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, np.float64)
    m = np.max(x, axis=-1, keepdims=True)
    return x - m - np.log(np.sum(np.exp(x - m), axis=-1, keepdims=True))


@dataclass
class DistillResult:
    losses: Dict[str, float]      # asr, native, dec, turn, total
    ce: np.ndarray                # [N] per-row cross-entropy (0 where not ASR)
    kl: np.ndarray                # [N] per-row T^2 KL (0 where not native)
    grad: np.ndarray              # [N][V + added] dL / d student logits


def row_weights(kind, dec_group, turn_group):
    """Per-row coefficients of the four means: ce weight and kl weight."""
    kind = np.asarray(kind)
    dec_group = np.asarray(dec_group)
    turn_group = np.asarray(turn_group)
    n = kind.shape[0]
    w_ce = np.zeros(n)
    w_kl = np.zeros(n)
    asr = kind == KIND_ASR
    nat = kind == KIND_NATIVE
    if asr.any():
        w_ce[asr] = 1.0 / asr.sum()
    if nat.any():
        w_kl[nat] += 1.0 / nat.sum()
    for groups, n_groups in ((dec_group, N_DEC_GROUPS), (turn_group, N_TURN_GROUPS)):
        members = [nat & (groups == g) for g in range(n_groups)]
        present = [m for m in members if m.any()]
        for m in present:
            w_kl[m] += 1.0 / (len(present) * m.sum())
    return w_ce, w_kl


def row_terms(student, teacher, target, temperature: float = 1.0):
    """Per-row cross-entropy (temperature 1) against ``target`` (rows with a
    negative target get 0) and T^2 KL(P_T || P_S) at temperature T, for every
    row given; student [n][V + added], teacher [n][V]."""
    s = np.asarray(student, np.float64)
    t = np.asarray(teacher, np.float64)
    target = np.asarray(target)
    n, vs = s.shape
    v = t.shape[1]
    T = float(temperature)
    logp_t = log_softmax(t / T)
    logp_sT = log_softmax(s / T)
    # the added tokens have zero teacher probability and contribute nothing
    kl = (T * T) * np.sum(np.exp(logp_t) * (logp_t - logp_sT[:, :v]), axis=1)
    logp_s1 = log_softmax(s)
    ce = np.zeros(n)
    has = target >= 0
    ce[has] = -logp_s1[np.flatnonzero(has), target[has]]
    return ce, kl


def row_gradient(student, teacher, target, w_ce, w_kl, temperature: float = 1.0):
    """dL/d student logits of the given rows with their coefficients:
    w_kl T (softmax(s/T) - P_T extended) + w_ce (softmax(s) - onehot(target))."""
    s = np.asarray(student, np.float64)
    t = np.asarray(teacher, np.float64)
    target = np.asarray(target)
    n, vs = s.shape
    v = t.shape[1]
    T = float(temperature)
    p_t = np.zeros((n, vs))
    p_t[:, :v] = np.exp(log_softmax(t / T))
    grad = (np.asarray(w_kl, np.float64) * T)[:, None] * (np.exp(log_softmax(s / T)) - p_t)
    onehot = np.zeros((n, vs))
    has = target >= 0
    onehot[np.flatnonzero(has), target[has]] = 1.0
    grad += np.asarray(w_ce, np.float64)[:, None] * (np.exp(log_softmax(s)) - onehot)
    return grad


def distill_losses(student, teacher, kind, target, dec_group, turn_group,
                   temperature: float = 1.0) -> DistillResult:
    kind = np.asarray(kind)
    target = np.asarray(target)
    dec_group = np.asarray(dec_group)
    turn_group = np.asarray(turn_group)
    asr = kind == KIND_ASR
    nat = kind == KIND_NATIVE
    ce, kl = row_terms(student, teacher, np.where(asr, target, -1), temperature)
    kl = np.where(nat, kl, 0.0)

    l_asr = float(ce[asr].mean()) if asr.any() else 0.0
    l_nat = float(kl[nat].mean()) if nat.any() else 0.0

    def balanced(groups, n_groups):
        means = [kl[nat & (groups == g)].mean() for g in range(n_groups)
                 if (nat & (groups == g)).any()]
        return float(np.mean(means)) if means else 0.0

    l_dec = balanced(dec_group, N_DEC_GROUPS)
    l_turn = balanced(turn_group, N_TURN_GROUPS)
    w_ce, w_kl = row_weights(kind, dec_group, turn_group)
    grad = row_gradient(student, teacher, np.where(asr, target, -1), w_ce, w_kl, temperature)
    losses = {"asr": l_asr, "native": l_nat, "dec": l_dec, "turn": l_turn,
              "total": l_asr + l_nat + l_dec + l_turn}
    return DistillResult(losses=losses, ce=ce, kl=kl, grad=grad)
