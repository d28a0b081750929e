"""Seeded synthetic batches for the adaptation objective (no loss arithmetic).

A batch holds the prediction rows of ``n_utt`` short utterances of ``units``
one-second units each.  Per unit (Sec. 3.1 order): the unit's first native
decision (a native row; listen / speak / other with probabilities 0.8 / 0.1 /
0.1), then the side-channel segment as transcription rows -- the opening
delimiter (target: first added token), t ~ Poisson(3) transcript tokens
(targets uniform over the teacher vocabulary) and the closing delimiter
(target: second added token) -- then m ~ Poisson(1) native non-decision rows
(turn end with probability 0.2, else continuation).  Teacher logits ~ N(0, 2^2)
over V tokens; student logits are the teacher's plus N(0, 0.5^2) noise, and
N(-2, 1) on the added tokens.  Values are float32, rounded to bf16 for bf16
batches.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .streams import bf16_round

KIND_NONE, KIND_ASR, KIND_NATIVE = 0, 1, 2


@dataclass
class DistillBatch:
    student: np.ndarray     # float32 [N][V + added]
    teacher: np.ndarray     # float32 [N][V]
    kind: np.ndarray        # int8 [N]
    target: np.ndarray      # int32 [N] (-1 where not a transcription row)
    dec_group: np.ndarray   # int8 [N]: 0 listen, 1 speak, 2 other, -1 none
    turn_group: np.ndarray  # int8 [N]: 1 turn end, 0 continuation, -1 none

    @property
    def n(self) -> int:
        return int(self.kind.shape[0])


def row_layout(seed: int, n_utt: int, units: int, vocab: int, added: int = 2):
    """Row metadata of a batch (kinds, targets, groups), drawn from ``seed``."""
    rng = np.random.default_rng([seed, 0])
    kind, target, dec, turn = [], [], [], []
    for _ in range(n_utt):
        for _ in range(units):
            kind.append(KIND_NATIVE)
            target.append(-1)
            dec.append(int(rng.choice(3, p=[0.8, 0.1, 0.1])))
            turn.append(-1)
            t = int(min(rng.poisson(3.0), 64))
            seg = [vocab] + [int(x) for x in rng.integers(0, vocab, size=t)] + [vocab + added - 1]
            for y in seg:
                kind.append(KIND_ASR)
                target.append(y)
                dec.append(-1)
                turn.append(-1)
            for _ in range(int(rng.poisson(1.0))):
                kind.append(KIND_NATIVE)
                target.append(-1)
                dec.append(-1)
                turn.append(int(rng.random() < 0.2))
    return (np.array(kind, np.int8), np.array(target, np.int32), np.array(dec, np.int8),
            np.array(turn, np.int8))


def make_distill_batch(seed: int, n_utt: int, units: int, vocab: int, added: int = 2,
                       dtype: str = "f32") -> DistillBatch:
    kind, target, dec, turn = row_layout(seed, n_utt, units, vocab, added)
    n = kind.shape[0]
    rng = np.random.default_rng([seed, 1])
    teacher = (2.0 * rng.standard_normal((n, vocab))).astype(np.float32)
    student = np.empty((n, vocab + added), np.float32)
    student[:, :vocab] = teacher + (0.5 * rng.standard_normal((n, vocab))).astype(np.float32)
    student[:, vocab:] = (-2.0 + rng.standard_normal((n, added))).astype(np.float32)
    if dtype == "bf16":
        teacher, student = bf16_round(teacher), bf16_round(student)
    return DistillBatch(student=student, teacher=teacher, kind=kind, target=target,
                        dec_group=dec, turn_group=turn)
