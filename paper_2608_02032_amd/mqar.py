"""Multi-query associative recall (MQAR) data, as the paper specifies it
(App. D.1, "Task construction" and "Lengths and number of pairs"): the
harder variant whose non-special positions carry random vocabulary tokens.

For a sequence of length L with R key-value pairs, R distinct keys are drawn
from the key vocabulary and R distinct values from a disjoint value
vocabulary; positions 1..2R (1-based) hold k_1, v_1, ..., k_R, v_R; of the
alternating candidate query slots 2R+1, 2R+3, ..., L-1, R distinct ones receive
a random permutation of the keys; every other position holds a random token
of the whole vocabulary.  The target at a query position holding k_i is v_i
(the model predicts it from the prefix ending at the query key); every other
label is ignored.  The curriculum trains with R in {L/16, L/8, 3L/16, L/4}
and evaluates at R = L/4, where all L/4 query slots are occupied.

Seeded numpy generation only; nothing of the model is here.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

IGNORE = -100


@dataclass(frozen=True)
class MqarVocab:
    """Token ids: keys [0, n_keys), values [n_keys, n_keys + n_values)."""
    n_keys: int = 64
    n_values: int = 64

    @property
    def size(self) -> int:
        return self.n_keys + self.n_values


def curriculum_pairs(L: int):
    """The four-stage pair-count curriculum R in {L/16, L/8, 3L/16, L/4}."""
    return [L // 16, L // 8, 3 * L // 16, L // 4]


def mqar_batch(rng: np.random.Generator, batch: int, L: int, R: int, vocab: MqarVocab = MqarVocab()):
    """Returns (tokens [batch][L] int64, labels [batch][L] int64, IGNORE where
    no target)."""
    if L % 2 != 0:
        raise ValueError("L must be even")
    slots = np.arange(2 * R, L, 2)  # 0-based candidate query slots (1-based 2R+1, 2R+3, ...)
    if R > vocab.n_keys or R > vocab.n_values or R > len(slots):
        raise ValueError("R = %d pairs do not fit L = %d and the vocabulary" % (R, L))
    tokens = rng.integers(0, vocab.size, size=(batch, L), dtype=np.int64)
    labels = np.full((batch, L), IGNORE, dtype=np.int64)
    for b in range(batch):
        keys = rng.choice(vocab.n_keys, size=R, replace=False)
        vals = vocab.n_keys + rng.choice(vocab.n_values, size=R, replace=False)
        tokens[b, 0:2 * R:2] = keys
        tokens[b, 1:2 * R:2] = vals
        qpos = np.sort(rng.choice(slots, size=R, replace=False))
        order = rng.permutation(R)
        tokens[b, qpos] = keys[order]
        labels[b, qpos] = vals[order]
    return tokens, labels
