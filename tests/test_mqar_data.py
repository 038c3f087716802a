"""The MQAR generator against the task construction of App. D.1: source
pairs in the first 2R positions, distinct keys and values from disjoint
vocabularies, queries at R distinct alternating slots after them carrying a
permutation of the keys, labels only there (the key's value)."""
import numpy as np
import pytest

from paper_2608_02032_amd import mqar


@pytest.mark.parametrize("L,R", [(256, 16), (256, 64), (512, 32), (64, 16)])
def test_mqar_batch_follows_the_task_construction(L, R):
    voc = mqar.MqarVocab(64, 64)
    tok, lab = mqar.mqar_batch(np.random.default_rng(L + R), 8, L, R, voc)
    assert tok.shape == (8, L) and lab.shape == (8, L)
    assert tok.min() >= 0 and tok.max() < voc.size
    for b in range(8):
        keys, vals = tok[b, 0:2 * R:2], tok[b, 1:2 * R:2]
        assert len(set(keys)) == R and len(set(vals)) == R
        assert np.all(keys < voc.n_keys) and np.all(vals >= voc.n_keys)
        q = np.nonzero(lab[b] != mqar.IGNORE)[0]
        assert len(q) == R
        # 1-based positions 2R+1, 2R+3, ...: 0-based even positions from 2R
        assert np.all(q >= 2 * R) and np.all(q % 2 == 0)
        assert sorted(tok[b, q]) == sorted(keys)
        pair = dict(zip(keys, vals))
        for p in q:
            assert lab[b, p] == pair[tok[b, p]]
        assert np.all(lab[b, :2 * R] == mqar.IGNORE)


def test_mqar_full_evaluation_setting_fills_every_slot():
    # R = L/4: the L/4 candidate slots are all query slots
    L = 256
    tok, lab = mqar.mqar_batch(np.random.default_rng(1), 4, L, L // 4)
    for b in range(4):
        assert np.array_equal(np.nonzero(lab[b] != mqar.IGNORE)[0], np.arange(L // 2, L, 2))
    assert mqar.curriculum_pairs(L) == [16, 32, 48, 64]


def test_mqar_rejects_pairs_that_do_not_fit():
    with pytest.raises(ValueError):
        mqar.mqar_batch(np.random.default_rng(0), 1, 64, 17)
