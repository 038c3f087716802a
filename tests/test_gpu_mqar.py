"""MQAR smoke training (App. D.1): a two-layer DART language model, chunk
size 16, state size 16, d_model 64, trained on the first curriculum stage
(L = 256, R = L/16 = 16 pairs) with every DART-layer op -- convolution,
step sizes, scan with its memories, state-memory attention with the gated
residual, gated RMSNorm -- forward and backward in libdart.  The loss must
fall far below its start and the query accuracy must reach recall levels
(chance is 1/64 per query); seeded, about ten seconds on one GPU."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def test_mqar_training_learns_recall():
    import torch
    from paper_2608_02032_amd import layer, mqar
    print("\n[gpu-case] mqar smoke training L=256 R=16 N=16 S=16 d_model=64, 1500 steps", flush=True)
    losses, accs = layer.train_mqar(1500, L=256, R=16, batch=64, d_model=64, d_state=16, chunk=16,
                                    lr=2e-3, seed=0, vocab=mqar.MqarVocab(64, 64), log_every=250)
    torch.cuda.synchronize()
    first = float(np.mean(losses[:10]))
    last = float(np.mean(losses[-100:]))
    acc = float(np.mean(accs[-100:]))
    print("  loss %.3f -> %.3f, query accuracy (last 100 steps) %.3f" % (first, last, acc), flush=True)
    assert np.all(np.isfinite(losses))
    assert last < first - 2.0
    assert acc > 0.5
