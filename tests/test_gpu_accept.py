"""GPU parity of bd_accept_len: bit-exact accepted lengths, bonus tokens and argmax."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import case, dev, i32_dev

pytestmark = pytest.mark.gpu


def _run(logits: np.ndarray, draft: np.ndarray, what: str):
    case(f"accept {what}")
    lg = torch.from_numpy(np.ascontiguousarray(logits, dtype=np.float32)).to(dev())
    acc, bonus, am = bd.bd_accept_len(lg, i32_dev(draft), return_argmax=True)
    torch.cuda.synchronize()
    ra, rb, ram = O.accept_len(logits, draft, draft.shape[1])
    assert np.array_equal(am.cpu().numpy(), ram), what
    assert np.array_equal(acc.cpu().numpy(), ra), what
    assert np.array_equal(bonus.cpu().numpy(), rb), what
    return ra


@pytest.mark.parametrize("name", ["tiny-4k-gqa4", "16k-collapse-b8"])
def test_accept_workloads(name):
    cfg = synth.workload(name)
    data = [synth.logits_and_drafts(cfg, s) for s in range(cfg.num_seqs)]
    logits = np.stack([d[0] for d in data])
    draft = np.stack([d[1] for d in data])
    ra = _run(logits, draft, name)
    assert ra.tolist() == [d[3] for d in data]                # planted prefix lengths


def test_accept_ties_signed_zero_and_gamma0():
    g = np.random.default_rng(7)
    S, gamma, V = 5, 4, 3001
    logits = np.floor(g.standard_normal((S, gamma + 1, V)) * 1.5).astype(np.float32)   # heavy ties
    logits[0, 0, :] = -1.0
    logits[0, 0, 1500] = -0.0
    logits[0, 0, 2999] = 0.0                                  # +0 ties -0: lowest index wins
    draft = g.integers(0, 3, (S, gamma)).astype(np.int32)
    am = np.array([[O.greedy_argmax(logits[s, i]) for i in range(gamma + 1)] for s in range(S)])
    draft[1] = am[1, :gamma]                                  # fully accepted sequence
    draft[2, :2] = am[2, :2]
    _run(logits, draft, "ties")
    _run(logits[:, :1], np.zeros((S, 0), np.int32), "gamma 0")


def test_accept_unaligned_rows_and_small_vocab():
    g = np.random.default_rng(8)
    for V in [1, 3, 1023, 4099]:
        logits = g.standard_normal((3, 3, V)).astype(np.float32)
        draft = g.integers(0, V, (3, 2)).astype(np.int32)
        _run(logits, draft, f"V={V}")
