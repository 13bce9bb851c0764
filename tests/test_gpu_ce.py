"""GPU parity of bd_top1_ce (Eqs. 5-7) and bd_sample_budgets (Cat(B, w)) against the oracle.

Targets and sampled budgets are integers: exact.  The loss and log-sum-exp are
fp32 accumulations of up to 128K terms (relative error of order 1e-6 on a
log-sum-exp of order 10): |gpu - oracle| <= 1e-4 + 1e-5 |oracle|.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
from gpu_utils import case, i32_dev

pytestmark = pytest.mark.gpu
ATOL, RTOL = 1e-4, 1e-5


def _close(gpu, ref, what):
    gpu = np.asarray(gpu, np.float64)
    bad = np.abs(gpu - ref) > ATOL + RTOL * np.abs(ref)
    assert not bad.any(), (what, np.argwhere(bad)[:4].tolist(), gpu[bad][:4], ref[bad][:4])


@pytest.mark.parametrize("R,V,stride", [(48, 32000, 32000), (6, 128256, 128256), (5, 1001, 1003), (7, 32002, 32004)])
def test_ce_with_teacher(R, V, stride):
    g = np.random.default_rng(R * 7 + V)
    st = np.zeros((R, stride), np.float32)
    te = np.zeros((R, stride), np.float32)
    st[:, :V] = g.standard_normal((R, V)) * 2
    te[:, :V] = np.round(g.standard_normal((R, V)) * 3)          # many ties in the teacher rows
    case(f"ce R={R} V={V} stride={stride}")
    sd, td = torch.from_numpy(st).cuda()[:, :V], torch.from_numpy(te).cuda()[:, :V]
    loss, tgt, lse = bd.bd_top1_ce(sd, teacher=td, return_targets=True, return_lse=True)
    torch.cuda.synchronize()
    ol, ot, ols = O.top1_ce(st[:, :V], teacher=te[:, :V])
    assert tgt.cpu().tolist() == ot.tolist()
    _close(loss.cpu().numpy(), ol, "loss")
    _close(lse.cpu().numpy(), ols, "lse")


def test_ce_with_given_targets_and_invalid_entries():
    R, V = 9, 50000
    g = np.random.default_rng(3)
    st = (g.standard_normal((R, V)) * 4).astype(np.float32)
    tg = g.integers(0, V, R).astype(np.int32)
    tg[2], tg[5] = -1, V                                           # outside the vocabulary
    case("ce with given targets")
    loss, tgt = bd.bd_top1_ce(torch.from_numpy(st).cuda(), targets=i32_dev(tg), return_targets=True)
    torch.cuda.synchronize()
    ok = np.ones(R, bool)
    ok[[2, 5]] = False
    ol, _, _ = O.top1_ce(st[ok], targets=tg[ok])
    got = loss.cpu().numpy()
    _close(got[ok], ol, "loss")
    assert np.isnan(got[~ok]).all()
    assert tgt.cpu().numpy()[~ok].tolist() == [-1, -1] and tgt.cpu().numpy()[ok].tolist() == tg[ok].tolist()


def test_ce_uniform_rows_give_log_vocab():
    R, V = 4, 32000
    case("ce uniform")
    loss = bd.bd_top1_ce(torch.zeros((R, V), device="cuda"), targets=i32_dev([0, 1, 31999, 17]))
    torch.cuda.synchronize()
    _close(loss.cpu().numpy(), np.full(R, np.log(V)), "uniform")


def test_sample_budgets_matches_oracle_exactly():
    budgets, w = [256, 512, 1024, 2048], [0.4, 0.3, 0.2, 0.1]
    thr = O.budget_thresholds(w)
    u = np.random.default_rng(4).random(100000).astype(np.float32)
    edge = np.concatenate([thr, [np.nextafter(t, np.float32(0)) for t in thr], [0.0, np.nextafter(np.float32(1), np.float32(0))]])
    u = np.concatenate([u, edge.astype(np.float32)])
    case("sample budgets")
    got = bd.bd_sample_budgets(torch.from_numpy(u).cuda(), budgets, w)
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy(), O.sample_budgets(u, budgets, w))
