"""Seeded sweep of multiview attention shapes against the fp64 oracle (block mode and the split kernel).

Each case draws the number of sequences, KV heads, group size, block length, views, their list
capacity and fill, the sequence lengths (down to shorter than the block) and whether the training
outputs are requested, so that workgroup ranges start and end at every offset of the tile pipeline
(odd and even tile counts, pieces ending between the paired barriers, one-tile and empty ranges) and
views hold absent, out-of-range and repeated entries.  Forward cases also draw the query magnitude
(standard deviation 1, 4 or 16: logits spanning up to tens of nats).  Outputs are poisoned with NaN first, so a row
that is never written fails.  Tolerances as elsewhere: bf16 outputs within 2e-2 + 1e-2 |oracle|, fp32
outputs within 1e-4 max|oracle| + 1e-4 |oracle|, log-sum-exps within 1e-3.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import assert_close, assert_lse, bf16_dev, bf16_host64, case, i32_dev

pytestmark = pytest.mark.gpu


def _draw(seed):
    g = np.random.default_rng(1000 + seed)
    S = int(g.integers(1, 4))
    Hkv = int(g.choice([1, 2, 4]))
    G = int(g.choice([1, 2, 4, 8]))
    C = int(g.integers(8, 97))
    V = int(g.integers(0, 6))
    full = bool(V == 0 or g.random() < 0.8)
    train = bool(g.random() < 0.4)
    lens = [int(g.integers(max(1, C // 2), 2600)) for _ in range(S)]
    ld = int(g.integers(1, 1200))
    idx = np.full((V, S, Hkv, ld), -1, np.int32)
    nsel = np.zeros((V, S), np.int32)
    for i in range(V):
        for s, L in enumerate(lens):
            n = int(g.integers(0, ld + 1))
            for h in range(Hkv):
                if g.random() < 0.7:
                    idx[i, s, h, :n] = np.sort(g.choice(L, min(n, L), replace=False)).tolist() + [-1] * (n - min(n, L))
                else:                               # repeats, absent and out-of-range entries
                    idx[i, s, h, :n] = g.integers(-2, L + 40, n)
            nsel[i, s] = n
    return S, Hkv, G, C, V, full, train, lens, ld, idx, nsel


def _bits(g, shape, sd=1.0):
    return synth.f32_to_bf16_bits((sd * g.standard_normal(shape, dtype=np.float32)).astype(np.float32))


@pytest.mark.parametrize("seed", list(range(16)))
def test_multiview_random_shapes(seed):
    S, Hkv, G, C, V, full, train, lens, ld, idx, nsel = _draw(seed)
    g = np.random.default_rng(2000 + seed)
    Lm = max(lens)
    k, v = _bits(g, (S, Hkv, Lm, 128)), _bits(g, (S, Hkv, Lm, 128))
    qsd = float(g.choice([1.0, 4.0, 16.0]))         # query magnitude: logits spanning up to tens of nats
    qb = _bits(g, (S, C, Hkv * G, 128), qsd)
    Hq = Hkv * G
    nan16 = lambda shape: torch.full(shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    nan32 = lambda shape: torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
    outs = (nan16((V, S, C, Hq, 128)) if V else None, nan16((S, C, Hq, 128)) if full else None,
            nan32((V, S, C, Hq, 128)) if (V and train) else None, nan32((V, S, C, Hq)) if (V and train) else None,
            nan32((S, C, Hq, 128)) if (full and train) else None, nan32((S, C, Hq)) if (full and train) else None)
    what = f"sweep {seed}: S={S} Hkv={Hkv} G={G} C={C} V={V} ld={ld} full={full} train={train} lens={lens} q_sd={qsd}"
    case(what)
    res = bd.bd_multiview_attn(bf16_dev(k), bf16_dev(v), bf16_dev(qb), i32_dev(idx) if V else None,
                               i32_dev(nsel) if V else None, i32_dev(lens), full=full, train=train, outputs=outs)
    torch.cuda.synchronize()
    rv, rf, lv, lf = O.multiview_attn(k, v, qb, list(idx), list(nsel), lens, with_full=full, return_lse=True)
    if V:
        assert_close(bf16_host64(res[0]), rv, what + " views")
    if full:
        assert_close(bf16_host64(res[1]), rf, what + " full")
    if train:
        def close32(gpu, ref, name):
            atol = 1e-4 * max(float(np.abs(ref).max(initial=0.0)), 1e-30)
            assert_close(gpu.double().cpu().numpy(), ref, name, atol=atol, rtol=1e-4)
        if V:
            close32(res[2], rv, what + " views fp32")
            assert_lse(res[3].cpu().numpy(), lv, what + " views lse")
        if full:
            close32(res[4], rf, what + " full fp32")
            assert_lse(res[5].cpu().numpy(), lf, what + " full lse")


def _draw_bwd(seed):
    g = np.random.default_rng(3000 + seed)
    S = int(g.integers(1, 3))
    Hkv = int(g.choice([1, 2]))
    G = int(g.choice([1, 2, 4]))
    C = int(g.integers(8, 300))                    # up to five 64-key passes of the dK/dV kernel
    V = int(g.integers(0, 4))
    full = bool(V == 0 or g.random() < 0.8)
    lens = [int(g.integers(max(1, C // 2), 1600)) for _ in range(S)]
    ld = int(g.integers(1, 900))
    idx = np.full((V, S, Hkv, ld), -1, np.int32)
    nsel = np.zeros((V, S), np.int32)
    for i in range(V):
        for s, L in enumerate(lens):
            n = int(g.integers(0, ld + 1))
            for h in range(Hkv):
                m = min(n, L)
                idx[i, s, h, :n] = np.sort(g.choice(L, m, replace=False)).tolist() + [-1] * (n - m)
            nsel[i, s] = n
    return S, Hkv, G, C, V, full, lens, idx, nsel


@pytest.mark.parametrize("seed", list(range(10)))
def test_multiview_backward_random_shapes(seed):
    """Training forward and backward (dQ over every branch, dK/dV of the block rows) on seeded shapes,
    gradients poisoned with NaN first; dq / dk / dv within 1e-3 max|oracle| + 1e-3 |oracle|."""
    from mv_check import _run
    S, Hkv, G, C, V, full, lens, idx, nsel = _draw_bwd(seed)
    g = np.random.default_rng(4000 + seed)
    Lm = max(lens)
    k, v = _bits(g, (S, Hkv, Lm, 128)), _bits(g, (S, Hkv, Lm, 128))
    qb = _bits(g, (S, C, Hkv * G, 128))
    nan32 = lambda shape: torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")
    grads = (nan32((S, C, Hkv * G, 128)), nan32((S, C, Hkv, 128)), nan32((S, C, Hkv, 128)))
    _run(k, v, qb, idx if V else None, nsel if V else None, lens,
         f"bwd sweep {seed}: S={S} Hkv={Hkv} G={G} C={C} V={V} full={full} lens={lens}", full=full, seed=seed,
         grads=grads)
