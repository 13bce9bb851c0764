"""GPU parity of the per-round cache updates (bd_cache_append, bd_cache_rollback) against the oracle.

Byte and integer work: every comparison is exact.  The last test runs one round
of Alg. 2 through the C ABI (select, gamma drafts with appends, verifier rows,
verify, accept, rollback of both caches) and checks each attention output and
the final lengths against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import assert_close, bf16_dev, bf16_host64, case, i32_dev

pytestmark = pytest.mark.gpu


def _bits(shape, seed):
    g = np.random.default_rng(seed)
    return synth.f32_to_bf16_bits(g.standard_normal(shape).astype(np.float32))


def _u16(t):
    return t.cpu().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("n", [8, 40])
def test_append_matches_oracle_with_clamps(n):
    # 8 rows: one launch (a workgroup per sequence); 40 rows: a workgroup per row and a second launch
    S, Hkv, cap, ld = 3, 2, 100, 20
    k, v = _bits((S, Hkv, cap, 128), 1), _bits((S, Hkv, cap, 128), 2)
    kn, vn = _bits((S, n, Hkv, 128), 3), _bits((S, n, Hkv, 128), 4)
    lens, nsel = [10, 95, 100], [5, 15, 18]
    idx = np.full((S, Hkv, ld), -1, np.int32)
    for s in range(S):
        idx[s, :, :nsel[s]] = np.arange(nsel[s])
    ok, ov, ol, oi, on = O.cache_append(k, v, lens, kn, vn, idx, nsel)
    case(f"append of {n} rows with capacity and list clamps")
    kd, vd, ld_, idd, nd = bf16_dev(k), bf16_dev(v), i32_dev(lens), i32_dev(idx), i32_dev(nsel)
    bd.bd_cache_append(kd, vd, ld_, bf16_dev(kn), bf16_dev(vn), idx=idd, nsel=nd)
    torch.cuda.synchronize()
    assert np.array_equal(_u16(kd), ok) and np.array_equal(_u16(vd), ov)
    assert ld_.cpu().tolist() == ol.tolist() == [10 + n, 100, 100]
    assert np.array_equal(idd.cpu().numpy(), oi) and nd.cpu().tolist() == on.tolist() == [min(5 + n, 20), 20, 18]


@pytest.mark.parametrize("n", [5, 20])
def test_append_paged_layout(n):
    S, Hkv, page, pages_per_seq = 2, 2, 16, 4
    num_pages = S * pages_per_seq
    g = np.random.default_rng(5)
    perm = g.permutation(num_pages).astype(np.int32)
    table = perm.reshape(S, pages_per_seq)
    pool_k, pool_v = _bits((num_pages, Hkv, page, 128), 6), _bits((num_pages, Hkv, page, 128), 7)
    kn, vn = _bits((S, n, Hkv, 128), 8), _bits((S, n, Hkv, 128), 9)
    lens = [30, 61]
    case("append into a paged cache")
    kd, vd, ld_ = bf16_dev(pool_k), bf16_dev(pool_v), i32_dev(lens)
    bd.bd_cache_append(kd, vd, ld_, bf16_dev(kn), bf16_dev(vn), page_table=i32_dev(table))
    torch.cuda.synchronize()
    # logical view of the pool before and after, compared with the oracle on that view
    def logical(pool):
        return np.stack([np.concatenate([pool[table[s, p]] for p in range(pages_per_seq)], axis=1) for s in range(S)])
    ok, ov, ol = O.cache_append(logical(pool_k), logical(pool_v), lens, kn, vn)
    assert np.array_equal(logical(_u16(kd)), ok) and np.array_equal(logical(_u16(vd)), ov)
    assert ld_.cpu().tolist() == ol.tolist() == [30 + n, 64]


def test_rollback_matches_oracle():
    lens, nsel, acc = [100, 100, 100, 3, 50], [20, 20, 20, 1, 9], [0, 2, 5, 9, -1]
    ol, on = O.cache_rollback(lens, acc, 5, nsel=nsel)
    case("rollback")
    ld_, nd = i32_dev(lens), i32_dev(nsel)
    bd.bd_cache_rollback(ld_, i32_dev(acc), 5, nsel=nd)
    torch.cuda.synchronize()
    assert ld_.cpu().tolist() == ol.tolist() and nd.cpu().tolist() == on.tolist()


def test_rollback_from_base_lengths_matches_oracle():
    lens, nsel, acc = [100, 100, 100, 3, 50, 64], [20, 20, 20, 1, 9, 64], [0, 2, 5, 9, -1, 3]
    base_l, base_n = [95, 97, 99, 0, 45, 64], [15, 18, 20, 0, 9, 62]
    ol, on = O.cache_rollback(lens, acc, 5, nsel=nsel, base_lens=base_l, base_nsel=base_n)
    case("rollback from base lengths")
    ld_, nd = i32_dev(lens), i32_dev(nsel)
    bd.bd_cache_rollback(ld_, i32_dev(acc), 5, nsel=nd, base_lens=i32_dev(base_l), base_nsel=i32_dev(base_n))
    torch.cuda.synchronize()
    assert ld_.cpu().tolist() == ol.tolist() and nd.cpu().tolist() == on.tolist()


def test_rounds_that_fill_the_list_and_the_cache():
    """Several rounds of speculative appends and rollbacks (from the lengths before each round) on a
    drafter list of fixed width and caches of fixed capacity: the list fills after a few rounds and the
    caches reach their capacity, and GPU lengths, lists and bytes follow the oracle round by round."""
    S, Hkv, cap, gamma, ld = 3, 2, 60, 4, 24
    g = np.random.default_rng(70)
    k, v = _bits((S, Hkv, cap, 128), 71), _bits((S, Hkv, cap, 128), 72)
    lens0, nsel0 = [30, 44, 52], [12, 16, 20]
    idx = np.full((S, Hkv, ld), -1, np.int32)
    for s in range(S):
        idx[s, :, :nsel0[s]] = np.sort(g.choice(lens0[s], nsel0[s], replace=False))
    kd, vd, lensd, idxd, nseld = bf16_dev(k), bf16_dev(v), i32_dev(lens0), i32_dev(idx), i32_dev(nsel0)
    ok, ov, ol, oi, on = k.copy(), v.copy(), np.array(lens0, np.int32), idx.copy(), np.array(nsel0, np.int32)
    for r in range(6):
        base_l, base_n = lensd.clone(), nseld.clone()
        ob_l, ob_n = ol.copy(), on.copy()
        for i in range(gamma):
            kn, vn = _bits((S, 1, Hkv, 128), 100 + 10 * r + i), _bits((S, 1, Hkv, 128), 200 + 10 * r + i)
            case(f"rounds: round {r} append {i}")
            bd.bd_cache_append(kd, vd, lensd, bf16_dev(kn), bf16_dev(vn), idx=idxd, nsel=nseld)
            ok, ov, ol, oi, on = O.cache_append(ok, ov, ol, kn, vn, oi, on)
        acc = g.integers(0, gamma + 1, size=S).astype(np.int32)
        bd.bd_cache_rollback(lensd, i32_dev(acc), gamma, nsel=nseld, base_lens=base_l, base_nsel=base_n)
        ol, on = O.cache_rollback(ol, acc, gamma, nsel=on, base_lens=ob_l, base_nsel=ob_n)
        torch.cuda.synchronize()
        assert lensd.cpu().tolist() == ol.tolist(), r
        assert nseld.cpu().tolist() == on.tolist(), r
        gi = idxd.cpu().numpy()
        for s in range(S):
            assert np.array_equal(gi[s, :, :on[s]], oi[s, :, :on[s]]), (r, s)
        assert np.array_equal(_u16(kd), ok) and np.array_equal(_u16(vd), ov)
    assert on.max() == ld and ol.max() == cap          # both limits were reached


def test_one_speculative_round_of_alg2():
    S, Hq, Hkv, L0, W, B, gamma = 2, 8, 2, 300, 16, 64, 4
    cap = L0 + gamma + 1
    g = np.random.default_rng(10)
    kS, vS = _bits((S, Hkv, cap, 128), 11), _bits((S, Hkv, cap, 128), 12)     # drafter cache (rows >= L0 unused)
    kL, vL = _bits((S, Hkv, cap, 128), 13), _bits((S, Hkv, cap, 128), 14)     # verifier cache
    q_win = _bits((S, W, Hq, 128), 15)
    lens0 = [L0, L0 - 7]
    dS_k, dS_v, dL_k, dL_v = bf16_dev(kS), bf16_dev(vS), bf16_dev(kL), bf16_dev(vL)
    lensS, lensL = i32_dev(lens0), i32_dev(lens0)
    case("round: select")
    idx_sel, nsel_sel = bd.bd_select_kv(dS_k, bf16_dev(q_win), lensS, B)
    ld = B + gamma
    idx = torch.full((S, Hkv, ld), -1, dtype=torch.int32, device=idx_sel.device)
    idx[:, :, :B] = idx_sel
    nsel = nsel_sel.clone()
    oi, on, _ = O.select_kv(kS, q_win, lens0, Hq, W, B)
    o_idx = np.full((S, Hkv, ld), -1, np.int32)
    o_idx[:, :, :B] = oi
    o_nsel, o_lensS = on.copy(), np.array(lens0, np.int32)
    ok, ov = kS.copy(), vS.copy()
    torch.cuda.synchronize()
    assert np.array_equal(idx_sel.cpu().numpy(), oi)          # exact at this size (no near-ties)
    # gamma drafts: decode with the current list, then append the drafted token's row
    for i in range(gamma):
        q = _bits((S, Hq, 128), 20 + i)
        case(f"round: draft {i}")
        out = bd.bd_sparse_decode_attn(dS_k, dS_v, bf16_dev(q), idx, nsel, lensS)
        torch.cuda.synchronize()
        ro, _ = O.sparse_decode_attn(ok, ov, q, o_idx, o_nsel, o_lensS)
        assert_close(bf16_host64(out), ro, f"draft {i}")
        kn, vn = _bits((S, 1, Hkv, 128), 30 + i), _bits((S, 1, Hkv, 128), 40 + i)
        bd.bd_cache_append(dS_k, dS_v, lensS, bf16_dev(kn), bf16_dev(vn), idx=idx, nsel=nsel)
        ok, ov, o_lensS, o_idx, o_nsel = O.cache_append(ok, ov, o_lensS, kn, vn, o_idx, o_nsel)
    # the verifier appends the committed token and the gamma drafts, then attends them
    kn, vn = _bits((S, gamma + 1, Hkv, 128), 50), _bits((S, gamma + 1, Hkv, 128), 51)
    bd.bd_cache_append(dL_k, dL_v, lensL, bf16_dev(kn), bf16_dev(vn))
    okL, ovL, o_lensL = O.cache_append(kL, vL, lens0, kn, vn)
    qv = _bits((S, gamma + 1, Hq, 128), 52)
    case("round: verify")
    outv = bd.bd_verify_attn(dL_k, dL_v, bf16_dev(qv), lensL)
    torch.cuda.synchronize()
    assert lensL.cpu().tolist() == o_lensL.tolist()
    rv, _ = O.verify_attn(okL, ovL, qv, o_lensL, gamma)
    assert_close(bf16_host64(outv), rv, "verify")
    # accept: planted greedy tokens make sequence s accept s+1 drafts
    V = 1000
    logits = g.standard_normal((S, gamma + 1, V)).astype(np.float32)
    am = g.integers(0, V, size=(S, gamma + 1))
    for s in range(S):
        for r in range(gamma + 1):
            logits[s, r, am[s, r]] = 9.0
    draft = am[:, :gamma].astype(np.int32).copy()
    for s in range(S):
        if s + 1 < gamma:
            draft[s, s + 1] = (am[s, s + 1] + 1) % V
    acc, _ = bd.bd_accept_len(torch.from_numpy(logits).cuda(), i32_dev(draft))
    oacc, _, _ = O.accept_len(logits, draft, gamma)
    torch.cuda.synchronize()
    assert acc.cpu().tolist() == oacc.tolist() == [1, 2]
    # rollback: the verifier's gamma draft rows are speculative; the drafter's appended rows are the
    # committed token and gamma-1 drafts, so gamma-1 of them are speculative
    case("round: rollback")
    bd.bd_cache_rollback(lensL, acc, gamma)
    bd.bd_cache_rollback(lensS, acc, gamma - 1, nsel=nsel)
    torch.cuda.synchronize()
    assert lensL.cpu().tolist() == O.cache_rollback(o_lensL, oacc, gamma).tolist()
    rl, rn = O.cache_rollback(o_lensS, oacc, gamma - 1, nsel=o_nsel)
    assert lensS.cpu().tolist() == rl.tolist() and nsel.cpu().tolist() == rn.tolist()
    assert lensL.cpu().tolist() == [L0 + 1 + 1, L0 - 7 + 1 + 2]
