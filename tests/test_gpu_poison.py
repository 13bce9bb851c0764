"""Every output element is written, and no scratch is read before it is written.

Before each call the outputs are filled with NaN (index outputs with a sentinel) and the workspace
past its counter region with 0xFF bytes (NaN as fp32).  The results must still match the oracle
element by element (a NaN fails every tolerance check), so a row, head, split or record that a
kernel skipped -- or scratch it read before writing -- shows up here.  The shapes take the split,
record and merge paths: several key splits per unit, block mode with partial records, paged caches,
multiple row blocks in selection.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import (assert_close, assert_lse, bf16_dev, bf16_host64, case, check_chunk_selection, check_selection,
                       config_data, i32_dev, oracle_chunk_selection, oracle_scores, paged_kv, poison_workspace)
from mv_check import _rand_bits, _run

pytestmark = pytest.mark.gpu

WS_BYTES = 512 << 20           # one poisoned workspace, larger than any call here requests
SENTINEL = 0x7FFFFFF0


def _nan(shape, dtype):
    return torch.full(shape, float("nan"), dtype=dtype, device="cuda")


def _sent(shape):
    return torch.full(shape, SENTINEL, dtype=torch.int32, device="cuda")


def test_poisoned_selection_token_and_chunks():
    cfg = synth.workload("multiview-train-b4-8k")
    qt, k, _ = config_data("multiview-train-b4-8k")
    S, Hkv, C = 2, cfg.num_kv_heads, cfg.block_len
    k = k[:S]
    lens = [cfg.seq_len, 5000]                     # the second sequence is shorter than the buffer
    qb = np.ascontiguousarray(qt[:S, -C:])        # 64 rows x G 4: two row blocks per KV head
    raws = oracle_scores(k, qb, lens, cfg.num_q_heads)
    kd = bf16_dev(k)
    ws = poison_workspace(WS_BYTES)
    for B in (256, 2048):
        case(f"poisoned token selection B={B}")
        outs = (_sent((S, Hkv, B)), _sent((S,)), _nan((S, Hkv, cfg.seq_len), torch.float32))
        idx, nsel, sc = bd.bd_select_kv(kd, bf16_dev(qb), i32_dev(lens), B, return_scores=True, workspace=ws,
                                        outputs=outs)
        torch.cuda.synchronize()
        gi, gn, gs = idx.cpu().numpy(), nsel.cpu().numpy(), sc.cpu().numpy()
        assert not np.isnan(gs[0]).any() and not np.isnan(gs[1, :, :lens[1]]).any()
        check_selection(gi, gn, gs, raws, lens, C, B, f"poisoned token B={B}", Hq=cfg.num_q_heads)
        case(f"poisoned chunk selection B={B}")
        outs = (_sent((S, Hkv, B + C)), _sent((S,)), _nan((S, Hkv, cfg.seq_len), torch.float32))
        idx, nsel, sc = bd.bd_select_kv_chunks(kd, bf16_dev(qb), i32_dev(lens), B, chunk=8, return_scores=True,
                                               workspace=ws, outputs=outs)
        torch.cuda.synchronize()
        gi, gn, gs = idx.cpu().numpy(), nsel.cpu().numpy(), sc.cpu().numpy()
        oi, on = oracle_chunk_selection(raws, lens, Hkv, C, B, 8, False)
        check_chunk_selection(gi, gn, gs, oi, on, raws, lens, C, B, 8, False, f"poisoned chunks B={B}")


def test_poisoned_decode_and_verify_16k_batch():
    cfg = synth.workload("16k-collapse-b8")
    qt, k, v = config_data("16k-collapse-b8")
    S, Hq, Hkv, L = cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.seq_len
    lens = [L] * S
    kd, vd = bf16_dev(k), bf16_dev(v)
    ws = poison_workspace(WS_BYTES)
    g = np.random.default_rng(5)
    B = 1024
    idx = np.stack([np.stack([np.sort(g.choice(L, B, replace=False)) for _ in range(Hkv)]) for _ in range(S)])
    idx = idx.astype(np.int32)
    case("poisoned decode 16K batch B=1024")
    out, lse = bd.bd_sparse_decode_attn(kd, vd, bf16_dev(qt[:, -1]), i32_dev(idx), i32_dev([B] * S), i32_dev(lens),
                                        return_lse=True, workspace=ws, out=_nan((S, Hq, 128), torch.bfloat16),
                                        lse=_nan((S, Hq), torch.float32))
    torch.cuda.synchronize()
    ro, rl = O.sparse_decode_attn(k, v, qt[:, -1], idx, [B] * S, lens)
    assert_close(bf16_host64(out), ro, "poisoned decode")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, "poisoned decode")
    g1 = cfg.gamma + 1
    case("poisoned verify 16K batch")
    out, lse = bd.bd_verify_attn(kd, vd, bf16_dev(qt[:, -g1:]), i32_dev(lens), return_lse=True, workspace=ws,
                                 out=_nan((S, g1, Hq, 128), torch.bfloat16), lse=_nan((S, g1, Hq), torch.float32))
    torch.cuda.synchronize()
    ro, rl = O.verify_attn(k, v, qt[:, -g1:], lens, cfg.gamma)
    assert_close(bf16_host64(out), ro, "poisoned verify")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, "poisoned verify")


@pytest.mark.parametrize("Hq,Hkv,gamma,paged", [(16, 2, 5, False), (8, 2, 5, True), (32, 32, 5, True), (8, 2, 0, False)])
def test_poisoned_verify_and_decode_ragged(Hq, Hkv, gamma, paged):
    # ragged lengths (one shorter than gamma + 1 rows would need), block mode (48 rows per KV head),
    # paged caches, empty decode sets
    lens = [3000, 1700, gamma + 1, 40]
    S, P = len(lens), 16
    ks = [_rand_bits((Hkv, L, 128), 300 + s) for s, L in enumerate(lens)]
    vs = [_rand_bits((Hkv, L, 128), 400 + s) for s, L in enumerate(lens)]
    q = _rand_bits((S, gamma + 1, Hq, 128), 500)
    if paged:
        maxp = (max(lens) + P - 1) // P
        npages = sum((L + P - 1) // P for L in lens)
        perm = np.random.default_rng(501).permutation(npages)
        table = np.full((S, maxp), -1, np.int32)
        c = 0
        for s, L in enumerate(lens):
            n = (L + P - 1) // P
            table[s, :n] = perm[c:c + n]
            c += n
        kd, vd = paged_kv(ks, vs, table, npages, P)
        pt = i32_dev(table)
    else:
        Lm = max(lens)
        kc = np.zeros((S, Hkv, Lm, 128), np.uint16)
        vc = np.zeros_like(kc)
        for s, L in enumerate(lens):
            kc[s, :, :L], vc[s, :, :L] = ks[s], vs[s]
        kd, vd, pt = bf16_dev(kc), bf16_dev(vc), None
    ws = poison_workspace(WS_BYTES)
    g1 = gamma + 1
    case(f"poisoned verify ragged Hq={Hq} Hkv={Hkv} gamma={gamma} paged={paged}")
    out, lse = bd.bd_verify_attn(kd, vd, bf16_dev(q), i32_dev(lens), return_lse=True, workspace=ws, page_table=pt,
                                 max_seq_len=max(lens), out=_nan((S, g1, Hq, 128), torch.bfloat16),
                                 lse=_nan((S, g1, Hq), torch.float32))
    torch.cuda.synchronize()
    ro, rl = O.verify_attn(ks, vs, q, lens, gamma)
    assert_close(bf16_host64(out), ro, "poisoned ragged verify")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, "poisoned ragged verify")
    ld = 900
    g = np.random.default_rng(502)
    idx = np.full((S, Hkv, ld), -1, np.int32)
    nsel = [900, 600, 0, 40]
    for s, L in enumerate(lens):
        n = min(nsel[s], L)
        for h in range(Hkv):
            idx[s, h, :n] = g.choice(L, n, replace=False)
    qd = np.ascontiguousarray(q[:, -1])
    case(f"poisoned decode ragged Hq={Hq} Hkv={Hkv} paged={paged}")
    out, lse = bd.bd_sparse_decode_attn(kd, vd, bf16_dev(qd), i32_dev(idx), i32_dev(nsel), i32_dev(lens),
                                        return_lse=True, workspace=ws, page_table=pt, max_seq_len=max(lens),
                                        out=_nan((S, Hq, 128), torch.bfloat16), lse=_nan((S, Hq), torch.float32))
    torch.cuda.synchronize()
    ro, rl = O.sparse_decode_attn(ks, vs, qd, idx, nsel, lens)
    assert_close(bf16_host64(out), ro, "poisoned ragged decode")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, "poisoned ragged decode")


def test_poisoned_multiview_forward_and_backward():
    """The multiview workload (views and full branch, training outputs) and its backward with every
    output and gradient pre-filled with NaN and the shared workspace poisoned."""
    cfg = synth.workload("multiview-train-b4-8k")
    qt, k, v = config_data("multiview-train-b4-8k")
    C, S, Hq, Hkv, L = cfg.block_len, cfg.num_seqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.seq_len
    budgets = [int(b) for b in synth.view_budgets(cfg)]
    V, ld = len(budgets), max(budgets)
    idx_v = np.full((V, S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((V, S), np.int32)
    for i, B in enumerate(budgets):
        for s in range(S):
            for h in range(Hkv):
                idx_v[i, s, h, :B] = np.r_[synth.random_index_set(cfg.config_id, s, h, L - C, B - C, tag_extra=7),
                                           np.arange(L - C, L)]
        nsel_v[i] = B
    f32, b16 = torch.float32, torch.bfloat16
    outputs = (_nan((V, S, C, Hq, 128), b16), _nan((S, C, Hq, 128), b16), _nan((V, S, C, Hq, 128), f32),
               _nan((V, S, C, Hq), f32), _nan((S, C, Hq, 128), f32), _nan((S, C, Hq), f32))
    grads = (_nan((S, C, Hq, 128), f32), _nan((S, C, Hkv, 128), f32), _nan((S, C, Hkv, 128), f32))
    _run(k, v, np.ascontiguousarray(qt[:, -C:]), idx_v, nsel_v, [L] * S, "poisoned multiview", seed=13,
         workspace=poison_workspace(WS_BYTES), outputs=outputs, grads=grads)


def test_poisoned_multiview_views_only_small_rows():
    """Views only, 24 rows per KV head (the split path rather than block mode), ragged lengths."""
    S, Hkv, G, C = 3, 2, 4, 6
    lens = [2500, 900, 6]
    Lm = max(lens)
    k, v = _rand_bits((S, Hkv, Lm, 128), 600), _rand_bits((S, Hkv, Lm, 128), 601)
    qb = _rand_bits((S, C, Hkv * G, 128), 602)
    g = np.random.default_rng(603)
    V, ld = 3, 700
    idx_v = np.full((V, S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((V, S), np.int32)
    for i in range(V):
        for s, L in enumerate(lens):
            n = min([700, 300, 0][i], L)
            for h in range(Hkv):
                idx_v[i, s, h, :n] = np.sort(g.choice(L, n, replace=False))
            nsel_v[i, s] = n
    ws = poison_workspace(WS_BYTES)
    case("poisoned multiview, views only, split path")
    ov, of = bd.bd_multiview_attn(bf16_dev(k), bf16_dev(v), bf16_dev(qb), i32_dev(idx_v), i32_dev(nsel_v),
                                  i32_dev(lens), full=False, workspace=ws,
                                  outputs=(_nan((V, S, C, Hkv * G, 128), torch.bfloat16),))
    torch.cuda.synchronize()
    assert of is None
    rv, _ = O.multiview_attn(k, v, qb, list(idx_v), list(nsel_v), lens, with_full=False)
    assert_close(bf16_host64(ov), rv, "poisoned views only")


def test_poisoned_accept():
    cfg = synth.workload("16k-collapse-b8")
    S, g1 = cfg.num_seqs, cfg.gamma + 1
    lg, dr = zip(*[synth.logits_and_drafts(cfg, s)[:2] for s in range(S)])
    lg, dr = np.stack(lg), np.stack(dr)
    case("poisoned accept 16K batch")
    acc, bonus, am = bd.bd_accept_len(torch.from_numpy(lg).cuda(), i32_dev(dr), return_argmax=True,
                                      workspace=poison_workspace(WS_BYTES),
                                      outputs=(_sent((S,)), _sent((S,)), _sent((S, g1))))
    torch.cuda.synchronize()
    ra, rb, ram = O.accept_len(lg, dr, cfg.gamma)
    assert np.array_equal(acc.cpu().numpy(), ra) and np.array_equal(bonus.cpu().numpy(), rb)
    assert np.array_equal(am.cpu().numpy(), ram)
