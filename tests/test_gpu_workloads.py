"""Every workload at full size against the fp64 oracle, through the C ABI.

Exact indices and accept lengths, floats within 2e-2 + 1e-2 |x| (bf16 outputs) and 1e-3 (lse):
  * the 16K batch (8 x 16,384, GQA 32/8): selection at B = 512 and 1024 under the two-part
    exact-index protocol (decode, verify and acceptance at full size are in the other files);
  * the multiview workload (4 x 8,192, C = 64): its four views selected on the GPU with the block as
    the observation window (W = C = 64, 256 scoring rows per KV head, two row blocks), then the
    multiview forward and backward over exactly those views, every sequence;
  * the ragged paged batch (64 MHA sequences of 4K-16K, 16-token pages): selection, decode over the
    GPU's selection, verify and acceptance, all 64 sequences.
Selection is compared in two parts: (i) the oracle's pooling and ranking applied to the GPU's own
fp32 scores give the GPU's indices bit for bit; (ii) GPU and oracle indices differ only where the
oracle's pooled scores are within a relative 1e-4 of its threshold (near ties, counted).
"""
import functools

import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import (assert_close, assert_lse, bf16_dev, bf16_host64, case, check_selection, config_data,
                       i32_dev, oracle_scores, paged_kv)
from mv_check import _run

pytestmark = pytest.mark.gpu


def _select(kd, q_win, lens, B, **kw):
    idx, nsel, scores = bd.bd_select_kv(kd, bf16_dev(q_win), i32_dev(lens), B, return_scores=True, **kw)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), nsel.cpu().numpy(), scores.cpu().numpy()


# ------------------------------------------------------------------ 16K batch

@functools.lru_cache(maxsize=1)
def _batch16k_scores():
    cfg = synth.workload("16k-collapse-b8")
    qt, k, _ = config_data("16k-collapse-b8")
    return oracle_scores(k, qt[:, -cfg.window:], [cfg.seq_len] * cfg.num_seqs, cfg.num_q_heads)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("B", [512, 1024])
def test_select_batch16k_full_size(B):
    cfg = synth.workload("16k-collapse-b8")
    qt, k, _ = config_data("16k-collapse-b8")
    lens = [cfg.seq_len] * cfg.num_seqs
    case(f"select 16K batch B={B}")
    gi, gn, gs = _select(bf16_dev(k), np.ascontiguousarray(qt[:, -cfg.window:]), lens, B)
    near = check_selection(gi, gn, gs, _batch16k_scores(), lens, cfg.window, B, f"16K batch B={B}",
                           Hq=cfg.num_q_heads)
    assert near <= 4, near


# ------------------------------------------------------------------ multiview workload

@pytest.mark.timeout(300)
def test_multiview_workload_gpu_selected_views_forward_backward():
    cfg = synth.workload("multiview-train-b4-8k")
    qt, k, v = config_data("multiview-train-b4-8k")
    C, S, Hkv = cfg.block_len, cfg.num_seqs, cfg.num_kv_heads
    lens = [cfg.seq_len] * S
    qb = np.ascontiguousarray(qt[:, -C:])
    raws = oracle_scores(k, qb, lens, cfg.num_q_heads)
    budgets = [int(b) for b in synth.view_budgets(cfg)]
    ld = max(budgets)
    idx_v = np.full((len(budgets), S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((len(budgets), S), np.int32)
    kd = bf16_dev(k)
    for i, B in enumerate(budgets):
        case(f"select multiview views W=C={C} B={B}")
        gi, gn, gs = _select(kd, qb, lens, B)
        near = check_selection(gi, gn, gs, raws, lens, C, B, f"view {i} B={B}", Hq=cfg.num_q_heads)
        assert near <= 2, near
        idx_v[i, :, :, :B] = gi
        nsel_v[i] = gn
    # the forward (bf16 and training outputs) and the backward over the GPU's views, every sequence
    _run(k, v, qb, idx_v, nsel_v, lens, "multiview workload, GPU-selected views", seed=11, kdev=kd)


# ------------------------------------------------------------------ ragged paged batch

@functools.lru_cache(maxsize=1)
def _ragged():
    cfg = synth.workload("ragged-paged-b64-mha")
    lens = synth.seq_lens(cfg)
    case("generating the ragged paged batch (64 sequences)")
    qs, ks, vs = synth.kv_batch(cfg, workers=16)
    table, npages = synth.page_table(cfg, lens)
    kd, vd = paged_kv(ks, vs, table, npages, cfg.page_size)
    return cfg, lens, qs, ks, vs, table, kd, vd


@pytest.mark.timeout(600)
def test_ragged_paged_batch_all_sequences():
    """Selection at B = 1024 over the page pool, decode over that selection, verify and acceptance, for
    all 64 sequences (the oracle reads the same sequences unpaged)."""
    cfg, lens, qs, ks, vs, table, kd, vd = _ragged()
    S, W, B = cfg.num_seqs, cfg.window, cfg.budgets[0]
    pt = i32_dev(table)
    q_win = np.stack([q[-W:] for q in qs])
    case("select ragged paged batch, 64 sequences")
    gi, gn, gs = _select(kd, q_win, lens, B, page_table=pt)
    case("oracle scores of the ragged paged batch")
    raws = oracle_scores(ks, q_win, lens, cfg.num_q_heads)
    near = check_selection(gi, gn, gs, raws, lens, W, B, "ragged paged", Hq=cfg.num_q_heads)
    assert near <= 16, near
    del raws, gs

    q = np.stack([x[-1] for x in qs])
    case("decode ragged paged batch over the GPU selection")
    out, lse = bd.bd_sparse_decode_attn(kd, vd, bf16_dev(q), i32_dev(gi), i32_dev(gn), i32_dev(lens),
                                        return_lse=True, page_table=pt)
    torch.cuda.synchronize()
    ro, rl = O.sparse_decode_attn(ks, vs, q, gi, gn, lens)
    assert_close(bf16_host64(out), ro, "ragged paged decode")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, "ragged paged decode")

    g1 = cfg.gamma + 1
    qv = np.stack([x[-g1:] for x in qs])
    case("verify ragged paged batch")
    out, lse = bd.bd_verify_attn(kd, vd, bf16_dev(qv), i32_dev(lens), return_lse=True, page_table=pt)
    torch.cuda.synchronize()
    ro, rl = O.verify_attn(ks, vs, qv, lens, cfg.gamma)
    assert_close(bf16_host64(out), ro, "ragged paged verify")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, "ragged paged verify")

    lg, dr = zip(*[synth.logits_and_drafts(cfg, s)[:2] for s in range(S)])
    lg, dr = np.stack(lg), np.stack(dr)
    case("accept ragged paged batch, vocab 32000")
    acc, bonus, am = bd.bd_accept_len(torch.from_numpy(lg).cuda(), i32_dev(dr), return_argmax=True)
    torch.cuda.synchronize()
    ra, rb, ram = O.accept_len(lg, dr, cfg.gamma)
    assert np.array_equal(acc.cpu().numpy(), ra) and np.array_equal(bonus.cpu().numpy(), rb)
    assert np.array_equal(am.cpu().numpy(), ram)
