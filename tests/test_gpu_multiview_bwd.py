"""GPU parity of bd_multiview_attn_bwd (and the forward's training outputs it consumes)
against the fp64 oracle, through the C ABI.

The backward takes the GPU forward's fp32 training outputs and log-sum-exps, as
a training step would; the oracle recomputes everything in fp64 from the same
bf16 inputs.  Tolerance: the kernels keep P and dS as bf16 pairs (relative
error about 2^-17) and accumulate in fp32, and the forward's fp32 output
carries its weights to about 2^-17, so an element's error is a few 1e-6 of
the sum of its terms' magnitudes.  The test bound |gpu - oracle| <=
1e-3 * max|oracle| + 1e-3 * |oracle| (per tensor) leaves a wide margin over
that and is far inside the 2e-2 + 1e-2 |x| bound of the path's outputs.
The fp32 forward outputs are held to 1e-4 * max|O| + 1e-4 |O|.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import (bf16_dev, case, check_chunk_selection, config_data, i32_dev, oracle_chunk_selection,
                       oracle_scores, paged_kv)
from mv_check import _rand_bits, _run

pytestmark = pytest.mark.gpu

def _selected_views(k, qb, lens, Hq, C, budgets):
    S, Hkv = k.shape[0], k.shape[1]
    ld = max(budgets)
    idx_v = np.full((len(budgets), S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((len(budgets), S), np.int32)
    for i, B in enumerate(budgets):
        idx, nsel, _ = O.select_kv(k, qb, lens, Hq, C, B)
        idx_v[i, :, :, :idx.shape[2]] = idx
        nsel_v[i] = nsel
    return idx_v, nsel_v


def test_bwd_small_selected_views_and_full():
    S, Hkv, G, L, C = 2, 2, 4, 1500, 64
    k, v = _rand_bits((S, Hkv, L, 128), 20), _rand_bits((S, Hkv, L, 128), 21)
    qb = _rand_bits((S, C, Hkv * G, 128), 22)
    idx_v, nsel_v = _selected_views(k, qb, [L, L], Hkv * G, C, [128, 256, 1024, 2048])
    _run(k, v, qb, idx_v, nsel_v, [L, L], "small", seed=1)


def test_bwd_block_above_64_rows():
    """C = 100 with G = 2: 7 key tiles of 16 (two passes over the dK/dV kernel's 4 key tiles per wave
    group) and 7 row tiles of 32 (an odd count, so the second wave group's last tile is padding)."""
    S, Hkv, G, L, C = 2, 2, 2, 1200, 100
    k, v = _rand_bits((S, Hkv, L, 128), 60), _rand_bits((S, Hkv, L, 128), 61)
    qb = _rand_bits((S, C, Hkv * G, 128), 62)
    idx_v, nsel_v = _selected_views(k, qb, [L, L], Hkv * G, C, [256, 512])
    _run(k, v, qb, idx_v, nsel_v, [L, L], "C=100 G=2", seed=6)


def test_bwd_ragged_lengths_odd_block_and_group():
    """C = 13 rows with G = 3 (39 rows per head: a ragged 32-row block), ragged L, one L below C."""
    S, Hkv, G, C = 3, 2, 3, 13
    lens = [900, 10, 377]
    Lm = max(lens)
    k, v = _rand_bits((S, Hkv, Lm, 128), 30), _rand_bits((S, Hkv, Lm, 128), 31)
    qb = _rand_bits((S, C, Hkv * G, 128), 32)
    g = np.random.default_rng(33)
    ld = 300
    idx_v = np.full((2, S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((2, S), np.int32)
    for s, L in enumerate(lens):
        for h in range(Hkv):
            a = np.sort(g.choice(L, min(L, 200), replace=False))
            idx_v[0, s, h, :len(a)] = a
            b = np.r_[g.choice(L, min(L, 150), replace=False), np.arange(max(0, L - C), L)]
            idx_v[1, s, h, :len(b)] = g.permutation(b)          # unsorted entries
        nsel_v[0, s] = min(L, 200)
        nsel_v[1, s] = min(L, 150) + min(L, C)
    _run(k, v, qb, idx_v, nsel_v, lens, "ragged C=13 G=3", seed=2)


def test_bwd_duplicates_absent_and_out_of_range_entries():
    """Entries -1, >= L and beyond nsel are skipped; a listed key counts as often as it is listed."""
    S, Hkv, G, L, C = 1, 1, 8, 600, 32
    k, v = _rand_bits((S, Hkv, L, 128), 40), _rand_bits((S, Hkv, L, 128), 41)
    qb = _rand_bits((S, C, Hkv * G, 128), 42)
    row = np.r_[np.arange(0, 400, 3), [-1, L, L + 7, 5, 5, L - 1, L - 1, L - 1, L - 2], np.arange(L - C, L)]
    idx_v = np.full((1, S, Hkv, len(row) + 40), 123, np.int32)   # slots past nsel hold a valid-looking key
    idx_v[0, 0, 0, :len(row)] = row
    nsel_v = np.array([[len(row)]], np.int32)
    _run(k, v, qb, idx_v, nsel_v, [L], "duplicates", seed=3)
    _run(k, v, qb, idx_v, nsel_v, [L], "duplicates views only", full=False, seed=4)


def test_bwd_single_branch_paths():
    """One view and no full branch (no partial records at all), then the full branch alone."""
    S, Hkv, G, L, C = 2, 2, 2, 700, 16
    k, v = _rand_bits((S, Hkv, L, 128), 50), _rand_bits((S, Hkv, L, 128), 51)
    qb = _rand_bits((S, C, Hkv * G, 128), 52)
    idx_v, nsel_v = _selected_views(k, qb, [L, L], Hkv * G, C, [128])
    _run(k, v, qb, idx_v, nsel_v, [L, L], "one view", full=False, seed=5)
    _run(k, v, qb, None, None, [L, L], "full only", seed=6)
    _run(k, v, qb, None, None, [L, L], "full only, dq only", seed=6, with_dkv=False)


def test_bwd_paged_cache():
    S, Hkv, G, C, P = 3, 2, 4, 32, 16
    lens = [1000, 517, 64]
    k = [_rand_bits((Hkv, L, 128), 60 + s) for s, L in enumerate(lens)]
    v = [_rand_bits((Hkv, L, 128), 70 + s) for s, L in enumerate(lens)]
    qb = _rand_bits((S, C, Hkv * G, 128), 80)
    g = np.random.default_rng(81)
    maxp = (max(lens) + P - 1) // P
    npages = sum((L + P - 1) // P for L in lens) + 5
    perm = g.permutation(npages)
    table = np.zeros((S, maxp), np.int32)
    c = 0
    for s, L in enumerate(lens):
        n = (L + P - 1) // P
        table[s, :n] = perm[c:c + n]
        c += n
    kd, vd = paged_kv(k, v, table, npages, P)
    ld = 256
    idx_v = np.full((2, S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((2, S), np.int32)
    for s, L in enumerate(lens):
        for h in range(Hkv):
            for i, B in enumerate((128, 256)):
                B = min(B, L)
                a = np.r_[g.choice(L - C, B - C, replace=False) if B > C else [], np.arange(L - C, L)][:B]
                idx_v[i, s, h, :len(a)] = a
                nsel_v[i, s] = len(a)
    _run(k, v, qb, idx_v, nsel_v, lens, "paged", seed=7, kdev=kd, vdev=vd, page_table=i32_dev(table))


def test_bwd_multiview4x8k_full_size():
    """The multi-view training block at full size (4 x 8,192, C = 64, four budgets + full) over seeded
    index lists; every sequence, head and branch is checked, forward and backward."""
    cfg = synth.workload("multiview-train-b4-8k")
    qt, k, v = config_data("multiview-train-b4-8k")
    C = cfg.block_len
    budgets = synth.view_budgets(cfg)
    S = cfg.num_seqs
    ld = int(budgets.max())
    idx_v = np.full((len(budgets), S, cfg.num_kv_heads, ld), -1, np.int32)
    nsel_v = np.zeros((len(budgets), S), np.int32)
    for i, B in enumerate(budgets):
        for s in range(S):
            for h in range(cfg.num_kv_heads):
                pre = synth.random_index_set(cfg.config_id, s, h, cfg.seq_len - C, int(B) - C)
                idx_v[i, s, h, :int(B)] = np.r_[pre, np.arange(cfg.seq_len - C, cfg.seq_len)]
        nsel_v[i] = B
    lens = [cfg.seq_len] * S
    _run(k, v, qt[:, -C:], idx_v, nsel_v, lens, "multiview 4x8K full size", seed=8)


def test_bwd_deterministic_and_workspace_reuse():
    """Two calls give bitwise-equal gradients; a workspace shared with forward calls of other shapes works."""
    S, Hkv, G, L, C = 2, 2, 4, 3000, 64
    k, v = _rand_bits((S, Hkv, L, 128), 90), _rand_bits((S, Hkv, L, 128), 91)
    qb = _rand_bits((S, C, Hkv * G, 128), 92)
    idx_v, nsel_v = _selected_views(k, qb, [L, L], Hkv * G, C, [256, 1024])
    ws = bd.Workspace()
    a = _run(k, v, qb, idx_v, nsel_v, [L, L], "det 1", seed=9, workspace=ws, check_fwd=False)
    # a forward of another shape on the same workspace in between
    case("multiview bwd: verify on the shared workspace")
    bd.bd_verify_attn(bf16_dev(k), bf16_dev(v), bf16_dev(qb[:, :6]), i32_dev([L, L]), workspace=ws)
    b = _run(k, v, qb, idx_v, nsel_v, [L, L], "det 2", seed=9, workspace=ws, check_fwd=False)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_bwd_two_row_groups_and_many_views():
    """C * G = 320 rows per KV head (two row groups of up to 8 row blocks, the second partly empty) and
    nine views of mixed lengths (two empty): the block-mode forward and both backward kernels."""
    S, Hkv, G, L, C = 2, 2, 5, 900, 64
    k, v = _rand_bits((S, Hkv, L, 128), 100), _rand_bits((S, Hkv, L, 128), 101)
    qb = _rand_bits((S, C, Hkv * G, 128), 102)
    g = np.random.default_rng(103)
    V, ld = 9, 400
    idx_v = np.full((V, S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((V, S), np.int32)
    for i in range(V):
        n = [0, 37, 400, 129, 0, 256, 64, 311, 100][i]
        for s in range(S):
            for h in range(Hkv):
                idx_v[i, s, h, :n] = np.sort(g.choice(L, n, replace=False))
            nsel_v[i, s] = n
    _run(k, v, qb, idx_v, nsel_v, [L, L - 3], "two row groups, nine views", seed=10)


@pytest.mark.timeout(600)
def test_training_shape_c256_16k_chunk_views():
    """Sec. 4's training shape: T = 16,384 (P = 16,128, C = 256), batch 1, GQA 32/8, so C * G = 1,024
    query rows per KV head (four row groups).  The views are the paper's TopKChunks selections (the top
    floor(B/8) chunks of the prefix, the block on top) for every budget of the training set, selected on
    the GPU with the block scoring the prefix; then the forward (bf16 and training outputs) and the
    backward over those views and the full branch, against the oracle."""
    cfg = synth.workload("train-c256-16k")
    qt, k, v = config_data("train-c256-16k")
    C, Hkv, s = cfg.block_len, cfg.num_kv_heads, 8
    lens = [cfg.seq_len]
    qb = np.ascontiguousarray(qt[:, -C:])
    raws = oracle_scores(k, qb, lens, cfg.num_q_heads)
    kd = bf16_dev(k)
    budgets = list(cfg.budgets)
    ld = max(budgets) + C
    idx_v = np.full((len(budgets), 1, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((len(budgets), 1), np.int32)
    for i, B in enumerate(budgets):
        case(f"training shape: chunk selection B={B}")
        idx, nsel, scores = bd.bd_select_kv_chunks(kd, bf16_dev(qb), i32_dev(lens), B, chunk=s, return_scores=True)
        torch.cuda.synchronize()
        gi, gn, gs = idx.cpu().numpy(), nsel.cpu().numpy(), scores.cpu().numpy()
        oi, on = oracle_chunk_selection(raws, lens, Hkv, C, B, s, False)
        near = check_chunk_selection(gi, gn, gs, oi, on, raws, lens, C, B, s, False, f"training shape B={B}")
        assert near <= 2, near
        assert ((gi >= 0).sum(axis=2) == s * (B // s) + C).all()
        idx_v[i, :, :, :B + C] = gi
        nsel_v[i] = gn
    _run(k, v, qb, idx_v, nsel_v, lens, "training shape C=256 16K", seed=12, kdev=kd)
