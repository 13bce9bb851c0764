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
from gpu_utils import assert_close, assert_lse, bf16_dev, bf16_host64, case, config_data, i32_dev, paged_kv

pytestmark = pytest.mark.gpu

GRAD_ATOL_FRAC, GRAD_RTOL = 1e-3, 1e-3


def _rand_bits(shape, seed, scale=1.0):
    g = np.random.default_rng(seed)
    return synth.f32_to_bf16_bits(scale * g.standard_normal(shape, dtype=np.float32))


def _grad_close(gpu, ref, what):
    atol = GRAD_ATOL_FRAC * max(float(np.abs(ref).max(initial=0.0)), 1e-30)
    return assert_close(gpu, ref, what, atol=atol, rtol=GRAD_RTOL)


def _out32_close(gpu, ref, what):
    atol = 1e-4 * max(float(np.abs(ref).max(initial=0.0)), 1e-30)
    return assert_close(gpu.cpu().numpy().astype(np.float64), ref, what, atol=atol, rtol=1e-4)


def _run(k, v, qb, idx_v, nsel_v, lens, what, full=True, seed=0, kdev=None, vdev=None, page_table=None,
         check_fwd=True, seqs=None, with_dkv=True, workspace=None):
    """Training forward, backward with seeded dO; compare dq / dk / dv (on `seqs`, default all) with the oracle."""
    S, C, Hq = qb.shape[0], qb.shape[1], qb.shape[2]
    V = 0 if idx_v is None else len(idx_v)
    kd = bf16_dev(k) if kdev is None else kdev
    vd = bf16_dev(v) if vdev is None else vdev
    iv = i32_dev(idx_v) if V else None
    nv = i32_dev(nsel_v) if V else None
    ld = i32_dev(lens)
    case(f"multiview bwd forward {what}")
    ov, of, o32v, lv, o32f, lf = bd.bd_multiview_attn(kd, vd, bf16_dev(qb), iv, nv, ld, full=full, train=True,
                                                      page_table=page_table, max_seq_len=int(max(lens)))
    dov_bits = _rand_bits((V, S, C, Hq, 128), 1000 + seed) if V else None
    dof_bits = _rand_bits((S, C, Hq, 128), 2000 + seed) if full else None
    case(f"multiview bwd {what}")
    dq, dk, dv = bd.bd_multiview_attn_bwd(kd, vd, bf16_dev(qb), iv, nv, ld, o32v, lv,
                                          bf16_dev(dov_bits) if V else None, o32f, lf,
                                          bf16_dev(dof_bits) if full else None, with_dkv=with_dkv,
                                          page_table=page_table, max_seq_len=int(max(lens)), workspace=workspace)
    torch.cuda.synchronize()
    seqs = list(range(S)) if seqs is None else seqs
    for s in seqs:
        sl = slice(s, s + 1)
        ks = [k[s]] if isinstance(k, list) else k[sl]
        vs = [v[s]] if isinstance(v, list) else v[sl]
        iv_s = [x[sl] for x in idx_v] if V else []
        nv_s = [x[sl] for x in nsel_v] if V else []
        dov = [synth.bf16_bits_to_f32(dov_bits[i, sl]).astype(np.float64) for i in range(V)]
        dof = synth.bf16_bits_to_f32(dof_bits[sl]).astype(np.float64) if full else None
        if check_fwd:
            rv, rf, rlv, rlf = O.multiview_attn(ks, vs, qb[sl], iv_s, nv_s, lens[s:s + 1], with_full=full,
                                                return_lse=True)
            if V:
                assert_close(bf16_host64(ov[:, sl]), rv, f"{what} seq {s} views out")
                assert_lse(lv[:, sl].cpu().numpy().astype(np.float64), rlv, f"{what} seq {s} views lse")
                _out32_close(o32v[:, sl], rv, f"{what} seq {s} views out32")
            if full:
                assert_close(bf16_host64(of[sl]), rf, f"{what} seq {s} full out")
                assert_lse(lf[sl].cpu().numpy().astype(np.float64), rlf, f"{what} seq {s} full lse")
                _out32_close(o32f[sl], rf, f"{what} seq {s} full out32")
        rq, rk, rvv = O.multiview_attn_bwd(ks, vs, qb[sl], iv_s, nv_s, lens[s:s + 1], dov, dof)
        _grad_close(dq[sl].cpu().numpy().astype(np.float64), rq, f"{what} seq {s} dq")
        if with_dkv:
            _grad_close(dk[sl].cpu().numpy().astype(np.float64), rk, f"{what} seq {s} dk")
            _grad_close(dv[sl].cpu().numpy().astype(np.float64), rvv, f"{what} seq {s} dv")
        else:
            assert dk is None and dv is None
    return dq, dk, dv


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


def test_bwd_multiview4x8k_full_size_sampled():
    """The multi-view training block at full size (4 x 8,192, C = 64, four budgets + full); the oracle
    checks one sequence, all heads and branches."""
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
    _run(k, v, qt[:, -C:], idx_v, nsel_v, lens, "multiview 4x8K full size", seed=8, seqs=[2], check_fwd=False)


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
