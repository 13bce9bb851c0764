"""GPU parity of the attention entry points (decode, verify, multiview) against the fp64 oracle.

Every call goes through the C ABI (ctypes binding).  Outputs are compared
element by element: |gpu - oracle| <= 2e-2 + 1e-2 |oracle| on bf16 outputs,
1e-3 absolute on fp32 log-sum-exp.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import (assert_close, assert_lse, bf16_dev, bf16_host64, case, config_data, i32_dev, paged_kv)

pytestmark = pytest.mark.gpu


def _rand_bits(shape, seed, scale=1.0):
    g = np.random.default_rng(seed)
    return synth.f32_to_bf16_bits(scale * g.standard_normal(shape, dtype=np.float32))


def _sparse_idx(cfg, S, Hkv, L, B, W=32):
    """Seeded index lists shaped like a selection: B-W prefix positions + the window."""
    idx = np.full((S, Hkv, B), -1, np.int32)
    for s in range(S):
        for g in range(Hkv):
            pre = synth.random_index_set(cfg.config_id, s, g, L - W, B - W)
            idx[s, g] = np.r_[pre, np.arange(L - W, L)]
    return idx


def _decode_check(k, v, q, idx, nsel, lens, what, kdev=None, vdev=None, page_table=None, **kw):
    kd = bf16_dev(k) if kdev is None else kdev
    vd = bf16_dev(v) if vdev is None else vdev
    case(f"decode {what}")
    out, lse = bd.bd_sparse_decode_attn(kd, vd, bf16_dev(q), i32_dev(idx), i32_dev(nsel), i32_dev(lens),
                                        return_lse=True, page_table=page_table, **kw)
    torch.cuda.synchronize()
    ro, rl = O.sparse_decode_attn(k, v, q, idx, nsel, lens)
    assert_close(bf16_host64(out), ro, what)
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, what)
    return out


# ------------------------------------------------------------------ decode

def test_decode_tiny4k_oracle_selection():
    cfg = synth.workload("tiny-4k-gqa4")
    qt, k, v = config_data("tiny-4k-gqa4")
    lens = [cfg.seq_len]
    idx, nsel, _ = O.select_kv(k, qt[:, -cfg.window:], lens, cfg.num_q_heads, cfg.window, 256)
    _decode_check(k, v, qt[:, -1], idx, nsel, lens, "tiny 4K B=256")


@pytest.mark.parametrize("B", [256, 512, 1024, 2048])
def test_decode_layer8k_budgets(B):
    cfg = synth.workload("llama3-8b-layer-8k")
    qt, k, v = config_data("llama3-8b-layer-8k")
    idx = _sparse_idx(synth.workload("llama3-8b-layer-8k"), 1, cfg.num_kv_heads, cfg.seq_len, B)
    _decode_check(k, v, qt[:, -1], idx, [B], [cfg.seq_len], f"8K layer B={B}")


def test_decode_batch16k_full_size():
    cfg = synth.workload("16k-collapse-b8")
    qt, k, v = config_data("16k-collapse-b8")
    for B in cfg.budgets:
        idx = _sparse_idx(synth.workload("16k-collapse-b8"), cfg.num_seqs, cfg.num_kv_heads, cfg.seq_len, B)
        _decode_check(k, v, qt[:, -1], idx, [B] * cfg.num_seqs, [cfg.seq_len] * cfg.num_seqs, f"16K batch B={B}")


def test_decode_edge_cases():
    S, Hkv, G, L = 3, 2, 4, 300
    k, v = _rand_bits((S, Hkv, L, 128), 1), _rand_bits((S, Hkv, L, 128), 2)
    q = _rand_bits((S, Hkv * G, 128), 3)
    lens = [300, 129, 17]
    idx = np.full((S, Hkv, 70), -1, np.int32)
    g = np.random.default_rng(4)
    idx[0] = g.permutation(L)[:70].reshape(1, 70).repeat(Hkv, 0)      # unsorted
    idx[1, :, :40] = g.integers(-5, 200, size=(Hkv, 40))              # -1s, negatives and >= L entries
    idx[2, :, :1] = 9                                                 # single entry
    nsel = [70, 1000, 1]                                              # nsel > ld clamps
    _decode_check(k, v, q, idx, nsel, lens, "edge mix")
    # no entries at all: output 0, lse -inf
    out = _decode_check(k, v, q, idx, [0, 0, 0], lens, "empty")
    assert torch.count_nonzero(out).item() == 0
    # a single entry returns its value row bit for bit
    out = bd.bd_sparse_decode_attn(bf16_dev(k), bf16_dev(v), bf16_dev(q), i32_dev(idx), i32_dev([1, 1, 1]), i32_dev(lens))
    torch.cuda.synchronize()
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got[2, :4], np.repeat(v[2, 0, 9][None], 4, 0))
    # V == 1: softmax weights are normalised on the device, output exactly 1.0
    ones = synth.f32_to_bf16_bits(np.ones((S, Hkv, L, 128), np.float32))
    out = bd.bd_sparse_decode_attn(bf16_dev(k), bf16_dev(ones), bf16_dev(q), i32_dev(idx), i32_dev([70, 40, 1]), i32_dev(lens))
    torch.cuda.synchronize()
    o = bf16_host64(out)
    assert np.all(o[0] == 1.0) and np.all(o[2] == 1.0)


def test_decode_permutation_and_determinism():
    cfg = synth.workload("llama3-8b-layer-8k")
    qt, k, v = config_data("llama3-8b-layer-8k")
    idx = _sparse_idx(synth.workload("llama3-8b-layer-8k"), 1, cfg.num_kv_heads, cfg.seq_len, 1024)
    perm = idx[:, :, np.random.default_rng(5).permutation(1024)]
    kd, vd, qd, lens = bf16_dev(k), bf16_dev(v), bf16_dev(qt[:, -1]), i32_dev([cfg.seq_len])
    case("decode permutation / determinism")
    a = bd.bd_sparse_decode_attn(kd, vd, qd, i32_dev(idx), i32_dev([1024]), lens)
    b = bd.bd_sparse_decode_attn(kd, vd, qd, i32_dev(idx), i32_dev([1024]), lens)
    c = bd.bd_sparse_decode_attn(kd, vd, qd, i32_dev(perm), i32_dev([1024]), lens)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    ref, _ = O.sparse_decode_attn(k, v, qt[:, -1], idx, [1024], [cfg.seq_len])
    assert_close(bf16_host64(c), ref, "permuted idx")


# ------------------------------------------------------------------ verify

def _verify_check(k, v, q, lens, gamma, what, kdev=None, vdev=None, page_table=None, **kw):
    kd = bf16_dev(k) if kdev is None else kdev
    vd = bf16_dev(v) if vdev is None else vdev
    case(f"verify {what}")
    out, lse = bd.bd_verify_attn(kd, vd, bf16_dev(q), i32_dev(lens), return_lse=True, page_table=page_table, **kw)
    torch.cuda.synchronize()
    ro, rl = O.verify_attn(k, v, q, lens, gamma)
    assert_close(bf16_host64(out), ro, what)
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, what)
    return out


@pytest.mark.parametrize("name", ["tiny-4k-gqa4", "llama3-8b-layer-8k"])
def test_verify_workloads(name):
    cfg = synth.workload(name)
    qt, k, v = config_data(name)
    g1 = cfg.gamma + 1
    _verify_check(k, v, qt[:, -g1:], [cfg.seq_len] * cfg.num_seqs, cfg.gamma, name)


def test_verify_batch16k_full_size():
    cfg = synth.workload("16k-collapse-b8")
    qt, k, v = config_data("16k-collapse-b8")
    g1 = cfg.gamma + 1
    _verify_check(k, v, qt[:, -g1:], [cfg.seq_len] * cfg.num_seqs, cfg.gamma, "16K batch 16K")


@pytest.mark.parametrize("Hq,Hkv,gamma", [(8, 2, 5), (4, 4, 5), (16, 2, 5), (8, 2, 0), (32, 8, 3)])
def test_verify_ragged_shapes(Hq, Hkv, gamma):
    S, Lmax = 4, 200
    k, v = _rand_bits((S, Hkv, Lmax, 128), 10), _rand_bits((S, Hkv, Lmax, 128), 11)
    q = _rand_bits((S, gamma + 1, Hq, 128), 12)
    lens = [200, 33, gamma + 1, 97]
    _verify_check(k, v, q, lens, gamma, f"ragged Hq={Hq} Hkv={Hkv} gamma={gamma}")


def test_verify_matches_decode_over_everything():
    cfg = synth.workload("tiny-4k-gqa4")
    qt, k, v = config_data("tiny-4k-gqa4")
    L, g1 = cfg.seq_len, cfg.gamma + 1
    kd, vd = bf16_dev(k), bf16_dev(v)
    idx = np.tile(np.arange(L, dtype=np.int32), (1, cfg.num_kv_heads, 1))
    case("verify vs decode over the whole cache")
    ov = bd.bd_verify_attn(kd, vd, bf16_dev(qt[:, -g1:]), i32_dev([L]))
    od = bd.bd_sparse_decode_attn(kd, vd, bf16_dev(qt[:, -1]), i32_dev(idx), i32_dev([L]), i32_dev([L]))
    torch.cuda.synchronize()
    assert_close(bf16_host64(od), bf16_host64(ov)[:, -1], "decode(all) vs verify row gamma")


def test_verify_paged_ragged_mha():
    cfg = synth.workload("ragged-paged-b64-mha")
    lens_all = synth.seq_lens(cfg)
    pick = [0, 1, 2, 3, 4, 5]
    lens = lens_all[pick]
    ks, vs, qs = [], [], []
    for s in pick:
        qt = synth.query_tail(cfg, s)
        k, v = synth.kv_sequence(cfg, s, q_tail=qt)
        ks.append(k), vs.append(v), qs.append(qt[-(cfg.gamma + 1):])
    table, npages = synth.page_table(cfg, lens)
    kd, vd = paged_kv(ks, vs, table, npages, cfg.page_size)
    _verify_check(ks, vs, np.stack(qs), lens, cfg.gamma, "paged ragged paged sample", kdev=kd, vdev=vd,
                  page_table=i32_dev(table))
    idx = np.stack([np.stack([np.r_[synth.random_index_set(cfg.config_id, s, g, int(lens[i]) - 32, 1024 - 32),
                                    np.arange(lens[i] - 32, lens[i])] for g in range(cfg.num_kv_heads)])
                    for i, s in enumerate(pick)]).astype(np.int32)
    _decode_check(ks, vs, np.stack([q[-1] for q in qs]), idx, [1024] * len(pick), lens, "paged ragged paged sample",
                  kdev=kd, vdev=vd, page_table=i32_dev(table))


def _paged_pool(k, v, lens, ps, seed):
    """Scatter [S][Hkv][Lmax][D] caches into a pool of ps-row pages under a seeded page order."""
    g = np.random.default_rng(seed)
    npg = [(int(L) + ps - 1) // ps for L in lens]
    perm = g.permutation(sum(npg)).astype(np.int32)
    table = np.full((len(lens), max(npg)), -1, np.int32)
    o = 0
    for s, n in enumerate(npg):
        table[s, :n] = perm[o:o + n]
        o += n
    ks = [k[s][:, :int(L)] for s, L in enumerate(lens)]
    vs = [v[s][:, :int(L)] for s, L in enumerate(lens)]
    kd, vd = paged_kv(ks, vs, table, int(sum(npg)), ps)
    return kd, vd, table


@pytest.mark.parametrize("ps", [8, 16, 48, 64, 1024])
def test_verify_paged_page_sizes(ps):
    """Pages that hold whole 16-key sub-tiles (16, 48, 64) read the full cache through a table of page
    offsets; other sizes (8) through the per-key table.  At 48 rows the pages straddle the splits'
    starts, and the 9,000-row sequence takes more than 8 splits per unit (the two-level merge)."""
    S, Hkv, G, gamma = 3, 2, 4, 5
    lens = [9000, 2049, 777]
    k = _rand_bits((S, Hkv, max(lens), 128), 910 + ps)
    v = _rand_bits((S, Hkv, max(lens), 128), 920 + ps)
    q = _rand_bits((S, gamma + 1, Hkv * G, 128), 930 + ps)
    kd, vd, table = _paged_pool(k, v, lens, ps, 940 + ps)
    _verify_check(k, v, q, lens, gamma, f"paged pages of {ps}", kdev=kd, vdev=vd, page_table=i32_dev(table))


@pytest.mark.parametrize("ps", [8, 32])
def test_verify_paged_page_outside_pool(ps):
    """A page number outside [0, num_pages) makes that page's keys absent: every row attends over the
    visible keys of the other pages (reference: the oracle's attention with those keys masked)."""
    S, Hkv, G, gamma = 2, 2, 4, 5
    lens = [3000, 1100]
    k = _rand_bits((S, Hkv, max(lens), 128), 950 + ps)
    v = _rand_bits((S, Hkv, max(lens), 128), 960 + ps)
    q = _rand_bits((S, gamma + 1, Hkv * G, 128), 970 + ps)
    kd, vd, table = _paged_pool(k, v, lens, ps, 980 + ps)
    npages = int(kd.shape[0])
    bad = [(0, 5, npages + 3), (1, 2, -2)]              # (sequence, page index, out-of-pool number)
    absent = [np.zeros(L, bool) for L in lens]
    for s, j, num in bad:
        table[s, j] = num
        absent[s][j * ps:(j + 1) * ps] = True
    case(f"verify paged, pages outside the pool, pages of {ps}")
    out, lse = bd.bd_verify_attn(kd, vd, bf16_dev(q), i32_dev(lens), return_lse=True, page_table=i32_dev(table))
    torch.cuda.synchronize()
    sc = 1.0 / np.sqrt(128.0)
    R, Hq = gamma + 1, Hkv * G
    ro = np.zeros((S, R, Hq, 128))
    rl = np.full((S, R, Hq), -np.inf)
    for s, L in enumerate(lens):
        pos = L - gamma - 1 + np.arange(R)
        vis = (np.arange(L)[None, :] <= pos[:, None]) & ~absent[s][None, :]
        qs = O.bf16_to_f64(q[s])
        for g in range(Hkv):
            o, l = O.attend(qs[:, g * G:(g + 1) * G].reshape(R * G, 128), O.bf16_to_f64(k[s][g, :L]),
                            O.bf16_to_f64(v[s][g, :L]), np.repeat(vis, G, axis=0), sc)
            ro[s, :, g * G:(g + 1) * G] = o.reshape(R, G, 128)
            rl[s, :, g * G:(g + 1) * G] = l.reshape(R, G)
    what = f"paged, pages outside the pool, pages of {ps}"
    assert_close(bf16_host64(out), ro, what)
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, what)


# ------------------------------------------------------------------ multiview

def _multiview_check(k, v, qb, idx_views, nsel_views, lens, what, full=True):
    case(f"multiview {what}")
    ov, of = bd.bd_multiview_attn(bf16_dev(k), bf16_dev(v), bf16_dev(qb), i32_dev(idx_views), i32_dev(nsel_views),
                                  i32_dev(lens), full=full)
    torch.cuda.synchronize()
    rv, rf = O.multiview_attn(k, v, qb, list(idx_views), list(nsel_views), lens, with_full=full)
    assert_close(bf16_host64(ov), rv, what + " views")
    if full:
        assert_close(bf16_host64(of), rf, what + " full")


def test_multiview_small_with_selected_views():
    S, Hkv, G, L, C = 2, 2, 4, 1500, 64
    k, v = _rand_bits((S, Hkv, L, 128), 20), _rand_bits((S, Hkv, L, 128), 21)
    qb = _rand_bits((S, C, Hkv * G, 128), 22)
    budgets = [128, 256, 1024, 2048]                  # the last keeps the whole cache
    ld = max(budgets)
    idx_v = np.full((len(budgets), S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((len(budgets), S), np.int32)
    for i, B in enumerate(budgets):
        idx, nsel, _ = O.select_kv(k, qb, [L, L], Hkv * G, C, B)
        idx_v[i, :, :, :idx.shape[2]] = idx
        nsel_v[i] = nsel
    _multiview_check(k, v, qb, idx_v, nsel_v, [L, L], "small")


def test_multiview_multiview4x8k_full_size():
    cfg = synth.workload("multiview-train-b4-8k")
    qt, k, v = config_data("multiview-train-b4-8k")
    C = cfg.block_len
    budgets = synth.view_budgets(cfg)
    ld = int(budgets.max())
    S = cfg.num_seqs
    idx_v = np.full((len(budgets), S, cfg.num_kv_heads, ld), -1, np.int32)
    nsel_v = np.zeros((len(budgets), S), np.int32)
    for i, B in enumerate(budgets):
        idx_v[i, :, :, :int(B)] = _sparse_idx(synth.workload("multiview-train-b4-8k"), S, cfg.num_kv_heads, cfg.seq_len, int(B), W=C)
        nsel_v[i] = B
    qb = qt[:, -C:]
    lens = [cfg.seq_len] * S
    case("multiview multiview 4x8K full size")
    ov, of = bd.bd_multiview_attn(bf16_dev(k), bf16_dev(v), bf16_dev(qb), i32_dev(idx_v), i32_dev(nsel_v), i32_dev(lens))
    torch.cuda.synchronize()
    gv, gf = bf16_host64(ov), bf16_host64(of)
    # every sequence, head, view and the full branch
    rv, rf = O.multiview_attn(k, v, qb, list(idx_v), list(nsel_v), lens)
    assert_close(gv, rv, "multiview 4x8K views")
    assert_close(gf, rf, "multiview 4x8K full")


def test_one_workspace_serves_every_operation_and_shape():
    """Counters must start at zero for every call even after calls of other shapes left scratch behind."""
    ws = bd.Workspace()
    g = np.random.default_rng(40)
    shapes = [(2, 8, 2, 300, 5), (6, 32, 32, 2000, 5), (1, 16, 2, 700, 0), (3, 32, 8, 4000, 3), (6, 32, 32, 1500, 5)]
    for it, (S, Hq, Hkv, L, gamma) in enumerate(shapes):
        k, v = _rand_bits((S, Hkv, L, 128), 50 + it), _rand_bits((S, Hkv, L, 128), 60 + it)
        q = _rand_bits((S, gamma + 1, Hq, 128), 70 + it)
        lens = g.integers(gamma + 1, L + 1, size=S).tolist()
        case(f"shared workspace verify {S}x{Hq}/{Hkv}x{L} gamma={gamma}")
        out = bd.bd_verify_attn(bf16_dev(k), bf16_dev(v), bf16_dev(q), i32_dev(lens), workspace=ws)
        torch.cuda.synchronize()
        assert_close(bf16_host64(out), O.verify_attn(k, v, q, lens, gamma)[0], f"shared ws verify {it}")
        B = min(256, L)
        idx = np.stack([np.stack([np.sort(g.choice(L, B, replace=False)) for _ in range(Hkv)]) for _ in range(S)]).astype(np.int32)
        case(f"shared workspace decode {S}x{Hq}/{Hkv}x{L}")
        out = bd.bd_sparse_decode_attn(bf16_dev(k), bf16_dev(v), bf16_dev(q[:, -1]), i32_dev(idx), i32_dev([B] * S),
                                       i32_dev(lens), workspace=ws)
        torch.cuda.synchronize()
        assert_close(bf16_host64(out), O.sparse_decode_attn(k, v, q[:, -1], idx, [B] * S, lens)[0], f"shared ws decode {it}")
        lg = g.standard_normal((S, gamma + 1, 5000)).astype(np.float32)
        dr = g.integers(0, 5000, (S, gamma)).astype(np.int32)
        case("shared workspace accept")
        acc, bonus = bd.bd_accept_len(torch.from_numpy(lg).cuda(), i32_dev(dr), workspace=ws)
        torch.cuda.synchronize()
        ra, rb, _ = O.accept_len(lg, dr, gamma)
        assert np.array_equal(acc.cpu().numpy(), ra) and np.array_equal(bonus.cpu().numpy(), rb)


def test_multiview_block_mode_unbalanced_views_and_empty_branches():
    """Block mode with views far shorter than the list capacity, an empty view, an all-absent view and a
    sequence shorter than the block: every branch's rows are written, empty ones as 0."""
    S, Hkv, G, C = 3, 2, 4, 48
    lens = [2000, 30, 777]
    Lm = max(lens)
    k, v = _rand_bits((S, Hkv, Lm, 128), 110), _rand_bits((S, Hkv, Lm, 128), 111)
    qb = _rand_bits((S, C, Hkv * G, 128), 112)
    g = np.random.default_rng(113)
    ld = 2048
    budgets = [64, 0, 5, 1500]
    idx_v = np.full((len(budgets), S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((len(budgets), S), np.int32)
    for i, B in enumerate(budgets):
        for s, L in enumerate(lens):
            n = min(B, L)
            for h in range(Hkv):
                idx_v[i, s, h, :n] = np.sort(g.choice(L, n, replace=False))
            nsel_v[i, s] = n
    idx_v[2, :, :, :5] = -1                            # view 2: five slots, all absent
    _multiview_check(k, v, qb, idx_v, nsel_v, lens, "block mode, unbalanced and empty views")


def test_multiview_many_small_views_share_one_range():
    """60 views of at most 8 entries and the full branch: the first workgroup's share of each unit's stream
    holds dozens of pieces, each padded to whole tiles of one slot table (up to 64 branches are
    accepted); the full branch is split across workgroups and merged by the second kernel.  One
    sequence is shorter than most views' entries, so their out-of-range entries are skipped."""
    S, Hkv, G, C = 2, 8, 4, 64
    lens = [4000, 700]
    Lm = max(lens)
    k, v = _rand_bits((S, Hkv, Lm, 128), 130), _rand_bits((S, Hkv, Lm, 128), 131)
    qb = _rand_bits((S, C, Hkv * G, 128), 132)
    g = np.random.default_rng(133)
    V, ld = 60, 8
    idx_v = np.full((V, S, Hkv, ld), -1, np.int32)
    nsel_v = np.zeros((V, S), np.int32)
    for i in range(V):
        for s in range(S):
            n = int(g.integers(0, ld + 1))
            for h in range(Hkv):
                idx_v[i, s, h, :n] = g.integers(0, lens[0], n)      # may repeat; past L_s for s = 1
            nsel_v[i, s] = n
    _multiview_check(k, v, qb, idx_v, nsel_v, lens, "60 small views")

