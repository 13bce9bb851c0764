"""Pins of the fp64 oracle to things other than itself (CPU only).

Each test ties one oracle function to a closed form, an invariant, a library
routine or brute force on a tiny input, chosen so that a plausible slip (a
dropped term, an off-by-one in the causal range, a wrong head grouping, a
transposed operand, a wrong tie rule) fails at least one of them.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle as O
import synth

SIG = float(np.float64(np.float32(1.0 / math.sqrt(128))))


def bits(x):
    return synth.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


# ---------------------------------------------------------------- widening

def test_bf16_widening_known_patterns():
    b = np.array([0x3F80, 0xC040, 0x0001, 0x7F7F, 0x8000, 0x0000], dtype=np.uint16)
    got = O.bf16_to_f64(b)
    want = [1.0, -3.0, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127, -0.0, 0.0]
    assert got.tolist() == want
    assert math.copysign(1.0, got[4]) == -1.0


def test_generator_rounding_is_rne():
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20], dtype=np.float32)
    assert synth.f32_to_bf16_bits(x).tolist() == [0x3F80, 0x3F82, 0xBF80, 0x3F81]


# ---------------------------------------------------------------- attention by definition

def _pyloop_attend(q, k, v, vis, scale):
    """Literal loops with math.exp: the textbook softmax-weighted sum."""
    R, D = q.shape
    out = [[0.0] * D for _ in range(R)]
    for r in range(R):
        ls = [(t, scale * sum(q[r][d] * k[t][d] for d in range(D))) for t in range(k.shape[0]) if vis[r][t]]
        if not ls:
            continue
        m = max(l for _, l in ls)
        z = sum(math.exp(l - m) for _, l in ls)
        for t, l in ls:
            w = math.exp(l - m) / z
            for d in range(D):
                out[r][d] += w * v[t][d]
    return np.array(out)


def test_attend_matches_python_loops_tiny():
    g = np.random.default_rng(1)
    q, k, v = g.standard_normal((3, 5)), g.standard_normal((7, 5)), g.standard_normal((7, 5))
    vis = g.random((3, 7)) < 0.6
    vis[:, 0] = True
    o, _ = O.attend(q, k, v, vis, 0.37)
    np.testing.assert_allclose(o, _pyloop_attend(q, k, v, vis, 0.37), rtol=1e-13, atol=1e-13)


def test_attend_matches_torch_sdpa_fp64():
    g = np.random.default_rng(2)
    q, k, v = g.standard_normal((6, 128)), g.standard_normal((50, 128)), g.standard_normal((50, 128))
    vis = g.random((6, 50)) < 0.5
    vis[:, 3] = True
    o, lse = O.attend(q, k, v, vis, SIG)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None],
        attn_mask=torch.from_numpy(vis)[None], scale=SIG)[0].numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)
    lg = SIG * q @ k.T
    ref_lse = [np.logaddexp.reduce(lg[r][vis[r]]) for r in range(6)]
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-13)


def test_attend_two_key_closed_form():
    # l1 = scale * a, l2 = 0 -> p1 = 1 / (1 + exp(-scale*a)); v1 = 1, v2 = 0 -> out = p1.
    a = 3.0
    q = np.zeros((1, 4)); q[0, 0] = 1.0
    k = np.zeros((2, 4)); k[0, 0] = a
    v = np.zeros((2, 4)); v[0, :] = 1.0
    o, lse = O.attend(q, k, v, np.ones((1, 2), bool), 0.5)
    assert abs(o[0, 0] - 1 / (1 + math.exp(-1.5))) < 1e-15
    assert abs(lse[0] - math.log(math.exp(1.5) + 1.0)) < 1e-14


def test_attend_empty_row():
    o, lse = O.attend(np.ones((2, 4)), np.ones((3, 4)), np.ones((3, 4)), np.zeros((2, 3), bool), 1.0)
    assert np.all(o == 0) and np.all(lse == -np.inf)


# ---------------------------------------------------------------- selection: scores

def _zero_k_raw(L, W, G):
    """K == 0: every logit is 0, row i (position L-W+i) is uniform over L-W+i+1 keys."""
    raw = np.zeros(L)
    for i in range(W):
        p = L - W + i
        raw[:p + 1] += G / (p + 1)
    return raw


def test_window_scores_zero_k_closed_form():
    L, W, G = 40, 6, 3
    g = np.random.default_rng(3)
    raw = O.window_scores(np.zeros((L, 16)), g.standard_normal((W, G, 16)), L, 0.25)
    np.testing.assert_allclose(raw, _zero_k_raw(L, W, G), rtol=1e-14)
    # prefix entries all equal; window entries strictly decreasing (fewer rows see later keys)
    assert np.all(raw[:L - W] == raw[0])
    assert np.all(np.diff(raw[L - W:]) < 0)


def test_window_scores_sum_is_rows_times_heads():
    g = np.random.default_rng(4)
    L, W, G = 300, 8, 4
    raw = O.window_scores(g.standard_normal((L, 32)), g.standard_normal((W, G, 32)), L, 0.3)
    assert abs(raw.sum() - W * G) < 1e-11


def test_window_scores_match_library_softmax():
    from scipy.special import softmax
    g = np.random.default_rng(5)
    L, W, G, D = 25, 4, 2, 8
    k, q = g.standard_normal((L, D)), g.standard_normal((W, G, D))
    want = np.zeros(L)
    for h in range(G):
        for i in range(W):
            p = L - W + i
            want[:p + 1] += softmax(0.4 * (k[:p + 1] @ q[i, h]))
    np.testing.assert_allclose(O.window_scores(k, q, L, 0.4), want, rtol=1e-13)


def test_window_scores_last_key_seen_only_by_last_row():
    # A key at L-1 with a huge logit: only row W-1 (at position L-1) sees it.
    L, W, D = 20, 4, 4
    k = np.zeros((L, D)); k[L - 1, 0] = 100.0
    q = np.zeros((W, 1, D)); q[:, 0, 0] = 1.0
    raw = O.window_scores(k, q, L, 1.0)
    e = math.exp(100.0)
    assert abs(raw[L - 1] - e / (e + L - 1)) < 1e-15
    # rows 0..W-2 are uniform over their ranges and never see L-1
    want0 = sum(1.0 / (L - W + i + 1) for i in range(W - 1)) + 1.0 / (e + L - 1)
    assert abs(raw[0] - want0) < 1e-14


# ---------------------------------------------------------------- selection: pooling and top-k

def test_max_pool_matches_sliding_window_max():
    from numpy.lib.stride_tricks import sliding_window_view
    g = np.random.default_rng(6)
    for n, kern in [(1, 7), (3, 7), (50, 7), (50, 1), (50, 3), (9, 9)]:
        x = g.random(n)
        r = kern // 2
        padded = np.concatenate([np.full(r, -np.inf), x, np.full(r, -np.inf)])
        want = sliding_window_view(padded, kern).max(axis=1)
        np.testing.assert_array_equal(O.max_pool(x, kern), want)


def _dominates(pooled, chosen):
    """Every chosen candidate ranks above every other under (-pooled, position)."""
    others = [t for t in range(len(pooled)) if t not in set(chosen)]
    return all((-pooled[a], a) < (-pooled[b], b) for a in chosen for b in others)


@pytest.mark.parametrize("seed", range(6))
def test_topk_brute_force_tiny(seed):
    g = np.random.default_rng(100 + seed)
    L, W, B = 14, 3, 7
    raw = np.round(g.random(L) * 4) / 4          # coarse values -> many exact ties
    sel, pooled = O.topk_from_scores(raw, L, W, B, 3)
    keep = B - W
    N = L - W
    winners = [c for c in itertools.combinations(range(N), keep) if _dominates(pooled, c)]
    assert len(winners) == 1
    assert sel[:keep].tolist() == list(winners[0])
    assert sel[keep:].tolist() == list(range(N, L))


def test_topk_equals_stable_argsort_and_nests():
    g = np.random.default_rng(7)
    L, W = 500, 16
    raw = np.floor(g.random(L) * 50)               # plenty of ties
    prev = None
    for B in [W, 40, 100, 200, 480]:
        sel, pooled = O.topk_from_scores(raw, L, W, B, 7)
        want = np.sort(np.argsort(-pooled, kind="stable")[:B - W])
        assert sel[:B - W].tolist() == want.tolist()
        if prev is not None:
            assert set(prev) <= set(sel.tolist())
        prev = sel.tolist()


def test_topk_ties_take_lowest_positions():
    sel, _ = O.topk_from_scores(np.ones(30), 30, 5, 12, 7)
    assert sel.tolist() == list(range(7)) + list(range(25, 30))


# ---------------------------------------------------------------- selection end to end

def _cfg_small(L=256, Hq=8, Hkv=2, W=16):
    g = np.random.default_rng(8)
    k = bits(g.standard_normal((1, Hkv, L, 128)))
    q = bits(g.standard_normal((1, W, Hq, 128)))
    return k, q


def test_select_identity_and_window_only():
    k, q = _cfg_small()
    idx, nsel, _ = O.select_kv(k, q, [256], 8, 16, 256)
    assert nsel[0] == 256 and np.all(idx[0] == np.arange(256))
    idx, nsel, _ = O.select_kv(k, q, [200], 8, 16, 300)
    assert nsel[0] == 200 and np.all(idx[0, :, :200] == np.arange(200)) and np.all(idx[0, :, 200:] == -1)
    idx, nsel, _ = O.select_kv(k, q, [256], 8, 16, 16)
    assert nsel[0] == 16 and np.all(idx[0] == np.arange(240, 256))


def test_select_zero_keys_takes_lowest_prefix():
    _, q = _cfg_small()
    k = np.zeros((1, 2, 256, 128), np.uint16)
    idx, _, raws = O.select_kv(k, q, [256], 8, 16, 64)
    assert np.all(idx[0] == np.r_[np.arange(48), np.arange(240, 256)])
    np.testing.assert_allclose(raws[0][0], _zero_k_raw(256, 16, 4), rtol=1e-14)


def test_select_single_spike_keeps_its_neighbourhood():
    L, W, t0 = 256, 16, 100
    g = np.random.default_rng(9)
    q = np.zeros((1, W, 8, 128), np.float32); q[..., 0] = 1.0
    k = 0.01 * g.standard_normal((1, 2, L, 128)).astype(np.float32)
    k[0, :, t0, 0] = 60.0
    idx, _, _ = O.select_kv(bits(k), bits(q), [L], 8, W, 32)
    for gg in range(2):
        assert set(range(t0 - 3, t0 + 4)) <= set(idx[0, gg].tolist())


def test_select_uses_contiguous_head_groups():
    # KV head 0 has one strong key; only query heads 4..7 (group 1 under h // G) point at it.
    L, W = 128, 8
    q = np.zeros((1, W, 8, 128), np.float32); q[0, :, 4:, 0] = 5.0
    k = np.zeros((1, 2, L, 128), np.float32); k[0, 0, 10, 0] = 5.0
    idx, _, raws = O.select_kv(bits(k), bits(q), [L], 8, W, 24)
    np.testing.assert_allclose(raws[0][0], _zero_k_raw(L, W, 4), rtol=1e-14)   # group 0: q == 0
    assert idx[0, 0, :16].tolist() == list(range(16))


def test_select_tiny4k_heavy_hitters_selected():
    cfg = synth.workload("tiny-4k-gqa4")
    L = cfg.seq_len
    qt = synth.query_tail(cfg, 0)
    k, _ = synth.kv_sequence(cfg, 0, q_tail=qt)
    idx, nsel, raws = O.select_kv([k], [qt[-cfg.window:]], [L], cfg.num_q_heads, cfg.window, 256)
    hh = synth.heavy_hitter_positions(cfg, L, 0)
    assert nsel[0] == 256
    for g in range(cfg.num_kv_heads):
        prefix = idx[0, g, :256 - 32]
        d = np.abs(prefix[:, None].astype(np.int64) - hh[None, :]).min(axis=1)
        assert np.all(d <= 3)                               # every kept prefix slot is next to a hitter
        assert abs(raws[0][g].sum() - 32 * 4) < 1e-9


def test_select_rejects_bad_arguments():
    k, q = _cfg_small()
    for W, B, P in [(0, 64, 7), (16, 8, 7), (16, 64, 4)]:
        with pytest.raises(ValueError):
            O.select_kv(k, q[:, :max(W, 1)], [256], 8, W, B, P)


# ---------------------------------------------------------------- chunk-level selection (TopKChunks)

def test_chunk_scores_partition_the_prefix():
    x = np.arange(1, 20, dtype=np.float64)            # 19 positions -> chunks of 8, 8, 3
    cs = O.chunk_scores(x, 8)
    assert cs.tolist() == [sum(range(1, 9)), sum(range(9, 17)), 17 + 18 + 19]
    assert abs(cs.sum() - x.sum()) < 1e-12


@pytest.mark.parametrize("counts_window", [False, True])
@pytest.mark.parametrize("seed", range(6))
def test_topk_chunks_brute_force_tiny(seed, counts_window):
    g = np.random.default_rng(300 + seed)
    L, W, s, B = 30, 4, 3, 13                         # prefix 26 -> 9 chunks (last has 2)
    raw = np.round(g.random(L) * 3) / 3                # coarse values -> ties between chunk sums
    sel, cs = O.topk_chunks_from_scores(raw, L, W, B, s, budget_counts_window=counts_window)
    # Sec. 3.4 keeps floor(B/s) = 4 chunks of the prefix; the other reading floor((B-W)/s) = 3
    nc, keep = 9, ((B - W) if counts_window else B) // s
    assert keep == (3 if counts_window else 4)
    # the kept set is the unique one ranking above every other chunk under (-score, index)
    winners = [c for c in itertools.combinations(range(nc), keep)
               if all((-cs[a], a) < (-cs[b], b) for a in c for b in set(range(nc)) - set(c))]
    assert len(winners) == 1
    want = [t for c in winners[0] for t in range(c * s, min((c + 1) * s, L - W))] + list(range(L - W, L))
    assert sel.tolist() == want


@pytest.mark.parametrize("counts_window", [False, True])
def test_topk_chunks_of_one_is_the_unpooled_token_selection(counts_window):
    g = np.random.default_rng(11)
    L, W = 400, 16
    raw = np.floor(g.random(L) * 40)
    for B in [16, 50, 200]:
        a, _ = O.topk_chunks_from_scores(raw, L, W, B, 1, budget_counts_window=counts_window)
        b, _ = O.topk_from_scores(raw, L, W, B, 1, budget_counts_window=counts_window)
        assert a.tolist() == b.tolist()


def test_topk_chunks_ties_take_lowest_chunks_and_nest():
    # 4 chunks tie: the paper's count keeps floor(24/8) = 3 (chunks 0, 1, 2), the other reading 2
    sel, _ = O.topk_chunks_from_scores(np.ones(40), 40, 8, 24, 8)
    assert sel.tolist() == list(range(24)) + list(range(32, 40))
    sel, _ = O.topk_chunks_from_scores(np.ones(40), 40, 8, 24, 8, budget_counts_window=True)
    assert sel.tolist() == list(range(16)) + list(range(32, 40))
    g = np.random.default_rng(12)
    raw = g.random(1000)
    for cw in (False, True):
        prev = None
        for B in [32, 96, 288, 800]:
            sel, cs = O.topk_chunks_from_scores(raw, 1000, 32, B, 8, budget_counts_window=cw)
            assert sel.size == 32 + 8 * (((B - 32) if cw else B) // 8)
            if prev is not None:
                assert set(prev) <= set(sel.tolist())
            prev = sel.tolist()


def test_topk_chunks_training_view_holds_floor_b_over_s_chunks_plus_the_block():
    # Alg. 1 step 4 at the training shape: a block of C = 64 continuation rows scores the prefix of
    # length P = L - C; the view is the top floor(B/8) chunks of the prefix, the block on top
    g = np.random.default_rng(13)
    L, C = 8192, 64
    raw = g.random(L)
    cs = O.chunk_scores(raw[:L - C], 8)
    for B in [256, 512, 1024, 2048, 1000]:
        sel, _ = O.topk_chunks_from_scores(raw, L, C, B, 8)
        assert sel.size == 8 * (B // 8) + C
        assert sel[-C:].tolist() == list(range(L - C, L))
        kept = sorted({int(t) // 8 for t in sel[:-C]})
        assert len(kept) == B // 8
        assert min(cs[kept]) >= max(np.delete(cs, kept))     # every kept chunk outranks every other


def test_select_chunks_zero_keys_and_spike():
    _, q = _cfg_small()
    k = np.zeros((1, 2, 256, 128), np.uint16)
    # equal scores: the lowest floor(64/8) = 8 chunks, then the window; B + W slots
    idx, nsel, _ = O.select_kv_chunks(k, q, [256], 8, 16, 64, 8)
    assert idx.shape == (1, 2, 80) and nsel[0] == 80
    assert np.all(idx[0] == np.r_[np.arange(64), np.arange(240, 256)])
    idx, nsel, _ = O.select_kv_chunks(k, q, [256], 8, 16, 64, 8, budget_counts_window=True)   # 6 chunks
    assert idx.shape == (1, 2, 64) and nsel[0] == 64
    assert np.all(idx[0] == np.r_[np.arange(48), np.arange(240, 256)])
    L, W, t0 = 256, 16, 100
    g = np.random.default_rng(9)
    qs = np.zeros((1, W, 8, 128), np.float32); qs[..., 0] = 1.0
    ks = 0.01 * g.standard_normal((1, 2, L, 128)).astype(np.float32)
    ks[0, :, t0, 0] = 60.0
    idx, _, _ = O.select_kv_chunks(bits(ks), bits(qs), [L], 8, W, 16, 8)
    for gg in range(2):                                # the spike's chunk [96, 104) is kept first
        assert set(range(96, 104)) <= set(idx[0, gg].tolist())
    idx, nsel, _ = O.select_kv_chunks(k, q, [200], 8, 16, 300, 8)     # B >= L: identity
    assert nsel[0] == 200 and np.all(idx[0, :, :200] == np.arange(200)) and np.all(idx[0, :, 200:] == -1)
    # B < L but B + W > L: slots past L are -1 and nsel = L
    idx, nsel, _ = O.select_kv_chunks(k, q, [200], 8, 16, 190, 8)
    assert idx.shape[2] == 206 and nsel[0] == 200
    assert np.all(idx[0, :, :200] == np.arange(200)) and np.all(idx[0, :, 200:] == -1)


def test_select_chunks_short_last_chunk_and_tail():
    # prefix of 21 positions: chunks of 8, 8, 5; the short chunk holds the spike and is kept
    L, W = 29, 8
    raw = np.full(L, 0.1)
    raw[18] = 50.0
    sel, cs = O.topk_chunks_from_scores(raw, L, W, 16, 8)
    assert sel.tolist() == list(range(8)) + list(range(16, 21)) + list(range(21, 29))
    assert cs.tolist() == pytest.approx([0.8, 0.8, 50.4])
    sel2, _ = O.topk_chunks_from_scores(raw, L, W, 8 + 16, 8, budget_counts_window=True)
    assert sel2.tolist() == sel.tolist()


# ---------------------------------------------------------------- sparse decode (Eq. 2)

def _kv(S, Hkv, L, seed, v_const=None):
    g = np.random.default_rng(seed)
    k = bits(g.standard_normal((S, Hkv, L, 128)))
    v = bits(g.standard_normal((S, Hkv, L, 128))) if v_const is None else bits(np.full((S, Hkv, L, 128), v_const))
    return k, v


def test_decode_single_entry_returns_its_value_row():
    k, v = _kv(1, 2, 64, 10)
    q = bits(np.random.default_rng(11).standard_normal((1, 8, 128)))
    idx = np.full((1, 2, 4), -1, np.int32); idx[0, 0, 0] = 17; idx[0, 1, 0] = 5
    out, lse = O.sparse_decode_attn(k, v, q, idx, [4], [64])
    np.testing.assert_array_equal(out[0, :4], np.repeat(O.bf16_to_f64(v[0, 0, 17])[None], 4, 0))
    np.testing.assert_array_equal(out[0, 4:], np.repeat(O.bf16_to_f64(v[0, 1, 5])[None], 4, 0))


def test_decode_zero_query_is_mean_and_lse_log_n():
    k, v = _kv(1, 2, 64, 12)
    q = np.zeros((1, 8, 128), np.uint16)
    idx = np.tile(np.array([1, 9, 30, 63, -1, 200], np.int32), (1, 2, 1))
    out, lse = O.sparse_decode_attn(k, v, q, idx, [6], [64])
    want = O.bf16_to_f64(v[0, 0, [1, 9, 30, 63]]).mean(0)
    np.testing.assert_allclose(out[0, 0], want, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(lse[0], math.log(4), rtol=1e-15)


def test_decode_value_one_and_grouping():
    S, Hkv, L = 2, 4, 32
    g = np.random.default_rng(13)
    k = bits(g.standard_normal((S, Hkv, L, 128)))
    v = np.zeros((S, Hkv, L, 128), np.float32)
    for gg in range(Hkv):
        v[:, gg] = gg + 1.0                      # V == KV-head number + 1
    q = bits(g.standard_normal((S, 8, 128)))
    idx = np.tile(np.arange(0, 32, 3, dtype=np.int32), (S, Hkv, 1))
    out, _ = O.sparse_decode_attn(k, bits(v), q, idx, [11, 11], [L, L])
    for h in range(8):
        np.testing.assert_allclose(out[:, h], h // 2 + 1.0, rtol=1e-14)


def test_decode_is_order_invariant_and_nsel_clamps():
    k, v = _kv(1, 2, 128, 14)
    q = bits(np.random.default_rng(15).standard_normal((1, 8, 128)))
    sel = np.random.default_rng(16).choice(128, 40, replace=False).astype(np.int32)
    a, la = O.sparse_decode_attn(k, v, q, np.tile(np.sort(sel), (1, 2, 1)), [40], [128])
    b, lb = O.sparse_decode_attn(k, v, q, np.tile(sel, (1, 2, 1)), [40], [128])
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)
    c, _ = O.sparse_decode_attn(k, v, q, np.tile(sel, (1, 2, 1)), [999], [128])   # nsel > ld_idx
    np.testing.assert_allclose(a, c, rtol=1e-12, atol=1e-13)
    e, le = O.sparse_decode_attn(k, v, q, np.tile(sel, (1, 2, 1)), [0], [128])
    assert np.all(e == 0) and np.all(le == -np.inf)


def test_decode_counts_a_repeated_entry_as_often_as_listed():
    """The index list is a multiset (R12): doubling every entry scales every weight's numerator and
    the normaliser alike (same output, log-sum-exp up by ln 2), and one key listed twice returns its
    value row with log-sum-exp = its logit + ln 2."""
    k, v = _kv(1, 2, 96, 17)
    q = bits(np.random.default_rng(18).standard_normal((1, 8, 128)))
    sel = np.random.default_rng(19).choice(96, 30, replace=False).astype(np.int32)
    a, la = O.sparse_decode_attn(k, v, q, np.tile(sel, (1, 2, 1)), [30], [96])
    b, lb = O.sparse_decode_attn(k, v, q, np.tile(np.r_[sel, sel[::-1]], (1, 2, 1)), [60], [96])
    np.testing.assert_allclose(b, a, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lb - la, math.log(2), rtol=1e-12)
    two = np.full((1, 2, 2), 41, np.int32)
    c, lc = O.sparse_decode_attn(k, v, q, two, [2], [96])
    scale = float(np.float32(1 / math.sqrt(128)))
    for h in range(8):
        g = h // 4
        np.testing.assert_allclose(c[0, h], O.bf16_to_f64(v[0, g, 41]), rtol=1e-14, atol=1e-15)
        logit = scale * float(O.bf16_to_f64(q[0, h]) @ O.bf16_to_f64(k[0, g, 41]))
        np.testing.assert_allclose(lc[0, h], logit + math.log(2), rtol=1e-12, atol=1e-12)


def test_decode_matches_torch_sdpa():
    S, Hkv, G, L = 2, 2, 4, 96
    k, v = _kv(S, Hkv, L, 17)
    q = bits(np.random.default_rng(18).standard_normal((S, Hkv * G, 128)))
    idx = np.stack([np.stack([synth.random_index_set(99, s, gg, L, 30) for gg in range(Hkv)]) for s in range(S)])
    out, _ = O.sparse_decode_attn(k, v, q, idx, [30, 30], [L, L])
    for s in range(S):
        for h in range(Hkv * G):
            J = idx[s, h // G]
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(O.bf16_to_f64(q[s, h]))[None, None],
                torch.from_numpy(O.bf16_to_f64(k[s, h // G, J]))[None],
                torch.from_numpy(O.bf16_to_f64(v[s, h // G, J]))[None], scale=SIG)[0, 0].numpy()
            np.testing.assert_allclose(out[s, h], ref, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- verify (Eq. 1)

def test_verify_causal_closed_form():
    # K == 0, V[t] = t: row j (position L-gamma-1+j) averages 0..position -> position / 2.
    S, Hkv, L, gamma = 1, 2, 50, 5
    k = np.zeros((S, Hkv, L, 128), np.uint16)
    v = bits(np.broadcast_to(np.arange(L, dtype=np.float32)[None, None, :, None], (S, Hkv, L, 128)))
    q = bits(np.random.default_rng(19).standard_normal((S, gamma + 1, 8, 128)))
    out, lse = O.verify_attn(k, v, q, [L], gamma)
    for j in range(gamma + 1):
        p = L - gamma - 1 + j
        np.testing.assert_allclose(out[0, j], p / 2.0, rtol=1e-14)
        np.testing.assert_allclose(lse[0, j], math.log(p + 1), rtol=1e-14)


def test_verify_rows_equal_truncated_full_decode_and_gamma0():
    S, Hkv, G, L, gamma = 1, 2, 4, 80, 4
    k, v = _kv(S, Hkv, L, 20)
    q = bits(np.random.default_rng(21).standard_normal((S, gamma + 1, Hkv * G, 128)))
    out, lse = O.verify_attn(k, v, q, [L], gamma)
    for j in range(gamma + 1):
        p = L - gamma - 1 + j
        idx = np.tile(np.arange(p + 1, dtype=np.int32), (S, Hkv, 1))
        d, dl = O.sparse_decode_attn(k, v, q[:, j], idx, [p + 1], [L])
        np.testing.assert_allclose(out[:, j], d, rtol=1e-12, atol=1e-13)
        o0, _ = O.verify_attn(k[:, :, :p + 1], v[:, :, :p + 1], q[:, j:j + 1], [p + 1], 0)
        np.testing.assert_allclose(o0[:, 0], d, rtol=1e-12, atol=1e-13)


def test_verify_matches_torch_sdpa_causal():
    S, Hkv, G, L, gamma = 2, 2, 2, 70, 5
    k, v = _kv(S, Hkv, L, 22)
    q = bits(np.random.default_rng(23).standard_normal((S, gamma + 1, Hkv * G, 128)))
    out, _ = O.verify_attn(k, v, q, [L, L], gamma)
    mask = np.arange(L)[None, :] <= (L - gamma - 1 + np.arange(gamma + 1))[:, None]
    for s in range(S):
        for h in range(Hkv * G):
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(O.bf16_to_f64(q[s, :, h]))[None],
                torch.from_numpy(O.bf16_to_f64(k[s, h // G]))[None],
                torch.from_numpy(O.bf16_to_f64(v[s, h // G]))[None],
                attn_mask=torch.from_numpy(mask)[None], scale=SIG)[0].numpy()
            np.testing.assert_allclose(out[s, :, h], ref, rtol=1e-12, atol=1e-13)


def test_verify_ragged_lengths():
    S, Hkv, Lmax, gamma = 2, 1, 40, 2
    k, v = _kv(S, Hkv, Lmax, 24)
    q = bits(np.random.default_rng(25).standard_normal((S, gamma + 1, 2, 128)))
    out, _ = O.verify_attn(k, v, q, [40, 17], gamma)
    o1, _ = O.verify_attn(k[1:, :, :17], v[1:, :, :17], q[1:], [17], gamma)
    np.testing.assert_array_equal(out[1:], o1)


# ---------------------------------------------------------------- multi-view (Alg. 1)

def test_multiview_cross_identities():
    S, Hkv, G, L, C = 1, 2, 2, 90, 8
    k, v = _kv(S, Hkv, L, 26)
    q = bits(np.random.default_rng(27).standard_normal((S, C, Hkv * G, 128)))
    full_idx = np.tile(np.arange(L, dtype=np.int32), (S, Hkv, 1))
    sub = np.stack([np.stack([np.r_[synth.random_index_set(5, 0, gg, L - C, 20), np.arange(L - C, L)]
                              for gg in range(Hkv)])]).astype(np.int32)
    ov, of = O.multiview_attn(k, v, q, [full_idx, sub], [[L], [28]], [L])
    np.testing.assert_allclose(ov[0], of, rtol=1e-12, atol=1e-13)           # B >= L view == full branch
    d, _ = O.sparse_decode_attn(k, v, q[:, C - 1], sub, [28], [L])          # last row == decode
    np.testing.assert_allclose(ov[1, :, C - 1], d, rtol=1e-12, atol=1e-13)
    vf, _ = O.verify_attn(k, v, q, [L], C - 1)                              # full branch == verify
    np.testing.assert_allclose(of, vf, rtol=1e-12, atol=1e-13)


def test_multiview_causal_closed_form():
    S, Hkv, L, C = 1, 1, 40, 6
    k = np.zeros((S, Hkv, L, 128), np.uint16)
    v = bits(np.broadcast_to(np.arange(L, dtype=np.float32)[None, None, :, None], (S, Hkv, L, 128)))
    q = bits(np.random.default_rng(28).standard_normal((S, C, 2, 128)))
    J = np.array([[[3, 11, 20, 34, 35, 36, 37, 38, 39]]], np.int32)
    ov, of = O.multiview_attn(k, v, q, [J], [[9]], [L])
    for c in range(C):
        p = L - C + c
        np.testing.assert_allclose(ov[0, 0, c], np.mean([t for t in J[0, 0] if t <= p]), rtol=1e-14)
        np.testing.assert_allclose(of[0, c], p / 2.0, rtol=1e-14)


# ---------------------------------------------------------------- accept (Eq. 3, Alg. 2)

def test_accept_planted_prefix_lengths():
    cfg = synth.workload("16k-collapse-b8")
    for s in range(cfg.num_seqs):
        lg, dr, tok, m = synth.logits_and_drafts(cfg, s, vocab=3000)
        acc, bonus, am = O.accept_len(lg[None], dr[None], cfg.gamma)
        assert am[0].tolist() == tok.tolist()
        assert acc[0] == m and bonus[0] == tok[m]


def test_accept_matches_numpy_argmax_and_range():
    g = np.random.default_rng(29)
    lg = np.floor(g.standard_normal((5, 4, 40)) * 2).astype(np.float32)     # many ties
    dr = g.integers(0, 40, (5, 3)).astype(np.int32)
    dr[0] = [int(np.argmax(lg[0, i])) for i in range(3)]                     # fully accepted row
    acc, bonus, am = O.accept_len(lg, dr, 3)
    assert am.tolist() == np.argmax(lg, axis=2).tolist()                     # first occurrence
    assert acc[0] == 3 and bonus[0] == am[0, 3]
    assert np.all((acc >= 0) & (acc <= 3))
    for s in range(5):
        kk = 0
        while kk < 3 and dr[s, kk] == am[s, kk]:
            kk += 1
        assert acc[s] == kk and bonus[s] == am[s, kk]


def test_accept_gamma0_and_signed_zero_tie():
    lg = np.zeros((1, 1, 8), np.float32)
    lg[0, 0, 2] = -0.0
    acc, bonus, am = O.accept_len(lg, np.zeros((1, 0), np.int32), 0)
    assert acc[0] == 0 and bonus[0] == 0 and am[0, 0] == 0
    lg = np.full((1, 1, 8), -1.0, np.float32); lg[0, 0, 5] = -0.0; lg[0, 0, 6] = 0.0
    assert O.accept_len(lg, np.zeros((1, 0), np.int32), 0)[1][0] == 5


def test_accept_rejects_nan():
    lg = np.zeros((1, 2, 4), np.float32); lg[0, 1, 1] = np.nan
    with pytest.raises(ValueError):
        O.accept_len(lg, np.zeros((1, 1), np.int32), 1)


# ---------------------------------------------------------------- hand-derived golden fixtures

def _golden():
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")) as f:
        return json.load(f)


def test_golden_select_zero_keys():
    gd = _golden()["select_zero_keys"]
    L, W, G, B = gd["L"], gd["W"], gd["G"], gd["B"]
    q = bits(np.random.default_rng(30).standard_normal((1, W, G, 128)))
    idx, nsel, raws = O.select_kv(np.zeros((1, 1, L, 128), np.uint16), q, [L], G, W, B)
    want = [n / d for n, d in gd["raw_num_den"]]
    np.testing.assert_allclose(raws[0][0], want, rtol=1e-15)
    assert idx[0, 0].tolist() == gd["idx"] and nsel[0] == B


def test_golden_accept_worked_example():
    gd = _golden()["accept_worked"]
    acc, bonus, am = O.accept_len(np.array([gd["logits"]], np.float32), np.array([gd["draft"]], np.int32), gd["gamma"])
    assert am[0].tolist() == gd["argmax"] and acc[0] == gd["accept"] and bonus[0] == gd["bonus"]


# ---------------------------------------------------------------- per-round cache updates (Alg. 2)

def test_append_then_decode_equals_decode_over_the_extended_cache():
    # the drafter's round: rows appended to a cache with spare capacity and to the sparse list
    # give the same attention as a cache built with those rows from the start
    S, Hkv, Hq, cap, L0, n = 2, 2, 8, 64, 40, 5
    g = np.random.default_rng(40)
    kf = bits(g.standard_normal((S, Hkv, cap, 128)))
    vf = bits(g.standard_normal((S, Hkv, cap, 128)))
    k0, v0 = kf.copy(), vf.copy()
    k0[:, :, L0:] = 0
    v0[:, :, L0:] = 0
    k_new = np.ascontiguousarray(kf[:, :, L0:L0 + n].transpose(0, 2, 1, 3))   # [S][n][Hkv][D]
    v_new = np.ascontiguousarray(vf[:, :, L0:L0 + n].transpose(0, 2, 1, 3))
    idx = np.full((S, Hkv, 32), -1, np.int32)
    idx[:, :, :10] = np.arange(0, 40, 4)
    k1, v1, lens, idx1, nsel1 = O.cache_append(k0, v0, [L0] * S, k_new, v_new, idx, [10] * S)
    assert lens.tolist() == [L0 + n] * S and nsel1.tolist() == [10 + n] * S
    assert np.array_equal(k1[:, :, :L0 + n], kf[:, :, :L0 + n]) and np.all(k1[:, :, L0 + n:] == 0)
    assert idx1[0, 1, 10:15].tolist() == list(range(L0, L0 + n)) and np.all(idx1[:, :, 15:] == -1)
    q = bits(g.standard_normal((S, Hq, 128)))
    want_idx = np.full((S, Hkv, 32), -1, np.int32)
    want_idx[:, :, :10] = np.arange(0, 40, 4)
    want_idx[:, :, 10:15] = np.arange(L0, L0 + n)
    a = O.sparse_decode_attn(k1, v1, q, idx1, nsel1, lens)
    b = O.sparse_decode_attn(kf, vf, q, want_idx, [15] * S, [L0 + n] * S)
    np.testing.assert_array_equal(a[0], b[0])


def test_append_clamps_at_capacity_and_index_width():
    S, Hkv, cap = 1, 1, 10
    k = np.zeros((S, Hkv, cap, 128), np.uint16)
    new = np.full((S, 4, Hkv, 128), 7, np.uint16)
    k1, v1, lens, idx1, nsel1 = O.cache_append(k, k, [8], new, new, np.full((S, Hkv, 5), -1, np.int32), [4])
    assert lens.tolist() == [10]                      # two of four rows fit
    assert np.all(k1[0, 0, 8:] == 7) and np.all(k1[0, 0, :8] == 0)
    assert nsel1.tolist() == [5] and idx1[0, 0, 4] == 8   # one of two slots fits


def test_rollback_keeps_the_accepted_prefix():
    # verifier: gamma speculative rows, accepted k -> L - (gamma - k); the drafter's list likewise
    lens, ns = O.cache_rollback([100, 100, 100, 3], [0, 2, 5, 9], 5, nsel=[20, 20, 20, 1])
    assert lens.tolist() == [95, 97, 100, 3] and ns.tolist() == [15, 17, 20, 1]
    assert O.cache_rollback([2], [0], 5).tolist() == [0]               # never below zero
    # append gamma rows then roll back after k accepted == append only the k accepted rows
    S, cap, gamma = 1, 32, 4
    g = np.random.default_rng(41)
    k = bits(g.standard_normal((S, 1, cap, 128)))
    new = bits(g.standard_normal((S, gamma, 1, 128)))
    for kacc in range(gamma + 1):
        _, _, l_all = O.cache_append(k, k, [10], new, new)
        l_rb = O.cache_rollback(l_all, [kacc], gamma)
        _, _, l_k = O.cache_append(k, k, [10], new[:, :kacc], new[:, :kacc])
        assert l_rb.tolist() == l_k.tolist()


@pytest.mark.parametrize("L0,nsel0,ld", [(10, 5, 32), (29, 5, 32), (10, 30, 32), (31, 31, 32), (32, 32, 32)])
def test_rollback_from_base_lengths_equals_appending_only_the_accepted_rows(L0, nsel0, ld):
    # capacity 32 rows, a list of ld slots: appending gamma speculative rows and rolling back to the
    # base lengths plus the accepted count must equal appending only the accepted rows, also where the
    # appends ran into the capacity or the end of the list (rows and slots that were never written)
    S, cap, gamma = 1, 32, 4
    g = np.random.default_rng(42)
    k = bits(g.standard_normal((S, 1, cap, 128)))
    new = bits(g.standard_normal((S, gamma, 1, 128)))
    idx = np.full((S, 1, ld), -1, np.int32)
    idx[0, 0, :nsel0] = np.arange(nsel0) % max(L0, 1)
    for kacc in range(gamma + 1):
        _, _, l_all, i_all, n_all = O.cache_append(k, k, [L0], new, new, idx, [nsel0])
        l_rb, n_rb = O.cache_rollback(l_all, [kacc], gamma, nsel=n_all, base_lens=[L0], base_nsel=[nsel0])
        _, _, l_k, i_k, n_k = O.cache_append(k, k, [L0], new[:, :kacc], new[:, :kacc], idx, [nsel0])
        assert l_rb.tolist() == l_k.tolist() and n_rb.tolist() == n_k.tolist(), kacc
        assert np.array_equal(i_all[0, 0, :n_rb[0]], i_k[0, 0, :n_k[0]])
    # the subtractive rule assumes every speculative row was written: with a full list it would
    # take committed entries off, the base rule does not
    if nsel0 + gamma > ld:
        _, _, l_all, _, n_all = O.cache_append(k, k, [L0], new, new, idx, [nsel0])
        _, n_sub = O.cache_rollback(l_all, [0], gamma, nsel=n_all)
        assert n_sub[0] < nsel0


# ---------------------------------------------------------------- top-1 CE (Eqs. 5-7) and budget sampling

def test_top1_ce_matches_torch_cross_entropy_and_targets():
    g = np.random.default_rng(50)
    R, V = 7, 300
    st = g.standard_normal((R, V)).astype(np.float32) * 3
    te = np.round(g.standard_normal((R, V)) * 2).astype(np.float32)      # ties in the teacher rows
    loss, tgt, lse = O.top1_ce(st, teacher=te)
    assert tgt.tolist() == [int(np.argmax(te[r])) for r in range(R)]       # first occurrence
    want = torch.nn.functional.cross_entropy(torch.from_numpy(st).double(), torch.from_numpy(tgt).long(),
                                             reduction="none").numpy()
    np.testing.assert_allclose(loss, want, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(lse, torch.logsumexp(torch.from_numpy(st).double(), 1).numpy(), rtol=1e-13)


def test_top1_ce_closed_forms():
    V = 1000
    loss, _, lse = O.top1_ce(np.zeros((2, V), np.float32), targets=[0, 999])
    np.testing.assert_allclose(loss, np.log(V), rtol=1e-14)                # uniform: log V
    st = np.zeros((1, V), np.float32); st[0, 5] = 40.0
    loss, _, _ = O.top1_ce(st, targets=[5])
    # target holds the max: loss = log(1 + 999 e^-40), about 4e-15, within fp64 rounding of lse = 40
    assert abs(loss[0] - np.log1p((V - 1) * np.exp(-40.0))) <= 2e-14
    a, _, _ = O.top1_ce(st + 3.5, targets=[7])                             # shift invariance
    b, _, _ = O.top1_ce(st, targets=[7])
    np.testing.assert_allclose(a, b, rtol=1e-12)
    np.testing.assert_allclose(b, 40.0 + np.log1p((V - 1) * np.exp(-40.0)), rtol=1e-12)


def test_budget_sampling_inverts_the_cdf():
    budgets, w = [256, 512, 1024, 2048], [0.4, 0.3, 0.2, 0.1]
    thr = O.budget_thresholds(w)
    assert thr.dtype == np.float32 and thr[-1] == 1.0
    assert O.sample_budgets([0.0], budgets, w).tolist() == [256]
    assert O.sample_budgets([np.nextafter(np.float32(1), np.float32(0))], budgets, w).tolist() == [2048]
    # a draw equal to a threshold falls in the next bucket; just below stays
    t0 = thr[0]
    assert O.sample_budgets([t0], budgets, w).tolist() == [512]
    assert O.sample_budgets([np.nextafter(t0, np.float32(0))], budgets, w).tolist() == [256]
    # frequencies follow the weights
    u = np.random.default_rng(51).random(200000).astype(np.float32)
    b = O.sample_budgets(u, budgets, w)
    freq = [(b == x).mean() for x in budgets]
    np.testing.assert_allclose(freq, w, atol=0.005)


# ---------------------------------------------------------------- multiview backward (Alg. 1 steps 3-5)

def _torch_multiview_grads(k, v, q, idx_views, nsel, lens, dov, dof, sc):
    """Reference gradients by fp64 autograd of a dense masked-softmax formulation (library routine)."""
    S, C, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    kt = torch.from_numpy(O.bf16_to_f64(k)).requires_grad_(True)
    vt = torch.from_numpy(O.bf16_to_f64(v)).requires_grad_(True)
    qt = torch.from_numpy(O.bf16_to_f64(q)).requires_grad_(True)
    total = 0
    for s in range(S):
        L = lens[s]
        pos = torch.arange(L - C, L)
        for h in range(Hq):
            g = h // G
            logits = sc * qt[s, :, h] @ kt[s, g, :L].T                       # [C][L]
            masks = []
            for vi in range(len(idx_views)):
                J = [int(t) for t in idx_views[vi][s, g, :nsel[vi][s]] if 0 <= t < L]
                m = torch.zeros((C, L), dtype=torch.bool)
                for t in J:
                    m[:, t] |= torch.tensor(True)
                masks.append((m & (torch.arange(L)[None, :] <= pos[:, None]), torch.from_numpy(dov[vi][s, :, h])))
            masks.append((torch.arange(L)[None, :] <= pos[:, None], torch.from_numpy(dof[s, :, h])))
            for m, do in masks:
                p = torch.softmax(logits.masked_fill(~m, float("-inf")), dim=1)
                total = total + (do * (p @ vt[s, g, :L])).sum()
    total.backward()
    return qt.grad.numpy(), kt.grad.numpy(), vt.grad.numpy()


def test_multiview_backward_matches_fp64_autograd():
    S, Hkv, Hq, L, C = 2, 2, 4, 40, 6
    g = np.random.default_rng(60)
    k, v = bits(g.standard_normal((S, Hkv, L, 128))), bits(g.standard_normal((S, Hkv, L, 128)))
    q = bits(g.standard_normal((S, C, Hq, 128)))
    lens = [40, 33]
    idx = [np.full((S, Hkv, 20), -1, np.int32) for _ in range(2)]
    for vi, B in enumerate([12, 20]):
        for s in range(S):
            for gg in range(Hkv):
                pre = np.sort(g.choice(lens[s] - C, B - C, replace=False))
                idx[vi][s, gg, :B] = np.r_[pre, np.arange(lens[s] - C, lens[s])]
    nsel = [np.array([12, 12]), np.array([20, 20])]
    dov = g.standard_normal((2, S, C, Hq, 128))
    dof = g.standard_normal((S, C, Hq, 128))
    sc = float(np.float32(1 / np.sqrt(128)))
    dq, dk, dv = O.multiview_attn_bwd(k, v, q, idx, nsel, lens, dov, dof)
    tq, tk, tv = _torch_multiview_grads(k, v, q, idx, nsel, lens, dov, dof, sc)
    np.testing.assert_allclose(dq, tq, rtol=1e-10, atol=1e-12)
    for s in range(S):
        blk = slice(lens[s] - C, lens[s])
        np.testing.assert_allclose(dk[s], tk[s, :, blk].transpose(1, 0, 2), rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(dv[s], tv[s, :, blk].transpose(1, 0, 2), rtol=1e-10, atol=1e-12)


def test_attend_backward_finite_differences():
    g = np.random.default_rng(61)
    R, N, D = 3, 5, 8
    q, k, v = g.standard_normal((R, D)), g.standard_normal((N, D)), g.standard_normal((N, D))
    vis = np.ones((R, N), bool); vis[0, 3:] = False
    dout = g.standard_normal((R, D))
    dq, dk, dv = O.attend_backward(q, k, v, vis, 0.3, dout)
    f = lambda q_, k_, v_: (O.attend(q_, k_, v_, vis, 0.3)[0] * dout).sum()
    eps = 1e-6
    for arr, grad, which in [(q, dq, 0), (k, dk, 1), (v, dv, 2)]:
        for idx in [(0, 1), (1, 4), (2, 0)]:
            if idx[0] >= arr.shape[0]:
                continue
            a2 = arr.copy(); a2[idx] += eps
            args = [q, k, v]; args[which] = a2
            b2 = arr.copy(); b2[idx] -= eps
            args2 = [q, k, v]; args2[which] = b2
            fd = (f(*args) - f(*args2)) / (2 * eps)
            assert abs(fd - grad[idx]) < 1e-6 * max(1.0, abs(fd)), (which, idx, fd, grad[idx])


def test_multiview_backward_counts_repeated_entries():
    """A view over a multiset: a key listed twice takes two softmax weights (the forward's reading)
    and its gradient is the sum over its entries.  fp64 autograd through index_select with a
    repeated index accumulates exactly that."""
    g = np.random.default_rng(62)
    S, Hkv, Hq, L, C = 1, 1, 2, 24, 4
    k, v = bits(g.standard_normal((S, Hkv, L, 128))), bits(g.standard_normal((S, Hkv, L, 128)))
    q = bits(g.standard_normal((S, C, Hq, 128)))
    J = np.array([0, 3, 3, 7, 21, 22, 22, 23, 9, -1, 30], np.int64)   # repeats, a block row twice, absent tails
    idx = [J.astype(np.int32).reshape(1, 1, -1)]
    nsel = [np.array([len(J)])]
    dov = g.standard_normal((1, S, C, Hq, 128))
    dq, dk, dv = O.multiview_attn_bwd(k, v, q, idx, nsel, [L], dov, None)
    sc = float(np.float32(1 / np.sqrt(128)))
    kt = torch.from_numpy(O.bf16_to_f64(k[0, 0])).requires_grad_(True)
    vt = torch.from_numpy(O.bf16_to_f64(v[0, 0])).requires_grad_(True)
    qt = torch.from_numpy(O.bf16_to_f64(q[0])).requires_grad_(True)               # [C][Hq][D]
    Jv = torch.from_numpy(J[(J >= 0) & (J < L)])
    kj, vj = kt.index_select(0, Jv), vt.index_select(0, Jv)
    pos = torch.arange(L - C, L)
    total = 0.0
    for h in range(Hq):
        logits = sc * qt[:, h] @ kj.T
        p = torch.softmax(logits.masked_fill(Jv[None, :] > pos[:, None], float("-inf")), dim=1)
        total = total + (torch.from_numpy(dov[0, 0, :, h]) * (p @ vj)).sum()
    total.backward()
    np.testing.assert_allclose(dq[0], qt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dk[0, :, 0], kt.grad.numpy()[L - C:], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dv[0, :, 0], vt.grad.numpy()[L - C:], rtol=1e-10, atol=1e-12)
    assert np.abs(kt.grad.numpy()[22]).max() > 0                                 # the repeated block row has a gradient
