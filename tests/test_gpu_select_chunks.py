"""GPU parity of bd_select_kv_chunks (TopKChunks) against the fp64 oracle.

Same two-part exact-index protocol as the token-level selection:
  (i) the chunk ranking is exact in the kernel's precision: chunk sums of the
      GPU's own fp32 scores, added left to right in fp32, ranked by (sum
      descending, chunk index ascending), reproduce the GPU indices bit for bit;
 (ii) end to end the GPU's kept chunks equal the oracle's, except chunks whose
      fp64 score lies within a relative 1e-4 of the oracle's threshold chunk.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import assert_close, assert_lse, bf16_dev, bf16_host64, case, config_data, i32_dev

pytestmark = pytest.mark.gpu
DELTA = 1e-4


def _fp32_chunk_sums(raw32, N, s):
    nc = (N + s - 1) // s
    pad = np.zeros(nc * s, np.float32)
    pad[:N] = raw32[:N]
    pad = pad.reshape(nc, s)
    acc = np.zeros(nc, np.float32)
    for j in range(s):                       # left to right, rounded to fp32 after every addition
        acc = (acc + pad[:, j]).astype(np.float32)
    return acc


def _kept_chunks(idx_row, N, s):
    return sorted({int(t) // s for t in idx_row if 0 <= t < N})


def _oracle(k, q_win, lens, Hq, W, B, s, cw, raws=None):
    """The oracle's selection; with raws (oracle scores per sequence, [Hkv][L]) given, only its
    ranking steps run (the scores do not depend on B)."""
    if raws is None:
        return O.select_kv_chunks(k, q_win, lens, Hq, W, B, s, budget_counts_window=cw)
    S, Hkv = len(lens), k.shape[1]
    ld = B if cw else B + W
    idx = np.full((S, Hkv, ld), -1, np.int32)
    nsel = np.zeros(S, np.int32)
    for si, L in enumerate(lens):
        if B >= L:
            idx[si, :, :L] = np.arange(L)
            nsel[si] = L
            continue
        for g in range(Hkv):
            sel, _ = O.topk_chunks_from_scores(raws[si][g], L, W, B, s, budget_counts_window=cw)
            idx[si, g, :sel.size] = sel
        nsel[si] = min(ld, L)
    return idx, nsel, raws


def _check(k, q_win, lens, Hq, W, B, s, what, cw=False, raws=None, lse_win=None):
    case(f"select chunks {what} B={B} s={s} counts_window={cw}")
    idx, nsel, scores = bd.bd_select_kv_chunks(bf16_dev(k), bf16_dev(q_win), i32_dev(lens), B, chunk=s,
                                               budget_counts_window=cw, return_scores=True,
                                               lse_win=None if lse_win is None else torch.from_numpy(lse_win).cuda())
    torch.cuda.synchronize()
    gi, gn, gs = idx.cpu().numpy(), nsel.cpu().numpy(), scores.cpu().numpy()
    oi, on, oraw = _oracle(k, q_win, lens, Hq, W, B, s, cw, raws)
    ld = B if cw else B + W
    assert gi.shape[2] == ld and oi.shape == gi.shape, what
    assert np.array_equal(gn, on), what
    near = 0
    for si in range(len(lens)):
        L = int(lens[si])
        for g in range(gi.shape[1]):
            if B >= L:
                assert np.array_equal(gi[si, g], oi[si, g]), (what, si, g)
                continue
            N = L - W
            keep = min(((B - W) if cw else B) // s, (N + s - 1) // s)
            # layout: kept chunk positions ascending, the window, then -1
            cs32 = _fp32_chunk_sums(gs[si, g], N, s)
            order = np.lexsort((np.arange(cs32.size), -cs32.astype(np.float64)))
            want_chunks = np.sort(order[:keep])
            want = [t for c in want_chunks for t in range(c * s, min((c + 1) * s, N))]
            want = want + list(range(N, L))
            want = want + [-1] * (ld - len(want))
            assert gi[si, g].tolist() == want, (what, "chunk ranking stage", si, g)
            # (ii) end to end
            diff = set(_kept_chunks(gi[si, g], N, s)) ^ set(_kept_chunks(oi[si, g], N, s))
            if diff:
                cs = O.chunk_scores(oraw[si][g][:N], s)
                thr = np.sort(cs)[::-1][keep - 1]
                for c in diff:
                    assert abs(cs[c] - thr) <= DELTA * thr, (what, si, g, c, cs[c], thr)
                near += 1
    return gi, near


@pytest.mark.parametrize("cw", [False, True])
def test_select_chunks_tiny4k(cw):
    cfg = synth.workload("tiny-4k-gqa4")
    qt, k, _ = config_data("tiny-4k-gqa4")
    _, near = _check(k, qt[:, -cfg.window:], [cfg.seq_len], cfg.num_q_heads, cfg.window, 256, 8, "tiny 4K", cw)
    assert near <= 1


@pytest.mark.parametrize("B", [256, 1024])
def test_select_chunks_layer8k(B):
    cfg = synth.workload("llama3-8b-layer-8k")
    qt, k, _ = config_data("llama3-8b-layer-8k")
    _, near = _check(k, qt[:, -cfg.window:], [cfg.seq_len], cfg.num_q_heads, cfg.window, B, 8, f"8K layer B={B}")
    assert near <= 2


@pytest.mark.parametrize("s", [1, 5, 8, 16])
def test_select_chunks_ragged_lengths_and_sizes(s):
    # L - W not a multiple of s (short last chunk), B - W not a multiple of s (-1 tail slots)
    S, Hkv, Hq, W = 3, 2, 8, 32
    lens = [2000, 1337, 77]
    g = np.random.default_rng(21)
    k = synth.f32_to_bf16_bits(g.standard_normal((S, Hkv, max(lens), 128)).astype(np.float32))
    q = synth.f32_to_bf16_bits(g.standard_normal((S, W, Hq, 128)).astype(np.float32))
    for cw in (False, True):
        _, near = _check(k, q, lens, Hq, W, 300, s, f"ragged s={s}", cw)
        assert near <= 1


@pytest.mark.parametrize("s", [5, 16])
def test_select_chunks_short_last_chunk_taken(s):
    # the prefix's last chunk is short and holds a key aligned with every query: it is kept, and the
    # window follows its last position directly (the kept count is not a multiple of s)
    S, Hkv, Hq, W, L, B = 2, 2, 8, 32, 1000, 200
    N = L - W
    assert N % s != 0
    g = np.random.default_rng(24 + s)
    kf = g.standard_normal((S, Hkv, L, 128)).astype(np.float32)
    qf = g.standard_normal((S, W, Hq, 128)).astype(np.float32)
    kf[:, :, N - 1] = 100.0 * qf.mean(axis=(1, 2))[:, None, :] / np.linalg.norm(qf.mean(axis=(1, 2)), axis=-1)[:, None, None]
    k, q = synth.f32_to_bf16_bits(kf), synth.f32_to_bf16_bits(qf)
    last = (N - 1) // s
    for cw in (False, True):
        gi, _ = _check(k, q, [L, L], Hq, W, B, s, f"short last chunk s={s}", cw=cw)
        for si in range(S):
            for h in range(Hkv):
                row = gi[si, h].tolist()
                assert last in _kept_chunks(row, N, s), (si, h)
                assert row[row.index(N - 1) + 1] == N, (si, h)    # the window follows the short chunk


def test_select_chunks_zero_keys_exact_and_decode_skips_unused_slots():
    S, Hkv, Hq, L, W = 1, 2, 8, 700, 16
    g = np.random.default_rng(22)
    q = synth.f32_to_bf16_bits(g.standard_normal((S, W, Hq, 128)).astype(np.float32))
    k = np.zeros((S, Hkv, L, 128), np.uint16)
    gi, _ = _check(k, q, [L], Hq, W, 100, 8, "zero keys", cw=True)   # 10 chunks of 8, 4 slots of -1
    assert gi[0, 0].tolist() == list(range(80)) + list(range(684, 700)) + [-1] * 4
    gp, _ = _check(k, q, [L], Hq, W, 100, 8, "zero keys")             # paper count: 12 chunks, 4 slots of -1
    assert gp[0, 0].tolist() == list(range(96)) + list(range(684, 700)) + [-1] * 4
    # the attention calls skip the -1 slots: decode over this selection equals the oracle's
    kr = synth.f32_to_bf16_bits(g.standard_normal((S, Hkv, L, 128)).astype(np.float32))
    v = synth.f32_to_bf16_bits(g.standard_normal((S, Hkv, L, 128)).astype(np.float32))
    qd = synth.f32_to_bf16_bits(g.standard_normal((S, Hq, 128)).astype(np.float32))
    case("decode over a chunk selection with -1 slots")
    out, lse = bd.bd_sparse_decode_attn(bf16_dev(kr), bf16_dev(v), bf16_dev(qd), i32_dev(gi), i32_dev([100]),
                                        i32_dev([L]), return_lse=True)
    torch.cuda.synchronize()
    ro, rl = O.sparse_decode_attn(kr, v, qd, gi, [100], [L])
    assert_close(bf16_host64(out), ro, "decode over chunks")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, "decode over chunks")


def test_select_chunks_identity_when_budget_covers_the_cache():
    S, Hkv, Hq, W = 2, 2, 8, 16
    g = np.random.default_rng(23)
    k = synth.f32_to_bf16_bits(g.standard_normal((S, Hkv, 300, 128)).astype(np.float32))
    q = synth.f32_to_bf16_bits(g.standard_normal((S, W, Hq, 128)).astype(np.float32))
    gi, _ = _check(k, q, [300, 120], Hq, W, 320, 8, "identity", cw=True)
    assert gi[1, 0].tolist() == list(range(120)) + [-1] * 200
    gi, _ = _check(k, q, [300, 120], Hq, W, 320, 8, "identity")
    assert gi[1, 0].tolist() == list(range(120)) + [-1] * 216
    # B < L <= B + W: every prefix chunk fits, slots past L are -1
    gi, _ = _check(k, q, [300, 120], Hq, W, 290, 8, "budget covers the prefix")
    assert gi[0, 0].tolist() == list(range(300)) + [-1] * 6


def _multiview_view_scores(cfg, qt, k):
    """Oracle scores of the multiview workload's block (W = C = 64 rows, G = 4: 256 rows per KV head)."""
    C, G = cfg.block_len, cfg.num_q_heads // cfg.num_kv_heads
    sc = float(np.float64(np.float32(1.0 / np.sqrt(128))))
    raws = []
    for si in range(cfg.num_seqs):
        qw = O.bf16_to_f64(qt[si, -C:])
        raws.append([O.window_scores(O.bf16_to_f64(k[si, g]), qw[:, g * G:(g + 1) * G], cfg.seq_len, sc)
                     for g in range(cfg.num_kv_heads)])
    return raws


def test_select_chunks_training_views_paper_count():
    """Alg. 1 step 4 at the multiview training shape: the 64-row block scores the 8,128-position
    prefix of each of the 4 sequences, and every budget B in {256, 512, 1024, 2048} keeps the top
    floor(B/8) chunks with the block on top (Sec. 3.4), B + 64 slots per head."""
    cfg = synth.workload("multiview-train-b4-8k")
    qt, k, _ = config_data("multiview-train-b4-8k")
    C = cfg.block_len
    raws = _multiview_view_scores(cfg, qt, k)
    lens = [cfg.seq_len] * cfg.num_seqs
    for B in (256, 512, 1024, 2048):
        gi, near = _check(k, np.ascontiguousarray(qt[:, -C:]), lens, cfg.num_q_heads, C, B, 8,
                          "multiview views", raws=raws)
        assert near <= 2
        for si in range(cfg.num_seqs):
            for g in range(cfg.num_kv_heads):
                row = gi[si, g]
                assert (row >= 0).sum() == 8 * (B // 8) + C        # floor(B/8) whole chunks + the block
                assert row[8 * (B // 8):8 * (B // 8) + C].tolist() == list(range(cfg.seq_len - C, cfg.seq_len))
        # the other reading at the same shape
        _check(k, np.ascontiguousarray(qt[:, -C:]), lens, cfg.num_q_heads, C, B, 8, "multiview views", cw=True,
               raws=raws)
