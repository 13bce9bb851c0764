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


def _check(k, q_win, lens, Hq, W, B, s, what):
    case(f"select chunks {what} B={B} s={s}")
    idx, nsel, scores = bd.bd_select_kv_chunks(bf16_dev(k), bf16_dev(q_win), i32_dev(lens), B, chunk=s,
                                               return_scores=True)
    torch.cuda.synchronize()
    gi, gn, gs = idx.cpu().numpy(), nsel.cpu().numpy(), scores.cpu().numpy()
    oi, on, oraw = O.select_kv_chunks(k, q_win, lens, Hq, W, B, s)
    assert np.array_equal(gn, on), what
    near = 0
    for si in range(len(lens)):
        L = int(lens[si])
        for g in range(gi.shape[1]):
            if B >= L:
                assert np.array_equal(gi[si, g], oi[si, g]), (what, si, g)
                continue
            N = L - W
            keep = min((B - W) // s, (N + s - 1) // s)
            # layout: kept chunk positions ascending, the window, then -1
            cs32 = _fp32_chunk_sums(gs[si, g], N, s)
            order = np.lexsort((np.arange(cs32.size), -cs32.astype(np.float64)))
            want_chunks = np.sort(order[:keep])
            want = [t for c in want_chunks for t in range(c * s, min((c + 1) * s, N))]
            want = want + list(range(N, L))
            want = want + [-1] * (B - len(want))
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


def test_select_chunks_tiny4k():
    cfg = synth.workload("tiny-4k-gqa4")
    qt, k, _ = config_data("tiny-4k-gqa4")
    _, near = _check(k, qt[:, -cfg.window:], [cfg.seq_len], cfg.num_q_heads, cfg.window, 256, 8, "tiny 4K")
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
    _, near = _check(k, q, lens, Hq, W, 300, s, f"ragged s={s}")
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
    gi, _ = _check(k, q, [L, L], Hq, W, B, s, f"short last chunk s={s}")
    last = (N - 1) // s
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
    gi, _ = _check(k, q, [L], Hq, W, 100, 8, "zero keys")          # 10 chunks of 8, 4 slots of -1
    assert gi[0, 0].tolist() == list(range(80)) + list(range(684, 700)) + [-1] * 4
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
    gi, _ = _check(k, q, [300, 120], Hq, W, 320, 8, "identity")
    assert gi[1, 0].tolist() == list(range(120)) + [-1] * 200
