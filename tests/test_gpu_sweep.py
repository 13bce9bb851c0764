"""Seeded sweeps of selection, decode, verify and acceptance over random shapes against the fp64 oracle.

Each case draws the batch, the KV head count and group size, and ragged cache lengths.  Selection
cases also draw:
  - the window (1..64 rows), budget (below, at and above the cache length), scale and pooling width;
  - the query magnitude (standard deviation 1 or 4);
  - token or chunk mode (chunk sizes 1..16), with both budget readings;
  - a contiguous or paged cache (random page order, page size 16 or 32).
Decode and verify cases also draw:
  - gamma (0..7), the list width and the query magnitude (standard deviation 1, 4 or 16: logits
    spanning tens of nats, so the lazily raised reference maximum moves often);
  - per-sequence entry counts (zero, partial, full), absent (-1) and out-of-range entries, and
    garbage past the count;
  - a contiguous or paged cache.
Acceptance cases draw the batch, gamma (0..15), vocabularies of 1..200K entries with padded rows,
ties and entries at the most negative float.
A last case runs verify and decode over one 131,072-row cache (the drafter model's context length).
Outputs are preallocated and poisoned first (indices with a sentinel, floats with NaN), so an
output the kernels never write fails.  Indices follow the two-part exact protocol of the selection
tests; bf16 outputs are within 2e-2 + 1e-2 |oracle|, log-sum-exps within 1e-3.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import (assert_close, assert_lse, bf16_dev, bf16_host64, case, check_chunk_selection,
                       check_selection, i32_dev, oracle_chunk_selection, oracle_scores, paged_kv)

pytestmark = pytest.mark.gpu


def _bits(g, shape, sd=1.0):
    return synth.f32_to_bf16_bits((sd * g.standard_normal(shape, dtype=np.float32)).astype(np.float32))


def _page_table(g, lens, ps):
    """A random page order for every sequence's pages: table [S][max_pages] (-1 past a sequence's
    last page) and the pool size."""
    npg = [(int(L) + ps - 1) // ps for L in lens]
    perm = g.permutation(sum(npg)).astype(np.int32)
    table = np.full((len(lens), max(npg)), -1, np.int32)
    o = 0
    for s, n in enumerate(npg):
        table[s, :n] = perm[o:o + n]
        o += n
    return table, int(sum(npg))


def _cache(g, k, v, lens, paged):
    """Device K/V (V may be None) as given, or scattered into a paged pool; the page table or None."""
    if not paged:
        return bf16_dev(k), (bf16_dev(v) if v is not None else None), None
    ps = int(g.choice([8, 16, 32, 48]))   # multiples of 16 take the per-page table, 8 the per-key one
    table, npages = _page_table(g, lens, ps)
    ks = [k[s][:, :int(L)] for s, L in enumerate(lens)]
    vs = [(v if v is not None else k)[s][:, :int(L)] for s, L in enumerate(lens)]
    kd, vd = paged_kv(ks, vs, table, npages, ps)
    return kd, (vd if v is not None else None), i32_dev(table)


def _draw_select(seed):
    g = np.random.default_rng(5000 + seed)
    S = int(g.integers(1, 4))
    Hkv = int(g.choice([1, 2, 4]))
    G = int(g.choice([1, 2, 4, 8]))
    W = int(g.choice([1, 4, 16, 32, 64]))
    while W * G > 256:                       # up to two 128-row blocks; keeps the oracle quick
        W //= 2
    lens = [int(g.integers(W, 3000)) for _ in range(S)]
    B = int(g.integers(W, 1400))
    pool = int(g.choice([1, 3, 5, 7, 9]))
    chunk = int(g.choice([0, 0, 1, 5, 8, 16]))   # 0: token mode
    cw = bool(g.random() < 0.5)
    paged = bool(g.random() < 0.35)
    scale = None if g.random() < 0.7 else float(g.uniform(0.03, 0.2))
    # query magnitude: up to sd 4, so the boundary scores stay normal fp32 numbers (where they would
    # underflow in fp32 but not in fp64, the two precisions rank them differently by definition)
    qsd = float(g.choice([1.0, 4.0]))
    return g, S, Hkv, G, W, lens, B, pool, chunk, cw, paged, scale, qsd


@pytest.mark.parametrize("seed", list(range(24)))
def test_select_random_shapes(seed):
    g, S, Hkv, G, W, lens, B, pool, chunk, cw, paged, scale, qsd = _draw_select(seed)
    Hq = Hkv * G
    k = _bits(g, (S, Hkv, max(lens), 128))
    q = _bits(g, (S, W, Hq, 128), qsd)
    kd, _, table = _cache(g, k, None, lens, paged)
    what = (f"select sweep {seed}: S={S} Hkv={Hkv} G={G} W={W} B={B} lens={lens} pool={pool} chunk={chunk} "
            f"cw={cw} paged={paged} scale={scale} q_sd={qsd}")
    case(what)
    ld = B if (chunk == 0 or cw) else B + W
    idx = torch.full((S, Hkv, ld), -7, dtype=torch.int32, device="cuda")
    nsel = torch.full((S,), -7, dtype=torch.int32, device="cuda")
    scores = torch.full((S, Hkv, max(lens)), float("nan"), dtype=torch.float32, device="cuda")
    if chunk == 0:
        bd.bd_select_kv(kd, bf16_dev(q), i32_dev(lens), B, pool_kernel=pool, scale=scale, return_scores=True,
                        page_table=table, max_seq_len=max(lens), outputs=(idx, nsel, scores))
    else:
        bd.bd_select_kv_chunks(kd, bf16_dev(q), i32_dev(lens), B, chunk=chunk, budget_counts_window=cw,
                               scale=scale, return_scores=True, page_table=table, max_seq_len=max(lens),
                               outputs=(idx, nsel, scores))
    torch.cuda.synchronize()
    gi, gn, gs = idx.cpu().numpy(), nsel.cpu().numpy(), scores.cpu().numpy()
    raws = oracle_scores(k, q, lens, Hq, scale)
    if chunk == 0:
        near = check_selection(gi, gn, gs, raws, lens, W, B, what, pool_kernel=pool, Hq=Hq)
    else:
        oi, on = oracle_chunk_selection(raws, lens, Hkv, W, B, chunk, cw)
        near = check_chunk_selection(gi, gn, gs, oi, on, raws, lens, W, B, chunk, cw, what)
    assert near <= S * Hkv, what


def _draw_attn(seed):
    g = np.random.default_rng(6000 + seed)
    S = int(g.integers(1, 5))
    Hkv = int(g.choice([1, 2, 4, 8]))
    G = int(g.choice([1, 2, 4, 8]))
    gamma = int(g.integers(0, 8))
    lens = [int(g.integers(gamma + 1, 5000)) for _ in range(S)]
    ld = int(g.integers(1, 2100))
    paged = bool(g.random() < 0.4)
    scale = None if g.random() < 0.7 else float(g.uniform(0.03, 0.2))
    qsd = float(g.choice([1.0, 4.0, 16.0]))
    return g, S, Hkv, G, gamma, lens, ld, paged, scale, qsd


def _lists(g, S, Hkv, lens, ld):
    """Decode lists: per sequence an entry count (zero, partial or the full width); per head distinct
    in-range positions with some absent (-1) and out-of-range (>= L) entries; garbage past the count."""
    idx = g.integers(-5, max(lens) + 60, (S, Hkv, ld)).astype(np.int32)
    nsel = np.zeros(S, np.int32)
    for s, L in enumerate(lens):
        r = g.random()
        n = 0 if r < 0.1 else (ld if r < 0.4 else int(g.integers(1, ld + 1)))
        nsel[s] = n
        for h in range(Hkv):
            m = min(n, L)
            row = g.choice(L, m, replace=False).astype(np.int32)
            if m:
                holes = g.random(m) < 0.05
                row[holes] = np.where(g.random(holes.sum()) < 0.5, -1, L + g.integers(0, 50, holes.sum()))
            idx[s, h, :m] = row
            idx[s, h, m:n] = -1
    return idx, nsel


@pytest.mark.parametrize("seed", list(range(24)))
def test_decode_verify_random_shapes(seed):
    g, S, Hkv, G, gamma, lens, ld, paged, scale, qsd = _draw_attn(seed)
    Hq = Hkv * G
    Lm = max(lens)
    k, v = _bits(g, (S, Hkv, Lm, 128)), _bits(g, (S, Hkv, Lm, 128))
    qv = _bits(g, (S, gamma + 1, Hq, 128), qsd)
    qd = _bits(g, (S, Hq, 128), qsd)
    idx, nsel = _lists(g, S, Hkv, lens, ld)
    if seed % 4 == 3:
        nsel[0] = 0                          # an empty list: zero output, -inf log-sum-exp
    kd, vd, table = _cache(g, k, v, lens, paged)
    what = (f"attn sweep {seed}: S={S} Hkv={Hkv} G={G} gamma={gamma} ld={ld} lens={lens} paged={paged} "
            f"scale={scale} q_sd={qsd}")
    nan16 = lambda shape: torch.full(shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    nan32 = lambda shape: torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")

    case(what + " decode")
    out, lse = nan16((S, Hq, 128)), nan32((S, Hq))
    bd.bd_sparse_decode_attn(kd, vd, bf16_dev(qd), i32_dev(idx), i32_dev(nsel), i32_dev(lens), scale=scale,
                             return_lse=True, page_table=table, max_seq_len=Lm, out=out, lse=lse)
    torch.cuda.synchronize()
    ro, rl = O.sparse_decode_attn(k, v, qd, idx, nsel, lens, scale=scale)
    assert_close(bf16_host64(out), ro, what + " decode")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, what + " decode")

    case(what + " verify")
    out, lse = nan16((S, gamma + 1, Hq, 128)), nan32((S, gamma + 1, Hq))
    bd.bd_verify_attn(kd, vd, bf16_dev(qv), i32_dev(lens), scale=scale, return_lse=True, page_table=table,
                      max_seq_len=Lm, out=out, lse=lse)
    torch.cuda.synchronize()
    ro, rl = O.verify_attn(k, v, qv, lens, gamma, scale=scale)
    assert_close(bf16_host64(out), ro, what + " verify")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, what + " verify")


def _draw_accept(seed):
    g = np.random.default_rng(7000 + seed)
    S = int(g.integers(1, 65))
    gamma = int(g.integers(0, 16))
    V = int(g.choice([int(g.integers(1, 64)), int(g.integers(64, 5000)), int(g.integers(5000, 200000))]))
    pad = int(g.choice([0, 0, 1, 3, 64]))    # row stride V + pad
    ties = bool(g.random() < 0.4)
    return g, S, gamma, V, pad, ties


@pytest.mark.parametrize("seed", list(range(24)))
def test_accept_random_shapes(seed):
    """Greedy acceptance on seeded shapes: vocabularies of 1..200K (vector and scalar scans), padded
    rows, heavy ties and entries at the most negative float, maxima at either end, drafts matching a
    planted prefix; accepted lengths, bonus tokens and argmax bit-exact against the oracle."""
    g, S, gamma, V, pad, ties = _draw_accept(seed)
    R = gamma + 1
    big = g.standard_normal((S, R, V + pad)).astype(np.float32)
    if ties:
        big = np.floor(big * 1.5).astype(np.float32)
    big[g.random(big.shape) < 0.01] = -np.finfo(np.float32).max   # logits are finite by contract
    for s in range(S):                       # maxima planted at the first or the last index of some rows
        i = int(g.integers(0, R))
        big[s, i, 0 if g.random() < 0.5 else V - 1] = 100.0
    logits = big[:, :, :V]
    am = np.array([[O.greedy_argmax(logits[s, i]) for i in range(R)] for s in range(S)], np.int32).reshape(S, R)
    draft = g.integers(0, V, (S, gamma)).astype(np.int32)
    for s in range(S):
        m = int(g.integers(0, gamma + 1))
        draft[s, :m] = am[s, :m]
    what = f"accept sweep {seed}: S={S} gamma={gamma} V={V} pad={pad} ties={ties}"
    case(what)
    dbig = torch.from_numpy(big).to("cuda")
    acc = torch.full((S,), -7, dtype=torch.int32, device="cuda")
    bonus = torch.full((S,), -7, dtype=torch.int32, device="cuda")
    gam = torch.full((S, R), -7, dtype=torch.int32, device="cuda")
    bd.bd_accept_len(dbig[:, :, :V], i32_dev(draft), return_argmax=True, outputs=(acc, bonus, gam))
    torch.cuda.synchronize()
    ra, rb, ram = O.accept_len(logits, draft, gamma)
    assert np.array_equal(gam.cpu().numpy(), ram), what
    assert np.array_equal(acc.cpu().numpy(), ra), what
    assert np.array_equal(bonus.cpu().numpy(), rb), what


def test_long_context_verify_and_decode():
    """One sequence with 131,072 cache rows (the drafter model's context length), GQA 32/8: verify at
    gamma = 5 over the whole cache, and decode over 2,048 entries spread across it, against the
    oracle; outputs poisoned first."""
    g = np.random.default_rng(8000)
    L, Hkv, G, gamma = 131072, 8, 4, 5
    Hq = Hkv * G
    k, v = _bits(g, (1, Hkv, L, 128)), _bits(g, (1, Hkv, L, 128))
    q = _bits(g, (1, gamma + 1, Hq, 128))
    idx = np.stack([np.sort(g.choice(L, 2048, replace=False)) for _ in range(Hkv)]).astype(np.int32)[None]
    kd, vd = bf16_dev(k), bf16_dev(v)
    what = f"long context L={L} Hkv={Hkv} G={G}"
    case(what + " verify")
    out = torch.full((1, gamma + 1, Hq, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((1, gamma + 1, Hq), float("nan"), dtype=torch.float32, device="cuda")
    bd.bd_verify_attn(kd, vd, bf16_dev(q), i32_dev([L]), return_lse=True, out=out, lse=lse)
    torch.cuda.synchronize()
    ro, rl = O.verify_attn(k, v, q, [L], gamma)
    assert_close(bf16_host64(out), ro, what + " verify")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, what + " verify")
    case(what + " decode")
    out = torch.full((1, Hq, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((1, Hq), float("nan"), dtype=torch.float32, device="cuda")
    qd = np.ascontiguousarray(q[:, -1])
    bd.bd_sparse_decode_attn(kd, vd, bf16_dev(qd), i32_dev(idx), i32_dev([2048]), i32_dev([L]), return_lse=True,
                             out=out, lse=lse)
    torch.cuda.synchronize()
    ro, rl = O.sparse_decode_attn(k, v, qd, idx, [2048], [L])
    assert_close(bf16_host64(out), ro, what + " decode")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, what + " decode")
