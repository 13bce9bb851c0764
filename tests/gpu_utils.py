"""Helpers for the GPU parity tests: device transfer, tolerance checks, case labels."""
import functools
import sys

import numpy as np
import torch

import synth

# Tolerance on bf16 attention outputs (fp32 accumulation): |gpu - oracle| <= ATOL + RTOL * |oracle|.
ATOL, RTOL = 2e-2, 1e-2
# Log-sum-exp outputs are fp32: the logits carry fp32 rounding of a 128-term dot
# product (|error| well below 1e-4 for |logit| < 20) and the sum of exponentials
# a relative error below 1e-5, so 1e-3 absolute leaves a wide margin.
LSE_ATOL = 1e-3


def case(msg: str) -> None:
    """Name the GPU step about to run (flushed, so a lost box still shows it)."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def dev():
    return torch.device("cuda:0")


def bf16_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev()).view(torch.bfloat16)


def bf16_host64(t: torch.Tensor) -> np.ndarray:
    b = t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def i32_dev(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).to(dev())


def assert_close(gpu: np.ndarray, ref: np.ndarray, what: str, atol=ATOL, rtol=RTOL):
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    err = np.abs(gpu - ref)
    bound = atol + rtol * np.abs(ref)
    bad = ~(err <= bound)                     # a NaN (an element never written) fails too
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; worst at {i}: "
                             f"gpu {gpu[i]} oracle {ref[i]}")
    return float(err.max()) if err.size else 0.0


def assert_lse(gpu: np.ndarray, ref: np.ndarray, what: str):
    assert not np.isnan(gpu).any(), f"{what}: NaN log-sum-exp"
    both_inf = np.isneginf(gpu) & np.isneginf(ref)
    assert np.array_equal(np.isneginf(gpu), np.isneginf(ref)), f"{what}: -inf pattern differs"
    d = np.abs(np.where(both_inf, 0.0, gpu) - np.where(both_inf, 0.0, ref))   # -inf - -inf is not a number
    assert d.max(initial=0.0) <= LSE_ATOL, f"{what}: lse error {d.max()}"


@functools.lru_cache(maxsize=4)
def config_data(name: str, verifier: bool = False):
    """Per-sequence bf16 bits of a fixed-length workload: (q_tail [S][T][Hq][D], k, v [S][Hkv][L][D])."""
    cfg = synth.workload(name)
    tags = (synth.TAG_K_VERIFIER, synth.TAG_V_VERIFIER) if verifier else (synth.TAG_K, synth.TAG_V)
    qs, ks, vs = synth.kv_batch(cfg, tag_k=tags[0], tag_v=tags[1])
    return np.stack(qs), np.stack(ks), np.stack(vs)


def contiguous_kv(k_bits: np.ndarray, v_bits: np.ndarray):
    return bf16_dev(k_bits), bf16_dev(v_bits)


def paged_kv(k_seqs, v_seqs, table: np.ndarray, num_pages: int, page_size: int):
    """Scatter per-sequence [Hkv][L_s][D] caches into a page pool [num_pages][Hkv][page_size][D]."""
    hkv = k_seqs[0].shape[0]
    kp = np.zeros((num_pages, hkv, page_size, 128), np.uint16)
    vp = np.zeros_like(kp)
    for s, (k, v) in enumerate(zip(k_seqs, v_seqs)):
        L = k.shape[1]
        for pi in range((L + page_size - 1) // page_size):
            pg = table[s, pi]
            n = min(page_size, L - pi * page_size)
            kp[pg, :, :n] = k[:, pi * page_size:pi * page_size + n]
            vp[pg, :, :n] = v[:, pi * page_size:pi * page_size + n]
    return bf16_dev(kp), bf16_dev(vp)


# ---- selection parity at scale: oracle scores computed once, ranked per budget ----------------

def oracle_scores(k_seqs, q_obs, lens, Hq, scale=None):
    """The oracle's raw window scores of every (sequence, KV head): list over s of [Hkv][L_s] float64.

    k_seqs: per sequence [Hkv][>=L_s][128] bf16 bits; q_obs: per sequence [W][Hq][128] bits.
    """
    import oracle as O
    sc = float(np.float64(np.float32(1.0 / np.sqrt(128) if scale is None else scale)))
    out = []
    for s, L in enumerate(lens):
        L = int(L)
        Hkv = k_seqs[s].shape[0]
        G = Hq // Hkv
        qw = O.bf16_to_f64(q_obs[s])
        out.append([O.window_scores(O.bf16_to_f64(k_seqs[s][g, :L]), qw[:, g * G:(g + 1) * G], L, sc)
                    for g in range(Hkv)])
    return out


def check_selection(gi, gn, gs, raws, lens, W, B, what, pool_kernel=7, delta=1e-4, Hq=None):
    """Two-part exact-index protocol of bd_select_kv against oracle scores `raws`.

    (i) the oracle's pooling and ranking applied to the GPU's own fp32 scores gs reproduce the GPU
    indices bit for bit; (ii) the GPU and oracle index sets differ only at positions whose fp64 pooled
    score lies within relative `delta` of the oracle's (B-W)-th score.  The GPU scores also sum to
    W*G per head and match the oracle's to 1e-3.  Returns the number of heads with a near tie.
    """
    import oracle as O
    assert gn.tolist() == [B if B < int(L) else int(L) for L in lens], what
    near = 0
    for s, L in enumerate(lens):
        L = int(L)
        for g in range(gi.shape[1]):
            if B >= L:
                assert gi[s, g].tolist() == list(range(L)) + [-1] * (B - L), (what, s, g)
                continue
            sel, _ = O.topk_from_scores(gs[s, g, :L].astype(np.float64), L, W, B, pool_kernel=pool_kernel)
            assert np.array_equal(gi[s, g], sel), (what, "top-B stage", s, g)
            if Hq is not None:
                G = Hq // gi.shape[1]
                np.testing.assert_allclose(gs[s, g, :L].sum(dtype=np.float64), W * G, rtol=1e-4)
            np.testing.assert_allclose(gs[s, g, :L], raws[s][g], rtol=1e-3, atol=1e-6)
            osel, pooled = O.topk_from_scores(raws[s][g], L, W, B, pool_kernel=pool_kernel)
            diff = set(gi[s, g].tolist()) ^ set(osel.tolist())
            if diff:
                thr = np.sort(pooled)[::-1][B - W - 1]
                for t in diff:
                    assert abs(pooled[t] - thr) <= delta * thr, (what, s, g, t, pooled[t], thr)
                near += 1
    return near


def poison_workspace(nbytes: int, device="cuda"):
    """A bd.Workspace whose bytes past the counter region are all 0xFF (NaN as fp32): scratch a
    kernel reads before writing would show up in its results."""
    import paper_2606_00144_amd as bd
    ws = bd.Workspace()
    buf = ws.get(nbytes, device)
    if buf is not None:
        start = (-buf.data_ptr()) % 256 + (1 << 20)     # the binding aligns the base to 256 bytes
        if buf.numel() > start:
            buf[start:].fill_(255)
    return ws


def fp32_chunk_sums(raw32, N, s):
    """Chunk sums of fp32 scores added left to right in fp32 (the kernel's order)."""
    nc = (N + s - 1) // s
    pad = np.zeros(nc * s, np.float32)
    pad[:N] = raw32[:N]
    pad = pad.reshape(nc, s)
    acc = np.zeros(nc, np.float32)
    for j in range(s):                       # rounded to fp32 after every addition
        acc = (acc + pad[:, j]).astype(np.float32)
    return acc


def check_chunk_selection(gi, gn, gs, oi, on, oraw, lens, W, B, s, cw, what, delta=1e-4):
    """Two-part protocol of bd_select_kv_chunks against the oracle's (oi, on, oraw).

    (i) chunk sums of the GPU's own fp32 scores, added left to right in fp32 and ranked by (sum
    descending, chunk index ascending), give the GPU's indices bit for bit (kept chunks ascending,
    the window, then -1); (ii) the GPU's kept chunks equal the oracle's except chunks whose fp64
    score lies within relative `delta` of the oracle's threshold chunk.  Returns the near-tie count.
    """
    import oracle as O
    ld = B if cw else B + W
    assert gi.shape[2] == ld and oi.shape == gi.shape, what
    assert np.array_equal(gn, on), what
    kept = lambda row, N: sorted({int(t) // s for t in row if 0 <= t < N})
    near = 0
    for si in range(len(lens)):
        L = int(lens[si])
        for g in range(gi.shape[1]):
            if B >= L:
                assert np.array_equal(gi[si, g], oi[si, g]), (what, si, g)
                continue
            N = L - W
            keep = min(((B - W) if cw else B) // s, (N + s - 1) // s)
            cs32 = fp32_chunk_sums(gs[si, g], N, s)
            order = np.lexsort((np.arange(cs32.size), -cs32.astype(np.float64)))
            want_chunks = np.sort(order[:keep])
            want = [t for c in want_chunks for t in range(c * s, min((c + 1) * s, N))]
            want = want + list(range(N, L))
            want = want + [-1] * (ld - len(want))
            assert gi[si, g].tolist() == want, (what, "chunk ranking stage", si, g)
            diff = set(kept(gi[si, g], N)) ^ set(kept(oi[si, g], N))
            if diff:
                cs = O.chunk_scores(oraw[si][g][:N], s)
                thr = np.sort(cs)[::-1][keep - 1]
                for c in diff:
                    assert abs(cs[c] - thr) <= delta * thr, (what, si, g, c, cs[c], thr)
                near += 1
    return near


def oracle_chunk_selection(raws, lens, Hkv, W, B, s, cw):
    """The oracle's TopKChunks lists from precomputed oracle scores (its ranking steps only)."""
    import oracle as O
    S = len(lens)
    ld = B if cw else B + W
    idx = np.full((S, Hkv, ld), -1, np.int32)
    nsel = np.zeros(S, np.int32)
    for si, L in enumerate(lens):
        L = int(L)
        if B >= L:
            idx[si, :, :L] = np.arange(L)
            nsel[si] = L
            continue
        for g in range(Hkv):
            sel, _ = O.topk_chunks_from_scores(raws[si][g], L, W, B, s, budget_counts_window=cw)
            idx[si, g, :sel.size] = sel
        nsel[si] = min(ld, L)
    return idx, nsel
