"""Plain, slow, fp64 reference of the BudgetDraft sparse-drafter / full-verifier path.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  It shares no code
with the HIP path: inputs arrive as bf16 bit patterns (``uint16``) or fp32
arrays and are widened here, exactly, to float64.

Every function states the passage of the paper it follows.  Where the paper
is silent, the reading taken is stated in the docstring (the selection
policy, window, pooling and tie rules come from the workload description the
kernels are measured on, not from the paper, which only names chunk-level
selection ranked by accumulated attention weight, in Sec. 3.4).

Conventions (shared with the C ABI):
  * Query head h reads KV head g(h) = h // G, G = Hq / Hkv (contiguous groups).
  * Causal rule: a key at position t is visible to a query at position p iff
    0 <= t <= p.  Sequence s holds cache rows 0 .. L_s-1, the query tail
    included; the last query row sits at position L_s - 1.
  * scale: the caller's fp32 softmax scale, promoted exactly to float64.
  * An empty key set gives output 0 and log-sum-exp -inf.

Parity status: every function here is pinned by the CPU tests in
``tests/test_oracle_pins.py`` (closed forms, invariants, library routines and
brute force on tiny inputs); none is "parity unpinned".
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np


# --------------------------------------------------------------------------
# Input widening
# --------------------------------------------------------------------------

def bf16_to_f64(bits) -> np.ndarray:
    """bf16 bit patterns -> float64, exactly: (bits << 16) viewed as float32, widened."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _scale64(scale: Optional[float], head_dim: int) -> float:
    if scale is None:
        scale = 1.0 / np.sqrt(head_dim)
    return float(np.float64(np.float32(scale)))


# --------------------------------------------------------------------------
# Attention by definition (Eq. 1 and Eq. 2)
# --------------------------------------------------------------------------

def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, visible: np.ndarray, scale: float):
    """Softmax attention of query rows over the keys each row may see.

    Eq. (1)/(2): a distribution conditions on a KV cache through attention;
    for one row, weights p_t = exp(l_t) / sum_u exp(l_u) with
    l_t = scale * <q, k_t> over the visible keys t, output sum_t p_t v_t.

    q [R][D], k [N][D], v [N][D] float64; visible [R][N] bool.
    Returns out [R][D] float64 and lse [R] (natural log of sum_t exp l_t).
    """
    R, D = q.shape
    out = np.zeros((R, D), dtype=np.float64)
    lse = np.full(R, -np.inf, dtype=np.float64)
    if k.shape[0] == 0:
        return out, lse
    visible = np.asarray(visible, dtype=bool)
    has = visible.any(axis=1)                        # rows with at least one key
    logits = scale * (q @ k.T)                       # [R][N]
    m = np.where(visible, logits, -np.inf).max(axis=1)
    m = np.where(has, m, 0.0)
    e = np.where(visible, np.exp(np.where(visible, logits, 0.0) - m[:, None]), 0.0)   # unnormalised weights
    z = e.sum(axis=1)
    out[has] = (e[has] @ v) / z[has, None]
    lse[has] = m[has] + np.log(z[has])
    return out, lse


# --------------------------------------------------------------------------
# Budgeted KV selection (Alg. 2 "sparsify"; Sec. 3.4: entries ranked by accumulated attention weight)
# --------------------------------------------------------------------------

def window_scores(k_g: np.ndarray, q_obs: np.ndarray, L: int, scale: float) -> np.ndarray:
    """Cumulative attention weight of every cached key under the observation rows.

    Sec. 3.4 ranks cache entries by the attention weight they accumulate; here the
    weights are those of the W observation rows of every query head of the
    group (reading: probabilities, each row normalised over its own causal
    key range, summed over rows and heads).

    k_g [L][D] float64 (one KV head), q_obs [W][G][D] float64 at positions
    L-W .. L-1.  Returns raw [L] float64.
    """
    W, G, _ = q_obs.shape
    raw = np.zeros(L, dtype=np.float64)
    for h in range(G):
        logits = scale * (q_obs[:, h, :] @ k_g.T)          # [W][L]
        for i in range(W):
            p = L - W + i                                 # position of row i
            row = logits[i, :p + 1]
            a = np.exp(row - row.max())
            a /= a.sum()
            raw[:p + 1] += a
    return raw


def max_pool(x: np.ndarray, kernel: int) -> np.ndarray:
    """Stride-1 centred max filter of odd width ``kernel``; windows are cut at both ends."""
    r = kernel // 2
    n = x.shape[0]
    out = x.copy()
    for o in range(1, r + 1):
        if o >= n:
            break
        out[:n - o] = np.maximum(out[:n - o], x[o:])
        out[o:] = np.maximum(out[o:], x[:n - o])
    return out


def topk_from_scores(raw: np.ndarray, L: int, window: int, budget: int, pool_kernel: int = 7,
                     budget_counts_window: bool = True) -> Tuple[np.ndarray, np.ndarray]:
    """Pool the prefix scores and keep the budget (selection steps after scoring).

    Candidates are the prefix positions [0, N), N = L - W; the W window
    positions are always kept.  Reading of the budget: B counts the window, so
    B - W prefix entries are kept (``budget_counts_window=False`` keeps B).
    Order: larger pooled score first, lower position first among equal scores.
    Returns (selected positions ascending, window appended) and pooled [N].
    """
    N = L - window
    pooled = max_pool(np.asarray(raw[:N], dtype=np.float64), pool_kernel)
    keep = budget - window if budget_counts_window else budget
    keep = max(0, min(keep, N))
    pos = np.arange(N)
    order = np.lexsort((pos, -pooled))                  # primary: -pooled, secondary: position
    chosen = np.sort(order[:keep])
    sel = np.concatenate([chosen, np.arange(N, L)]).astype(np.int32)
    return sel, pooled


def select_kv(k, q_win, seq_lens, num_q_heads: int, window: int, budget: int, pool_kernel: int = 7,
              scale: Optional[float] = None, budget_counts_window: bool = True):
    """K_S^sp(B) as an index set per (sequence, KV head): Alg. 2 "sparsify".

    k: per sequence [Hkv][>=L_s][D] bf16 bits; q_win: per sequence [W][Hq][D]
    bf16 bits (the last W query rows).  Returns idx [S][Hkv][B] int32 (tail -1; B + W slots with
    ``budget_counts_window=False``), nsel [S] int32 (min(slots, L_s)) and raw scores (list of
    [Hkv][L_s] float64).

    B >= L_s keeps every position (the sparse cache equals the full cache).
    """
    if window < 1 or budget < window or pool_kernel < 1 or pool_kernel % 2 == 0:
        raise ValueError("invalid selection arguments")
    S = len(seq_lens)
    Hkv = k[0].shape[0]
    G = num_q_heads // Hkv
    D = k[0].shape[-1]
    sc = _scale64(scale, D)
    out_budget = budget if budget_counts_window else budget + window
    idx = np.full((S, Hkv, out_budget), -1, dtype=np.int32)
    nsel = np.zeros(S, dtype=np.int32)
    raws = []
    for s in range(S):
        L = int(seq_lens[s])
        if window > L:
            raise ValueError("window longer than the sequence")
        qw = bf16_to_f64(q_win[s])                       # [W][Hq][D]
        raw_s = np.zeros((Hkv, L))
        if budget >= L:
            idx[s, :, :L] = np.arange(L, dtype=np.int32)
            nsel[s] = L
            raws.append(raw_s)
            continue
        for g in range(Hkv):
            kg = bf16_to_f64(k[s][g, :L])
            raw = window_scores(kg, qw[:, g * G:(g + 1) * G, :], L, sc)
            sel, _ = topk_from_scores(raw, L, window, budget, pool_kernel, budget_counts_window)
            idx[s, g, :sel.size] = sel
            raw_s[g] = raw
        nsel[s] = min(out_budget, L)
        raws.append(raw_s)
    return idx, nsel, raws


def chunk_scores(raw_prefix: np.ndarray, chunk: int) -> np.ndarray:
    """Score of every chunk of the prefix: the sum of its positions' cumulative attention weight.

    Sec. 3.4 partitions the prefix cache into chunks of ``chunk`` positions and scores each
    chunk by cumulative attention weight.  Chunk c covers [c*chunk, min((c+1)*chunk, N)); the
    last chunk is shorter when N is not a multiple of ``chunk``.
    """
    x = np.asarray(raw_prefix, dtype=np.float64)
    N = x.shape[0]
    nc = (N + chunk - 1) // chunk
    out = np.zeros(nc, dtype=np.float64)
    for c in range(nc):
        out[c] = x[c * chunk:min((c + 1) * chunk, N)].sum()
    return out


def topk_chunks_from_scores(raw: np.ndarray, L: int, window: int, budget: int,
                            chunk: int = 8, budget_counts_window: bool = False) -> Tuple[np.ndarray, np.ndarray]:
    """TopKChunks (Sec. 3.4; Alg. 1 step 4, Alg. 2 "sparsify"): the chunk-level selection.

    Sec. 3.4 cuts the prefix cache into chunks of s = ``chunk`` positions, scores every chunk by
    cumulative attention weight and retains the top floor(B / s) chunks; the continuation rows
    (here the W scoring rows at positions N .. L-1, N = L - W) attend on top of them (Alg. 1
    step 4).  So the prefix [0, N) is cut into chunks (the last one shorter when s does not divide
    N), the top floor(B / s) chunks are kept (larger score first, lower chunk index among equal
    scores), their positions returned in ascending order, and the W window positions appended.
    ``budget_counts_window=True`` takes the other reading, where B also pays for the window:
    floor((B - W) / s) chunks.  A kept short last chunk contributes fewer than s positions.
    Returns (positions, chunk scores).
    """
    N = L - window
    cs = chunk_scores(raw[:N], chunk)
    nc = cs.shape[0]
    prefix_budget = budget - window if budget_counts_window else budget
    keep = max(0, min(prefix_budget // chunk, nc))
    order = np.lexsort((np.arange(nc), -cs))            # primary: -score, secondary: chunk index
    chosen = np.sort(order[:keep])
    parts = [np.arange(c * chunk, min((c + 1) * chunk, N)) for c in chosen]
    sel = np.concatenate(parts + [np.arange(N, L)]).astype(np.int32)
    return sel, cs


def select_kv_chunks(k, q_win, seq_lens, num_q_heads: int, window: int, budget: int, chunk: int = 8,
                     scale: Optional[float] = None, budget_counts_window: bool = False):
    """K_S^sp(B) by TopKChunks per (sequence, KV head): scoring as select_kv, chunk selection.

    Each head's list has ``ld`` slots, ld = B + W (the paper's count: B pays for prefix chunks
    only) or B (``budget_counts_window``).  Returns idx [S][Hkv][ld] int32 (slots past a head's
    kept positions hold -1), nsel [S] = min(ld, L_s) (slots, not kept positions) and the raw
    scores.  B >= L_s keeps every position (nsel = L_s).
    """
    if window < 1 or budget < window or chunk < 1:
        raise ValueError("invalid selection arguments")
    S = len(seq_lens)
    Hkv = k[0].shape[0]
    G = num_q_heads // Hkv
    D = k[0].shape[-1]
    sc = _scale64(scale, D)
    ld = budget if budget_counts_window else budget + window
    idx = np.full((S, Hkv, ld), -1, dtype=np.int32)
    nsel = np.zeros(S, dtype=np.int32)
    raws = []
    for s in range(S):
        L = int(seq_lens[s])
        if window > L:
            raise ValueError("window longer than the sequence")
        qw = bf16_to_f64(q_win[s])
        raw_s = np.zeros((Hkv, L))
        if budget >= L:
            idx[s, :, :L] = np.arange(L, dtype=np.int32)
            nsel[s] = L
            raws.append(raw_s)
            continue
        for g in range(Hkv):
            kg = bf16_to_f64(k[s][g, :L])
            raw = window_scores(kg, qw[:, g * G:(g + 1) * G, :], L, sc)
            sel, _ = topk_chunks_from_scores(raw, L, window, budget, chunk, budget_counts_window)
            idx[s, g, :sel.size] = sel
            raw_s[g] = raw
        nsel[s] = min(ld, L)
        raws.append(raw_s)
    return idx, nsel, raws


# --------------------------------------------------------------------------
# Drafter decode attention over the selected entries (Eq. 2; Alg. 2 "draft")
# --------------------------------------------------------------------------

def _valid_entries(idx_row: np.ndarray, n: int, L: int) -> np.ndarray:
    n = max(0, min(int(n), idx_row.shape[0]))
    j = idx_row[:n].astype(np.int64)
    return j[(j >= 0) & (j < L)]


def sparse_decode_attn(k, v, q, idx, nsel, seq_lens, scale: Optional[float] = None):
    """p_S(. | x_<t; K_S^sp(B)) attention for one decode query per head (Eq. 2).

    q [S][Hq][D] bits at position L_s-1; idx [S][Hkv][ld] positions (entries
    outside [0, L_s) are skipped), nsel [S] used entries.  Returns out
    [S][Hq][D] float64, lse [S][Hq].
    """
    S, Hq, D = q.shape
    Hkv = k[0].shape[0]
    G = Hq // Hkv
    sc = _scale64(scale, D)
    out = np.zeros((S, Hq, D))
    lse = np.full((S, Hq), -np.inf)
    for s in range(S):
        L = int(seq_lens[s])
        qs = bf16_to_f64(q[s])
        for g in range(Hkv):
            J = _valid_entries(idx[s, g], nsel[s], L)
            kg = bf16_to_f64(k[s][g][J])
            vg = bf16_to_f64(v[s][g][J])
            vis = np.ones((G, J.size), dtype=bool)
            o, l = attend(qs[g * G:(g + 1) * G], kg, vg, vis, sc)
            out[s, g * G:(g + 1) * G] = o
            lse[s, g * G:(g + 1) * G] = l
    return out, lse


# --------------------------------------------------------------------------
# Verifier full-KV attention at the gamma+1 draft positions (Eq. 1; Alg. 2 "verify")
# --------------------------------------------------------------------------

def verify_attn(k, v, q, seq_lens, gamma: int, scale: Optional[float] = None):
    """p_L(. | x_<t; K_L^full) attention for the gamma+1 verifier rows (Eq. 1).

    Row j of q [S][gamma+1][Hq][D] sits at position L_s - gamma - 1 + j and
    sees keys 0 .. that position.  Returns out [S][gamma+1][Hq][D], lse [S][gamma+1][Hq].
    """
    S, R, Hq, D = q.shape
    assert R == gamma + 1
    Hkv = k[0].shape[0]
    G = Hq // Hkv
    sc = _scale64(scale, D)
    out = np.zeros((S, R, Hq, D))
    lse = np.full((S, R, Hq), -np.inf)
    for s in range(S):
        L = int(seq_lens[s])
        qs = bf16_to_f64(q[s])                           # [R][Hq][D]
        pos = L - gamma - 1 + np.arange(R)
        t = np.arange(L)
        vis_rows = t[None, :] <= pos[:, None]            # [R][L]
        for g in range(Hkv):
            kg = bf16_to_f64(k[s][g, :L])
            vg = bf16_to_f64(v[s][g, :L])
            qg = qs[:, g * G:(g + 1) * G, :].reshape(R * G, D)        # row-major (j, h)
            vis = np.repeat(vis_rows, G, axis=0)
            o, l = attend(qg, kg, vg, vis, sc)
            out[s, :, g * G:(g + 1) * G] = o.reshape(R, G, D)
            lse[s, :, g * G:(g + 1) * G] = l.reshape(R, G)
    return out, lse


# --------------------------------------------------------------------------
# Multi-view block attention (Alg. 1 steps 3-4: full-cache and sparse-cache branches)
# --------------------------------------------------------------------------

def multiview_attn(k, v, q_blk, idx_views, nsel_views, seq_lens, scale: Optional[float] = None,
                   with_full: bool = True, return_lse: bool = False):
    """Continuation block attended under several sparse views and the full cache.

    Alg. 1: the continuation rows attend Clone(K_S^full) (full branch, step 3)
    and K_S^sp(B) for a sampled budget (sparse branch, step 4), with real
    position ids.  Row c of q_blk [S][C][Hq][D] sits at position L_s - C + c.
    View v sees {t in idx_views[v, s, g, :nsel] : t <= position}; the full
    branch sees {t <= position}.
    Returns out_views [V][S][C][Hq][D] and out_full [S][C][Hq][D] (or None);
    with return_lse also their log-sum-exps [V][S][C][Hq] and [S][C][Hq] (or None).
    """
    S, C, Hq, D = q_blk.shape
    nv = len(idx_views)
    Hkv = k[0].shape[0]
    G = Hq // Hkv
    sc = _scale64(scale, D)
    out_v = np.zeros((nv, S, C, Hq, D))
    out_f = np.zeros((S, C, Hq, D)) if with_full else None
    lse_v = np.zeros((nv, S, C, Hq))
    lse_f = np.zeros((S, C, Hq)) if with_full else None
    for s in range(S):
        L = int(seq_lens[s])
        qs = bf16_to_f64(q_blk[s])
        pos = L - C + np.arange(C)
        for g in range(Hkv):
            qg = qs[:, g * G:(g + 1) * G, :].reshape(C * G, D)
            kg_all = bf16_to_f64(k[s][g, :L])
            vg_all = bf16_to_f64(v[s][g, :L])
            for vi in range(nv):
                J = _valid_entries(idx_views[vi][s, g], nsel_views[vi][s], L)
                vis = np.repeat(J[None, :] <= pos[:, None], G, axis=0)
                o, lse = attend(qg, kg_all[J], vg_all[J], vis, sc)
                out_v[vi, s, :, g * G:(g + 1) * G] = o.reshape(C, G, D)
                lse_v[vi, s, :, g * G:(g + 1) * G] = lse.reshape(C, G)
            if with_full:
                t = np.arange(L)
                vis = np.repeat(t[None, :] <= pos[:, None], G, axis=0)
                o, lse = attend(qg, kg_all, vg_all, vis, sc)
                out_f[s, :, g * G:(g + 1) * G] = o.reshape(C, G, D)
                lse_f[s, :, g * G:(g + 1) * G] = lse.reshape(C, G)
    return (out_v, out_f, lse_v, lse_f) if return_lse else (out_v, out_f)


def attend_backward(q, k, v, visible, scale: float, dout):
    """Gradients of ``attend`` with respect to q, k and v for an upstream gradient dout [R][D].

    With p_rt the softmax weights of row r over its visible keys and out_r = sum_t p_rt v_t:
    dv_t = sum_r p_rt dout_r; dp_rt = <dout_r, v_t>; D_r = <dout_r, out_r>;
    ds_rt = p_rt (dp_rt - D_r); dq_r = scale sum_t ds_rt k_t; dk_t = scale sum_r ds_rt q_r.
    Returns dq [R][D], dk [N][D], dv [N][D] float64.
    """
    R, D = q.shape
    N = k.shape[0]
    dq, dk, dv = np.zeros((R, D)), np.zeros((N, D)), np.zeros((N, D))
    if N == 0:
        return dq, dk, dv
    out, lse = attend(q, k, v, visible, scale)
    visible = np.asarray(visible, dtype=bool)
    has = visible.any(axis=1)
    logits = scale * (q @ k.T)
    p = np.where(visible & has[:, None], np.exp(np.where(visible, logits, 0.0) - np.where(has, lse, 0.0)[:, None]), 0.0)
    dv = p.T @ dout
    dp = dout @ v.T
    Dr = (dout * out).sum(axis=1)
    ds = p * (dp - Dr[:, None])
    dq = scale * (ds @ k)
    dk = scale * (ds.T @ q)
    return dq, dk, dv


def multiview_attn_bwd(k, v, q_blk, idx_views, nsel_views, seq_lens, dout_views, dout_full,
                       scale: Optional[float] = None):
    """Backward of ``multiview_attn`` for the drafter's training losses.

    Alg. 1 back-propagates L_A and L_C through the continuation's full-cache and
    sparse-cache branches (steps 3-5); the prefix cache is computed without
    gradient (step 2), so of the keys and values only the block's own rows,
    positions L_s-C .. L_s-1, receive gradients.  Gradients of the views and the
    full branch add up.  dout_views [V][S][C][Hq][D], dout_full [S][C][Hq][D]
    (or None): upstream gradients of the two outputs.
    Returns dq [S][C][Hq][D], dk_blk [S][C][Hkv][D], dv_blk [S][C][Hkv][D] float64.
    """
    S, C, Hq, D = q_blk.shape
    nv = len(idx_views)
    Hkv = k[0].shape[0]
    G = Hq // Hkv
    sc = _scale64(scale, D)
    dq = np.zeros((S, C, Hq, D))
    dk = np.zeros((S, C, Hkv, D))
    dv = np.zeros((S, C, Hkv, D))
    for s in range(S):
        L = int(seq_lens[s])
        qs = bf16_to_f64(q_blk[s])
        pos = L - C + np.arange(C)
        for g in range(Hkv):
            qg = qs[:, g * G:(g + 1) * G, :].reshape(C * G, D)
            kg_all = bf16_to_f64(k[s][g, :L])
            vg_all = bf16_to_f64(v[s][g, :L])
            branches = []
            for vi in range(nv):
                J = _valid_entries(idx_views[vi][s, g], nsel_views[vi][s], L)
                branches.append((J, np.asarray(dout_views[vi][s][:, g * G:(g + 1) * G], dtype=np.float64)))
            if dout_full is not None:
                branches.append((np.arange(L), np.asarray(dout_full[s][:, g * G:(g + 1) * G], dtype=np.float64)))
            for J, do in branches:
                vis = np.repeat(J[None, :] <= pos[:, None], G, axis=0)
                gq, gk, gv = attend_backward(qg, kg_all[J], vg_all[J], vis, sc, do.reshape(C * G, D))
                dq[s, :, g * G:(g + 1) * G] += gq.reshape(C, G, D)
                for j, t in enumerate(J):
                    if t >= L - C:                        # a block row: it carries a gradient
                        dk[s, t - (L - C), g] += gk[j]
                        dv[s, t - (L - C), g] += gv[j]
    return dq, dk, dv


# --------------------------------------------------------------------------
# Greedy acceptance (Eq. 3; Alg. 2 accept and bonus token)
# --------------------------------------------------------------------------

def greedy_argmax(row: np.ndarray) -> int:
    """argmax_v of one logit row, lowest index among equal maxima (Eq. 3, Eq. 5)."""
    r = np.asarray(row, dtype=np.float64)
    if not np.all(np.isfinite(r)):
        raise ValueError("logits must be finite")
    m = r.max()
    return int(np.nonzero(r == m)[0][0])


def accept_len(logits, draft, gamma: int):
    """Accepted-prefix length and bonus token of greedy speculative decoding.

    Eq. (3): draft i is accepted iff it equals the verifier's greedy token.
    Alg. 2: k is the largest count with every draft i <= k accepted; the
    verifier's token after the accepted prefix is appended as a bonus.
    Indexing (0-based): logits row i is the verifier's prediction for draft i
    (row 0 belongs to the last committed token); bonus = greedy token of row k.

    logits [S][gamma+1][V] (any float), draft [S][gamma] int.
    Returns accept [S], bonus [S], argmax [S][gamma+1], all int32.
    """
    S = len(logits)
    am = np.zeros((S, gamma + 1), dtype=np.int32)
    acc = np.zeros(S, dtype=np.int32)
    bonus = np.zeros(S, dtype=np.int32)
    for s in range(S):
        for i in range(gamma + 1):
            am[s, i] = greedy_argmax(logits[s][i])
        kk = 0
        while kk < gamma and int(draft[s][kk]) == am[s, kk]:
            kk += 1
        acc[s] = kk
        bonus[s] = am[s, kk]
    return acc, bonus, am


# --------------------------------------------------------------------------
# Per-round cache updates (Alg. 2: the drafter's sparse cache grows with the
# drafted tokens; after verification both caches keep the accepted tokens)
# --------------------------------------------------------------------------

def cache_append(k, v, seq_lens, k_new, v_new, idx=None, nsel=None):
    """Write n new rows per sequence at positions L_s .. L_s+n-1 and advance L_s.

    k, v: [S][Hkv][cap][D] bf16 bits (copies are returned); k_new, v_new: [S][n][Hkv][D].
    Rows at or past the capacity cap are dropped and L_s stops at cap.  With idx
    [S][Hkv][ld] and nsel [S] (the drafter's sparse cache), each written position
    is also appended to every head's index list at slots nsel[s] .. (dropped past
    ld), and nsel advances by the number of appended slots.
    Returns (k, v, seq_lens[, idx, nsel]).
    """
    k, v = np.array(k, copy=True), np.array(v, copy=True)
    lens = np.array(seq_lens, dtype=np.int32, copy=True)
    S, Hkv, cap = k.shape[0], k.shape[1], k.shape[2]
    n = k_new.shape[1]
    if idx is not None:
        idx, nsel = np.array(idx, dtype=np.int32, copy=True), np.array(nsel, dtype=np.int32, copy=True)
    for s in range(S):
        L = int(lens[s])
        rows = [i for i in range(n) if L + i < cap]
        for i in rows:
            for g in range(Hkv):
                k[s, g, L + i] = k_new[s, i, g]
                v[s, g, L + i] = v_new[s, i, g]
        if idx is not None:
            m = int(nsel[s])
            slots = [j for j in range(len(rows)) if m + j < idx.shape[2]]
            for j in slots:
                idx[s, :, m + j] = L + rows[j]
            nsel[s] = m + len(slots)
        lens[s] = L + len(rows)
    return (k, v, lens) if idx is None else (k, v, lens, idx, nsel)


def cache_rollback(seq_lens, accept, spec: int, nsel=None, base_lens=None, base_nsel=None):
    """Drop the rejected speculative rows after verification (Alg. 2, cache update).

    Each sequence ends in ``spec`` speculative rows, of which the first accept[s] were accepted
    (accept is clamped to [0, spec]).  Without base lengths, spec - accept[s] rows are dropped from
    L_s (and from nsel[s], the drafter's sparse list, when given), never below zero.  With the
    lengths from before the speculative appends (``base_lens``, and ``base_nsel`` for the list),
    L_s becomes min(L_s, base_lens[s] + accept[s]) and nsel[s] min(nsel[s], base_nsel[s] + accept[s]):
    an accepted row is kept only if it was written, so rows an append dropped at the capacity (or
    list entries dropped past the list's end) are never taken off a second time.
    Returns (seq_lens[, nsel]).
    """
    lens = np.array(seq_lens, dtype=np.int64)
    acc = np.clip(np.asarray(accept, dtype=np.int64), 0, spec)
    if base_lens is None:
        lens = np.maximum(lens - (spec - acc), 0).astype(np.int32)
    else:
        lens = np.minimum(lens, np.asarray(base_lens, dtype=np.int64) + acc).astype(np.int32)
    if nsel is None:
        return lens
    ns = np.asarray(nsel, dtype=np.int64)
    if base_nsel is None:
        ns = np.maximum(ns - (spec - acc), 0)
    else:
        ns = np.minimum(ns, np.asarray(base_nsel, dtype=np.int64) + acc)
    return lens, ns.astype(np.int32)


# --------------------------------------------------------------------------
# Training-side neighbours of the acceptance rule (Sec. 3.3-3.4)
# --------------------------------------------------------------------------

def top1_ce(student, teacher=None, targets=None):
    """Top-1 cross-entropy of the drafter against the verifier's greedy targets.

    Eq. (5) gives the target of each continuation row, the lowest-index argmax of
    the verifier's logits (``teacher``; or ``targets`` given directly); the summand
    of L_A (Eq. 6) and L_C (Eq. 7) for that row is -log softmax(student row)[target]
    = logsumexp(student row) - student[target] (natural log).
    student, teacher: [R][V] fp32; returns (loss [R], target [R] int32, lse [R]) in float64.
    """
    x = np.asarray(student, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("student logits must be finite")
    R = x.shape[0]
    if teacher is not None:
        tgt = np.array([greedy_argmax(np.asarray(teacher[r])) for r in range(R)], dtype=np.int32)
    else:
        tgt = np.asarray(targets, dtype=np.int32)
    m = x.max(axis=1)
    lse = m + np.log(np.exp(x - m[:, None]).sum(axis=1))
    loss = lse - x[np.arange(R), tgt]
    return loss, tgt, lse


def budget_thresholds(weights) -> np.ndarray:
    """Cumulative thresholds of Cat(B, w) in fp32: prefix sums of w in order, divided by their total.

    The sampling rule compares fp32 numbers, so both implementations take the
    decision in fp32 (Sec. 3.4 draws B ~ Cat(B, w) each training step).
    """
    w = np.asarray(weights, dtype=np.float32)
    c = np.zeros(w.size, dtype=np.float32)
    acc = np.float32(0.0)
    for i in range(w.size):
        acc = np.float32(acc + w[i])
        c[i] = acc
    return (c / c[-1]).astype(np.float32)


def sample_budgets(u, budgets, weights) -> np.ndarray:
    """B ~ Cat(budgets, weights) by inversion: the first budget whose fp32 cumulative threshold
    exceeds the uniform draw u in [0, 1) (the last budget if none does)."""
    thr = budget_thresholds(weights)
    u = np.asarray(u, dtype=np.float32)
    out = np.empty(u.size, dtype=np.int32)
    for i, x in enumerate(u.ravel()):
        j = 0
        while j < thr.size - 1 and not (x < thr[j]):
            j += 1
        out[i] = budgets[j]
    return out
