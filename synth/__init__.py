"""Seeded synthetic inputs for the BudgetDraft sparse-drafter / full-verifier path.

This module is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It only *draws* inputs: it holds none of the method's arithmetic
(no attention, no scoring, no pooling, no top-k, no argmax).  Everything is
numpy; bf16 tensors are carried as ``uint16`` bit patterns.

Workload shapes stand in for the paper's long-context prompts (Sec. 4,
"Context Lengths": 3.8K / 8K / 16K-token prompts of PG-19, QMSum and
NarrativeQA).  Those datasets are not used: only the tensor shapes and the
attention structure matter to the kernels, so K, V and Q are i.i.d. N(0, 1)
with a small fraction of "heavy-hitter" keys planted along the mean query
direction, imitating the observation (Appendix, budget paradox) that next-token
attention is dominated by a small subset of the prefix.

Random streams: ``numpy.random.Generator(PCG64(SeedSequence([ROOT_SEED,
config_id, tag, *extra])))``.  Every (config, tensor, sequence) has its own
stream, so any one sequence of a batch can be regenerated on its own.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

ROOT_SEED = 20260601

# Stream tags (one per tensor kind).
TAG_K, TAG_V, TAG_Q, TAG_HH, TAG_LOGITS, TAG_DRAFT, TAG_LENS, TAG_PAGES, TAG_BUDGETS = range(9)
TAG_K_VERIFIER, TAG_V_VERIFIER = 9, 10
TAG_IDX = 11

HEAD_DIM = 128


def rng(config_id: int, tag: int, *extra: int) -> np.random.Generator:
    """Independent PCG64 stream for (config, tensor tag, extra ids)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([ROOT_SEED, config_id, tag, *extra])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round-to-nearest-even), returned as uint16 bits.

    Inputs must be finite.  Storage conversion for generated data only.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = (u >> 16) & 1            # finite inputs: u + 0x8000 cannot wrap in uint32
    r += 0x7FFF
    r += u
    r >>= 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bits to float32 (storage conversion)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass(frozen=True)
class Config:
    """Shape and data recipe of one synthetic workload."""

    config_id: int
    name: str
    num_seqs: int
    num_q_heads: int
    num_kv_heads: int
    seq_len: int                 # fixed length, or the upper bound when ragged
    hh_frac: float               # fraction of prefix positions planted as heavy hitters
    window: int                  # observation window W (selection)
    budgets: Sequence[int]       # drafter KV budgets B
    gamma: int                   # draft length
    vocab: int                   # logits width for the accept step (0: none)
    accept_m: Optional[int] = None   # fixed accepted-prefix plant (None: seeded per sequence)
    block_len: int = 0           # multi-view continuation block C (0: none)
    num_views: int = 0
    ragged_min_len: int = 0      # >0: lengths ~ U{ragged_min_len .. seq_len}
    page_size: int = 0           # >0: paged KV layout

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def obs_rows(self) -> int:
        """Rows of the query tail that score the cache (W, or C for the block)."""
        return self.block_len if self.block_len else self.window

    @property
    def q_rows(self) -> int:
        """Tail query rows kept per sequence: covers W, gamma+1 and C."""
        return max(self.window, self.gamma + 1, self.block_len, 1)


CONFIGS: List[Config] = [
    Config(0, "tiny-4k-gqa4", 1, 8, 2, 4096, 0.01, 32, (256,), 5, 32000, accept_m=3),
    Config(1, "llama3-8b-layer-8k", 1, 32, 8, 8192, 0.01, 32, (256, 512, 1024, 2048), 5, 128256),
    Config(2, "16k-collapse-b8", 8, 32, 8, 16384, 0.005, 32, (512, 1024), 5, 128256),
    Config(3, "multiview-train-b4-8k", 4, 32, 8, 8192, 0.01, 64, (), 5, 0, block_len=64, num_views=4),
    Config(4, "ragged-paged-b64-mha", 64, 32, 32, 16384, 0.01, 32, (1024,), 5, 32000,
           ragged_min_len=4096, page_size=16),
    # the paper's training shape (Sec. 4: T = 16,384 = P + C with C = 256, batch size 1): one
    # sequence, the 256-row continuation block scores the prefix, and the views take every budget of
    # the training set {256, 512, 1024, 2048} (Sec. 3.4) beside the full branch
    Config(5, "train-c256-16k", 1, 32, 8, 16384, 0.01, 256, (256, 512, 1024, 2048), 5, 0, block_len=256),
]
WORKLOADS = {c.name: c for c in CONFIGS}


def workload(name: str) -> Config:
    """The synthetic workload of that name (its config_id seeds its generators)."""
    return WORKLOADS[name]


def seq_lens(cfg: Config) -> np.ndarray:
    """Per-sequence context lengths (cache rows, including the query tail)."""
    if cfg.ragged_min_len:
        return rng(cfg.config_id, TAG_LENS).integers(cfg.ragged_min_len, cfg.seq_len + 1,
                                                     size=cfg.num_seqs).astype(np.int32)
    return np.full(cfg.num_seqs, cfg.seq_len, dtype=np.int32)


def view_budgets(cfg: Config) -> np.ndarray:
    """Budgets of the multi-view block, drawn Uniform{256, 512, 1024, 2048}."""
    if not cfg.num_views:
        return np.zeros(0, dtype=np.int32)
    choices = np.array([256, 512, 1024, 2048], dtype=np.int32)
    return choices[rng(cfg.config_id, TAG_BUDGETS).integers(0, 4, size=cfg.num_views)]


def query_tail(cfg: Config, s: int) -> np.ndarray:
    """Post-RoPE query rows of sequence s: bf16 bits [q_rows][Hq][128].

    Row r sits at position L_s - q_rows + r: the last W rows are the
    observation window, the last gamma+1 rows the verifier's draft positions,
    the last row the drafter's decode query, the last C rows the block.
    """
    g = rng(cfg.config_id, TAG_Q, s)
    return f32_to_bf16_bits(g.standard_normal((cfg.q_rows, cfg.num_q_heads, HEAD_DIM), dtype=np.float32))


def heavy_hitter_positions(cfg: Config, L: int, s: int) -> np.ndarray:
    """Sorted planted positions of sequence s, sampled from the prefix [0, L - obs_rows)."""
    n_prefix = L - cfg.obs_rows
    n_hh = int(round(cfg.hh_frac * L))
    n_hh = max(0, min(n_hh, n_prefix))
    pos = rng(cfg.config_id, TAG_HH, s).choice(n_prefix, size=n_hh, replace=False)
    return np.sort(pos).astype(np.int64)


def kv_sequence(cfg: Config, s: int, L: Optional[int] = None, tag_k: int = TAG_K, tag_v: int = TAG_V,
                q_tail: Optional[np.ndarray] = None, plant: bool = True):
    """K and V of sequence s as bf16 bits [Hkv][L][128] each.

    Heavy hitters: for KV head g the direction u_g is the normalised sum of the
    observation-window queries of its query heads (taken in float64 from the
    bf16 queries); a planted key becomes 4 * ||k_t|| * u_g, then bf16.  The
    positions are shared by all KV heads.  V is left N(0, 1).
    """
    if L is None:
        L = int(seq_lens(cfg)[s])
    hkv, G = cfg.num_kv_heads, cfg.group
    k = rng(cfg.config_id, tag_k, s).standard_normal((hkv, L, HEAD_DIM), dtype=np.float32)
    if plant and cfg.hh_frac > 0:
        if q_tail is None:
            q_tail = query_tail(cfg, s)
        qo = bf16_bits_to_f32(q_tail[-cfg.obs_rows:]).astype(np.float64)   # [obs][Hq][D]
        pos = heavy_hitter_positions(cfg, L, s)
        for g in range(hkv):
            d = qo[:, g * G:(g + 1) * G, :].sum(axis=(0, 1))
            u = d / np.linalg.norm(d)
            norms = np.linalg.norm(k[g, pos, :].astype(np.float64), axis=1, keepdims=True)
            k[g, pos, :] = (4.0 * norms * u[None, :]).astype(np.float32)
    v = rng(cfg.config_id, tag_v, s).standard_normal((hkv, L, HEAD_DIM), dtype=np.float32)
    return f32_to_bf16_bits(k), f32_to_bf16_bits(v)


def logits_and_drafts(cfg: Config, s: int, vocab: Optional[int] = None, gamma: Optional[int] = None):
    """Verifier logits [gamma+1][V] fp32 and drafts [gamma] int32 of sequence s.

    Logits are N(0, 1) clipped to [-6, 6]; each row r gets a planted unique
    maximum 7.0 at a seeded token t_r, so its greedy token is t_r by
    construction.  Drafts copy t_0..t_{m-1}, then take a token != t_m, then
    random tokens; the accepted-prefix length is therefore m by construction.
    Returns (logits, drafts, planted_tokens, m).
    """
    V = cfg.vocab if vocab is None else vocab
    gm = cfg.gamma if gamma is None else gamma
    g = rng(cfg.config_id, TAG_LOGITS, s)
    logits = np.clip(g.standard_normal((gm + 1, V), dtype=np.float32), -6.0, 6.0)
    tok = g.integers(0, V, size=gm + 1)
    logits[np.arange(gm + 1), tok] = 7.0
    d = rng(cfg.config_id, TAG_DRAFT, s)
    m = cfg.accept_m if cfg.accept_m is not None else int(d.integers(0, gm + 1))
    m = min(m, gm)
    drafts = d.integers(0, V, size=gm)
    drafts[:m] = tok[:m]
    if m < gm:
        off = int(d.integers(1, V))
        drafts[m] = (tok[m] + off) % V
    return logits, drafts.astype(np.int32), tok.astype(np.int32), m


def page_table(cfg: Config, lens: np.ndarray):
    """Seeded page assignment for a paged cache.

    Returns (table [S][max_pages] int32, -1 for unused, num_pages).  The pool
    holds exactly sum_s ceil(L_s / page_size) pages, handed out under a seeded
    permutation.
    """
    ps = cfg.page_size
    npages = [(int(L) + ps - 1) // ps for L in lens]
    total = int(sum(npages))
    max_pages = (cfg.seq_len + ps - 1) // ps
    perm = rng(cfg.config_id, TAG_PAGES).permutation(total).astype(np.int32)
    table = np.full((len(lens), max_pages), -1, dtype=np.int32)
    off = 0
    for s, n in enumerate(npages):
        table[s, :n] = perm[off:off + n]
        off += n
    return table, total


def random_index_set(config_id: int, s: int, g: int, L: int, n: int, tag_extra: int = 0) -> np.ndarray:
    """A seeded ascending set of n distinct positions in [0, L) (for sparse-attention inputs)."""
    n = min(n, L)
    return np.sort(rng(config_id, TAG_IDX, s, g, tag_extra).choice(L, size=n, replace=False)).astype(np.int32)


def kv_batch(cfg: Config, seqs: Optional[Sequence[int]] = None, tag_k: int = TAG_K, tag_v: int = TAG_V,
             workers: int = 8):
    """Query tails, K and V of several sequences, generated in parallel (one stream per sequence).

    Returns lists (q_tail, k, v) in the order of ``seqs``.
    """
    import concurrent.futures

    seqs = list(range(cfg.num_seqs)) if seqs is None else list(seqs)

    def one(s):
        qt = query_tail(cfg, s)
        k, v = kv_sequence(cfg, s, q_tail=qt, tag_k=tag_k, tag_v=tag_v)
        return qt, k, v

    with concurrent.futures.ThreadPoolExecutor(max_workers=max(1, workers)) as ex:
        res = list(ex.map(one, seqs))
    return [r[0] for r in res], [r[1] for r in res], [r[2] for r in res]
