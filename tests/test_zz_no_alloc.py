"""bd_verify_attn_noalloc (fixed in-library scratch) against bd_verify_attn (caller workspace).

Both run the same kernels, so outputs and log-sum-exps must agree bit for bit; the
second call of each pair uses a smaller input than the first, so stale scratch from a
larger call must not leak into a smaller one.  The smaller case is also checked against
the fp64 oracle (the verify tolerance of the other parity tests).
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import assert_close, assert_lse, bf16_dev, bf16_host64, case, config_data, i32_dev

pytestmark = pytest.mark.gpu


def _pair(name, S=None):
    cfg = synth.workload(name)
    qt, k, v = config_data(name, True)
    if S is not None:
        qt, k, v = qt[:S], k[:S], v[:S]
    lens = [cfg.seq_len] * k.shape[0]
    q = np.ascontiguousarray(qt[:, -(cfg.gamma + 1):])
    return cfg, q, k, v, lens


def _run_both(cfg, q, k, v, lens, what):
    case(f"verify noalloc vs workspace: {what}")
    kd, vd, qd, ld = bf16_dev(k), bf16_dev(v), bf16_dev(q), i32_dev(lens)
    # outputs filled with NaN first: every element must be written
    out_n = torch.full(qd.shape, float("nan"), dtype=torch.bfloat16, device=qd.device)
    lse_n = torch.full(qd.shape[:3], float("nan"), dtype=torch.float32, device=qd.device)
    bd.bd_verify_attn_noalloc(kd, vd, qd, ld, out=out_n, lse=lse_n)
    out_w, lse_w = bd.bd_verify_attn(kd, vd, qd, ld, return_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(out_n.view(torch.int16), out_w.view(torch.int16)), what
    assert torch.equal(lse_n.view(torch.int32), lse_w.view(torch.int32)), what
    return out_n, lse_n


def test_noalloc_matches_workspace_entry_point_two_calls_large_then_small():
    # first the 16K batch (8 x 16384, the launch configuration the benchmark times), then a
    # smaller input (the 4K single sequence), with the same fixed scratch
    cfg, q, k, v, lens = _pair("16k-collapse-b8")
    _run_both(cfg, q, k, v, lens, "16K batch")
    cfg, q, k, v, lens = _pair("tiny-4k-gqa4")
    out, lse = _run_both(cfg, q, k, v, lens, "4K single sequence")
    ro, rl = O.verify_attn(k, v, q, lens, cfg.gamma)
    assert_close(bf16_host64(out), ro, "noalloc verify vs oracle")
    assert_lse(lse.cpu().numpy().astype(np.float64), rl, "noalloc verify lse vs oracle")


def test_noalloc_repeated_calls_and_oversized_shape_rejected():
    # three calls in a row on one shape (each leaves the counters zero for the next), then a
    # two-sequence slice of the 8K layer shape; a paged shape whose plan needs more than the
    # fixed scratch is refused before anything runs
    cfg, q, k, v, lens = _pair("llama3-8b-layer-8k")
    first = _run_both(cfg, q, k, v, lens, "8K layer, call 1")
    for i in (2, 3):
        again = _run_both(cfg, q, k, v, lens, f"8K layer, call {i}")
        assert torch.equal(first[0].view(torch.int16), again[0].view(torch.int16))
    cfg, q, k, v, lens = _pair("16k-collapse-b8", S=2)
    _run_both(cfg, q, k, v, lens, "16K, two sequences")
    # 64 sequences x 32 KV heads, paged at 8 tokens a page (the per-key table bounds the splits to
    # 2,048 keys), up to 16384 rows: 133 MiB of records
    S, H, P = 64, 32, 8
    pages = torch.zeros((1, H, P, 128), dtype=torch.bfloat16, device="cuda")
    table = torch.zeros((S, 16384 // P), dtype=torch.int32, device="cuda")
    qq = torch.zeros((S, 6, H, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(bd.BdError) as e:
        bd.bd_verify_attn_noalloc(pages, pages, qq, torch.full((S,), 16, dtype=torch.int32, device="cuda"),
                                  out=torch.empty_like(qq), page_table=table)
    assert e.value.status == bd.BD_ERR_UNSUPPORTED and "scratch" in str(e.value)
