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
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; worst at {i}: "
                             f"gpu {gpu[i]} oracle {ref[i]}")
    return float(err.max()) if err.size else 0.0


def assert_lse(gpu: np.ndarray, ref: np.ndarray, what: str):
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
