"""Multiview forward (training outputs) + backward against the fp64 oracle, shared by the GPU tests.

Tolerances: the backward's dq / dk / dv (fp32) within 1e-3 * max|oracle| + 1e-3 |oracle| per tensor
(the kernels keep P and dS as bf16 pairs, relative error about 2^-17, and accumulate in fp32);
the forward's fp32 training outputs within 1e-4 * max|O| + 1e-4 |O|; bf16 outputs and lse as in
every attention test.
"""
import numpy as np
import torch

import oracle as O
import paper_2606_00144_amd as bd
import synth
from gpu_utils import assert_close, assert_lse, bf16_dev, bf16_host64, case, i32_dev

GRAD_ATOL_FRAC, GRAD_RTOL = 1e-3, 1e-3


def _rand_bits(shape, seed, scale=1.0):
    g = np.random.default_rng(seed)
    return synth.f32_to_bf16_bits(scale * g.standard_normal(shape, dtype=np.float32))


def _grad_close(gpu, ref, what):
    atol = GRAD_ATOL_FRAC * max(float(np.abs(ref).max(initial=0.0)), 1e-30)
    return assert_close(gpu, ref, what, atol=atol, rtol=GRAD_RTOL)


def _out32_close(gpu, ref, what):
    atol = 1e-4 * max(float(np.abs(ref).max(initial=0.0)), 1e-30)
    return assert_close(gpu.cpu().numpy().astype(np.float64), ref, what, atol=atol, rtol=1e-4)


def _run(k, v, qb, idx_v, nsel_v, lens, what, full=True, seed=0, kdev=None, vdev=None, page_table=None,
         check_fwd=True, seqs=None, with_dkv=True, workspace=None, outputs=None, grads=None):
    """Training forward, backward with seeded dO; compare dq / dk / dv (on `seqs`, default all) with the oracle.
    outputs / grads: optional preallocated forward outputs and gradients (e.g. filled with NaN)."""
    S, C, Hq = qb.shape[0], qb.shape[1], qb.shape[2]
    V = 0 if idx_v is None else len(idx_v)
    kd = bf16_dev(k) if kdev is None else kdev
    vd = bf16_dev(v) if vdev is None else vdev
    iv = i32_dev(idx_v) if V else None
    nv = i32_dev(nsel_v) if V else None
    ld = i32_dev(lens)
    case(f"multiview bwd forward {what}")
    ov, of, o32v, lv, o32f, lf = bd.bd_multiview_attn(kd, vd, bf16_dev(qb), iv, nv, ld, full=full, train=True,
                                                      page_table=page_table, max_seq_len=int(max(lens)),
                                                      workspace=workspace, outputs=outputs)
    dov_bits = _rand_bits((V, S, C, Hq, 128), 1000 + seed) if V else None
    dof_bits = _rand_bits((S, C, Hq, 128), 2000 + seed) if full else None
    case(f"multiview bwd {what}")
    dq, dk, dv = bd.bd_multiview_attn_bwd(kd, vd, bf16_dev(qb), iv, nv, ld, o32v, lv,
                                          bf16_dev(dov_bits) if V else None, o32f, lf,
                                          bf16_dev(dof_bits) if full else None, with_dkv=with_dkv,
                                          page_table=page_table, max_seq_len=int(max(lens)), workspace=workspace,
                                          grads=grads)
    torch.cuda.synchronize()
    seqs = list(range(S)) if seqs is None else seqs
    for s in seqs:
        sl = slice(s, s + 1)
        ks = [k[s]] if isinstance(k, list) else k[sl]
        vs = [v[s]] if isinstance(v, list) else v[sl]
        iv_s = [x[sl] for x in idx_v] if V else []
        nv_s = [x[sl] for x in nsel_v] if V else []
        dov = [synth.bf16_bits_to_f32(dov_bits[i, sl]).astype(np.float64) for i in range(V)]
        dof = synth.bf16_bits_to_f32(dof_bits[sl]).astype(np.float64) if full else None
        if check_fwd:
            rv, rf, rlv, rlf = O.multiview_attn(ks, vs, qb[sl], iv_s, nv_s, lens[s:s + 1], with_full=full,
                                                return_lse=True)
            if V:
                assert_close(bf16_host64(ov[:, sl]), rv, f"{what} seq {s} views out")
                assert_lse(lv[:, sl].cpu().numpy().astype(np.float64), rlv, f"{what} seq {s} views lse")
                _out32_close(o32v[:, sl], rv, f"{what} seq {s} views out32")
            if full:
                assert_close(bf16_host64(of[sl]), rf, f"{what} seq {s} full out")
                assert_lse(lf[sl].cpu().numpy().astype(np.float64), rlf, f"{what} seq {s} full lse")
                _out32_close(o32f[sl], rf, f"{what} seq {s} full out32")
        rq, rk, rvv = O.multiview_attn_bwd(ks, vs, qb[sl], iv_s, nv_s, lens[s:s + 1], dov, dof)
        _grad_close(dq[sl].cpu().numpy().astype(np.float64), rq, f"{what} seq {s} dq")
        if with_dkv:
            _grad_close(dk[sl].cpu().numpy().astype(np.float64), rk, f"{what} seq {s} dk")
            _grad_close(dv[sl].cpu().numpy().astype(np.float64), rvv, f"{what} seq {s} dv")
        else:
            assert dk is None and dv is None
    return dq, dk, dv
