"""Distortion-model mismatch in weighted distortion J (Appendix
"Cross-Quantizer Transfer", Sec. 3.4 "Distortion calibration"), on
synthetic KV instead of perplexity on real models.

Every family is swept on the same 64 components (32 outlier-scaled key
components, 32 value components, 512 tokens each) through the C-ABI, fitted,
and allocated with each family's fitted parameters (and uniformly); each
allocation is then scored on every family's measured distortion table:
    J[A][B] = sum_i w_i D_i^B(b_i^A).
The same matrix from the oracle's sweep, fit and greedy allocation must
agree, and the claims that hold on these inputs are checked: every
allocation beats uniform, and at 3 and 4 bits the matched parameters give
the lowest J for every quantizer."""
import numpy as np
import pytest

import paper_2605_06675_amd as rq
import workloads
from oracle import alloc as oalloc
from oracle import calib as ocalib
from oracle import fit as ofit
from tests import gpu_helpers as gh

pytestmark = pytest.mark.gpu

N, T = 64, 512
BITS = [2, 3, 4, 5, 6]
FAMS = {"turbo": workloads.TURBO, "kivi": workloads.KIVI,
        "quarot": workloads.QUAROT, "rtn": workloads.RTN}


def _inputs():
    dtype = workloads.BF16
    x16 = workloads.calib_cpu(N, T, dtype)
    r16 = np.stack([workloads.turbo_rotation(42, i // 8, i % 8) for i in range(N)])
    w = np.random.default_rng([42, 9]).lognormal(0.0, 0.76, size=N)
    return dtype, x16, r16, w


def _gpu_tables(dtype, x16, r16):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    cb = torch.from_numpy(rq.rq_turbo_codebook().reshape(-1)).cuda()
    out = {}
    for name, fam in FAMS.items():
        print(f"transfer sweep {name}", flush=True)
        parts = []
        for is_value, sl in ((0, slice(0, N // 2)), (1, slice(N // 2, N))):
            turbo = fam == workloads.TURBO
            parts.append(rq.rq_calibrate_distortion(
                fam, dtype, gh.dev(np.ascontiguousarray(x16[sl]), dtype),
                is_value, BITS,
                rotation=gh.dev(np.ascontiguousarray(r16[sl]), workloads.BF16)
                if turbo else None, codebook=cb if turbo else None))
        out[name] = tuple(np.concatenate([p[k] for p in parts]) for k in range(3))
    return out


def _oracle_tables(dtype, x16, r16):
    x = workloads.u16_to_f32(x16, dtype)
    rf = workloads.u16_to_f32(r16, workloads.BF16).astype(np.float64)
    out = {}
    for name, fam in FAMS.items():
        rot = (lambda sl: rf[sl]) if fam == workloads.TURBO else (lambda sl: None)
        m = np.concatenate([
            ocalib.sweep(fam, x[: N // 2], BITS, False, rot(slice(0, N // 2))),
            ocalib.sweep(fam, x[N // 2:], BITS, True, rot(slice(N // 2, N)))])
        a, b, _ = ofit.fit_distortion(m, BITS)
        out[name] = (m, a, b)
    return out


def _matrix(tables, w, avg, allocate):
    J = lambda D, b: float(np.sum(w * D[np.arange(N), np.asarray(b) - BITS[0]]))
    rows = {}
    for an, (_, a, b) in tables.items():
        bits = allocate(w, a, b, avg)
        rows[an] = [J(tables[qn][0], bits) for qn in tables]
    if avg == int(avg):
        u = np.full(N, int(avg))
        rows["uniform"] = [J(tables[qn][0], u) for qn in tables]
    return rows


def _lib_alloc(w, a, b, avg):
    return rq.rq_allocate_bits(w, a, b, avg, 2, 6, want_cont=False)[0]


def _oracle_alloc(w, a, b, avg):
    return oalloc.greedy(w, a, b, oalloc.budget(N, avg), 2, 6)


def test_transfer_matrix_in_weighted_distortion():
    dtype, x16, r16, w = _inputs()
    gpu = _gpu_tables(dtype, x16, r16)
    ora = _oracle_tables(dtype, x16, r16)
    names = list(FAMS)
    for avg in (2.5, 3.0, 4.0):
        G = _matrix(gpu, w, avg, _lib_alloc)
        O = _matrix(ora, w, avg, _oracle_alloc)
        print(f"avg {avg}: alloc \\ quant " + " ".join(names))
        for r in G:
            print(f"  {r:>8} " + " ".join(f"{v:9.5f}" for v in G[r]))
            np.testing.assert_allclose(G[r], O[r], rtol=1e-3)
        if avg == int(avg):
            for j, qn in enumerate(names):
                col = {r: G[r][j] for r in G}
                assert all(col[r] < col["uniform"] for r in names), (avg, qn)
                assert col[qn] == min(col[r] for r in names), (avg, qn, col)
