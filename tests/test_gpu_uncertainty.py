"""GPU parity of arbor_uncertainty (Eq. 1) against the oracle's fp64 entropy.

Tolerance: |u_gpu - u_oracle| <= 1e-5.  The kernel sums at most 2^31 terms
2^(x - m) <= 1 in fp32, a thread's share sequentially and the shares in a
tree; for the vocabularies here (<= 128256) the relative error of S and T
stays near 1e-6, i.e. about 1e-6 / ln|V| in u, well inside the bar.
"""
import math

import numpy as np
import pytest
import torch

from oracle import arbor_oracle as O
from paper_2605_22106_amd import _lib as L
from paper_2605_22106_amd import synth
from tests.gpu_helpers import check_rc, status

pytestmark = pytest.mark.gpu
TOL = 1e-5


def ws_for(z):
    dt = L.BF16 if z.dtype == torch.bfloat16 else L.F32
    n = L.arbor_uncertainty_workspace_size(z.shape[0], z.shape[1], dt)
    return torch.empty(n, dtype=torch.uint8, device="cuda")


def run(z, top_k, dst=None, n_out=None):
    n_out = n_out if n_out is not None else z.shape[0]
    u = torch.full((n_out,), -7.0, device="cuda")
    st = status()
    check_rc(L.arbor_uncertainty(z, top_k, u, st, ws_for(z), dst=dst))
    torch.cuda.synchronize()
    return u.cpu().numpy(), int(st)


def oracle_u(z, top_k):
    zz = z.float().cpu().numpy().astype(np.float64)
    return np.array([O.uncertainty(row, top_k=top_k if top_k else None) for row in zz])


@pytest.mark.parametrize("vocab", [1000, 4096, 65536])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("top_k", [0, 1, 7, 50, 999, 5000])
def test_uncertainty_rows(vocab, dtype, top_k):
    z = synth.boundary_logits(12, vocab, seed=vocab + top_k, dtype=dtype, device="cuda")
    u, s = run(z, top_k)
    assert s == L.OK
    k = top_k if 0 < top_k < vocab else 0
    ref = oracle_u(z, k)
    assert np.max(np.abs(u - ref)) <= TOL, np.max(np.abs(u - ref))


@pytest.mark.parametrize("top_k", [1, 40, 255, 256, 257])
def test_uncertainty_top_k_chunked_edges(top_k):
    # rows split over several chunks (64 rows of 65536): K at and around the
    # chunked path's limit; constant rows (every value ties with the bound, so
    # the chunks fall back to a select over all their values), a row whose
    # top K all sit in one chunk, and the synthetic mix
    rows, vocab = 64, 65536
    z = synth.boundary_logits(rows, vocab, seed=top_k, dtype="bf16", device="cuda")
    z[0] = 0.25
    z[1, :300] = 9.0
    z[2] = torch.arange(vocab, device="cuda").float().remainder(7).to(torch.bfloat16)
    u, s = run(z, top_k)
    assert s == L.OK
    ref = oracle_u(z, top_k)
    assert np.max(np.abs(u - ref)) <= TOL, np.max(np.abs(u - ref))
    u2, _ = run(z, top_k)
    assert np.array_equal(u.view(np.uint32), u2.view(np.uint32))


def test_uncertainty_closed_forms():
    # uniform row -> 0; a near one-hot row -> 1; two equal logits among -inf-like ones
    z = torch.zeros(3, 1024, device="cuda")
    z[1] = -80.0
    z[1, 17] = 0.0
    z[2] = -200.0
    z[2, 3] = z[2, 900] = 5.0
    u, s = run(z, 0)
    assert s == L.OK
    assert abs(u[0]) <= TOL and abs(u[1] - 1.0) <= TOL
    assert abs(u[2] - (1 - math.log(2) / math.log(1024))) <= TOL


def test_uncertainty_dst_and_reproducibility():
    z = synth.boundary_logits(9, 2048, seed=3, device="cuda")
    dst = torch.tensor([8, 0, 12, 3, 5, 1, 14, 2, 7], dtype=torch.int32, device="cuda")
    u1, s1 = run(z, 20, dst=dst, n_out=16)
    u2, s2 = run(z, 20, dst=dst, n_out=16)
    assert s1 == s2 == L.OK
    assert np.array_equal(u1.view(np.uint32), u2.view(np.uint32))
    ref = oracle_u(z, 20)
    d = dst.cpu().numpy()
    assert np.max(np.abs(u1[d] - ref)) <= TOL
    untouched = np.setdiff1d(np.arange(16), d)
    assert np.all(u1[untouched] == -7.0)


def test_uncertainty_rejects_non_finite_and_bad_dst():
    z = synth.boundary_logits(4, 512, seed=1, device="cuda")
    z[2, 100] = float("nan")
    u, s = run(z, 0)
    assert s == L.ENONFINITE
    assert u[2] == -7.0
    z = synth.boundary_logits(2, 512, seed=2, device="cuda")
    u, s = run(z, 0, dst=torch.tensor([0, 5], dtype=torch.int32, device="cuda"), n_out=4)
    assert s == L.EINVAL
    # host-side: a vocabulary that is not a multiple of 8 bf16 values
    bad = torch.zeros(2, 1001, dtype=torch.bfloat16, device="cuda")
    assert L.arbor_uncertainty(bad, 0, torch.zeros(2, device="cuda"), status(),
                               torch.empty(4096, dtype=torch.uint8, device="cuda")) == L.EUNSUPPORTED
    # a workspace too small for the split rows
    z = synth.boundary_logits(4, 65536, seed=3, device="cuda")
    tiny = torch.empty(16, dtype=torch.uint8, device="cuda")
    assert L.arbor_uncertainty(z, 0, torch.zeros(4, device="cuda"), status(), tiny) == L.EWORKSPACE


@pytest.mark.parametrize("top_k", [0, 40])
def test_uncertainty_full_vocabulary(top_k):
    # one boundary row per block of the 8B-shaped tree, Llama-3 vocabulary
    z = synth.boundary_logits(85, 128256, seed=11, dtype="bf16", device="cuda")
    u, s = run(z, top_k)
    assert s == L.OK
    ref = oracle_u(z, top_k)
    assert np.max(np.abs(u - ref)) <= TOL, np.max(np.abs(u - ref))
