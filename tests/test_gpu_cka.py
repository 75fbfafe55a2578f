"""Parity of ace_pairwise_cka (the HIP library, through the C-ABI) with the
fp64 oracle's pairwise linear CKA on the same seeded inputs.

The library takes the probe and adapters in the storage type (bf16 or fp32);
the oracle works in fp64 on exactly those values.  Both sides then differ by
fp32 accumulation only (X A^T on the matrix cores and the Gram over the
probe); for probes of up to 10^4 rows that keeps every entry of S within
1e-4 of the fp64 value (S lies in [0, 1]), the bound asserted here.
"""
import numpy as np
import pytest
import torch

from oracle import consolidation_oracle as C
from paper_2609_06072_amd import workloads as W

pytestmark = pytest.mark.gpu
ATOL = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    from paper_2609_06072_amd import ace  # noqa: F401  (fails loudly if libace.so is missing)


def _f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def _case(dtype, N, d_in, d_out, E, r, seed=0, noise=0.5):
    base = W.CONFIGS["olmoe_bf16" if dtype == "bf16" else "tiny_fp32"]
    cfg = base.scaled(d_model=d_in, d_ffn=d_out, E=E, r_e=r, groups=("consecutive", 3))
    return W.make_probe_adapters(cfg, "gate", N=N, noise=noise, seed=seed, device="cuda")


def _gpu_cka(pa):
    from paper_2609_06072_amd import ace
    print(f"cka N={pa.X.shape[0]} d_in={pa.d_in} d_out={pa.d_out} E={pa.E} r={pa.r} "
          f"{pa.X.dtype}", flush=True)
    S = ace.ace_pairwise_cka(pa.X, pa.A, pa.B, pa.E, pa.r)
    torch.cuda.synchronize()
    return _f64(S)


SMALL = [  # N, d_in, d_out, E, r: ragged against the projection tiles (64 probe
           # rows x 256 adapter rows), the Gram tiles (128 for bf16, 64 for
           # fp32), the probe chunks (400 rows or more) and the 256-row chunks
           # of B^T B; ranks up to 8 take the one-wave pair kernel (B^T B
           # partials formed in the msum launch), larger ranks the block one
    (300, 40, 24, 6, 3),
    (700, 72, 600, 7, 5),
    (1500, 136, 72, 9, 8),
    (130, 64, 16, 20, 16),
    (2100, 96, 40, 4, 64),
    (77, 8, 1, 5, 1),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_cka_parity_small(dtype, shape):
    N, d_in, d_out, E, r = shape
    pa = _case(dtype, N, d_in, d_out, E, r)
    S = _gpu_cka(pa)
    ref = C.cka_matrix(_f64(pa.X), _f64(pa.A), _f64(pa.B), E, r)
    err = np.abs(S - ref).max()
    print(f"  max |S - ref| = {err:.2e}", flush=True)
    assert err <= ATOL
    assert np.array_equal(S, S.T)


def test_cka_full_size_sampled():
    """The OLMoE-like gate adapters (E = 64, rank 8, 2048 -> 1024) on the
    paper's probe size N = 10,000: the diagonal, symmetry and range hold
    everywhere, and sampled pairs match the oracle evaluated on those two
    experts alone."""
    cfg = W.CONFIGS["olmoe_bf16"]
    pa = W.make_probe_adapters(cfg, "gate", N=10000, seed=0, device="cuda")
    S = _gpu_cka(pa)
    assert np.abs(np.diag(S) - 1.0).max() <= ATOL
    assert np.array_equal(S, S.T) and S.min() >= -ATOL and S.max() <= 1 + ATOL
    X, A, B = _f64(pa.X), _f64(pa.A), _f64(pa.B)
    r, d_out = pa.r, pa.d_out
    same = [(i, j) for i in range(pa.E) for j in range(i + 1, pa.E) if pa.clusters[i] == pa.clusters[j]]
    diff = [(i, j) for i in range(pa.E) for j in range(i + 1, pa.E) if pa.clusters[i] != pa.clusters[j]]
    for i, j in (same[0], diff[0], diff[len(diff) // 2]):
        sub_A = np.concatenate([A[i * r:(i + 1) * r], A[j * r:(j + 1) * r]])
        sub_B = np.concatenate([B[d_out * r * i:d_out * r * (i + 1)], B[d_out * r * j:d_out * r * (j + 1)]])
        ref = C.cka_matrix(X, sub_A, sub_B, 2, r)[0, 1]
        print(f"  pair ({i},{j}) same cluster={pa.clusters[i] == pa.clusters[j]}: "
              f"gpu {S[i, j]:.6f} ref {ref:.6f}", flush=True)
        assert abs(S[i, j] - ref) <= ATOL


def test_cka_degenerate_and_deterministic():
    from paper_2609_06072_amd import ace
    pa = _case("bf16", 400, 64, 32, 5, 4)
    S1 = _gpu_cka(pa)
    S2 = _gpu_cka(pa)
    assert np.array_equal(S1, S2)
    # an expert with B = 0 has no defined CKA: zero row and column
    B = pa.B.clone()
    B[32 * 4 * 2:32 * 4 * 3] = 0
    S0 = ace.ace_pairwise_cka(pa.X, pa.A, B, 5, 4)
    torch.cuda.synchronize()
    S0 = _f64(S0)
    assert np.all(S0[2] == 0) and np.all(S0[:, 2] == 0)
    ref = C.cka_matrix(_f64(pa.X), _f64(pa.A), _f64(B), 5, 4)
    assert np.abs(S0 - ref).max() <= ATOL
    # a probe of one row (nothing left after centring) or none gives S = 0
    for n in (1, 0):
        S = ace.ace_pairwise_cka(pa.X[:n].contiguous(), pa.A, pa.B, 5, 4)
        torch.cuda.synchronize()
        assert np.all(_f64(S) == 0)
