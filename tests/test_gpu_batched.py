"""GPU: the batched entry points equal the single-problem calls bit for bit
(same kernels, one problem after another) and match the fp64 oracle; shared
key sets (stride 0) and empty batches."""
import numpy as np
import pytest

import oracle
import parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    from paper_2609_04910_amd import gauss_sum as gs
    gs.load()
    yield


def clouds(seed, B, M, N, D, C, shared=False):
    """B independent N(0, I)/sqrt(D) clouds (the paper's benchmark inputs), fp16."""
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((B, M, D)) / np.sqrt(D)).astype(np.float16)
    kb = 1 if shared else B
    k = (rng.standard_normal((kb, N, D)) / np.sqrt(D)).astype(np.float16)
    v = rng.standard_normal((kb, N, C)).astype(np.float32)
    g = rng.standard_normal((B, M, C)).astype(np.float32)
    if shared:
        k, v = k[0], v[0]
    return q, k, v, g


@pytest.mark.parametrize("B,M,N,D,C", [(4, 300, 517, 32, 1), (3, 64, 1000, 64, 3), (5, 129, 97, 17, 2)])
def test_batched_equals_single_calls_and_oracle(B, M, N, D, C):
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, g = clouds(B * 100 + D, B, M, N, D, C)
    tq, tk, tv, tg = (parity.to_torch(a) for a in (q, k, v, g))
    tau = 1.0
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, tau)
    dq, dk, dv = gs.gauss_sum_bwd_batched(tq, tk, tv, tau, tg)
    torch.cuda.synchronize()
    for b in range(B):
        s1 = gs.gauss_sum_fwd(tq[b], tk[b], tv[b], tau)
        d1 = gs.gauss_sum_bwd(tq[b], tk[b], tv[b], tau, tg[b])
        torch.cuda.synchronize()
        assert torch.equal(out[b], s1)
        for x, y in zip((dq, dk, dv), d1):
            assert torch.equal(x[b], y)
    b = B - 1
    ref, scale = oracle.fwd(q[b], k[b], v[b], tau, threads=parity.oracle_threads())
    parity.compare("batched fwd", out[b].cpu().numpy(), ref, scale, parity.TOL["f16"])
    ref, scale = oracle.dk(q[b], k[b], v[b], g[b], tau, threads=parity.oracle_threads())
    parity.compare("batched dk", dk[b].cpu().numpy(), ref, scale, parity.TOL["f16"])


def test_batched_shared_keys_and_empty():
    import torch
    from paper_2609_04910_amd import gauss_sum as gs
    q, k, v, g = clouds(7, 6, 200, 333, 48, 2, shared=True)
    tq, tk, tv, tg = (parity.to_torch(a) for a in (q, k, v, g))
    out = gs.gauss_sum_fwd_batched(tq, tk, tv, 1.0)
    dq, _, _ = gs.gauss_sum_bwd_batched(tq, tk, tv, 1.0, tg, want=(True, False, False))
    torch.cuda.synchronize()
    for b in range(6):
        assert torch.equal(out[b], gs.gauss_sum_fwd(tq[b], tk, tv, 1.0))
        assert torch.equal(dq[b], gs.gauss_sum_bwd(tq[b], tk, tv, 1.0, tg[b], want=(True, False, False))[0])
    empty = gs.gauss_sum_fwd_batched(tq[:0], tk, tv, 1.0)
    assert empty.shape == (0, 200, 2)
