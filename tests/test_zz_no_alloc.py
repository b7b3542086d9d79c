"""The no-allocation signature call (carnator_signature_sim_noalloc) against
the workspace call (carnator_signature_sim) and the oracle, through the C ABI:
two calls in a row, the second with a smaller input, share the library's
scratch; top-k indices must match exactly and cosines bit for bit between the
two entry points (the same kernels), and within 1e-6 of the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_32420_amd as P

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _case(m, dim, nq, k, seed):
    g = torch.Generator(device=DEV).manual_seed(seed)
    bank = torch.randn(m, dim, generator=g, device=DEV)
    q = torch.randn(nq, dim, generator=g, device=DEV)
    q[-1] = bank[m // 3] + 0.5 * torch.randn(dim, generator=g, device=DEV)  # planted near-duplicate
    return q, bank


def _compare(q, bank, k):
    i1, s1, a1 = P.signature_sim(q, bank, k, return_all=True)
    i2, s2, a2 = P.signature_sim_noalloc(q, bank, k, return_all=True)
    torch.cuda.synchronize()
    assert torch.equal(i1, i2)
    assert torch.equal(s1.view(torch.int32), s2.view(torch.int32))
    assert torch.equal(a1.view(torch.int32), a2.view(torch.int32))
    wi, wv, frag = oracle.topk_cosine(q.cpu().numpy(), bank.cpu().numpy(), k)
    gi, gv = i2.cpu().numpy(), s2.cpu().numpy().astype(np.float64)
    for r in range(q.shape[0]):
        if frag[r]:
            assert set(gi[r]) == set(wi[r])
        else:
            assert gi[r].tolist() == wi[r].tolist()
        assert np.abs(gv[r] - wv[r]).max() <= 1e-6
    assert int(gi[-1, 0]) == bank.shape[0] // 3


def test_noalloc_two_calls_second_smaller():
    # the CogVideoX-shaped bank (one launch, two queries), then a smaller one
    q, bank = _case(4096, 3072, 2, 8, 1)
    _compare(q, bank, 8)
    q, bank = _case(1000, 256, 1, 5, 2)
    _compare(q, bank, 5)


def test_noalloc_query_groups_and_limit():
    # six queries: a scan per group of four and a top-k launch, same scratch
    q, bank = _case(3000, 128, 6, 17, 3)
    _compare(q, bank, 17)
    q, bank = _case(700, 64, 3, 64, 4)
    _compare(q, bank, 64)
    # nq * m beyond the scratch: rejected, nothing enqueued
    bank = torch.zeros(524289, 4, device=DEV)
    with pytest.raises(P.CarnatorError) as e:
        P.signature_sim_noalloc(torch.ones(1, 4, device=DEV), bank, 1)
    assert e.value.status == -5
