"""Cache lookup parity on the GPU: ac_lookup against the oracle's exhaustive fp64
cosine search. The index must match bit-exactly except where the oracle's top-2
scores differ by less than 1e-6 (then either of the tied rows is accepted)."""

import numpy as np
import pytest
import torch

from oracle import lookup as OL
from paper_2511_06724_amd import dn, workloads as W
from tests.gpu_util import DEV, announce

pytestmark = pytest.mark.gpu


def _check(q, cache, qd, cd):
    i, s = dn.ac_lookup(qd, cd)
    ri, rs = OL.top1(q, cache)
    if i != ri:
        sc = OL.cosine_scores(q, cache)
        assert abs(sc[i] - sc[ri]) < 1e-6, (i, ri, sc[i], sc[ri])
    assert abs(s - rs) < 1e-5
    return i


def test_planted_neighbours_full_cache():
    announce("lookup: 100000 x 768 planted")
    cache = W.cache_embeddings(100_000, 768, seed=7)
    qs, rows = W.planted_queries(cache, 16, seed=9)
    cd = torch.from_numpy(cache.view(np.uint16)).to(DEV)
    for q, j in zip(qs, rows):
        qd = torch.from_numpy(q.view(np.uint16).copy()).to(DEV)
        assert _check(q, cache, qd, cd) == j


@pytest.mark.parametrize("n,dim", [(1, 768), (1001, 768), (4097, 64), (300, 77), (257, 1), (5000, 1536)])
def test_ragged_sizes_and_odd_dims(n, dim):
    announce(f"lookup: n={n} dim={dim}")
    rng = np.random.default_rng(n + dim)
    cache = rng.standard_normal((n, dim)).astype(np.float16)
    for k in range(3):
        q = rng.standard_normal(dim).astype(np.float16)
        _check(q, cache, torch.from_numpy(q.view(np.uint16).copy()).to(DEV),
               torch.from_numpy(cache.view(np.uint16).copy()).to(DEV))


def test_duplicates_give_lowest_index():
    announce("lookup: duplicates")
    cache = W.cache_embeddings(20_000, 768, seed=3)
    for j in (17, 9999, 19_999):
        cache[j - 10 if j >= 10 else j + 5] = cache[j]
    cache[12_345] = cache[17]
    cd = torch.from_numpy(cache.view(np.uint16)).to(DEV)
    for j, want in ((17, 7), (9999, 9989), (19_999, 19_989)):
        qd = torch.from_numpy(cache[j].view(np.uint16).copy()).to(DEV)
        i, _ = dn.ac_lookup(qd, cd)
        assert i == min(want, j)
    qd = torch.from_numpy(cache[12_345].view(np.uint16).copy()).to(DEV)
    assert dn.ac_lookup(qd, cd)[0] == 7


def test_zero_query_is_an_error_and_fetch_is_exact():
    cache = torch.from_numpy(W.cache_embeddings(100, 64, seed=1).view(np.uint16)).to(DEV)
    zq = torch.zeros(64, dtype=torch.int16, device=DEV)
    code, idx, _ = dn.ac_lookup_raw(zq.data_ptr(), cache.data_ptr(), 100, 64)
    assert code == dn.DN_EINVAL and idx == -7
    lat = torch.randn((10, 4, 8, 8), device=DEV).to(torch.bfloat16)
    out = torch.empty((4, 8, 8), device=DEV)
    dn.ac_fetch_latent(lat, 6, out)
    torch.cuda.synchronize()
    assert torch.equal(out, lat[6].float())
