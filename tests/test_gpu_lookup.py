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


# ----------------------------------------------------------------------------- batched search

def _dev16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.uint16)).to(DEV)


def _check_batch(qs, cache, idx, score):
    """Index bit-exact unless the oracle's scores of the two rows differ by < 1e-6;
    cosine within 1e-5; -1 exactly where the oracle has no defined cosine."""
    ridx, rsc = OL.top1_batch(qs, cache)
    s = OL.cosine_scores_batch(qs, cache)
    for j in range(len(ridx)):
        if ridx[j] < 0:
            assert idx[j] == -1, (j, idx[j])
            continue
        assert 0 <= idx[j] < cache.shape[0]
        if idx[j] != ridx[j]:
            assert abs(s[j, idx[j]] - s[j, ridx[j]]) < 1e-6, (j, idx[j], ridx[j])
        assert abs(score[j] - rsc[j]) < 1e-5, (j, score[j], rsc[j])
    return ridx


def test_batch_planted_full_cache():
    announce("lookup batch: 100000 x 768, 64 planted queries")
    cache = W.cache_embeddings(100_000, 768, seed=7)
    qs, rows = W.planted_queries(cache, 64, seed=11)
    qs = np.stack(qs)
    idx, score = dn.ac_lookup_batch(_dev16(qs), _dev16(cache))
    _check_batch(qs, cache, idx, score)
    assert list(idx) == list(rows)


@pytest.mark.parametrize("nq,n,dim", [(1, 1, 768), (5, 17, 256), (64, 1001, 512), (70, 4097, 768),
                                      (3, 300, 1024), (2, 15, 768), (7, 200, 77), (9, 33, 1536),
                                      (8, 60001, 256), (4, 40003, 512), (5, 70001, 1024)])
def test_batch_ragged_sizes_zero_rows_and_queries(nq, n, dim):
    announce(f"lookup batch: nq={nq} n={n} dim={dim}")
    rng = np.random.default_rng(nq * 1000 + n + dim)
    cache = rng.standard_normal((n, dim)).astype(np.float16)
    qs = rng.standard_normal((nq, dim)).astype(np.float16)
    if n > 3:
        cache[n // 2] = 0
        qs[0] = cache[n // 2 + 1]
    if nq > 2:
        qs[nq - 2] = 0
    idx, score = dn.ac_lookup_batch(_dev16(qs), _dev16(cache))
    ridx = _check_batch(qs, cache, idx, score)
    if nq > 2:
        assert idx[nq - 2] == -1 and ridx[nq - 2] == -1
    if n > 3:
        assert idx[0] == n // 2 + 1


def test_batch_agrees_with_single_query_search():
    announce("lookup batch vs ac_lookup: 20000 x 768")
    cache = W.cache_embeddings(20_000, 768, seed=5)
    rng = np.random.default_rng(2)
    qs = rng.standard_normal((16, 768)).astype(np.float16)
    cd = _dev16(cache)
    idx, score = dn.ac_lookup_batch(_dev16(qs), cd)
    s = OL.cosine_scores_batch(qs, cache)
    for j in range(16):
        i1, s1 = dn.ac_lookup(_dev16(qs[j]), cd)
        if i1 != idx[j]:
            assert abs(s[j, i1] - s[j, idx[j]]) < 1e-6
        assert abs(s1 - score[j]) < 2e-6


def test_batch_duplicates_give_lowest_index_and_errors_touch_nothing():
    announce("lookup batch: duplicates, argument errors")
    cache = W.cache_embeddings(20_000, 768, seed=3)
    for j in (17, 9999, 19_999):
        cache[j - 10] = cache[j]
    cache[12_345] = cache[17]
    qs = np.stack([cache[17], cache[9999], cache[19_999], cache[12_345]])
    idx, score = dn.ac_lookup_batch(_dev16(qs), _dev16(cache))
    assert list(idx) == [7, 9989, 19_989, 7]
    assert all(abs(v - 1.0) < 1e-6 for v in score)
    import ctypes as C
    out = (C.c_int64 * 2)(-7, -7)
    assert dn.lib.ac_lookup_batch(None, 2, 1, 5, 768, out, None) == dn.DN_EINVAL
    assert dn.lib.ac_lookup_batch(1, 0, 1, 5, 768, out, None) == dn.DN_EINVAL
    assert list(out) == [-7, -7]


# ----------------------------------------------------------------------------- similarity-driven K

K_THR = [0.80, 0.85, 0.90, 0.93]
K_LEV = [0, 5, 10, 15, 25]


@pytest.mark.parametrize("n,dim,nq", [(100_000, 768, 70), (5000, 77, 9)])
def test_lookup_batch_k_matches_oracle_levels(n, dim, nq):
    """ac_lookup_batch_k: indices and cosines bitwise those of ac_lookup_batch; the level
    of each query bit-exactly the oracle's select_k on the reported fp32 cosine, and the
    oracle's select_k on its own fp64 cosine (rounded to fp32) except within 1e-6 of a
    threshold; a zero query gets index -1 and K = 0. dim 77 runs the per-query scan."""
    announce(f"lookup batch + K: n={n} dim={dim} nq={nq}")
    cache = W.cache_embeddings(n, dim, seed=7)
    qs, rows = W.planted_queries(cache, nq, seed=9, cos_lo=0.75, cos_hi=0.97)
    qs[3] = 0
    cd = torch.from_numpy(cache.view(np.uint16)).to(DEV)
    qd = torch.from_numpy(qs.view(np.uint16).copy()).to(DEV)
    idx, score, k = dn.ac_lookup_batch_k(qd, cd, K_THR, K_LEV)
    bidx, bscore = dn.ac_lookup_batch(qd, cd)
    assert idx == bidx
    assert np.array_equal(np.asarray(score, np.float32).view(np.uint32), np.asarray(bscore, np.float32).view(np.uint32))
    assert idx[3] == -1 and k[3] == 0
    assert list(OL.select_k(np.asarray(score, np.float32), K_THR, K_LEV)) == k
    ridx, rscore = OL.top1_batch(qs, cache)
    rk = OL.select_k(rscore.astype(np.float32), K_THR, K_LEV)
    for j in range(nq):
        if j == 3:
            continue
        assert idx[j] == rows[j]
        if rk[j] != k[j]:
            assert min(abs(rscore[j] - t) for t in K_THR) < 1e-6, (j, rscore[j], k[j], rk[j])
    assert len(set(k)) >= 3   # the planted cosines span several levels


def test_lookup_batch_k_rejects_bad_tables():
    announce("lookup batch + K: table errors")
    cache = torch.from_numpy(W.cache_embeddings(256, 256, seed=1).view(np.uint16)).to(DEV)
    q = cache[:2].clone()
    for thr, lev in (([0.9, 0.8], [0, 5, 10]), ([0.8, float("nan")], [0, 5, 10]), ([0.8], [5, 0]),
                     ([0.8], [-1, 5]), ([0.1 * i for i in range(15)] + [2.0], list(range(17)))):
        t = dn.k_table(thr[:15], lev[:16])
        t.n_thresholds = len(thr)
        idx = (dn.C.c_int64 * 2)(-7, -7)
        kk = (dn.C.c_int32 * 2)(-7, -7)
        code = dn.lib.ac_lookup_batch_k(q.data_ptr(), 2, cache.data_ptr(), 256, 256, dn.C.byref(t), idx, None, kk)
        assert code == dn.DN_EINVAL, (thr, lev)
        assert list(idx) == [-7, -7] and list(kk) == [-7, -7]
