"""ac_lookup_batch_noalloc (the entry point for callers that cannot allocate) against
ac_lookup_batch through the C ABI: indices bit-exact and cosines bitwise equal (the same
kernels run), on consecutive calls where the second is smaller than the first (the
library's fixed scratch then holds the first call's winners), with and without a
cosine output, on the matrix-core widths and on a per-query width."""

import numpy as np
import pytest
import torch

from paper_2511_06724_amd import dn, workloads as W
from tests.gpu_util import DEV, announce

pytestmark = pytest.mark.gpu


def _dev16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.uint16)).to(DEV)


def _noalloc(q, cache, with_score=True):
    nq = q.shape[0]
    idx = torch.full((nq,), -7, device=DEV, dtype=torch.int64)
    score = torch.full((nq,), float("nan"), device=DEV) if with_score else None
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    dn.ac_lookup_batch_noalloc(q, cache, idx, score, stream=s)
    s.synchronize()
    return idx.cpu().tolist(), (score.cpu().numpy() if with_score else None)


def _check_call(q, cache, with_score=True):
    ridx, rscore = dn.ac_lookup_batch(q, cache)
    idx, score = _noalloc(q, cache, with_score)
    assert idx == ridx
    if with_score:
        assert np.array_equal(score.view(np.uint32), np.asarray(rscore, np.float32).view(np.uint32))
    return idx


@pytest.mark.parametrize("dim", [768, 77])
def test_noalloc_matches_batch_on_two_calls_second_smaller(dim):
    announce(f"no-alloc lookup vs ac_lookup_batch, dim={dim}")
    n1, nq1 = (100_000, 70) if dim == 768 else (20_000, 9)
    cache = W.cache_embeddings(n1, dim, seed=7)
    qs, rows = W.planted_queries(cache, nq1, seed=9)
    cd, qd = _dev16(cache), _dev16(qs)
    idx = _check_call(qd, cd)
    assert idx == [int(r) for r in rows]
    # second call, smaller: fewer rows and queries (fewer scan workgroups than the first)
    n2, nq2 = 4097, 5
    small = W.cache_embeddings(n2, dim, seed=17)
    sq, srows = W.planted_queries(small, nq2, seed=19)
    sd = _dev16(small)
    idx2 = _check_call(_dev16(sq), sd, with_score=False)
    assert idx2 == [int(r) for r in srows]
    # a zero query reports -1, as in ac_lookup_batch
    sq[1] = 0
    idx3 = _check_call(_dev16(sq), sd)
    assert idx3[1] == -1


def test_noalloc_argument_errors_enqueue_nothing():
    announce("no-alloc lookup argument errors")
    cache = _dev16(W.cache_embeddings(64, 256, seed=3))
    q = cache[:2].clone()
    out = torch.full((2,), -7, device=DEV, dtype=torch.int64)
    for bad in (dict(nq=0), dict(n=0), dict(dim=0), dict(out=None)):
        code = dn.lib.ac_lookup_batch_noalloc(q.data_ptr(), bad.get("nq", 2), cache.data_ptr(), bad.get("n", 64),
                                              bad.get("dim", 256),
                                              None if "out" in bad else out.data_ptr(), None,
                                              torch.cuda.current_stream().cuda_stream)
        assert code == dn.DN_EINVAL
    torch.cuda.synchronize()
    assert out.cpu().tolist() == [-7, -7]
