"""The allocation-free top-q entry point against the ordinary one, through the
C ABI: on the same scores and masks both must give the same indices, scores
and eligible count, bit for bit, on two calls in a row (the second on a
smaller input, so stale lists from the first call would show)."""
import ctypes as C
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2408_04323_amd import F32, F64  # noqa: E402
from paper_2408_04323_amd._native import lib  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def _scores(n, dt, seed):
    rng = np.random.default_rng(seed)
    s = rng.standard_normal(n)
    s[rng.integers(0, n, max(1, n // 100))] = 0.25          # ties: lowest index first
    s[rng.integers(0, n, max(1, n // 500))] = np.nan         # never eligible
    mask = (rng.random(n) < 0.7).astype(np.uint8)
    td = torch.float32 if dt == F32 else torch.float64
    return torch.as_tensor(s).to(td).to(DEV), torch.as_tensor(mask).to(DEV)


def _call(fn, score, mask, dt, q):
    idx = torch.full((q,), -7, dtype=torch.int64, device=DEV)
    sc = torch.full((q,), 7.0, dtype=score.dtype, device=DEV)
    nv = torch.full((1,), -7, dtype=torch.int32, device=DEV)
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = fn(C.c_void_p(score.data_ptr()), C.c_void_p(0 if mask is None else mask.data_ptr()), score.numel(), dt, q,
            C.c_void_p(idx.data_ptr()), C.c_void_p(sc.data_ptr()), C.c_void_p(nv.data_ptr()), stream)
    assert rc == 0, lib().scoot_last_error().decode()
    torch.cuda.synchronize()
    return idx.cpu().numpy(), sc.cpu().numpy(), int(nv.cpu()[0])


@pytest.mark.parametrize("dt", [F32, F64], ids=["f32", "f64"])
@pytest.mark.parametrize("masked", [True, False], ids=["mask", "nomask"])
@pytest.mark.parametrize("sizes", [(1_000_003, 64, 262_144, 8), (262_144, 4, 5_000, 1), (70_000, 1, 17, 3)])
def test_noalloc_topq_matches_topq(dt, masked, sizes):
    L = lib()
    n1, q1, n2, q2 = sizes
    for k, (n, q) in enumerate(((n1, q1), (n2, q2))):
        say("noalloc topq", dt, masked, n, q)
        score, mask = _scores(n, dt, 7 * n + k)
        m = mask if masked else None
        want = _call(L.scoot_suggest_topq, score, m, dt, q)
        got = _call(L.scoot_suggest_topq_noalloc, score, m, dt, q)
        np.testing.assert_array_equal(got[0], want[0])
        np.testing.assert_array_equal(got[1], want[1])   # NaN where no pick, in both
        assert got[2] == want[2]
        assert (want[0] >= 0).sum() == min(q, want[2])


def test_noalloc_topq_argument_errors():
    L = lib()
    idx = torch.empty(4, dtype=torch.int64, device=DEV)
    s = torch.zeros(10, device=DEV)
    st = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    for n, q in ((10, 0), (10, 65), (-1, 4), (1 << 31, 4)):
        rc = L.scoot_suggest_topq_noalloc(C.c_void_p(s.data_ptr()), None, n, F32, q, C.c_void_p(idx.data_ptr()),
                                          None, None, st)
        assert rc == -1 and L.scoot_last_error().decode().startswith("topq (no allocation)")
