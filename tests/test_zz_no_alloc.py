"""m2c_predict_rank_noalloc, through the C ABI, against m2c_predict_rank: the
same scores and tier maps bit for bit on two calls in a row, the second with
a smaller input, with the scratch holding z only and z plus the scores; and
the size limit is refused on the host with nothing enqueued."""
import ctypes

import numpy as np
import pytest

from paper_2410_14740_amd import m2c
from paper_2410_14740_amd import workloads as W

from helpers import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SCRATCH = 4 << 20  # M2C_NOALLOC_SCRATCH_BYTES


def _layer(ld, k, batch):
    return m2c.Layer(m2c.make_desc(ld.d_model, ld.d_ff, ld.pred_rank, k, ld.d_ff // 2,
                                   max_batch=batch), ld)


def _x(ld):
    return torch.from_numpy(np.ascontiguousarray(ld.x[0].view(np.uint16))).cuda()


def _both(L, x, batch, k, n16, n8, with_scores):
    d_ff = L.desc.d_ff
    lib = m2c.load()
    s = torch.cuda.current_stream().cuda_stream
    s_ref = torch.empty((batch, d_ff), dtype=torch.float32, device="cuda")
    t_ref = torch.empty((batch, d_ff), dtype=torch.uint8, device="cuda")
    s_new = torch.full((batch, d_ff), float("nan"), dtype=torch.float32, device="cuda")
    t_new = torch.full((batch, d_ff), 0xEE, dtype=torch.uint8, device="cuda")
    assert lib.m2c_predict_rank(L.handle, x.data_ptr(), batch, k, n16, n8, s_ref.data_ptr(),
                                t_ref.data_ptr(), s) == m2c.M2C_OK
    rc = lib.m2c_predict_rank_noalloc(L.handle, x.data_ptr(), batch, k, n16, n8,
                                      s_new.data_ptr() if with_scores else None,
                                      t_new.data_ptr(), s)
    assert rc == m2c.M2C_OK, m2c.m2c_last_error()
    torch.cuda.synchronize()
    assert torch.equal(t_new, t_ref)
    if with_scores:
        assert torch.equal(s_new.view(torch.int32), s_ref.view(torch.int32))


def test_noalloc_matches_predict_rank_twice_smaller_second():
    big = W.make_layer(W.WORKLOADS["tiny"].seed, 7, 1024, 2752, 128, 1,
                       rhos=(0.9, 0.5, 0.95, 0.7), zipf_bias=True)
    small = W.make_layer(55, 7, 512, 900, 32, 1)
    Lb, Ls = _layer(big, 688, 4), _layer(small, 225, 1)
    for with_scores in (False, True):
        say(f"noalloc: batch 4, d_ff 2752, scores buffer {with_scores}")
        _both(Lb, _x(big), 4, 688, 229, 229, with_scores)
        say(f"noalloc: batch 1, d_ff 900 (smaller), scores buffer {with_scores}")
        _both(Ls, _x(small), 1, 225, 75, 75, with_scores)
    Lb.close()
    Ls.close()


def test_noalloc_rejects_scratch_beyond_limit():
    """batch 4 x 262144 scores need 4 MiB plus z of scratch: refused on the
    host (nothing enqueued, the output untouched); with a scores buffer the
    same call fits (only z is scratch)."""
    # the widest layer (262144 neurons), rank 8 and d 128 keep the weights small
    d_ff, batch = 262144, 4
    assert 4 * batch * d_ff + 256 > SCRATCH  # the scores alone are exactly the limit; z exceeds it
    lw = W.make_layer(66, 0, 128, d_ff, 8, 1, rhos=(0.9,) * batch)
    L = m2c.Layer(m2c.make_desc(128, d_ff, 8, 100, 1000, max_batch=batch), lw)
    x = _x(lw)
    tiers = torch.full((batch, d_ff), 0xEE, dtype=torch.uint8, device="cuda")
    lib = m2c.load()
    s = torch.cuda.current_stream().cuda_stream
    rc = lib.m2c_predict_rank_noalloc(L.handle, x.data_ptr(), batch, 100, 10, 30, None,
                                      tiers.data_ptr(), s)
    assert rc == m2c.M2C_ERR_CAPACITY and "M2C_NOALLOC_SCRATCH_BYTES" in m2c.m2c_last_error()
    torch.cuda.synchronize()
    assert bool((tiers == 0xEE).all())
    say("noalloc: 262144 neurons with a scores buffer")
    _both(L, x, batch, 100, 10, 30, True)
    L.close()
