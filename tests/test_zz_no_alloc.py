"""The no-allocation decode entry point (paged_decode_attention_noalloc) against
the entry point it is a variant of (paged_decode_attention with a caller
workspace): same kernels and work split, so the outputs must be bitwise equal.
Two calls in a row, the second with a smaller batch, then a batch too large for
the scratch array, which must be refused before anything is launched."""

import sys

import numpy as np
import pytest
import torch

from helpers import Case, build_gpu, to_device, to_host, tolerance_check

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _noalloc(kv, pool, layer, q, sl, pt, out):
    B, Hq, D = q.shape
    kv.paged_decode_attention_noalloc(pool.handle, layer, q.data_ptr(), pt.data_ptr(), pt.shape[1],
                                      sl.data_ptr(), B, Hq, D ** -0.5, out.data_ptr(),
                                      torch.cuda.current_stream().cuda_stream)


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("dtype,hq,hkv,d", [("bf16", 32, 4, 128), ("f32", 8, 2, 64)])
def test_noalloc_matches_workspace_entry_point(dev, fused, dtype, hq, hkv, d):
    from paper_2609_25782_amd import hotcold_kv as kv
    lens = [4000, 17, 1, 2500, 0, 16, 9000, 333]
    case = Case(2, hq, hkv, d, dtype, lens, seed=91, layer=1)
    pool = build_gpu(case, dev, pool_kwargs={"max_sessions": 8})
    pool.set_combine(fused)
    q = to_device(case.q, dtype, dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    pt = pool.page_table[:len(lens)].contiguous()
    ref = case.oracle_out()
    for rows in (slice(0, 8), slice(1, 4)):       # the second call is smaller
        _say("%s hq=%d hkv=%d d=%d fused=%s rows %s" % (dtype, hq, hkv, d, fused, rows))
        qa, sa, pa = q[rows].contiguous(), sl[rows].contiguous(), pt[rows].contiguous()
        want = pool.decode(1, qa, sa, page_table=pa).clone()
        got = torch.full_like(want, float("nan"))
        _noalloc(kv, pool, 1, qa, sa, pa, got)
        torch.cuda.synchronize()
        assert torch.equal(got, want)
        tolerance_check(to_host(got), ref[rows], max_norm=1e-2 if dtype == "bf16" else 1e-5)
    pool.close()


def test_noalloc_refuses_batches_beyond_its_scratch(dev):
    from paper_2609_25782_amd import hotcold_kv as kv
    case = Case(1, 32, 4, 128, "bf16", [100], seed=92)
    pool = build_gpu(case, dev, pool_kwargs={"max_sessions": 1})
    B = 4096                                      # needs about 70 MB of partials
    need = kv.paged_decode_workspace_bytes(pool.handle, B, 32)
    assert need > kv.KV_DECODE_SCRATCH_BYTES
    q = torch.zeros((B, 32, 128), dtype=torch.bfloat16, device=dev)
    sl = torch.zeros(B, dtype=torch.int32, device=dev)
    pt = torch.full((B, 8), -1, dtype=torch.int32, device=dev)
    out = torch.full_like(q, 7.0)
    torch.cuda.synchronize()
    with pytest.raises(kv.KVError) as e:
        _noalloc(kv, pool, 0, q, sl, pt, out)
    assert e.value.status == kv.KV_ERR_INVALID
    assert "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())               # nothing was launched
    # the largest batch that fits still decodes, equal to the workspace call
    fit = next(b for b in range(B, 0, -64) if kv.paged_decode_workspace_bytes(pool.handle, b, 32)
               <= kv.KV_DECODE_SCRATCH_BYTES)
    _say("largest batch of 64-row steps that fits the scratch: %d" % fit)
    sl[:fit] = torch.tensor(np.full(fit, 100, np.int32), device=dev)
    pt[:fit, :7] = pool.page_table[0, :7]
    qa, sa, pa = q[:fit].contiguous(), sl[:fit].contiguous(), pt[:fit].contiguous()
    qa.copy_(to_device(np.repeat(case.q, fit, axis=0), "bf16", dev))
    want = pool.decode(0, qa, sa, page_table=pa).clone()
    got = torch.empty_like(want)
    _noalloc(kv, pool, 0, qa, sa, pa, got)
    torch.cuda.synchronize()
    assert torch.equal(got, want)
    tolerance_check(to_host(got[:1]), case.oracle_out())
    pool.close()
