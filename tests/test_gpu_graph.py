"""Decode steps captured in a HIP graph (GPU).

A serving loop replays a captured decode step instead of launching 2 x layers
kernels from the host.  Every replay must equal the eager decode bit for bit,
with the program's own eager work and synchronisations between replays, and a
replay must read the inputs as they are at replay time (new lengths, new
queries)."""

import numpy as np
import pytest
import torch

import synth
from helpers import Case, to_device, to_host, tolerance_check

pytestmark = pytest.mark.gpu

SEED = 5


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


@pytest.mark.parametrize("vector,many", [(False, False), (True, False), (False, True)])
def test_decode_step_graph_replays_match_eager(dev, vector, many):
    """Both forms of the split kernel: matrix cores and the vector ALU.  With
    many short rows (400 rows: more (row, KV head) segments than waves) the
    merge walks the waves' split-segment entries, which every replay rewrites."""
    from paper_2609_25782_amd.pool import HotColdPool
    layers, lens = 4, [300, 1000, 57, 2000, 16, 777]
    if many:
        lens = [int(x) for x in np.random.default_rng(9).integers(1, 600, size=400)]
    n_pages = sum(synth.pages_for(L) for L in lens)
    pool = HotColdPool(layers, 2, 128, "bf16", n_pages + 10, 0, len(lens), synth.pages_for(2100))
    pool.set_compute(vector)
    for b, L in enumerate(lens):
        pool.create_session(L)
        pool.fill_synthetic(b, b, SEED, float(synth.value_multiplier(1.0)))
    B = len(lens)
    cases = [Case(layers, 8, 2, 128, "bf16", lens, seed=SEED, layer=l) for l in range(layers)]
    qs = [to_device(c.q, "bf16", dev) for c in cases]
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    pt = pool.page_table[:B]

    def eager():
        return [pool.decode(l, qs[l], sl, page_table=pt).clone() for l in range(layers)]

    ref = eager()
    torch.cuda.synchronize()
    tolerance_check(to_host(ref[layers - 1]), cases[layers - 1].oracle_out())
    outs = [torch.empty_like(q) for q in qs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):                       # workspace allocated before capture
        pool.decode(0, qs[0], sl, page_table=pt, out=outs[0], stream=s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for l in range(layers):
            pool.decode(l, qs[l], sl, page_table=pt, out=outs[l], stream=s)
    for rep in range(4):
        for o in outs:
            o.fill_(7.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for l in range(layers):
            assert torch.equal(outs[l], ref[l]), "replay %d layer %d" % (rep, l)
        eager()                                      # the program's own work between replays
        torch.cuda.synchronize()
    # inputs changed in place: the replay reads them as they are now
    new_lens = [L // 2 + 1 for L in lens]
    sl.copy_(torch.tensor(new_lens, dtype=torch.int32, device=dev))
    for q in qs:
        q.mul_(-1.0)
    ref2 = eager()
    g.replay()
    torch.cuda.synchronize()
    for l in range(layers):
        assert torch.equal(outs[l], ref2[l])
    pool.close()
