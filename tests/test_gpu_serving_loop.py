"""Data paths 1-4 composed as a serving loop uses them: each step extends the
decoding sessions by one token, appends that token's K/V in every layer with
one batched call, gathers the batch table and decodes every layer.  Midway two
sessions are evicted, others keep decoding, and the two are resumed on a second
stream and rejoin.  Every checked step matches the fp64 oracle on the same
logical KV (the counter-based generator's prefix)."""

import numpy as np
import pytest
import torch

import synth
from helpers import Case, to_device, to_host, tolerance_check

pytestmark = pytest.mark.gpu

SEED = 43
NL, HKV, HQ, D, DT = 2, 2, 8, 128, "bf16"


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def test_append_decode_evict_resume_loop(dev):
    from paper_2609_25782_amd.pool import HotColdPool
    prompts = [31, 16, 1, 200, 47, 15]
    steps = 40
    final = [L + steps for L in prompts]
    kv = {(b, layer): synth.session_kv(SEED, b, final[b], layer, HKV, D, 1.0, DT)
          for b in range(len(prompts)) for layer in range(NL)}
    pages = sum(synth.pages_for(L) for L in final)
    pool = HotColdPool(NL, HKV, D, DT, pages + 4, pages + 4, len(prompts), max(synth.pages_for(L) for L in final))
    sids = []
    for b, L in enumerate(prompts):                      # the prompts (prefill stand-in)
        sid = pool.create_session(L)
        for layer in range(NL):
            k, v = kv[(b, layer)]
            pool.write_tokens(sid, layer, 0, to_device(k[:L], DT, dev), to_device(v[:L], DT, dev))
        sids.append(sid)
    lens = list(prompts)
    side = torch.cuda.Stream()
    active = list(range(len(prompts)))
    q = {layer: synth.queries(SEED + 1 + layer, len(prompts), HQ, D, 1.0, DT, layer) for layer in range(NL)}
    checked = 0
    for step in range(steps):
        if step == 12:                                   # two sessions pause; their pages go cold
            pool.evict([sids[1], sids[3]])
            active = [b for b in active if b not in (1, 3)]
        if step == 20:                                   # and come back, resumed on another stream
            pool.resume([sids[1], sids[3]], stream=side)
            torch.cuda.current_stream().wait_stream(side)
            active = sorted(active + [1, 3])
        for b in active:
            pool.extend(sids[b], lens[b] + 1)
        rows = [sids[b] for b in active]
        table = pool.gather_table(torch.tensor(rows, dtype=torch.int32, device=dev))
        sl = torch.tensor([lens[b] + 1 for b in active], dtype=torch.int32, device=dev)
        outs = []
        for layer in range(NL):
            k = np.stack([kv[(b, layer)][0][lens[b]] for b in active])
            v = np.stack([kv[(b, layer)][1][lens[b]] for b in active])
            pool.append_tokens(layer, rows, [lens[b] for b in active], to_device(k, DT, dev), to_device(v, DT, dev))
            qb = to_device(q[layer][active], DT, dev)
            outs.append(pool.decode(layer, qb, sl, page_table=table))
        for b in active:
            lens[b] += 1
        if step % 7 == 6 or step == steps - 1:
            torch.cuda.synchronize()
            for layer in range(NL):
                case = Case(NL, HQ, HKV, D, DT, [lens[b] for b in active], seed=SEED, layer=layer)
                case.kv = [(kv[(b, layer)][0][:lens[b]], kv[(b, layer)][1][:lens[b]]) for b in active]
                case.q = q[layer][active]
                tolerance_check(to_host(outs[layer]), case.oracle_out())
            checked += 1
    assert checked >= 6 and lens[1] < final[1] and lens[0] == final[0]
    st = pool.stats()
    assert st["pages_to_cold"] > 0 and st["pages_to_hot"] > 0
    pool.close()
