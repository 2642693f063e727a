"""The agentic replay over a device pool (GPU).

The device pool must take every decision the metadata-only pool takes on the
same replay (equal summaries and session tables), and after hundreds of steps of
LRU eviction, write-back and partial resumes the sessions' pages must still hold
exactly their own KV: the last step's decode of the running sessions, and the
decode of paused sessions resumed afterwards, match the oracle on KV
regenerated from each session's generator id.
"""

import numpy as np
import pytest

import synth
from helpers import Case, to_device, to_host, tolerance_check

pytestmark = pytest.mark.gpu

SEED = 91


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)


def _cfg(spill=False):
    from paper_2609_25782_amd import replay as rp
    cfg = rp.ReplayConfig(n_active=6, num_layers=2, num_kv_heads=2, head_dim=64, elt_bytes=2,
                          weight_bytes=0.0, tbt_s=1.0, warmup_s=80, plateau_s=320, sample_s=1.0,
                          prompt0=(10, 40), turn_prompt=(5, 30), turn_decode=(5, 40), peak=(60, 160),
                          gap_median_s=6.0, gap_mean_s=15.0, max_sessions=64, seed=3,
                          spill=spill, promote_s=7.0)
    cfg.hbm_bytes = 40 * cfg.page_bytes       # LRU pressure, partial resumes and preemptions
    cfg.cold_bytes = 2000 * cfg.page_bytes
    return cfg


def _oracle(lens, gens, q, layer):
    case = Case(2, 4, 2, 64, "bf16", lens, seed=SEED, layer=layer)
    case.kv = [synth.session_kv(SEED, g, n, layer, 2, 64, 1.0, "bf16") for g, n in zip(gens, lens)]
    case.q = q
    return case.oracle_out()


@pytest.mark.timeout(300)
@pytest.mark.parametrize("spill", [False, True])
def test_device_replay_follows_metadata_and_keeps_kv(dev, spill):
    import torch
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd import replay as rp
    from paper_2609_25782_amd.pool import HotColdPool

    cfg = _cfg(spill)
    print("replay, spill %s" % spill, flush=True)
    meta = rp.Replay(cfg)
    want = meta.run()
    print("metadata replay:", want["plateau_counts"], flush=True)

    hp = HotColdPool(2, 2, 64, "bf16", cfg.num_hot_pages, cfg.num_cold_pages, cfg.max_sessions,
                     cfg.stride)
    dp = rp.DevicePool(cfg, hp, SEED, float(synth.value_multiplier(1.0)))
    q_host = synth.queries(SEED + 1, cfg.n_active, 4, 64, 1.0, "bf16", 0)
    dec = rp.DeviceDecode(hp, to_device(q_host, "bf16", dev))
    r = rp.Replay(cfg, dp)
    got = r.run(dec)
    torch.cuda.synchronize()
    print("device replay:", got["plateau_counts"], flush=True)
    assert got == want
    for sid in range(cfg.max_sessions):
        assert kv.kv_session_info(dp.h, sid) == kv.kv_session_info(meta.pool.h, sid)
    c = got["plateau_counts"]
    assert c["pages_to_cold"] > 0 and 0 < c["resume_pages_resident"] < c["resume_pages_total"]
    if spill:                      # decode read spilled pages in place, then they came back
        assert got["preemptions"] == 0 and c["spilled_pages"] > 0 and c["promoted_pages"] > 0
        assert got["spill"]["cold_share_of_hot_set"] > 0
    t = dec.timings()
    assert len(t["step_ms"]) == int(cfg.plateau_s / cfg.step_s) and np.all(t["decode_ms"] > 0)

    # the last step's decode (layer 1 is the last one decoded) against the oracle;
    # a session that ended at that step has no generator id any more
    sids, lens = dec.last_batch()
    rows = [i for i, s in enumerate(sids) if s in dp.gen]
    assert len(rows) >= 3
    ref = _oracle([lens[i] for i in rows], [dp.gen[sids[i]] for i in rows], q_host[rows], 1)
    tolerance_check(to_host(dec.out)[rows], ref)

    # paused sessions, resumed one by one (fetching whatever LRU evicted)
    paused = [s for s in range(cfg.max_sessions)
              if kv.kv_session_info(dp.h, s)[0] == kv.KV_SESSION_PAUSED]
    assert paused
    checked = 0
    for s in paused[:8]:
        hot_before = kv.kv_session_info(dp.h, s)[2]
        kv.kv_resume_session(dp.h, s)
        n = kv.kv_session_info(dp.h, s)[1]
        table = hp.gather_table(torch.tensor([s], dtype=torch.int32, device=dev))
        lens_dev = torch.tensor([n], dtype=torch.int32, device=dev)
        out = to_host(hp.decode(0, dec.q[:1], lens_dev, page_table=table))
        tolerance_check(out, _oracle([n], [dp.gen[s]], q_host[:1], 0))
        checked += -1 in hot_before
        kv.kv_session_pause(dp.h, s)
    print("resumed and checked %d paused sessions, %d with evicted pages" % (len(paused[:8]), checked),
          flush=True)
    meta.close()
    hp.close()


def test_gather_table_rows(dev):
    """The batch table holds the pool's rows of the listed sessions, bit for bit
    (the oracle's pool model predicts them), and -1 rows for ids out of range."""
    import torch
    from oracle.pool_model import PoolModel
    from paper_2609_25782_amd.pool import HotColdPool

    hp = HotColdPool(1, 1, 64, "f32", 40, 40, 5, 6)
    m = PoolModel(40, 40, 5, 6)
    for L in (33, 90, 16, 5):
        assert hp.create_session(L) == m.create(L)
    hp.evict(1)
    m.evict(1)
    hp.resume(1)
    m.resume([1])
    sids = [3, 1, -1, 0, 7, 2, 3]
    got = hp.gather_table(torch.tensor(sids, dtype=torch.int32, device=dev)).cpu().numpy()
    want = np.array([m.row(s) if 0 <= s < 5 else [-1] * 6 for s in sids], np.int32)
    assert np.array_equal(got, want)
    hp.close()
