"""The library's page writers produce the documented page layout, byte for byte:
kv_write_tokens and kv_fill_synthetic against the oracle's own packer fed with
the seeded generator's values."""

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import ORACLE_DTYPE, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


@pytest.mark.parametrize("dtype,D,NL,hkv", [("bf16", 128, 3, 4), ("bf16", 64, 1, 1),
                                             ("f32", 64, 2, 2), ("f32", 128, 1, 1)])
def test_fill_synthetic_matches_generator(dev, dtype, D, NL, hkv):
    from paper_2609_25782_amd.pool import HotColdPool
    print("fill case", dtype, D, NL, hkv, flush=True)
    L = 16 * 5 + 3
    pool = HotColdPool(NL, hkv, D, dtype, 12, 0, 2, 8)
    pages = [7, 2, 11, 0, 5, 9]
    sid = pool.create_session(L, pages)
    mult = float(synth.value_multiplier(0.7))
    pool.fill_synthetic(sid, 5, 1234, mult)
    torch.cuda.synchronize()
    got = pool.hot_page_bytes().cpu().numpy().reshape(-1)
    od = ORACLE_DTYPE[dtype]
    want = np.zeros_like(got)
    n_tok = 16 * len(pages)  # the fill writes every slot of every page
    for layer in range(NL):
        k, v = synth.session_kv(1234, 5, n_tok, layer, hkv, D, 0.7, dtype)
        oracle.pack_pool(want, NL, hkv, D, od, layer, np.array(pages), k, v)
    pb = pool.page_bytes
    for p in pages:
        assert np.array_equal(got[p * pb:(p + 1) * pb], want[p * pb:(p + 1) * pb]), "page %d" % p
    pool.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_write_tokens_matches_packer(dev, dtype):
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, D, L = 2, 2, 64, 16 * 3 + 9
    pool = HotColdPool(NL, hkv, D, dtype, 6, 0, 1, 4)
    pool.hot.zero_()
    sid = pool.create_session(L, [4, 1, 5, 0])
    k, v = synth.session_kv(9, 0, L, 1, hkv, D, 1.0, dtype)
    # two writes: a prefix and the rest, to exercise tok_begin
    pool.write_tokens(sid, 1, 0, to_device(k[:20], dtype, dev), to_device(v[:20], dtype, dev))
    pool.write_tokens(sid, 1, 20, to_device(k[20:], dtype, dev), to_device(v[20:], dtype, dev))
    torch.cuda.synchronize()
    want = np.zeros(pool.hot.numel(), np.uint8)
    oracle.pack_pool(want, NL, hkv, D, ORACLE_DTYPE[dtype], 1, np.array([4, 1, 5, 0]), k, v)
    assert np.array_equal(pool.hot_page_bytes().cpu().numpy().reshape(-1), want)
    pool.close()


def test_decode_reads_oracle_packed_pool(dev):
    """A pool packed on the host by the oracle's packer and uploaded raw decodes
    to the oracle's answer: the kernel reads the documented layout."""
    from helpers import Case, tolerance_check, to_host
    from paper_2609_25782_amd.pool import HotColdPool
    case = Case(2, 16, 2, 128, "bf16", [700, 33], seed=31, layer=1)
    pool = HotColdPool(2, 2, 128, "bf16", case.hot_pages, 0, 2, case.stride)
    host = np.zeros(pool.hot.numel(), np.uint8)
    for b in range(case.batch):
        k, v = case.kv[b]
        oracle.pack_pool(host, 2, 2, 128, oracle.BF16, 1, case.placement[b], k, v)
    pool.hot_pages().copy_(torch.from_numpy(host).to(dev).view(pool.num_hot_pages, pool.num_layers, -1))
    for b, L in enumerate(case.seq_lens):
        pool.create_session(L, [int(p) for p in case.placement[b]])
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(case.seq_lens, dtype=torch.int32, device=dev)
    got = to_host(pool.decode(1, q, sl))
    torch.cuda.synchronize()
    tolerance_check(got, case.oracle_out())
    pool.close()
