"""The streaming-read probe (kv_read_probe) reads every byte it is given: the
XOR of its per-block words equals the XOR of all 32-bit words of the buffer,
for sizes that exercise the unrolled loop and the tail, and for several grids.
Bad arguments are refused."""

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


@pytest.mark.parametrize("nbytes,blocks", [(16, 1), (4096 + 48, 3), (1 << 20, 7), ((1 << 24) + 16 * 1001, 64),
                                           ((1 << 27) + 16 * 37, 4096)])
def test_probe_reads_every_word(dev, nbytes, blocks):
    from paper_2609_25782_amd import hotcold_kv as kv
    rng = np.random.default_rng(nbytes % 1000 + blocks)
    host = rng.integers(0, 2 ** 32, size=nbytes // 4, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).to(dev)
    out = torch.full((blocks,), -1, dtype=torch.int32, device=dev)
    kv.kv_read_probe(buf.data_ptr(), nbytes, out.data_ptr(), blocks, 0)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)


def test_probe_refuses_bad_arguments(dev):
    from paper_2609_25782_amd import hotcold_kv as kv
    buf = torch.zeros(1024, dtype=torch.uint8, device=dev)
    out = torch.zeros(4, dtype=torch.int32, device=dev)
    for args in ((buf.data_ptr(), 1000, out.data_ptr(), 1),      # not a multiple of 16
                 (buf.data_ptr() + 4, 512, out.data_ptr(), 1),   # misaligned
                 (buf.data_ptr(), 1024, out.data_ptr(), 0),      # no blocks
                 (buf.data_ptr(), 0, out.data_ptr(), 1),
                 (0, 1024, out.data_ptr(), 1)):
        with pytest.raises(kv.KVError) as e:
            kv.kv_read_probe(*args, 0)
        assert e.value.status == kv.KV_ERR_INVALID
