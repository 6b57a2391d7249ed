"""The read-only streaming reference (sparrow_stream_read): every 32-bit word of the
buffer is read once - its checksum equals the wrap-around sum computed on the host."""
import numpy as np
import pytest
import torch

from paper_2606_08446_amd import sparrow as S

from parity import log

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(autouse=True)
def _need_gpu(gpu_device):
    S.load()
    yield


@pytest.mark.parametrize("nbytes", [16, 4096 + 16, 3 * 2**20 + 48, 2**28])
def test_stream_read_checksum(nbytes):
    log(f"case stream read {nbytes} bytes")
    g = torch.Generator(device=DEV)
    g.manual_seed(nbytes % 1000)
    words = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), generator=g, dtype=torch.int32,
                          device=DEV)
    got = S.stream_read(words)
    again = S.stream_read(words, checksum=got.clone())       # adds on top of the given value
    torch.cuda.synchronize()
    want = int(words.cpu().numpy().view(np.uint32).astype(np.uint64).sum() % 2**32)
    assert int(got.cpu().numpy().view(np.uint32)[0]) == want
    assert int(again.cpu().numpy().view(np.uint32)[0]) == (2 * want) % 2**32
