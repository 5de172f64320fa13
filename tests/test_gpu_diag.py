"""The streaming-read measurement helper reads every byte: its XOR fold
equals the host's."""
import numpy as np
import pytest
import torch

from paper_2607_24260_amd import kap as K

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (1 << 24) + 1024 * 16 + 16, 3 << 27])
def test_stream_read_folds_every_word(nbytes):
    g = torch.Generator(device="cuda").manual_seed(nbytes % 1000)
    buf = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), generator=g, dtype=torch.int32,
                        device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    K.stream_read(buf, sink)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(buf.cpu().numpy().view(np.uint32))
    assert int(sink.item()) & 0xFFFFFFFF == int(want)
