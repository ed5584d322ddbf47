"""The stream-read calibration kernel on the GPU: every work group reads
exactly its part of the buffer (the sink words equal the XOR of each part,
computed on the host), including uneven and empty parts."""
import numpy as np
import pytest
import torch

from paper_2605_30574_amd import calib

pytestmark = pytest.mark.gpu


def expected_words(data: np.ndarray, blocks: int) -> np.ndarray:
    units = data.view(np.uint32).reshape(-1, 4)
    per = -(-units.shape[0] // blocks)
    out = np.zeros(blocks, dtype=np.uint32)
    for b in range(blocks):
        part = units[b * per:(b + 1) * per]
        if part.size:
            out[b] = np.bitwise_xor.reduce(part.reshape(-1))
    return out


@pytest.mark.parametrize("units,blocks", [(1, 1), (5, 8), (1000003, 7), (1 << 20, 1024), (3 * 2048 + 11, 2048)])
def test_every_part_is_read(units, blocks):
    rng = np.random.default_rng(units * 31 + blocks)
    data = rng.integers(0, 2**32, size=units * 4, dtype=np.uint32).view(np.uint8)
    dev = torch.device("cuda:0")
    buf = torch.from_numpy(data).to(dev)
    sink = torch.full((blocks + 3,), -1, dtype=torch.int32, device=dev)
    calib.stream_read(buf, sink, blocks)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    assert np.array_equal(got[:blocks], expected_words(data, blocks))
    assert np.all(got[blocks:] == np.uint32(0xFFFFFFFF))   # nothing past the last work group's word
