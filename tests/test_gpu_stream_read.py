"""GPU check of the read-ceiling probe (peat_stream_read): every 32-bit word
of the buffer is read exactly once, so each 2 MiB span's XOR checksum equals
the host XOR of the same bytes (full spans, a ragged last span, and a buffer
smaller than one span)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2609_13544_amd as P

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes", [16, 4096, (2 << 20) - 16, (5 << 20) + 48, 3 * (2 << 20)])
def test_stream_read_checksum(nbytes):
    print(f"stream_read {nbytes} bytes", flush=True)
    rng = np.random.default_rng(nbytes)
    host = rng.integers(0, 2 ** 32, size=nbytes // 4, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    nspan = -(-nbytes // P.STREAM_SPAN)
    sink = torch.zeros(nspan, dtype=torch.int32, device="cuda")
    P.stream_read(buf, sink)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    words = P.STREAM_SPAN // 4
    want = [int(np.bitwise_xor.reduce(host[k * words:(k + 1) * words])) for k in range(nspan)]
    assert [int(x) for x in got] == want
