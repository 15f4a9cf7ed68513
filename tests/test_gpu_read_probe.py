"""td_read_probe (measurement only): every word of the buffer is read exactly once by both
methods, whatever the WG count and the buffer's ragged tail (the XOR of the WGs' sink
words equals the XOR of the buffer, computed on the host)."""
import numpy as np
import pytest

import paper_2502_00085_amd.binding as B
from gpu_harness import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, 16384 * 8 + 16, 3 * (1 << 20) + 48])
@pytest.mark.parametrize("method", [0, 1])
@pytest.mark.parametrize("wgs", [1, 3, 256, 1000])
def test_read_probe_reads_every_word_once(nbytes, method, wgs):
    import torch
    log(f"read probe: {nbytes} B, method {method}, {wgs} WGs")
    rng = np.random.default_rng(nbytes * 7 + method * 3 + wgs)
    host = rng.integers(0, 2**32, nbytes // 4, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(wgs, dtype=torch.int32, device="cuda")
    B.td_read_probe(buf, method, wgs, sink)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(host)
    assert got == want, f"xor {got:#x} != {want:#x}"
