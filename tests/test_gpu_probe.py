"""The read-bandwidth probe (ss_probe_read) on the GPU: each workgroup's
sink word is the XOR of its slice's 32-bit words, computed here on the CPU
from the same bytes (slices of ceil(bytes / 16 / workgroups) * 16 bytes,
trailing ones possibly empty)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2609_33184_amd import specstream as ss

pytestmark = pytest.mark.gpu


def _expected(words: np.ndarray, nbytes: int, groups: int) -> np.ndarray:
    share = (nbytes // 16 + groups - 1) // groups * 16
    out = np.zeros(groups, dtype=np.uint32)
    for g in range(groups):
        a, b = min(nbytes, g * share) // 4, min(nbytes, (g + 1) * share) // 4
        if b > a:
            out[g] = np.bitwise_xor.reduce(words[a:b])
    return out


@pytest.mark.parametrize("nbytes,groups", [(16, 1), (4096 * 3 + 48, 1), (3 * 1048576 + 4144, 7),
                                           (3 * 1048576 + 4144, 256), (1048576 + 16, 5000), (64 << 20, 1024)])
def test_probe_folds_every_slice(nbytes, groups):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    print(f"read probe: {nbytes} bytes, {groups} workgroups", flush=True)
    g = torch.Generator().manual_seed(nbytes ^ groups)
    host = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), dtype=torch.int32, generator=g)
    buf = host.to("cuda")
    sink = torch.full((groups,), -1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.Stream()
    ss.ss_probe_read(buf.data_ptr(), nbytes, sink.data_ptr(), groups, stream.cuda_stream)
    stream.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    want = _expected(host.numpy().view(np.uint32), nbytes, groups)
    assert np.array_equal(got, want)
