"""The streaming-read probe reads exactly the bytes it is asked for: its XOR checksum
equals the XOR of the same 32-bit words computed on the host, for a contiguous buffer and
for record prefixes with a stride."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("per,stride,n", [(4096, 4096, 1000), (1456, 3328, 777), (16, 48, 5), (4000, 4096, 3)])
def test_probe_checksum(per, stride, n):
    from paper_2503_18599_amd import binding as B
    g = torch.Generator().manual_seed(per + n)
    host = torch.randint(0, 256, ((n - 1) * stride + per + 64,), generator=g, dtype=torch.uint8)
    ck = B.probe_read(host.to("cuda"), per, stride, n)
    words = np.concatenate([host.numpy()[r * stride:r * stride + per] for r in range(n)]).view(np.uint32)
    want = np.bitwise_xor.reduce(words)
    assert int(ck.cpu().numpy().view(np.uint32)[0]) == int(want)
