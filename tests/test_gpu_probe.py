"""The streaming-bandwidth probe moves exactly the bytes its header states.

ptstore_bandwidth_probe measures the practical HBM ceiling the copies are
compared with. It is not a store operation, but what it moves must be what
the header says: kind 2 copies `bytes` from a to b, kind 1 writes 16-byte
vectors (1, 2, 3, 4) over `bytes` of b, kind 0 only reads a and leaves b
(its sink) as it was, and nothing past `bytes` is touched. Sizes that are not
whole 16-byte vectors, misaligned buffers and unknown kinds are refused on
the host before any launch.
"""
from __future__ import annotations

import pytest
import torch

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2607_22648_amd import ptstore as P

    DEV = torch.device("cuda:0")

TAIL = 64  # bytes after `bytes` that must keep their fill


@pytest.mark.parametrize("nbytes", [16, 32768 - 16, 32768, 3 * 32768 + 48, 1 << 22])
def test_probe_kinds_move_what_they_state(nbytes):
    g = torch.Generator(device=DEV)
    g.manual_seed(nbytes)
    a = torch.randint(0, 256, (nbytes + TAIL,), dtype=torch.uint8, device=DEV, generator=g)
    a_before = a.clone()
    b = torch.full((nbytes + TAIL,), 0x5A, dtype=torch.uint8, device=DEV)
    P.ptstore_bandwidth_probe(2, a, b, nbytes)  # copy
    torch.cuda.synchronize()
    assert torch.equal(b[:nbytes], a[:nbytes])
    assert bool((b[nbytes:] == 0x5A).all())
    b.fill_(0x5A)
    P.ptstore_bandwidth_probe(1, a, b, nbytes)  # write
    torch.cuda.synchronize()
    vec = torch.tensor([1, 2, 3, 4], dtype=torch.int32, device=DEV).view(torch.uint8)
    assert torch.equal(b[:nbytes].view(-1, 16), vec.expand(nbytes // 16, 16))
    assert bool((b[nbytes:] == 0x5A).all())
    b.fill_(0x5A)
    P.ptstore_bandwidth_probe(0, a, b, nbytes)  # read
    torch.cuda.synchronize()
    assert bool((b == 0x5A).all())
    assert torch.equal(a, a_before)


def test_probe_refuses_bad_arguments():
    a = torch.zeros(4096, dtype=torch.uint8, device=DEV)
    b = torch.zeros(4096, dtype=torch.uint8, device=DEV)
    for kind, x, y, n in [(3, a, b, 1024), (-1, a, b, 1024), (2, a, b, 8), (2, a, b, 1000),
                          (2, a[1:], b, 1024), (2, a, b[8:], 1024), (0, a, b, (32 << 30) + 16)]:
        with pytest.raises(P.PTStoreError) as ei:
            P.ptstore_bandwidth_probe(kind, x, y, n)
        assert ei.value.code == P.PTSTORE_ERR_INVALID, (kind, n)
    torch.cuda.synchronize()
    assert bool((b == 0).all())
