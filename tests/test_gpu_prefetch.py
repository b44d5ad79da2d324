"""GPU tests of the cross-layer weight prefetcher (Sec. 4.3, App. E): every tensor a
consumer sees through a reused slot is the host tensor bit for bit, with a consumer
slow enough that a missing dependency would let the next copy overwrite the slot
first; misuse is refused on the host."""
import numpy as np
import pytest

import paper_2509_18344_amd as ss

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


class _DevView:
    """A device address seen as a torch tensor (no copy)."""

    def __init__(self, ptr, n):
        self.__cuda_array_interface__ = {"shape": (n,), "typestr": "|u1", "data": (ptr, False), "version": 2}


def _view(ptr, n):
    return torch.as_tensor(_DevView(ptr, n), device="cuda")


@pytest.mark.parametrize("slots", [2, 3])
def test_prefetch_ring_delivers_every_tensor_intact(slots):
    rng = np.random.default_rng(slots)
    slot_bytes = 4 << 20
    sizes = [int(s) for s in rng.integers(1, slot_bytes + 1, 12)]
    sizes[3] = slot_bytes
    host = [torch.from_numpy(rng.integers(0, 256, n, dtype=np.uint8)).pin_memory() for n in sizes]
    out = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in sizes]
    a = torch.randn(2048, 2048, device="cuda")
    pf = ss.Prefetcher(slot_bytes, slots)
    comp = torch.cuda.Stream()
    tickets = [pf.begin(host[i]) for i in range(slots - 1)]
    with torch.cuda.stream(comp):
        for i in range(len(sizes)):
            ptr = pf.acquire(tickets[i], comp)
            for _ in range(4):  # a slow consumer before the slot is read
                a = (a @ a).clamp_(-1, 1)
            out[i].copy_(_view(ptr, sizes[i]))
            pf.release(tickets[i], comp)
            if i + slots - 1 < len(sizes):
                tickets.append(pf.begin(host[i + slots - 1]))
    torch.cuda.synchronize()
    pf.close()
    for i in range(len(sizes)):
        assert torch.equal(out[i].cpu(), host[i]), i


def test_prefetch_refuses_misuse():
    pf = ss.Prefetcher(1 << 20, 2)
    h = [torch.zeros(1 << 20, dtype=torch.uint8).pin_memory() for _ in range(3)]
    t0 = pf.begin(h[0])
    t1 = pf.begin(h[1])
    with pytest.raises(ss.SubspecError, match="still holds"):
        pf.begin(h[2])  # slot of ticket 2 still holds ticket 0
    s = torch.cuda.current_stream()
    pf.acquire(t0, s)
    pf.release(t0, s)
    with pytest.raises(ss.SubspecError, match="released"):
        pf.acquire(t0, s)
    with pytest.raises(ss.SubspecError, match="not begun"):
        pf.acquire(7, s)
    t2 = pf.begin(h[2])
    assert (t0, t1, t2) == (0, 1, 2)
    with pytest.raises(ss.SubspecError, match="pinned"):
        pf.begin(np.zeros(16, np.uint8), 16)  # pageable host memory
    with pytest.raises(ss.SubspecError, match="do not fit"):
        pf.begin(torch.zeros(2 << 20, dtype=torch.uint8).pin_memory())
    for t in (t1, t2):
        pf.acquire(t, s)
        pf.release(t, s)
    torch.cuda.synchronize()
    pf.close()
