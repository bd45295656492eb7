"""GPU: the benchmark's streaming copy helper (trivance_copy_device) copies exactly, also when
its grid is issued as many dispatches, and writes nothing past the destination range."""

import sys

import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


class _Limit:
    def __init__(self, items):
        self.items = items

    def __enter__(self):
        import paper_2602_17254_amd as T

        self.prev = T.trivance_set_dispatch_limit(self.items) if self.items else None

    def __exit__(self, *exc):
        import paper_2602_17254_amd as T

        if self.prev is not None:
            T.trivance_set_dispatch_limit(self.prev)


@pytest.mark.parametrize("limit", [None, 1024])
@pytest.mark.parametrize("nbytes", [16, 1024 + 16, 64 * 1024 * 16 + 48, 1 << 26])
def test_copy_helper_copies_exactly(nbytes, limit):
    import paper_2602_17254_amd as T

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    print(f"[copy] bytes={nbytes} limit={limit}", flush=True)
    sys.stdout.flush()
    n = nbytes // 4
    g = torch.Generator(device="cuda")
    g.manual_seed(nbytes)
    src = torch.randint(-(2 ** 31), 2 ** 31 - 1, (n,), dtype=torch.int32, device="cuda", generator=g)
    dst_full = torch.zeros(n + 64, dtype=torch.int32, device="cuda")
    dst = dst_full[:n]
    with _Limit(limit):
        T.trivance_copy_device(dst, src)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    assert int(dst_full[n:].abs().sum()) == 0


def test_copy_helper_rejects_mismatched_tensors():
    import paper_2602_17254_amd as T

    a = torch.zeros(64, dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):
        T.trivance_copy_device(a, torch.zeros(60, dtype=torch.float32, device="cuda"))
    with pytest.raises(T.TrivanceError):
        T.trivance_copy_device(a[:6], a[8:14])  # 24 bytes: not a multiple of 16
