"""GPU: the benchmark's streaming copy helper (trivance_copy_device) copies exactly, also when
its grid is larger than one dispatch holds, and writes nothing past the destination range."""

import sys

import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.mark.parametrize("nbytes", [16, 1024 + 16, 64 * 1024 * 16 + 48, 1 << 26])
def test_copy_helper_copies_exactly(nbytes):
    import paper_2602_17254_amd as T

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    print(f"[copy] bytes={nbytes}", flush=True)
    sys.stdout.flush()
    n = nbytes // 4
    g = torch.Generator(device="cuda")
    g.manual_seed(nbytes)
    src = torch.randint(-(2 ** 31), 2 ** 31 - 1, (n,), dtype=torch.int32, device="cuda", generator=g)
    dst_full = torch.zeros(n + 64, dtype=torch.int32, device="cuda")
    dst = dst_full[:n]
    T.trivance_copy_device(dst, src)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    assert int(dst_full[n:].abs().sum()) == 0


def test_copy_helper_above_32_bit_work_items():
    """A copy of 34 GiB: 2^31 + 2^27 sixteen-byte lanes, more work-items than one dispatch holds,
    so the grid goes out as two dispatches. Checked on both sides of the dispatch boundary and at
    seeded positions, plus the guard words after the destination."""
    import paper_2602_17254_amd as T

    lanes = (1 << 31) + (1 << 27)
    n = lanes * 4  # int32 elements
    print(f"[copy] bytes={lanes * 16} (two dispatches)", flush=True)
    torch.cuda.empty_cache()
    src = torch.empty(n, dtype=torch.int32, device="cuda")
    dst_full = torch.zeros(n + 64, dtype=torch.int32, device="cuda")
    try:
        dst = dst_full[:n]
        # a pattern that differs per element: the counter-based generator's values
        T.trivance_fill_hash_uniform(src.view(torch.float32).view(1, n), 123)
        T.trivance_copy_device(dst, src)
        torch.cuda.synchronize()
        edge = (1 << 31) * 4  # first element of the second dispatch
        idx = torch.cat([torch.arange(0, 4096), torch.arange(edge - 4096, edge + 4096),
                         torch.arange(n - 4096, n),
                         torch.randint(0, n, (1 << 20,), generator=torch.Generator().manual_seed(5))])
        idx = idx.to("cuda")
        assert torch.equal(dst[idx], src[idx])
        assert int(dst_full[n:].abs().sum()) == 0
        assert bool((dst[edge:edge + 4096] != 0).any())
    finally:
        del src, dst_full
        torch.cuda.empty_cache()


def test_copy_helper_rejects_mismatched_tensors():
    import paper_2602_17254_amd as T

    a = torch.zeros(64, dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):
        T.trivance_copy_device(a, torch.zeros(60, dtype=torch.float32, device="cuda"))
    with pytest.raises(T.TrivanceError):
        T.trivance_copy_device(a[:6], a[8:14])  # 24 bytes: not a multiple of 16
