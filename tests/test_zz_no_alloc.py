"""The entry point that allocates nothing (sdsat_linear_noalloc) against the
one that takes a scratch buffer (sdsat_linear): identical outputs, bit for
bit, on two calls in a row, the second with a smaller input (so any value the
first call left in the shared static array would show), for both element
types; and its size limit is an error, not an overrun."""
import numpy as np
import pytest

from paper_2403_18647_amd import binding as B

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()


def _case(dtype, M, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(M, K, generator=g).cuda()
    w = (torch.randn(N, K, generator=g) * 0.05).to(torch.bfloat16 if dtype == 1 else torch.float32).cuda()
    packed = torch.empty(B.sdsat_linear_packed_bytes(dtype, N, K), dtype=torch.uint8, device="cuda")
    B.sdsat_linear_pack(dtype, N, K, w, packed)
    return x, packed


@pytest.mark.parametrize("dtype", [1, 0])
def test_noalloc_linear_matches_scratch_linear_twice(dtype):
    for M, N, K, seed in [(37, 1000, 4000, 1), (5, 272, 96, 2)]:      # second call smaller (M and K)
        print(f"noalloc dtype={dtype} M={M} N={N} K={K}", flush=True)
        x, packed = _case(dtype, M, N, K, seed)
        y_ref = torch.empty(M, N, device="cuda")
        scratch = torch.empty(B.sdsat_linear_scratch_bytes(M, N, K), dtype=torch.uint8, device="cuda")
        B.sdsat_linear(dtype, M, N, K, x, packed, y_ref, scratch)
        y = torch.full((M, N), float("nan"), device="cuda")
        B.sdsat_linear_noalloc(dtype, M, N, K, x, packed, y)
        torch.cuda.synchronize()
        assert torch.equal(y, y_ref)
        assert torch.isfinite(y).all()


def test_noalloc_linear_rejects_inputs_past_its_static_scratch():
    x = torch.zeros(64, 16416, device="cuda")            # 64 x 16416 x 4 bytes > 4 MiB
    packed = torch.zeros(B.sdsat_linear_packed_bytes(0, 16, 16416), dtype=torch.uint8, device="cuda")
    y = torch.zeros(64, 16, device="cuda")
    with pytest.raises(B.SdsatError) as e:
        B.sdsat_linear_noalloc(0, 64, 16, 16416, x, packed, y)
    assert e.value.code == -1
    assert b"4 MiB" in B.lib().sdsat_last_error(None)
    B.sdsat_linear_noalloc(0, 64, 16, 16384, x[:, :16384].contiguous(), packed, y)   # exactly 4 MiB fits
    torch.cuda.synchronize()
    assert torch.equal(y, torch.zeros_like(y))
