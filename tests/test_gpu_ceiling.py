"""The device-ceiling measurements (reporting only, not part of the method):
the copy stream moves the bytes it claims to, and both report plausible
rates (positive, below physical limits of the part)."""
import pytest
import torch

from paper_2606_04484_amd import capi

pytestmark = pytest.mark.gpu


def test_copy_ceiling_copies_and_reports_rates():
    n = 32 << 20                                    # bytes; halves of 16 MiB
    buf = torch.empty(n, dtype=torch.uint8, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(7)
    buf[: n // 2] = torch.randint(0, 256, (n // 2,), dtype=torch.uint8, device="cuda", generator=g)
    src = buf[: n // 2].clone()
    copy, read = capi.aj_ceiling_copy(buf)
    torch.cuda.synchronize()
    # the copy runs first, then the read-only stream; the read stream stores
    # one word only when its fold hits a fixed constant, so compare all but
    # the first 16 bytes of the destination
    assert torch.equal(buf[: n // 2], src)
    assert torch.equal(buf[n // 2 + 16:], src[16:])
    assert 10.0 < copy < 20000.0 and 10.0 < read < 20000.0     # GB/s


def test_mfma_ceiling_rates():
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.empty(2 * cus * 256, dtype=torch.float32, device="cuda")
    rnd = capi.aj_ceiling_mfma_bf16(True, out)
    const = capi.aj_ceiling_mfma_bf16(False, out)
    assert torch.isfinite(out).all()
    assert 100.0 < rnd < 3500.0 and 100.0 < const < 3500.0   # TFLOP/s
    small = torch.empty(16, dtype=torch.float32, device="cuda")
    with pytest.raises(capi.AjError, match="out holds"):
        capi.aj_ceiling_mfma_bf16(True, small)
