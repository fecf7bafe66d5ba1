"""The device number encoders against their integer definitions, over every fp32 bit pattern.

The compress kernels encode FP8 E4M3 coefficients (Section 3's quantised shared and residual
coefficients) with the gfx950 conversion instruction on inputs clamped to +-448, and every
device-side bf16 rounding uses the bf16 pair conversion; fdkv_check_conversions runs both over
all 2^32 fp32 bit patterns except NaN against round to nearest even written in integer
arithmetic (fp8.h's f32_to_e4m3, which the host tests pin to the enumerated E4M3 grid, and the
bit-pattern rounding of fdkv_common.h).
"""
import pytest

from paper_2607_06519_amd import binding as B

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    B.load()
    return torch


def test_device_encoders_equal_their_integer_definitions(torch_dev):
    print("[case] fdkv_check_conversions over all fp32 bit patterns", flush=True)
    e4m3, bf16 = B.check_conversions()
    print(f"  mismatches: E4M3 {e4m3}, bf16 {bf16}", flush=True)
    assert e4m3 == 0 and bf16 == 0
