"""The fp64 oracle pinned against the paper's printed sizes, library routines,
closed forms and invariants (CPU only)."""
import pytest

from oracle_checks import ALL_CHECKS


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_pin(orc, check):
    check(orc)


def test_fp16_rounding_is_ieee_rne():
    # the fp16 path's inputs are torch .half() of the fp32 draws: IEEE
    # round-to-nearest-even, which numpy's float16 cast also implements
    import numpy as np
    import torch
    x = torch.rand(1 << 16, generator=torch.Generator().manual_seed(0)) * 8 - 4
    assert np.array_equal(x.half().numpy(), x.numpy().astype(np.float16))
    # halfway case rounds to even: 1 + 2^-11 -> 1.0, 1 + 3*2^-11 -> 1 + 2^-9
    assert torch.tensor([1 + 2 ** -11]).half().item() == 1.0
    assert torch.tensor([1 + 3 * 2 ** -11]).half().item() == 1 + 2 ** -9
