"""CPU tests: the fp64 oracle against its pins (closed forms, identities,
finite differences, special cases, an independent autograd route)."""
import numpy as np
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_bf16_inputs_upcast_exactly(orc):
    """The oracle consumes exact fp64 upcasts of the bf16 bytes the GPU reads."""
    import torch

    from workloads import lora_inputs

    inp = lora_inputs(5, 16, 8, 2, seed=3)
    X64 = inp["x"].to(torch.float64).numpy()
    # bf16 has 8 significant bits: every value is exactly representable and
    # survives a float32 round trip unchanged.
    assert np.array_equal(X64, X64.astype(np.float32).astype(np.float64))
    U = orc.u(inp["x"], inp["A"])
    assert np.allclose(U, X64 @ inp["A"].to(torch.float64).numpy().T, rtol=0, atol=1e-12)


def test_threads_reported(orc):
    assert orc.threads() >= 1
