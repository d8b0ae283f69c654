"""Host checks of the autograd layers: padding arithmetic, argument validation, and that a CPU
tensor is refused (the layers have no CPU path)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2209_04161_amd import modules


@pytest.mark.parametrize("size,k,s,want", [
    (28, 5, 1, (2, 2)),    # LeNet-5 conv1 with SAME padding
    (224, 7, 2, (2, 3)),   # ResNet stem: TF pads 2 before, 3 after
    (14, 3, 1, (1, 1)),
    (14, 1, 1, (0, 0)),
    (7, 3, 2, (1, 1)),
    (8, 3, 2, (0, 1)),
])
def test_same_pads_follow_tf(size, k, s, want):
    assert modules.same_pads(size, k, s) == want
    before, after = want
    out = (size + before + after - k) // s + 1
    assert out == -(-size // s)  # SAME keeps ceil(size / stride) outputs


def test_layers_validate_their_table():
    lut = torch.zeros(1 << 14, dtype=torch.int32)
    with pytest.raises(ValueError):
        modules.AMLinear(4, 3, lut, 12)
    with pytest.raises(ValueError):
        modules.AMLinear(4, 3, lut[:100], 7)
    with pytest.raises(ValueError):
        modules.AMConv2d(1, 6, 5, lut.to(torch.float32), 7)
    layer = modules.AMConv2d(3, 8, (3, 5), lut, 7, stride=2, padding="same")
    assert tuple(layer.weight.shape) == (3, 5, 3, 8)
    assert layer.pads(224, 224) == modules.same_pads(224, 3, 2) + modules.same_pads(224, 5, 2)
    assert modules.AMConv2d(3, 8, 3, lut, 7, padding=(1, 2, 0, 1)).pads(9, 9) == (1, 2, 0, 1)


def test_cpu_tensors_are_refused():
    lut = torch.zeros(1 << 14, dtype=torch.int32)
    lin = modules.AMLinear(4, 3, lut, 7)
    with pytest.raises(ValueError):
        lin(torch.ones(2, 4))
    conv = modules.AMConv2d(1, 2, 3, lut, 7, padding="same")
    with pytest.raises(ValueError):
        conv(torch.ones(1, 5, 5, 1))
