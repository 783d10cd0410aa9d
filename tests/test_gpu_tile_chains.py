"""Whole-layer parity where every workgroup of the tiled GEMMs runs several
tiles in a row, so the copy pipeline crosses tile boundaries.  The second
product has more tiles than workgroups here (at least 17 row tiles x 16
column tiles), and its number of K steps per tile sits on either side of
the point where the next tile's first steps stop being issued together
with the current tile's last step and start being issued in stride: 5
steps (issued together) and 6 steps (in stride) with three stages, and a
four-stage kernel (MXFP8 activations, 128-element steps) with 9 steps."""
import pytest

import synth
from tests.gpu_util import check_forward, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


@pytest.mark.parametrize("I", [320, 384])     # bf16 second product: 5 and 6 K steps of 64
def test_bf16_chained_tiles(dev, I):
    check_forward(synth.tiny_config(3, T=600, H=4096, E=8, I=I, top_k=4))


def test_mxfp8_four_stage_chained_tiles(dev):
    # I = 1152 is a multiple of 128 but not of 256: the second product takes
    # 128-element steps on the four-stage kernel, 9 per tile
    check_forward(synth.tiny_config(9, T=600, H=4096, E=16, I=1152, top_k=4))
