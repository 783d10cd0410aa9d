"""GPU parity of the whole layer with bf16 experts against the fp64 oracle
(quantisation points mirrored): bit-exact routing and permutation, and
max|out - oracle| <= 2e-2 * rms(oracle out)."""
import numpy as np
import pytest

import synth
from tests.gpu_util import check_forward, require_gpu, run_forward

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _check(cfg, inp=None, out_dtype="f32"):
    return check_forward(cfg, inp, out_dtype)


def test_tiny_config_full_size(dev):
    _check(synth.config(1))


@pytest.mark.parametrize("T", [1, 7, 77, 300])
def test_small_shapes_skinny_and_tiled(dev, T):
    # E=4, k=2: T=300 gives 150 rows per expert (tiled kernels), small T the skinny ones
    _check(synth.tiny_config(1, T=T, H=384, I=256, E=4, top_k=2))


@pytest.mark.parametrize("T", [5, 400])
def test_minimum_k(dev, T):
    # H = I = 128: two K steps per tile, fewer than the pipeline has stages
    _check(synth.tiny_config(1, T=T, H=128, I=128, E=4, top_k=2))


@pytest.mark.parametrize("H,I", [(1024, 1024), (2048, 3072), (3072, 2048), (4096, 4096),
                                 (640, 1920), (1920, 640), (896, 1664), (1664, 896),
                                 (1152, 1536), (1536, 1152), (1280, 1792), (1792, 1280)])
def test_streamed_decode_kernel(dev, H, I):
    # decode-sized batches (<= 32 rows per expert on average) take the
    # streamed kernel in both products when K is a multiple of 1024 up to
    # 4096 (one to four 512-byte pieces per wave and row) or below 2048 (one
    # piece of K/2 bytes): every piece width from 320 to 960 bytes appears
    # here; T = 37 leaves ragged 16-row tiles, E = 9 an odd expert count
    _check(synth.tiny_config(2, T=37, H=H, I=I, E=9, top_k=3))


def test_many_experts_ragged(dev):
    _check(synth.tiny_config(1, T=201, H=512, I=384, E=40, top_k=5))


def test_bf16_output_format(dev):
    _check(synth.tiny_config(1, T=50), out_dtype="bf16")


def test_decode_config_full_size(dev):
    _check(synth.config(2))


def test_prefill_config_full_size(dev):
    _check(synth.config(3))


def test_run_twice_bit_identical(dev):
    cfg = synth.tiny_config(1, T=300, E=4, top_k=2)
    inp = synth.make_inputs(cfg)
    a, ws, _, _ = run_forward(cfg, inp)
    b, _, _, _ = run_forward(cfg, inp, workspace=ws)
    assert np.array_equal(a, b)


def test_token_order_permutes_output(dev):
    cfg = synth.tiny_config(1, T=120, E=8, top_k=3)
    inp = synth.make_inputs(cfg)
    perm = np.random.default_rng(1).permutation(cfg.T)
    a, _, _, _ = run_forward(cfg, inp)
    b, _, _, _ = run_forward(cfg, dict(inp, hidden=inp["hidden"][perm], logits=inp["logits"][perm]))
    assert np.array_equal(b, a[perm])


@pytest.mark.parametrize("H,I", [(392, 200), (4104, 1416), (8, 8), (136, 1032)])
@pytest.mark.parametrize("T", [5, 300])
def test_shapes_multiple_of_8(dev, H, I, T):
    # bf16 H and I multiples of 8 but not of 128: every batch runs the tiled
    # kernels with a ragged last K step (zero chunks past K) and a ragged last
    # column tile (masked stores); T = 5 would take the decode kernels at
    # 128-aligned shapes
    _check(synth.tiny_config(1, T=T, H=H, I=I, E=6, top_k=2))
