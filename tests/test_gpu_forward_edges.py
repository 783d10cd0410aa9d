"""GPU parity of the whole layer on routing and shape edge cases (every
weight format): a single expert with top_k = 1, routing skewed onto one
expert (many row tiles of one segment), sigmoid scores without
renormalisation, hundreds of experts, and top_k = E."""
import numpy as np
import pytest

import synth
from tests.gpu_util import check_forward, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


# fp8 output-level cases use I = 1024: see test_gpu_forward_quant for why the
# fp8 comparison needs I of the workload's order (its intermediate codes are
# pinned there at small I).
def _I(wcfg):
    return 1024 if wcfg in (4, 9) else 256


@pytest.mark.parametrize("wcfg", [1, 4, 5, 7, 9])
@pytest.mark.parametrize("T", [3, 700])
def test_single_expert_top1(dev, wcfg, T):
    # E = 1, k = 1: every token through the one expert with weight 1 (x2.5 in
    # sigmoid mode); T = 3 takes the small-batch kernels, T = 700 the tiled ones
    check_forward(synth.tiny_config(wcfg, T=T, E=1, top_k=1, I=_I(wcfg), logit_bias="none", sel_bias_std=0.0))


@pytest.mark.parametrize("wcfg", [1, 4, 5, 7, 9])
def test_skew_onto_one_expert(dev, wcfg):
    # a steep Zipf bias sends most rows to one expert: one segment spans more
    # row tiles than the scheduler groups together
    cfg = synth.tiny_config(wcfg, T=1500, E=8, top_k=2, I=_I(wcfg), logit_bias="zipf:6.0", sel_bias_std=0.0)
    out, ref, L = check_forward(cfg)
    counts = np.bincount(ref["ids"].ravel(), minlength=cfg.E)
    assert counts.max() > 10 * L["block_m"]


def test_sigmoid_without_renormalisation(dev):
    check_forward(synth.tiny_config(1, T=300, E=12, top_k=3, mode="sigmoid", renormalize=False,
                                    routed_scale=2.5, sel_bias_std=0.2))


def test_softmax_full_probabilities_scaled(dev):
    check_forward(synth.tiny_config(1, T=250, E=10, top_k=4, renormalize=False, routed_scale=1.7))


def test_hundreds_of_experts(dev):
    # E = 300: the permute runs several chunks; most experts get a few rows
    check_forward(synth.tiny_config(1, T=600, E=300, top_k=4, H=256, I=128))


def test_top_k_equals_e(dev):
    check_forward(synth.tiny_config(1, T=120, E=6, top_k=6))


@pytest.mark.parametrize("k", [12, 32])
def test_many_routed_rows_per_token(dev, k):
    # more than eight routed rows per token: the weighted sum takes the
    # slots eight at a time, in slot order
    check_forward(synth.tiny_config(1, T=90, E=48, top_k=k, H=256, I=128))


@pytest.mark.parametrize("wcfg", [1, 5, 7])
@pytest.mark.parametrize("T", [20, 2000])
def test_max_experts_and_top_k(dev, wcfg, T):
    # the ABI's limits E = 1024 and top_k = 32 (bf16, int4, MXFP4); T = 20
    # takes the decode kernels where the format has them, T = 2000 (64000
    # routed rows) the tiled ones
    check_forward(synth.tiny_config(wcfg, T=T, E=1024, top_k=32, H=256, I=128))


@pytest.mark.parametrize("wcfg", [1, 5])
@pytest.mark.parametrize("T", [8, 200])
def test_max_hidden_size(dev, wcfg, T):
    # H = 65536, the ABI's limit: 512 (bf16 tiled) to 1024 K steps of GEMM1
    check_forward(synth.tiny_config(wcfg, T=T, E=4, top_k=2, H=65536, I=256))
