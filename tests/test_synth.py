"""The seeded input generator: determinism, substream independence and the
storage formats' shapes and value recipe."""
import numpy as np
import torch

import synth
from synth import moe_inputs as S


def test_deterministic_and_subset_independent():
    cfg = synth.tiny_config(5)
    a = synth.make_inputs(cfg, threads=1)
    b = synth.make_inputs(cfg, threads=4)
    for k in a:
        if a[k] is not None:
            assert np.array_equal(a[k], b[k]), k
    sub = synth.make_expert_weights(cfg, experts=[7, 2])
    assert np.array_equal(sub["w1"][0], a["w1"][7]) and np.array_equal(sub["w2_scale"][1], a["w2_scale"][2])


def test_shapes_per_format():
    for n in (1, 4, 5):
        cfg = synth.tiny_config(n)
        x = synth.make_inputs(cfg)
        E, H, I, T = cfg.E, cfg.H, cfg.I, cfg.T
        assert x["hidden"].shape == (T, H) and x["hidden"].dtype == np.uint16
        assert x["logits"].shape == (T, E) and x["logits"].dtype == np.float32
        if cfg.wfmt == "bf16":
            assert x["w1"].shape == (E, 2 * I, H) and x["w1"].dtype == np.uint16 and x["w1_scale"] is None
        if cfg.wfmt == "fp8":
            assert x["w1"].shape == (E, 2 * I, H) and x["w1"].dtype == np.uint8
            assert x["w1_scale"].shape == (E, 2 * I // 128, H // 128) and x["w2_scale"].shape == (E, H // 128, I // 128)
            assert x["sel_bias"].shape == (E,)
        if cfg.wfmt == "int4":
            assert x["w1"].shape == (E, 2 * I, H // 8) and x["w1"].dtype == np.int32
            assert x["w1_scale"].shape == (E, 2 * I, H // 128) and x["w1_scale"].dtype == np.uint16


def test_value_recipe_statistics():
    cfg = synth.tiny_config(1, T=256, H=1024, I=512, E=4)
    x = synth.make_inputs(cfg)
    h = torch.from_numpy(x["hidden"].view(np.int16)).view(torch.bfloat16).float().numpy()
    assert abs(h.std() - 1) < 0.02 and abs(h.mean()) < 0.02
    w1 = torch.from_numpy(x["w1"].view(np.int16)).view(torch.bfloat16).float().numpy()
    w2 = torch.from_numpy(x["w2"].view(np.int16)).view(torch.bfloat16).float().numpy()
    assert abs(w1.var() * cfg.H - 1) < 0.02 and abs(w2.var() * cfg.I - 1) < 0.02


def test_skewed_routing_bias():
    r = synth.make_routing_inputs(synth.config(5))
    # Zipf bias: expert with rank 1 has bias 0, rank E has -1.1*ln(E)
    b = r["logits"].mean(0)
    assert b.max() > -0.5 and b.min() < -1.1 * np.log(128) + 0.5
    cfg3 = synth.config(3)
    assert synth.make_routing_inputs(cfg3)["logits"].shape == (cfg3.T, cfg3.E)
    assert S.CONFIGS[4].sel_bias_std == 0.1
