"""Pins of the oracle's MoE Gate and permute steps: hand-worked closed forms,
brute-force selection loops, crafted ties and invariants."""
import math

import numpy as np
import pytest

import synth
from oracle import moe_oracle as O

E1 = math.e


def test_softmax_worked_example_ties_and_renorm():
    lg = np.array([[0.0, 1.0, 2.0, 3.0, 2.0]], dtype=np.float32)
    ids, w = O.gate(lg, None, 2, "softmax", True, 1.0)
    assert ids.tolist() == [[3, 2]]                         # tie 2 vs 4 -> index 2
    assert np.allclose(w, [[E1 / (1 + E1), 1 / (1 + E1)]], rtol=0, atol=1e-15)
    ids, w = O.gate(lg, None, 3, "softmax", True, 1.0)
    assert ids.tolist() == [[3, 2, 4]]
    assert np.allclose(w, [[E1 / (E1 + 2), 1 / (E1 + 2), 1 / (E1 + 2)]], rtol=0, atol=1e-15)
    # full softmax (no renormalisation): p_e = exp(l_e) / sum exp(l)
    ids, w = O.gate(lg, None, 2, "softmax", False, 1.0)
    z = 1 + E1 + 2 * E1 ** 2 + E1 ** 3
    assert np.allclose(w, [[E1 ** 3 / z, E1 ** 2 / z]], rtol=0, atol=1e-15)


def test_sigmoid_worked_example_bias_selects_only():
    lg = np.array([[0.0, 0.0, 2.0, -1.0]], dtype=np.float32)
    b = np.array([0.5, 0.0, 0.0, 1.0], dtype=np.float32)
    # keys: 1.0, 0.5, sigmoid(2)=0.881, sigmoid(-1)+1=1.269 -> experts 3, 0
    ids, w = O.gate(lg, b, 2, "sigmoid", True, 2.5)
    assert ids.tolist() == [[3, 0]]
    s3 = 1 / (1 + E1)                                       # sigmoid(-1), unbiased
    assert np.allclose(w, [[2.5 * s3 / (s3 + 0.5), 2.5 * 0.5 / (s3 + 0.5)]], rtol=0, atol=1e-15)
    ids, w = O.gate(lg, b, 2, "sigmoid", False, 1.0)
    assert np.allclose(w, [[s3, 0.5]], rtol=0, atol=1e-15)


def _brute_topk(key_row, k):
    """Selection by repeated scan: largest key, lowest index on ties."""
    chosen = []
    for _ in range(k):
        best = None
        for e, v in enumerate(key_row):
            if e in chosen:
                continue
            if best is None or v > key_row[best]:
                best = e
        chosen.append(best)
    return chosen


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_gate_ids_vs_brute_force(n):
    cfg = synth.config(n)
    if cfg.T * cfg.E > 300000:
        cfg = synth.tiny_config(n, T=600, E=cfg.E)
    r = synth.make_routing_inputs(cfg)
    ids, w = O.gate(r["logits"], r["sel_bias"], cfg.top_k, cfg.mode, cfg.renormalize, cfg.routed_scale)
    lg = r["logits"].astype(np.float64)
    b = np.zeros(cfg.E) if r["sel_bias"] is None else r["sel_bias"].astype(np.float64)
    key = lg + b if cfg.mode == "softmax" else 1 / (1 + np.exp(-lg)) + b
    for t in range(0, cfg.T, max(1, cfg.T // 64)):
        assert ids[t].tolist() == _brute_topk(key[t].tolist(), cfg.top_k)
    # invariants: weights sum to routed_scale, positive, distinct ids
    assert np.allclose(w.sum(1), cfg.routed_scale, rtol=0, atol=1e-12)
    assert np.all(w > 0)
    assert all(len(set(row)) == cfg.top_k for row in ids.tolist())


def test_gate_masked_experts_vs_brute_force():
    # -inf keys (masked experts): a row with fewer than k finite keys takes
    # its remaining experts among the masked ones by lowest index, as the
    # repeated scan does; masked experts get weight 0
    rng = np.random.default_rng(11)
    lg = rng.standard_normal((300, 40)).astype(np.float32)
    keep = np.argsort(rng.random((300, 40)), axis=1) < rng.integers(1, 9, size=300)[:, None]
    lg[~keep] = -np.inf
    ids, w = O.gate(lg, None, 6, "softmax", True, 1.0)
    for t in range(300):
        assert ids[t].tolist() == _brute_topk(lg[t].tolist(), 6)
    assert np.allclose(w.sum(1), 1.0, rtol=0, atol=1e-12)
    assert np.all((w == 0) == ~np.take_along_axis(keep, ids, axis=1))
    b = np.where(keep[0], 0.0, -np.inf).astype(np.float32)
    lg = rng.standard_normal((300, 40)).astype(np.float32)
    ids, w = O.gate(lg, b, 6, "sigmoid", True, 2.5)
    assert np.allclose(w.sum(1), 2.5, rtol=0, atol=1e-12)
    key = 1 / (1 + np.exp(-lg.astype(np.float64))) + b
    for t in range(300):
        assert ids[t].tolist() == _brute_topk(key[t].tolist(), 6)


def test_gate_crafted_integer_ties():
    rng = np.random.default_rng(3)
    lg = rng.integers(-2, 3, (500, 16)).astype(np.float32)   # many exact ties
    ids, _ = O.gate(lg, None, 5, "softmax", True, 1.0)
    for t in range(500):
        assert ids[t].tolist() == _brute_topk(lg[t].tolist(), 5)
    # all-equal row: ids are 0..k-1 in order, weights uniform
    ids, w = O.gate(np.zeros((1, 16), np.float32), None, 4, "softmax", True, 1.0)
    assert ids.tolist() == [[0, 1, 2, 3]] and np.allclose(w, 0.25, rtol=0, atol=1e-15)
    ids, w = O.gate(np.zeros((1, 16), np.float32), np.zeros(16, np.float32), 4, "sigmoid", True, 2.5)
    assert ids.tolist() == [[0, 1, 2, 3]] and np.allclose(w, 0.625, rtol=0, atol=1e-15)


def test_gate_single_expert_weight_is_one():
    lg = np.random.default_rng(4).standard_normal((9, 1)).astype(np.float32)
    ids, w = O.gate(lg, None, 1, "softmax", True, 1.0)
    assert np.all(ids == 0) and np.all(w == 1.0)


def _brute_permute(flat, E, block_m):
    n = len(flat)
    offsets, sorted_ids, inv = [0], [], [None] * n
    for e in range(E):
        seg = [f for f in range(n) if flat[f] == e]
        for f in seg:
            inv[f] = len(sorted_ids)
            sorted_ids.append(f)
        while len(sorted_ids) % block_m:
            sorted_ids.append(n)
        offsets.append(len(sorted_ids))
    cap = n + E * (block_m - 1)
    sorted_ids += [n] * (cap - len(sorted_ids))
    return offsets, sorted_ids, inv


@pytest.mark.parametrize("block_m", [1, 4, 16, 64])
@pytest.mark.parametrize("n", [1, 2, 5])
def test_permute_vs_brute_force(n, block_m):
    cfg = synth.config(n)
    cfg = synth.tiny_config(n, T=min(cfg.T, 97), E=cfg.E, top_k=cfg.top_k)
    r = synth.make_routing_inputs(cfg)
    ids, _ = O.gate(r["logits"], r["sel_bias"], cfg.top_k, cfg.mode)
    off, sid, inv = O.permute(ids, cfg.E, block_m)
    b_off, b_sid, b_inv = _brute_permute(ids.reshape(-1).tolist(), cfg.E, block_m)
    assert off.tolist() == b_off and sid.tolist() == b_sid and inv.tolist() == b_inv


def test_permute_invariants_large():
    cfg = synth.config(4)
    r = synth.make_routing_inputs(synth.tiny_config(4, T=4096, E=256, top_k=8))
    ids, _ = O.gate(r["logits"], r["sel_bias"], 8, "sigmoid")
    for bm in (1, 128):
        off, sid, inv = O.permute(ids, 256, bm)
        n = ids.size
        assert np.all(np.diff(off) >= 0) and np.all(off % bm == 0)
        real = sid[sid < n]
        assert np.array_equal(np.sort(real), np.arange(n))
        assert np.array_equal(sid[inv], np.arange(n))
        assert len(sid) == O.permute_capacity(4096, 8, 256, bm)
        flat = ids.reshape(-1)
        for e in (0, 17, 255):
            seg = sid[off[e]:off[e + 1]]
            seg = seg[seg < n]
            assert np.all(flat[seg] == e) and np.all(np.diff(seg) > 0)
    del cfg


def test_permute_degenerate():
    off, sid, inv = O.permute(np.zeros((0, 2), np.int32), 4, 16)
    assert off.tolist() == [0] * 5 and sid.tolist() == [0] * (4 * 15) and inv.size == 0
    ids = np.full((10, 1), 3, np.int32)                     # every token -> one expert
    off, sid, inv = O.permute(ids, 4, 8)
    assert off.tolist() == [0, 0, 0, 0, 16] and sid[:10].tolist() == list(range(10))
    assert sid[10:16].tolist() == [10] * 6
