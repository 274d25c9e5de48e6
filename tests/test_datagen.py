"""The seeded input generators: published RNG test vector, slice determinism,
and the shape/structure of the synthetic workloads."""
import numpy as np
import torch

import datagen
from datagen import configs, inputs, rng


def test_splitmix64_published_sequence():
    # SplitMix64 seeded with 1234567 (test vector of the reference C implementation)
    got = rng.raw64(1234567, 5).numpy().view(np.uint64).tolist()
    assert got == [6457827717110365317, 3203168211198807973, 9817491932198370423,
                   4593380528125082431, 16408922859458223821]


def test_stream_slices_regenerate_exactly():
    key = rng.stream_key(7, 3, 1)
    full = rng.normal(key, 1000)
    part = rng.normal(key, 100, start=450)
    assert torch.equal(full[450:550], part)
    u = rng.uniform(key, 10000)
    assert float(u.min()) > 0.0 and float(u.max()) < 1.0
    assert abs(float(u.mean()) - 0.5) < 0.02


def test_normals_look_standard():
    z = rng.normal(rng.stream_key(1), 200000)
    assert abs(float(z.mean())) < 0.01
    assert abs(float(z.std()) - 1.0) < 0.01


def test_choice_without_replacement():
    c = rng.choice_without_replacement(rng.stream_key(5), 10, 50, 20)
    assert len(set(c.tolist())) == 20 and int(c.min()) >= 10 and int(c.max()) < 50
    assert (c[1:] > c[:-1]).all()


def test_budget_rule():
    assert configs.budget_k(8192, 1000) == 819
    assert configs.budget_k(32768, 500) == 1638
    assert configs.budget_k(16384, 1000) == 1638
    assert configs.budget_k(2048, 1000) == 204
    assert configs.budget_k(5, 1000) == 1          # at least one row
    assert configs.extras_count(32768, 200) == 655


def test_tiny_prefill_structure():
    cfg = datagen.get("tiny")
    pre = inputs.make_prefill(cfg)
    assert pre["q_win"].shape == (1, 1, 8, 32, 64) and pre["q_win"].dtype == torch.float32
    assert pre["k"].shape == (1, 8, 2048, 64)
    k = pre["k"].double()
    mu = pre["mu"]
    for h in range(8):
        u = mu[0, 0, h] / mu[0, 0, h].norm()
        pos = pre["heavy"][(0, 0, h)]
        assert len(pos) == 32 and int(pos.max()) < 2048 - 32
        proj = k[0, h] @ u
        np.testing.assert_allclose(proj[pos].numpy(), 4.0, atol=1e-5)   # planted +4 along u


def test_bf16_config_rounds_and_varlen():
    cfg = datagen.get("batched64").with_(B=3, L=2, varlen_lo=100, varlen_hi=300, W=8)
    lens = inputs.seqlens(cfg)
    assert len(lens) == 3 and all(100 <= n <= 300 for n in lens)
    pre = inputs.make_prefill(cfg)
    assert pre["k"].dtype == torch.bfloat16 and pre["k"].shape[0] == 1   # shared across layers
    q = inputs.decode_queries(cfg, 0, mu=pre["mu"])
    assert q.shape == (3, 2, 32, 128)


def test_extras_avoid_selection():
    cfg = datagen.get("llama8b_32k").with_(L=1, seqlens=(1000,), extra_bp=500)
    lens = [1000]
    b = inputs.make_budget(cfg, lens)
    sel = inputs.random_selection(cfg, lens, b["k"])
    ex = inputs.extras_for_step(cfg, 3, lens, sel[0], b["cu_k"], 0)
    assert len(ex) == cfg.Hkv
    for h in range(cfg.Hkv):
        s = set(sel[0, h].tolist())
        e = ex[h].tolist()
        assert len(e) == 50 and len(set(e)) == 50 and not (s & set(e))


def test_extras_layer_matches_per_unit_draws():
    cfg = datagen.get("batched64").with_(B=4, L=2, varlen_lo=300, varlen_hi=900, extra_bp=700)
    lens = inputs.seqlens(cfg)
    b = inputs.make_budget(cfg, lens)
    sel = inputs.random_selection(cfg, lens, b["k"])
    for layer in range(cfg.L):
        for step in (0, 5):
            ids, cu_e = inputs.extras_layer(cfg, step, lens, sel[layer], b["cu_k"], layer)
            ref = inputs.extras_for_step(cfg, step, lens, sel[layer], b["cu_k"], layer)
            for h in range(cfg.Hkv):
                for r in range(cfg.B):
                    got = ids[h, cu_e[r]:cu_e[r + 1]]
                    assert torch.equal(got.to(torch.int64), ref[h * cfg.B + r])


def test_extras_layers_matches_single_layer_calls():
    cfg = datagen.get("llama8b_32k").with_(L=3, seqlens=(700,), extra_bp=300)
    lens = [700]
    b = inputs.make_budget(cfg, lens)
    sel = inputs.random_selection(cfg, lens, b["k"])
    ids, cu_e = inputs.extras_layers(cfg, 2, lens, sel, b["cu_k"], [0, 1, 2])
    for layer in range(3):
        one, _ = inputs.extras_layer(cfg, 2, lens, sel[layer], b["cu_k"], layer)
        assert torch.equal(ids[layer], one)
        ref = inputs.extras_for_step(cfg, 2, lens, sel[layer], b["cu_k"], layer)
        for h in range(cfg.Hkv):
            assert torch.equal(ids[layer, h].to(torch.int64), ref[h])
