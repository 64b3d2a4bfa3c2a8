"""The seeded input generator: reproducibility, slicing, distribution, skew."""
import numpy as np
import torch

from synth import BY_NAME, CONFIGS, gen, mini


def test_mix64_reference_values():
    # SplitMix64 with state 0: the first outputs of the published generator
    # (Steele, Lea & Flood 2014; also java.util.SplittableRandom)
    z = 0
    outs = []
    for _ in range(3):
        z = (z + gen.GAMMA) & gen.MASK64
        outs.append(gen.mix64_int(z))
    assert outs == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_numpy_stream_matches_scalar_definition():
    key = gen.stream_key(20260001, gen.KIND_GU, 3)
    tab = gen.normal_table()
    v = gen.normal_f32(key, 1000, 64, np.float32(0.02))
    for i in range(64):
        u = gen.mix64_int(key + (1000 + i + 1) * gen.GAMMA)
        assert v[i] == np.float32(tab[u >> 48]) * np.float32(0.02)


def test_slices_are_consistent():
    cfg = mini(BY_NAME["qwen_moe_bf16"])
    gate, up = gen.expert_gate_up(cfg, 1, 5)
    full = gen.tensor_values(cfg, gen.KIND_GU, 1, 0, (cfg.E + cfg.S) * 2 * cfg.F * cfg.H)
    full = full.reshape(cfg.E + cfg.S, 2 * cfg.F, cfg.H)
    assert np.array_equal(gate, full[5, :cfg.F]) and np.array_equal(up, full[5, cfg.F:])
    x = gen.x_all(cfg)
    assert np.array_equal(gen.x_rows(cfg, 3, 17, 5), x[3, 17:22])


def test_bf16_bits_match_torch():
    rng = np.random.default_rng(0)
    v = (rng.normal(size=10000) * 10.0 ** rng.uniform(-5, 5, size=10000)).astype(np.float32)
    ours = gen.bf16_bits_to_f32(gen.f32_to_bf16_bits(v))
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)


def test_normal_moments():
    v = gen.normal_f32(gen.stream_key(1, 1, 0), 0, 1 << 20, np.float32(1.0)).astype(np.float64)
    assert abs(v.mean()) < 5e-3 and abs(v.std() - 1.0) < 5e-3
    tab = gen.normal_table()
    assert np.all(np.diff(tab) > 0) and tab[0] == -tab[-1]


def test_router_bias_skew_models():
    for cfg in CONFIGS:
        b = gen.router_bias(cfg)
        assert b.shape == (cfg.L, cfg.E) and b.dtype == np.float32
        p = np.exp(b.astype(np.float64))
        assert np.allclose(p.sum(axis=1), 1.0, rtol=1e-5)
        if cfg.skew.startswith("zipf"):
            zipf = np.arange(1, cfg.E + 1) ** (-cfg.skew_param)
            zipf /= zipf.sum()
            assert np.allclose(np.sort(p, axis=1)[:, ::-1], zipf[None], rtol=1e-5)
    # drift: hot experts persist between consecutive layers
    cfg = BY_NAME["dsv3_share_bf16"]
    b = gen.router_bias(cfg)
    top = [set(np.argsort(-b[l])[:16]) for l in range(cfg.L)]
    assert all(len(top[l] & top[l + 1]) >= 8 for l in range(cfg.L - 1))


def test_config_shapes():
    for cfg in CONFIGS:
        assert cfg.E % cfg.D == 0 and cfg.H % 256 == 0 and cfg.F % 128 == 0
    assert [c.m for c in CONFIGS] == [1, 3, 6, 12, 6]


def test_compiled_host_generator_matches_numpy_definition():
    assert gen._host_lib() is not None, "synth/libsynthhost.so is not built"
    for kind, dt in [(gen.KIND_X, False), (gen.KIND_GU, True), (gen.KIND_WG, True)]:
        key = gen.stream_key(20260003, kind, 5)
        sig = gen.sigma_of(kind, 2048)
        ref = gen.normal_f32(key, 123456789, 300001, sig)
        if dt:
            ref = gen.bf16_bits_to_f32(gen.f32_to_bf16_bits(ref))
        assert np.array_equal(gen.normal_values(key, 123456789, 300001, sig, dt), ref)
