"""Seeded input recipes: determinism, shapes, placement rules, work counters (CPU only)."""
import numpy as np

from paper_2609_39819_amd.workloads import (
    BLOCK_SIZE, algorithmic_flops, bf16_bits_to_f32, config_shapes, f32_to_bf16_bits, forked_lengths,
    kv_bytes, make_config)


def test_bf16_rounding_is_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, 1.0 + 2**-9, -2.5, np.inf, 3.0e38], dtype=np.float32)
    r = bf16_bits_to_f32(f32_to_bf16_bits(x))
    # 1+2^-8 is a tie between 1 and 1+2^-7 -> even (1.0); 1+3*2^-8 ties up to 1+2^-6
    assert r.tolist()[:5] == [1.0, 1.0, 1.0 + 2**-6, 1.0, -2.5]
    assert np.isinf(r[5]) and np.isfinite(r[6])
    assert np.isnan(bf16_bits_to_f32(f32_to_bf16_bits(np.array([np.nan], np.float32))))[0]


def test_tiny_config_matches_its_description():
    w = make_config("tiny")
    assert (w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype) == (4, 1, 64, "f32")
    assert w.prefix_len.tolist() == [240] and w.suffix_len.tolist() == [16]
    assert w.block_table.shape == (1, 16)
    # the 16 used ids are the first 16 of one seeded permutation of the 64-block pool
    perm = np.random.default_rng(1).permutation(64)
    assert w.block_table[0].tolist() == perm[:16].tolist()
    assert np.isnan(w.k_pool_c[w.compact_table[0, 15]]).all()     # suffix block empty before append
    assert np.isfinite(w.k_pool_c[w.compact_table[0, :15]]).all()
    assert abs(w.scale - 1 / 8) < 1e-15


def test_generation_is_deterministic():
    a, b = make_config("tiny"), make_config("tiny")
    for f in ("block_table", "k_pool_c", "v_pool_c", "k_new", "v_new", "q"):
        assert np.array_equal(getattr(a, f), getattr(b, f), equal_nan=True)


def test_gqa_8k_placement():
    w = make_config("gqa_8k")
    assert w.block_table.shape == (1, 544)
    ids = w.block_table[0]
    assert len(np.unique(ids)) == 544 and ids.min() >= 0 and ids.max() < 65536
    assert w.q.dtype == np.uint16 and w.q.shape == (512, 32, 128)
    assert w.k_new.shape == (512, 8, 128)


def test_forked_lengths_and_shared_blocks():
    c = config_shapes("forked_agents")
    rng = np.random.default_rng(c["seed"])
    P, S = forked_lengths(rng, 16, 4096, c["private_prefix"], c["suffix"])
    assert ((P >= 8192) & (P <= 4096 + 65536)).all()
    assert ((S >= 256) & (S <= 4096)).all()
    # structure on a scaled-down instance of the same recipe
    from paper_2609_39819_amd.workloads import build_workload
    w = build_workload(name="f", seed=4, prefix_len=[40, 70, 33], suffix_len=[5, 9, 30], num_q_heads=4,
                       num_kv_heads=2, head_dim=8, num_blocks=1000, shared_prefix_blocks=2)
    assert (w.block_table[:, :2] == w.block_table[0, :2]).all()
    rest = np.concatenate([w.block_table[b, 2:(w.prefix_len[b] + w.suffix_len[b] + 15) // 16] for b in range(3)])
    assert len(np.unique(np.concatenate([rest, w.block_table[0, :2]]))) == len(rest) + 2


def test_flop_and_byte_counters_match_hand_values():
    # (prefix, suffix, Hq, D) -> flops; hand values: 4*D*Hq*(S*P + S(S+1)/2)
    assert algorithmic_flops([240], [16], 4, 64) == 4_071_424
    assert algorithmic_flops([8192], [512], 32, 128) == 70_871_154_688
    assert algorithmic_flops([131072], [2048], 96, 128) == 13_297_269_080_064
    assert algorithmic_flops([204800], [57344], 96, 128) == 658_059_118_510_080
    assert algorithmic_flops([131072], [2048], 24, 128) == 3_324_317_270_016
    assert kv_bytes([240], [16], 1, 64, 4) == 131_072
    assert kv_bytes([8192], [512], 8, 128, 2) == 35_651_584
    assert kv_bytes([131072], [2048], 8, 128, 2) == 545_259_520
    assert kv_bytes([204800], [57344], 8, 128, 2) == 1_073_741_824


def test_block_size_is_sixteen():
    assert BLOCK_SIZE == 16


def test_tp4_shard_shape():
    """One GPU's share of the 128K turn under 4-way head parallelism: a quarter
    of the heads and of the work, same lengths."""
    from paper_2609_39819_amd.workloads import algorithmic_flops, config_shapes
    c, full = config_shapes("react_128k_tp4"), config_shapes("react_128k")
    assert (c["num_q_heads"], c["num_kv_heads"]) == (full["num_q_heads"] // 4, full["num_kv_heads"] // 4)
    assert (c["prefix"], c["suffix"]) == (full["prefix"], full["suffix"])
    f4 = algorithmic_flops([c["prefix"]], [c["suffix"]], c["num_q_heads"], c["head_dim"])
    f1 = algorithmic_flops([full["prefix"]], [full["suffix"]], full["num_q_heads"], full["head_dim"])
    # 4*D*Hq*(S*P + S(S+1)/2) = 4*128*96*(2048*131072 + 2048*2049/2)
    assert 4 * f4 == f1 == 49152 * 270533632
