"""The seeded input generator: reproducible, random-access, bf16 rounding and value recipe."""
import numpy as np
import torch

import synth
from synth import inputs as I


def test_bf16_round_to_nearest_even_matches_torch():
    g = np.random.default_rng(0)
    a = np.concatenate([
        g.standard_normal(100000).astype(np.float32) * 10,
        np.array([0.0, -0.0, 1.0, 3.0e38, -1e-40, 1.00390625, 1.01171875, 65504.0], dtype=np.float32),
    ])
    ours = I.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    # widening is exact
    back = I.bf16_bits_to_f32(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(a).to(torch.bfloat16).float().numpy())


def test_reproducible_and_random_access():
    w = synth.get_workload("qwen", n_prompts=3, seq_len=300, d=128, V=700)
    X1 = I.hidden_rows(w, 7)
    X2 = I.hidden_rows(w, 7)
    np.testing.assert_array_equal(X1, X2)
    rows = np.array([899, 0, 257, 256, 255, 512])
    np.testing.assert_array_equal(I.hidden_rows(w, 7, rows=rows), X1[rows])
    W = I.lm_head_rows(w, 7)
    np.testing.assert_array_equal(I.lm_head_rows(w, 7, rows=np.array([699, 3])), W[[699, 3]])
    q = I.qk_layer(w, "q", 0, 7)
    np.testing.assert_array_equal(I.qk_layer(w, "q", 0, 7, rows=np.array([5, 600])), q[[5, 600]])
    assert not np.array_equal(I.hidden_rows(w, 8), X1)


def test_hidden_recipe_rms_and_outliers():
    w = synth.get_workload("llama", n_prompts=3, seq_len=200, d=256)
    X = I.bf16_bits_to_f32(I.hidden_rows(w, 42)).astype(np.float64)
    rms = np.sqrt((X ** 2).mean(axis=1))
    big = rms > 2.5
    # exactly round(0.05 * 200) = 10 outliers per prompt, each with RMS 4, others RMS 1 (bf16 rounding)
    assert [int(big[b * 200:(b + 1) * 200].sum()) for b in range(3)] == [10, 10, 10]
    np.testing.assert_allclose(rms[~big], 1.0, atol=5e-3)
    np.testing.assert_allclose(rms[big], 4.0, atol=2e-2)


def test_weight_and_qk_distributions():
    w = synth.get_workload("qwen", n_prompts=2, seq_len=512, d=256, V=4096)
    W = I.bf16_bits_to_f32(I.lm_head_rows(w, 1)).astype(np.float64)
    assert abs(W.std() - 0.02) < 5e-4 and abs(W.mean()) < 5e-4
    s = I.query_head_scales(w, 1)
    assert s.shape == (1, 12) and s.min() >= 0.5 and s.max() <= 2.0
    q = I.bf16_bits_to_f32(I.qk_layer(w, "q", 0, 1)).astype(np.float64)
    np.testing.assert_allclose(q.std(axis=(0, 2)), s[0], rtol=0.03)
    k = I.bf16_bits_to_f32(I.qk_layer(w, "k", 0, 1)).astype(np.float64)
    assert k.shape == (1024, 2, 128) and abs(k.std() - 1.0) < 0.02


def test_ragged_lengths():
    w = synth.get_workload("ragged")
    lens = I.prompt_lengths(w, 42)
    assert len(lens) == 256 and lens.min() >= 32 and lens.max() <= 4096
    # log-uniform: the median is near sqrt(32 * 4096) = 362
    assert 250 < np.median(lens) < 520
    cu = I.cu_seqlens_from_lengths(lens)
    assert cu.dtype == np.int32 and cu[0] == 0 and cu[-1] == lens.sum()
    np.testing.assert_array_equal(lens, I.prompt_lengths(w, 42))


def test_tiny_is_fp32():
    w = synth.get_workload("tiny")
    inp = I.make_inputs(w, 42)
    assert inp["X"].dtype == np.float32 and inp["X"].shape == (128, 64)
    assert inp["W"].shape == (1000, 64) and inp["Q"].shape == (1, 128, 2, 32) and inp["K"].shape == (1, 128, 2, 32)
    assert inp["W1"].shape == (32, 64) and inp["W2"].shape == (1, 32)
