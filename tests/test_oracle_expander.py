"""Pins of the expander / prior-head oracle (Sec. "Architecture", Table 4)."""
import numpy as np
import torch

from oracle import expander as EX


def test_added_parameters_reproduce_table_4():
    # Qwen3-4B and Qwen3-8B hidden sizes with 4 categories: 26.2M and 67.1M added parameters.
    assert EX.added_parameters(2560, 4) == 26_234_884
    assert EX.added_parameters(4096, 4) == 67_141_636


def test_zero_expander_copies_the_trunk_state_into_every_branch():
    """With W = 0 and c = 0 every branch equals h (initialisation from a DFlash checkpoint)."""
    rng = np.random.default_rng(1)
    H, R = 16, 3
    h = rng.normal(size=(2, 5, H))
    out = EX.expand_branches(h, np.zeros((R * H, H)), np.zeros(R * H))
    assert out.shape == (2, 5, R, H)
    for z in range(R):
        assert np.array_equal(out[:, :, z], h)


def test_branch_z_uses_its_own_block_of_rows_and_bias():
    """W_z = a_z I and c_z = b_z 1 give h_{k,z} = (1 + a_z) h_k + b_z (z-major features)."""
    rng = np.random.default_rng(2)
    H, R = 8, 4
    a = np.array([0.5, -1.0, 2.0, 0.0])
    b = np.array([1.0, 0.25, -3.0, 7.0])
    W = np.concatenate([a[z] * np.eye(H) for z in range(R)])
    c = np.repeat(b, H)
    h = rng.normal(size=(3, H))
    out = EX.expand_branches(h, W, c)
    for z in range(R):
        np.testing.assert_allclose(out[:, z], (1 + a[z]) * h + b[z], rtol=0, atol=1e-15)


def test_prior_head_one_hot_and_bias():
    H, R = 6, 3
    U = np.arange(R * H, dtype=np.float64).reshape(R, H)
    e = np.array([0.5, -1.0, 2.0])
    h = np.zeros((2, H))
    h[0, 4] = 1.0
    np.testing.assert_array_equal(EX.prior_logits(h, U, e), [U[:, 4] + e, e])


def test_bf16_rounding_matches_torch_on_binary32_inputs():
    """For binary32 inputs the single rounding equals torch's float32 -> bfloat16 conversion
    (round to nearest even), including ties and binade carries."""
    rng = np.random.default_rng(3)
    x = rng.normal(size=20000).astype(np.float32) * np.float32(3.0)
    ties = (np.arange(-64, 64, dtype=np.float32) + np.float32(0.5)) * np.float32(2.0 ** -7)
    x = np.concatenate([x, ties, np.float32([255.5, 1.99609375, -0.0, 0.0, 1e-20])])
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(EX.bf16_round(x.astype(np.float64)), want)
