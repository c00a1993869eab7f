"""CPU tests of the seeded input generator (shared by the oracle and the HIP path)."""
import numpy as np
import torch

from paper_2106_06899_amd import workloads as wl


def test_bf16_rounding_matches_torch():
    rng = np.random.Generator(np.random.PCG64(3))
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1.0, -1.0, 1.00390625, 1.01171875, 3.4e38, -3.4e38, 1e-40],
                                 dtype=np.float32)])
    bits = wl.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.uint16).numpy()
    assert np.array_equal(bits, ref)
    back = wl.bf16_bits_to_f32(bits)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_inputs_are_seeded_and_shaped():
    w = wl.WORKLOADS["c2"].scaled(B=1, H=2, Lq=64, Lk=64)
    a = wl.make_inputs(w)
    b = wl.make_inputs(w)
    for key in ("Q", "K", "V"):
        assert a[key].values.shape == (1, 2, 64, 64)
        assert a[key].bits.dtype == np.uint16
        assert np.array_equal(a[key].bits, b[key].bits)
        assert np.array_equal(wl.bf16_bits_to_f32(a[key].bits), a[key].values)
    c = wl.make_inputs(w, seed=7)
    assert not np.array_equal(a["Q"].bits, c["Q"].bits)


def test_planted_queries_point_at_their_keys():
    """Generator check: each planted query is the sum of 4 key rows plus N(0, 0.5) noise,
    so those keys score far above the rest (not a parity criterion)."""
    w = wl.WORKLOADS["c3"].scaled(H=2, Lq=256, Lk=1024)
    x = wl.make_inputs(w)
    Q, K, pidx = x["Q"].values.astype(np.float64), x["K"].values.astype(np.float64), x["planted_idx"]
    assert pidx.shape == (1, 2, 256, 4)
    assert all(len(set(r)) == 4 for r in pidx.reshape(-1, 4).tolist())
    s = np.einsum("bhid,bhjd->bhij", Q, K)
    top = np.argsort(-s, axis=-1)[..., :w.k]
    hit = np.mean([np.isin(pidx[0, h, i], top[0, h, i]).all() for h in range(2) for i in range(256)])
    assert hit > 0.95


def test_ffn_inputs_std():
    w = wl.WORKLOADS["c5"].scaled(N=64, d_model=256, d_ff=2048)
    x = wl.make_inputs(w)
    assert x["W1"].values.shape == (2048, 256) and x["X"].values.shape == (64, 256)
    assert abs(float(x["W1"].values.std()) - 0.02) < 0.001
    assert abs(float(x["X"].values.std()) - 1.0) < 0.05
