"""T12: the seeded input generator rounds like the reference casts (RNE)."""

import numpy as np
import torch

import synthetic as S
from synthetic import workloads as W


def test_fp16_rounding_matches_numpy_cast():
    x = S.draw(7, (100000,), "normal", 0.0, 30.0)
    assert np.array_equal(S.round_to_storage(x, "f16"), x.astype(np.float16))


def test_bf16_rne_matches_torch_on_random_and_ties():
    x = S.draw(8, (1_000_000,), "normal", 0.0, 3.0)
    # exact ties between two bf16 neighbours (low 16 bits == 0x8000), both parities
    base = np.arange(1, 2001, dtype=np.uint32) << 16
    ties = (base | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, -ties, np.array([0.0, -0.0, 1e-40, 3.4e38], np.float32)])
    got = S.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref)
    back = S.bf16_bits_to_f32(got)
    assert np.array_equal(back, torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_seeds_and_distributions():
    specs = W.specs("conv", hh=16, ww=16)
    names = [s[0] for s in specs]
    assert names == ["X", "W", "scale", "shift"] and [s[1] for s in specs] == [4001, 4002, 4003, 4004]
    t = W.inputs("conv", hh=64, ww=64)
    sc = t["scale"].astype(np.float64)
    assert sc.min() >= 0.5 and sc.max() <= 1.5
    x = S.draw(4001, (200000,), "normal", 0.0, 0.05)
    assert abs(x.std() - 0.05) < 1e-3 and abs(x.mean()) < 1e-3
    a = W.inputs("attention")
    b = W.inputs("attention")
    assert all(np.array_equal(a[k], b[k]) for k in a)
    assert a["Q"].dtype == np.float32 and W.inputs("linattn", n=8)["Q"].dtype == np.uint16
