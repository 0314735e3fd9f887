"""The seeded input generator: determinism, row subsets, bf16 rounding and the
structure each preset promises."""
import numpy as np
import torch

from paper_2603_13180_amd import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100_000).astype(np.float32) * 1e3,
                        np.array([0.0, -0.0, 448.0, 1e-40, -3.4e38], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(synth.f32_to_bf16_bits(x), ref)
    assert np.array_equal(synth.bf16_bits_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_row_subset_equals_full_tensor_rows():
    full = synth.generate("llama3-125m-d768")
    rows = np.array([0, 5, 511, 1023])
    sub = synth.generate("llama3-125m-d768", rows=rows)
    assert full.x.shape == (1024, 768)
    assert np.array_equal(sub.x, full.x[rows]) and np.array_equal(sub.gamma, full.gamma)
    again = synth.generate("llama3-125m-d768")
    assert np.array_equal(again.x, full.x)


def test_outlier_channels_and_row_scales():
    w = synth.generate("llama3-8b-d4096", rows=np.arange(0, 4096, 64))
    xf = synth.bf16_bits_to_f32(w.x)
    col_rms = np.sqrt((xf.astype(np.float64) ** 2).mean(0))
    assert (col_rms > 8).sum() == 41
    w = synth.generate("llama3-1b-d2048", rows=np.arange(0, 16384, 97))
    row_rms = np.sqrt((synth.bf16_bits_to_f32(w.x).astype(np.float64) ** 2).mean(1))
    assert row_rms.min() > 0.09 and row_rms.max() < 11 and row_rms.max() / row_rms.min() > 20


def test_stress_preset_structure():
    p = synth.PRESETS["llama3-8b-longctx-stress"]
    aux = synth._aux(p, 0)
    assert len(aux["zero_rows"]) == p.T // 100 == len(aux["const_rows"])
    assert not set(aux["zero_rows"]) & set(aux["const_rows"])
    rows = np.concatenate([aux["zero_rows"][:3], aux["const_rows"][:3], [1, 2]])
    rows.sort()
    w = synth.generate("llama3-8b-longctx-stress", rows=rows)
    xf = synth.bf16_bits_to_f32(w.x)
    for i, r in enumerate(rows):
        if r in aux["zero_rows"]:
            assert np.all(xf[i] == 0)
        elif r in aux["const_rows"]:
            assert np.all(xf[i] == xf[i, 0])
        else:
            assert 0 < (np.abs(xf[i]) == 448).sum() < 20
    g = synth.bf16_bits_to_f32(w.gamma)
    assert g.min() >= 0.5 and g.max() <= 1.5
