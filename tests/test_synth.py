"""The seeded input module: bf16 rounding and reproducible draws."""
import numpy as np

import synth


def test_bf16_round_to_nearest_even():
    one = 1.0
    ulp = 2.0 ** -7                      # bf16 spacing at 1.0
    vals = np.array([one, one + ulp / 2, one + 3 * ulp / 2, one + ulp / 2 + 2.0 ** -20, -2.5, 0.0, -0.0,
                     np.inf, np.finfo(np.float32).max], dtype=np.float32)
    bits = synth.f32_to_bf16_bits(vals)
    back = synth.bf16_bits_to_f64(bits)
    # ties go to the even mantissa; above the tie rounds up
    assert back[0] == 1.0
    assert back[1] == 1.0
    assert back[2] == one + 2 * ulp
    assert back[3] == one + ulp
    assert back[4] == -2.5
    assert bits[5] == 0 and bits[6] == 0x8000
    assert np.isinf(back[7])
    assert np.isinf(back[8])            # beyond the largest bf16: rounds to inf
    nan = synth.f32_to_bf16_bits(np.array([np.nan], dtype=np.float32))
    assert np.isnan(synth.bf16_bits_to_f64(nan))[0]


def test_bf16_matches_torch_rounding():
    import torch
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 10
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_draw_is_reproducible_and_masked():
    wl = synth.tiny("bf16")
    a = synth.draw(wl)
    b = synth.draw(wl)
    assert np.array_equal(a.x.dev, b.x.dev)
    assert np.array_equal(a.params[0][0].R.dev, b.params[0][0].R.dev)
    mask = np.zeros(wl.B, dtype=bool)
    mask[1] = True
    c = synth.draw(wl, row_mask=mask)
    assert np.array_equal(c.x.dev, a.x.dev)
    assert np.all(c.dy.f64[:, ~mask] == 0) and np.array_equal(c.dy.f64[:, mask], a.dy.f64[:, mask])
    # the tiny config: forget-gate bias 1.0, everything else 0
    bb = a.params[0][0].b
    assert np.all(bb[64:128] == 1.0) and np.all(bb[:64] == 0) and np.all(bb[128:] == 0)
    # only the last step carries the loss weights
    assert np.all(a.dy.f64[:-1] == 0)


def test_flop_count_headline():
    # 4 layers x 3 x 2*T*B*4H*(I+H) with T=50, B=128, I=H=1024
    assert abs(synth.gnmt4().gemm_flops() - 1288.49e9) < 0.01e9


def test_block_sample_covers_every_share_and_block():
    for B in (1, 3, 16, 20, 32, 64, 128, 256, 264, 512):
        rows = synth.sample_rows_blocks(B, seed=B)
        assert rows[0] == 0 and rows[-1] == B - 1 and len(set(rows.tolist())) == len(rows)
        share = (B + 7) // 8
        for p in range(8):
            for b0 in range(p * share, min(B, p * share + share), 16):
                b1 = min(B, p * share + share, b0 + 16)
                assert np.any((rows >= b0) & (rows < b1)), (B, p, b0)
    # 32 (share, block) pairs at B = 512, up to two rows each
    assert 48 <= len(synth.sample_rows_blocks(512, seed=2)) <= 66
