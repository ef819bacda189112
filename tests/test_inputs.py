"""The seeded input generators: bf16 rounding and workload recipes."""

import numpy as np
import pytest

from paper_2608_07524_amd import inputs as I


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.array([0.0, -0.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 3.0e38], dtype=np.float32)])
    x = x.astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(I.bf16_bits(x), ref)
    back = I.bf16_to_f64(ref)
    assert np.array_equal(back, torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).double().numpy())


def test_workload_recipes():
    assert I.tiny().cu_seqlens.tolist() == [0, 37, 101, 229, 429]
    rng = np.random.default_rng(0)
    w = I.video_short_mix(rng)
    assert len(w.lengths) == 32 and set(w.lengths) <= {1024, 2048, 4096, 8192}
    assert I.video_tokens_per_frame(256, 256) == 256
    assert I.video_tokens_per_frame(480, 854) == 1620
    assert I.video_tokens_per_frame(720, 1280) == 3600
    packs = I.video_long_tail_packs(np.random.default_rng(0), n_packs=3)
    assert len(packs) == 3 and all(p.total_tokens <= 131072 for p in packs)
    t = I.text_packs(np.random.default_rng(0), 2)
    assert all(p.total_tokens <= 262144 and p.causal for p in t)
    assert all(128 <= s <= 131072 for p in t for s in p.lengths)
    assert I.greedy_pack([5, 5, 3, 9, 1], 10) == [[5, 5], [3], [9, 1]]
