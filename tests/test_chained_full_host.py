"""Host-side pieces of the full-size layer checks: the bf16 rounding they use
equals the oracle's, and the block sampling covers every block."""
import numpy as np

from chained_full import block_samples, rnd_bf16
from oracle.bf16 import round_bf16


def test_fast_bf16_rounding_equals_the_oracle_rounding():
    rng = np.random.default_rng(3)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.float32([0.0, -0.0, 1.0, 65504.0, 1e-40, -3.4e38])])
    # exact ties: the low 16 bits 0x8000, both parities of the kept part
    ties = (np.arange(1, 2000, dtype=np.uint32) << 16 | np.uint32(0x8000)).view(np.float32)
    for v in (a, ties, -ties):
        np.testing.assert_array_equal(rnd_bf16(v), round_bf16(v))


def test_block_samples_cover_every_block():
    rng = np.random.default_rng(0)
    for rows, cols in [(1, 1), (64, 64), (65, 3), (1000, 257), (4096, 25088)]:
        idx = block_samples(rows, cols, rng, cap=10 ** 9)
        r, c = idx // cols, idx % cols
        assert idx.min() >= 0 and idx.max() < rows * cols
        seen = set(zip((r // 64).tolist(), (c // 64).tolist()))
        assert len(seen) == (-(-rows // 64)) * (-(-cols // 64))
    idx = block_samples(4096, 25088, rng, cap=1000)
    assert 1000 <= idx.size <= 1002
    r, c = idx // 25088, idx % 25088
    assert np.any(r // 64 == 63) and np.any(c // 64 == 391)     # ragged edge blocks kept
