"""Host-side logic of the layer driver (CPU)."""
import numpy as np

from paper_2601_05296_amd import layer


def test_recompute_chunks_keep_routing_rows_aligned():
    """Every chunk of the full-recompute policy starts at a token whose rows
    of the [T, k] int32 / float32 routing arrays are 16-byte aligned (the C
    ABI rejects other pointers), for any requested chunk size and any k."""
    rng = np.random.default_rng(5)
    for _ in range(2000):
        T = int(rng.integers(1, 5000))
        want = int(rng.integers(1, 6000))
        c = layer.aligned_chunk(want, T)
        assert 1 <= c <= max(want, 4) or c == T
        assert c == T or (c % 4 == 0 and c >= 4)
        for k in range(1, 17):
            for t0, t1 in layer._chunks(T, c):
                assert (t0 * k * 4) % 16 == 0
                assert 0 < t1 - t0 <= c
    assert layer.aligned_chunk(659, 856) == 656
    assert layer.aligned_chunk(3, 856) == 4
    assert layer.aligned_chunk(900, 856) == 856
