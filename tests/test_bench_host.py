"""Host-side helpers of the benchmark (no GPU)."""
import bench


def test_byte_lru_hit_rate_hand_worked():
    # capacity of two 10-byte models: 1 miss, 2 miss, 1 hit, 3 miss (evicts 2, the least
    # recently used), 1 hit, 2 miss (evicts 3) -> 2 hits of 6
    assert bench.byte_lru_hit_rate([1, 2, 1, 3, 1, 2], {1: 10, 2: 10, 3: 10}, 20) == 2 / 6
    # a model larger than half the capacity evicts everything else; sizes, not counts, decide
    assert bench.byte_lru_hit_rate([1, 2, 3, 1, 2], {1: 10, 2: 10, 3: 25}, 30) == 0.0
    assert bench.byte_lru_hit_rate([1, 2, 1, 2], {1: 10, 2: 10}, 20) == 0.5
