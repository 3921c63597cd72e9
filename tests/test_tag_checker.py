"""The tagged-pattern checker used by the GPU parity tests, checked on the CPU:
it accepts a correct gather (built with numpy indexing) and rejects planted
mistakes -- two heads swapped, a block in the wrong slot -- naming where."""
import numpy as np
import pytest

from gpu_util import check_tags, tag_cache

SENT = np.int16(-21555)


def _gather(tags, src_slots, dst_slots, n_dst):
    L, _, S, H, bs, D = tags.shape
    dst = np.full((L, 2, n_dst, H, bs, D), SENT, np.int16)
    dst[:, :, dst_slots] = tags[:, :, src_slots]
    return dst


def test_correct_gather_passes():
    tags = tag_cache(3, 9, 2, 4, 16)
    src, dst_slots = np.array([4, 0, 7]), np.array([2, 5, 1])
    check_tags(tags, _gather(tags, src, dst_slots, 6), src, dst_slots, SENT)


def test_swapped_heads_are_caught_and_located():
    tags = tag_cache(3, 9, 2, 4, 16)
    src, dst_slots = np.array([4, 0, 7]), np.array([2, 5, 1])
    dst = _gather(tags, src, dst_slots, 6)
    dst[1, 0, 5] = dst[1, 0, 5][::-1].copy()                    # block 1, layer 1, K: heads swapped
    with pytest.raises(AssertionError, match=r"block 1, slot 5, \(layer, kv, head, token, vector\) \[1, 0, 0, 0, 0\]"):
        check_tags(tags, dst, src, dst_slots, SENT)


def test_block_in_the_wrong_slot_is_caught():
    tags = tag_cache(2, 6, 1, 2, 8)
    src, dst_slots = np.array([1, 2]), np.array([0, 3])
    dst = _gather(tags, src, np.array([0, 4]), 5)               # block 1 written to slot 4, not 3
    with pytest.raises(AssertionError):
        check_tags(tags, dst, src, dst_slots, SENT)
