"""The reference dispatch order that the GPU tests compare the planner's
exported order with, checked on constructed plans."""
import numpy as np

from tests.gpu_util import expected_dispatch


def _tasks(lists, bhs=None):
    """Tasks over consecutive ranges of one tile list, one task per entry of `lists`."""
    tasks, kv, lo = [], [], 0
    for i, l in enumerate(lists):
        tasks.append([0 if bhs is None else bhs[i], i, lo, lo + len(l), 0, 1])
        kv += l
        lo += len(l)
    return np.array(tasks, dtype=np.int64), np.array(kv, dtype=np.int32)


def test_equal_lists_move_up_to_their_first_occurrence():
    A, B, C = [0, 1, 2], [1, 2, 3], [0, 1]
    t, kv = _tasks([A, B, A, C, B, A])
    assert expected_dispatch(t, kv, None).tolist() == [0, 2, 5, 1, 4, 3]


def test_unique_lists_keep_row_order():
    t, kv = _tasks([[0], [0, 1], [1], [1, 2], [2]])
    assert expected_dispatch(t, kv, None).tolist() == [0, 1, 2, 3, 4]


def test_heads_and_member_bits_separate_equal_tile_lists():
    A = [4, 5]
    t, kv = _tasks([A, A, A], bhs=[0, 1, 0])
    assert expected_dispatch(t, kv, None).tolist() == [0, 2, 1]
    mem = np.array([1, 3, 1, 2, 1, 3], dtype=np.uint64)  # task 1 differs in its second tile's bits
    t, kv = _tasks([A, A, A])
    assert expected_dispatch(t, kv, mem).tolist() == [0, 2, 1]


def test_window_grid_groups_each_frame_by_column():
    """A (3, 2, 4) grid window whose middle half-width covers both rows: the
    two query blocks of a (frame, column) pair read the same list and are
    dispatched together, columns 1 and 2 (whose column windows both cover the
    whole row) as one group of four."""
    from workloads.gen import window_mask
    m = window_mask((3, 2, 4), (1, 1, 2))
    lists = [list(np.nonzero(row)[0]) for row in m]
    t, kv = _tasks(lists)
    got = expected_dispatch(t, kv, None).tolist()
    frame0 = [0, 4, 1, 2, 5, 6, 3, 7]  # (h, w) = (0,0),(1,0), (0,1),(0,2),(1,1),(1,2), (0,3),(1,3)
    assert got[:8] == frame0
    assert sorted(got) == list(range(24))
