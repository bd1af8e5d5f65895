"""Pins of the oracle's frame gather and scatter (the query gather of a
skip step and the write-back of its keyframe rows; App. B.2: keyframe
queries only, non-keyframe outputs not computed) on hand-built cases whose
expected rows are written out by hand, not derived from the row map."""
import numpy as np
import pytest

import oracle


def _frames():
    # 3 frames of 2 rows, each row 2 x 2 uint16 bit patterns whose value names
    # (frame, row, element): 100 * frame + 10 * row + element
    src = np.zeros((6, 2, 2), dtype=np.uint16)
    for f in range(3):
        for r in range(2):
            src[2 * f + r] = (100 * f + 10 * r + np.arange(4)).reshape(2, 2)
    return src


def test_gather_hand_built():
    src = _frames()
    keep = src.copy()
    out = oracle.gather_frames(src, [0, 2], 2)
    expect = np.array([[[0, 1], [2, 3]], [[10, 11], [12, 13]],
                       [[200, 201], [202, 203]], [[210, 211], [212, 213]]], dtype=np.uint16)
    assert out.dtype == np.uint16 and np.array_equal(out, expect)
    assert np.array_equal(src, keep)                 # input not mutated
    out[0] = 7                                       # result does not alias the input
    assert np.array_equal(src, keep)


def test_gather_single_middle_frame():
    out = oracle.gather_frames(_frames(), [1], 2)
    assert np.array_equal(out[:, 0, 0], np.array([100, 110], dtype=np.uint16))


def test_scatter_hand_built_leaves_other_rows():
    compact = np.array([[[7, 7], [7, 7]], [[8, 8], [8, 8]],
                        [[9, 9], [9, 9]], [[6, 6], [6, 6]]], dtype=np.uint16)
    dst = np.full((6, 2, 2), 0xBEEF, dtype=np.uint16)   # sentinel everywhere
    keep_c, keep_d = compact.copy(), dst.copy()
    out = oracle.scatter_frames(compact, dst, [0, 2], 2)
    expect = np.full((6, 2, 2), 0xBEEF, dtype=np.uint16)
    expect[0], expect[1], expect[4], expect[5] = 7, 8, 9, 6
    assert np.array_equal(out, expect)
    # frame 1 (rows 2, 3) untouched, inputs not mutated
    assert (out[2:4] == 0xBEEF).all()
    assert np.array_equal(compact, keep_c) and np.array_equal(dst, keep_d)


def test_scatter_of_gather_restores_listed_frames_only():
    src = _frames()
    dst = np.full_like(src, 0xFFFF)
    out = oracle.scatter_frames(oracle.gather_frames(src, [1, 2], 2), dst, [1, 2], 2)
    assert np.array_equal(out[2:], src[2:])
    assert (out[:2] == 0xFFFF).all()


def test_float_bits_are_moved_unchanged():
    # bit patterns of NaNs with payloads and negative zero survive both copies
    bits = np.array([0x7FC1, 0xFFC3, 0x8000, 0x0001, 0x7F80, 0x3F80], dtype=np.uint16).reshape(6, 1)
    g = oracle.gather_frames(bits, [0, 2], 2)
    assert g.ravel().tolist() == [0x7FC1, 0xFFC3, 0x7F80, 0x3F80]
    s = oracle.scatter_frames(g, np.zeros_like(bits), [0, 2], 2)
    assert s.ravel().tolist() == [0x7FC1, 0xFFC3, 0, 0, 0x7F80, 0x3F80]


def test_scatter_rejects_a_wrong_row_count():
    with pytest.raises(ValueError):
        oracle.scatter_frames(np.zeros((3, 2), np.uint16), np.zeros((6, 2), np.uint16), [0, 2], 2)
