"""Pins for the prefix-tree and routing oracle (Sec. 5), on hand-built traces."""
import pytest

from oracle.scheduler import PrefixTreeRef, route_ref

EDGES = [1000, 4000]          # bins: [0, 1000), [1000, 4000), [4000, inf)
S_OK, S_FAIL, S_BIG = 0b0000, 0b0001, 0b0110   # (type 0 ok), (type 0 failed), (type 1 large)


def tree():
    t = PrefixTreeRef(EDGES)
    # prompt 7: three traces
    t.insert(7, [S_OK], [1500, 300])            # short after a success
    t.insert(7, [S_FAIL, S_FAIL], [6000, 5000, 4200])
    t.insert(7, [S_FAIL], [3000, 2500])
    # prompt 9: one trace without tools
    t.insert(9, [], [800])
    return t


def test_histograms_by_hand():
    t = tree()
    # root: residual[0] of all four traces: 1500, 6000, 3000, 800 -> bins 1, 2, 1, 0
    assert t.lookup(123, []) == ([0.25, 0.5, 0.25], -1)
    # prompt 7 at depth 0: 1500, 6000, 3000 -> bins 1, 2, 1
    assert t.lookup(7, []) == ([0.0, 2 / 3, 1 / 3], 0)
    # after one failure: 5000 and 2500 -> bins 2, 1
    assert t.lookup(7, [S_FAIL]) == ([0.0, 0.5, 0.5], 1)
    # after two failures: 4200 -> bin 2
    assert t.lookup(7, [S_FAIL, S_FAIL]) == ([0.0, 0.0, 1.0], 2)
    # after a success: 300 -> bin 0
    assert t.lookup(7, [S_OK]) == ([1.0, 0.0, 0.0], 1)


def test_back_off_to_parent():
    t = tree()
    # unseen third return after two failures -> the depth-2 node
    assert t.lookup(7, [S_FAIL, S_FAIL, S_BIG]) == ([0.0, 0.0, 1.0], 2)
    # unseen first return -> the prompt node
    assert t.lookup(7, [S_BIG]) == ([0.0, 2 / 3, 1 / 3], 0)
    # a seen state after an unseen one does not skip the gap
    assert t.lookup(7, [S_BIG, S_FAIL]) == ([0.0, 2 / 3, 1 / 3], 0)
    # unseen prompt -> root
    assert t.lookup(5, [S_FAIL])[1] == -1


def test_bin_edges_are_half_open():
    t = PrefixTreeRef(EDGES)
    for r in (0, 999, 1000, 3999, 4000, 10 ** 9):
        t.insert(1, [], [r])
    assert t.lookup(1, [])[0] == [2 / 6, 2 / 6, 2 / 6]


def test_empty_tree_is_an_error():
    with pytest.raises(ValueError):
        PrefixTreeRef(EDGES).lookup(1, [])


def test_route_by_hand():
    hist = [0.5, 0.5]
    t_dec = [[10.0, 30.0],     # small bucket: expected 20
             [8.0, 14.0],      # medium: expected 11
             [9.0, 10.0]]      # large: expected 9.5
    c_mig = [[99.0, 1.0, 2.0],  # diagonal ignored
             [1.0, 0.0, 1.0],
             [3.0, 3.0, 0.0]]
    # from bucket 0: small 20 + 0, medium 11 + 1 = 12, large 9.5 + 2 = 11.5
    assert route_ref(hist, t_dec, c_mig, 0) == (2, 11.5)
    # from bucket 1: small 20 + 1, medium 11 + 0, large 9.5 + 1 = 10.5
    assert route_ref(hist, t_dec, c_mig, 1) == (2, 10.5)
    # from bucket 2: small 20 + 3, medium 11 + 3, large 9.5
    assert route_ref(hist, t_dec, c_mig, 2) == (2, 9.5)
    # a costly move keeps the request where it is: medium 11 + 0 < large 9.5 + 2.5
    c_mig[1][2] = 2.5
    assert route_ref(hist, t_dec, c_mig, 1) == (1, 11.0)
    # staying is free even with a non-zero diagonal entry
    assert route_ref([1.0, 0.0], [[5.0, 0.0], [5.0, 0.0]], [[7.0, 0.0], [1.0, 7.0]], 1) == (1, 5.0)
    # ties go to the lowest index
    assert route_ref([1.0], [[2.0], [1.0], [1.0]], [[0, 0, 0]] * 3, 0) == (1, 1.0)
