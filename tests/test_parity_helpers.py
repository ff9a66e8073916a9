"""CPU pins of the GPU tests' own helpers: the near-tie detector that decides
which tokens escape the bit-exact index comparison, and the flip bookkeeping
that decides which tokens and experts a comparison leaves out."""
import numpy as np

from oracle import moe_oracle as O
from tests.parity import row_pairs, touched_experts


def test_near_ties_flags_exactly_the_close_gaps():
    # token 0: clear gaps; 1: k-th vs (k+1)-th within 1e-4 (set tie);
    # 2: two selected within 1e-4 (order tie); 3: both; 4: masked
    z = np.array([[3.0, 2.0, 1.0, 0.0],
                  [3.0, 1.00005, 1.0, 0.0],
                  [3.0, 2.99995, 1.0, 0.0],
                  [2.0, 1.99995, 1.99990, 0.0],
                  [1.0, 1.0, 1.0, 1.0]])
    mask = np.array([1, 1, 1, 1, 0], dtype=bool)
    st, ot = O.near_ties(z, 2, gap=1e-4, mask=mask)
    assert st.tolist() == [False, True, False, True, False]
    assert ot.tolist() == [False, False, True, True, False]
    # the gap is measured on fp32 keys: a 1e-9 difference that fp32 keeps is still a tie
    st, _ = O.near_ties(np.array([[1.0, 1.0 + 2 ** -20, 0.0]]), 1)
    assert st.tolist() == [True]
    # k = E: no (k+1)-th logit, so no set tie
    st, ot = O.near_ties(np.array([[1.0, 1.0]]), 2)
    assert st.tolist() == [False] and ot.tolist() == [True]
    # far gaps never count, whatever the scale
    st, ot = O.near_ties(np.array([[1e6, 0.0, -1e6]]), 2)
    assert not st.any() and not ot.any()


def test_touched_experts_is_the_union_of_both_selections():
    gpu = np.array([[0, 1], [2, 3], [4, 5]])
    ref = np.array([[0, 1], [2, 6], [4, 5]])
    flipped = np.array([False, True, False])
    t = touched_experts(flipped, gpu, ref, 8)
    assert np.nonzero(t)[0].tolist() == [2, 3, 6]
    assert not touched_experts(np.zeros(3, bool), gpu, ref, 8).any()


def test_row_pairs_follow_experts_across_slot_orders():
    # token 0's slots are swapped between the two runs (an order tie)
    gpu_idx = np.array([[1, 0], [0, 1]])
    gpu_row = np.array([[2, 0], [1, 3]])
    ref_idx = np.array([[0, 1], [0, 1]])
    ref_row = np.array([[0, 2], [1, 3]])
    g, r = row_pairs(gpu_idx, gpu_row, ref_idx, ref_row, [0, 1])
    assert g.tolist() == [2, 0, 1, 3] and r.tolist() == [2, 0, 1, 3]
