"""Host rules of the runtime: the swap policy and the budget allocation of
Sec. 3 ("Swap", "AllocateLLMBudget"), called through the C ABI (pure host
functions, no GPU)."""
import pytest

from paper_2607_20501_amd import mk


def test_swap_marks_subkernels_below_tau():
    # speedups ref/sel: 2.0, 0.5, 0.95, 0.85
    sw, trig = mk.mk_swap_decide([1.0, 2.0, 1.0, 1.0], [2.0, 1.0, 0.95, 0.85], 0.9)
    assert trig and sw == [0, 1, 0, 1]


def test_swap_threshold_is_strict():
    sw, trig = mk.mk_swap_decide([1.0, 1.0], [1.0, 0.9], 0.9)
    assert trig and sw == [0, 0]          # 0.9 is not below 0.9
    sw, _ = mk.mk_swap_decide([1.0, 1.0], [1.0, 0.8999], 0.9)
    assert sw == [0, 1]


def test_swap_needs_two_subkernels():
    sw, trig = mk.mk_swap_decide([2.0], [1.0], 0.9)
    assert not trig and sw == [0]


def test_swap_not_triggered_when_every_subkernel_is_slower():
    sw, trig = mk.mk_swap_decide([2.0, 3.0, 4.0], [1.0, 1.0, 1.0], 0.9)
    assert not trig and sw == [0, 0, 0]


def test_swap_skips_subkernels_without_reference():
    sw, trig = mk.mk_swap_decide([1.0, 5.0, 1.0], [2.0, -1.0, 0.1], 0.9)
    assert trig and sw == [0, 0, 1]


def test_swap_rejects_bad_arguments():
    lib = mk.load()
    assert lib.mk_swap_decide(-1, None, None, 0.9, None, None) != 0
    assert lib.mk_swap_decide(2, None, None, 0.9, None, None) != 0


def test_budget_proportional_to_runtime():
    shares = mk.mk_budget_shares([1.0, 3.0, 0.0, 4.0])
    assert shares == pytest.approx([0.125, 0.375, 0.0, 0.5])
    assert sum(shares) == pytest.approx(1.0)


def test_budget_even_among_subkernels_needing_work():
    shares = mk.mk_budget_shares([1.0, 3.0, 2.0, 4.0], [0, 1, 0, 1])
    assert shares == pytest.approx([0.0, 0.5, 0.0, 0.5])


def test_budget_degenerate_cases():
    assert mk.mk_budget_shares([0.0, 0.0]) == [0.0, 0.0]
    assert mk.mk_budget_shares([]) == []
    with pytest.raises(mk.MkError):
        mk.mk_budget_shares([1.0, -1.0])
