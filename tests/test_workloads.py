"""The seeded input generator: determinism, nesting of hot sets, and the derived budgets."""
import numpy as np
import pytest

from workloads import CONFIGS, get, make_layer


def test_same_seed_same_bytes_and_layers_differ():
    w = get("C1")
    a, b = make_layer(w, 0), make_layer(w, 0)
    for name in "qkv":
        for r in range(w.loops):
            assert np.array_equal(getattr(a, name)[r], getattr(b, name)[r])
    c = make_layer(w, 1)
    assert not np.array_equal(a.k[0], c.k[0])


def test_hot_sets_are_nested_and_sized():
    w = get("C2").replace(seq=1000, heads=2, head_dim=16)
    st = make_layer(w)
    prev = set(range(w.seq))
    for r in range(2, w.loops + 1):
        hot = set(st.hot[r - 2][0].tolist())
        assert hot <= prev and len(hot) == w.n_hot(r)
        prev = hot


def test_budgets_of_the_five_workloads():
    assert [get("C1").k(2)] == [64]
    assert [get("C2").k(r) for r in (2, 3, 4)] == [410, 410, 410]
    assert [get("C3").k(r) for r in (2, 3, 4)] == [1229, 550, 246]
    assert [get("C4").k(r) for r in (2, 3, 4)] == [1638, 1638, 1638]
    assert [get("C5").k(r) for r in range(2, 9)] == [3277, 2232, 1521, 1036, 706, 481, 328]
    assert get("C4").top_cols == 1532 and get("C4").c_list == 1536 and get("C4").window == 512
    assert get("C1").c_list == 32 and get("C2").c_list == 512 and get("C5").c_list == 1024
    assert [get("C5").bits_at(r) for r in range(2, 9)] == [4, 4, 2, 2, 2, 2, 2]
    for w in CONFIGS.values():
        assert w.head_dim in (64, 128)


def test_decaying_column_budget_is_nested_and_validated():
    w = get("C4").replace(seq=2000, window=128, col_budget=4 + 128 + 300,
                          col_decay=(4 + 128 + 300, 4 + 128 + 400, 4 + 128 + 100))
    assert [w.top_cols_at(r) for r in (2, 3, 4)] == [300, 300, 100]     # a larger budget cannot regrow the list
    assert get("C4").top_cols_at(4) == get("C4").top_cols                  # no schedule: constant
    with pytest.raises(ValueError):
        get("C4").replace(col_decay=(2048, 1024))                         # R - 1 = 3 entries needed
    with pytest.raises(ValueError):
        get("C4").replace(col_decay=(1024, 1024, 512))                    # must start at col_budget
