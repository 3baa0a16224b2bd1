"""Pins for the compatibility predicate, probe and gate (not GPU).  Token
translations of the worked examples of Section 3 and Appendix C."""
import numpy as np
import pytest

from oracle import gate

# token ids standing for text pieces of the paper's examples
I, CANNOT, CANT, M_SORRY, THINK, HELP, DOT = 1, 2, 3, 4, 5, 6, 7


def test_partial_start_and_passed_opening_are_compatible():
    table = [[I, CANNOT, HELP]]
    assert gate.compatible([I], table)                     # "I" may still become a refusal
    assert gate.compatible([I, CANNOT, HELP, DOT], table)  # passed a known opening
    assert not gate.compatible([I, THINK], table)


def test_soft_gate_example_alternatives():
    table = [[I, CANNOT], [I, CANT], [I, M_SORRY]]
    assert not gate.compatible([I, THINK], table)
    for alt in (CANNOT, CANT, M_SORRY):
        assert gate.compatible([I, alt], table)


def test_min_match_ignores_short_entries():
    assert not gate.compatible([I], [[I]])
    assert gate.compatible([I], [[I]], min_match=1)
    assert not gate.compatible([9], [])                    # empty table: never compatible


@pytest.mark.parametrize("seed", range(20))
def test_prefix_closure(seed):
    g = np.random.default_rng(seed)
    table = [list(g.integers(0, 4, size=g.integers(2, 6))) for _ in range(4)]
    q = list(g.integers(0, 4, size=8))
    for n in range(1, 9):
        if gate.compatible(q[:n], table):
            assert all(gate.compatible(q[:j], table) for j in range(1, n + 1))


def _scripted(seq):
    """logits whose argmax follows `seq`."""
    def lg(t):
        z = np.zeros(10)
        z[t] = 1.0
        return z
    return lg(seq[0]), (lambda q: lg(seq[len(q)]))


def test_probe_events_and_early_exit():
    table = [[1, 2, 3]]
    first, nxt = _scripted([1, 2, 3, 4, 5, 6, 7, 8, 9])
    assert gate.probe(first, nxt, table, k=6) == ([1, 2, 3, 4, 5, 6], gate.MAXLEN)
    first, nxt = _scripted([1, 5, 3, 4])
    assert gate.probe(first, nxt, table, k=6) == ([1, 5], gate.INCOMPAT)
    first, nxt = _scripted([1, 2, 9, 9])
    assert gate.probe(first, nxt, table, k=6, eos=9) == ([1, 2, 9], gate.INCOMPAT)
    first, nxt = _scripted([1, 2, 3, 9, 9])
    assert gate.probe(first, nxt, table, k=6, eos=9) == ([1, 2, 3, 9], gate.STOP)
    first, nxt = _scripted([7])
    assert gate.probe(first, nxt, [], k=6) == ([7], gate.INCOMPAT)


@pytest.mark.parametrize("seed", range(20))
def test_early_exit_decision_equals_full_probe(seed):
    """Prefix closure makes 'stop at the first incompatible token' and 'decode k
    tokens then check once' the same decision."""
    g = np.random.default_rng(100 + seed)
    table = [list(g.integers(0, 3, size=g.integers(2, 5))) for _ in range(3)]
    seq = list(g.integers(0, 3, size=12))
    first, nxt = _scripted(seq)
    q, ev = gate.probe(first, nxt, table, k=8)
    full_hit = gate.compatible(seq[:8], table)
    assert gate.is_hit(ev) == full_hit
    if not full_hit:
        assert not gate.compatible(q, table) and gate.compatible(q[:-1], table) or len(q) == 1


def test_table_entries_csr():
    assert gate.table_entries(np.array([0, 2, 5]), np.array([4, 5, 6, 7, 8])) == [[4, 5], [6, 7, 8]]
