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


def test_gate_decision_per_event():
    """Algorithm 1 returns the greedy probe on STOP and MAXLEN and samples on INCOMPAT."""
    assert gate.is_hit(gate.STOP) and gate.is_hit(gate.MAXLEN) and not gate.is_hit(gate.INCOMPAT)


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


def _counting(seq):
    """Scripted logits plus a counter of the decode steps asked for."""
    first, nxt = _scripted(seq)
    calls = []

    def counted(q):
        calls.append(len(q))
        return nxt(q)
    return first, counted, calls


def test_fixed_probe_decodes_k_tokens_then_applies_the_detector():
    """Appendix B: the probe always runs k greedy tokens, then the detector
    decides once; Section 3's naive approach is the same with k = L."""
    table = [[1, 2, 3]]
    seq = [1, 5, 3, 4, 6, 7, 8, 2, 2]
    first, nxt, calls = _counting(seq)
    assert gate.fixed_probe(first, nxt, table, k=6) == (seq[:6], gate.INCOMPAT)
    assert calls == [1, 2, 3, 4, 5]            # k - 1 decode steps after the prompt's own logits
    # the early-exit probe stops at the second token with the same decision
    first, nxt, calls = _counting(seq)
    assert gate.probe(first, nxt, table, k=6) == ([1, 5], gate.INCOMPAT)
    assert calls == [1]
    first, nxt, calls = _counting([1, 2, 3, 4, 5, 6, 7])
    assert gate.fixed_probe(first, nxt, table, k=6) == ([1, 2, 3, 4, 5, 6], gate.MAXLEN)
    # a stop token ends decoding; compatible -> STOP (a greedy refusal), else INCOMPAT
    first, nxt, calls = _counting([1, 2, 3, 9, 4])
    assert gate.fixed_probe(first, nxt, table, k=6, eos=9) == ([1, 2, 3, 9], gate.STOP)
    assert calls == [1, 2, 3]
    first, nxt, _ = _counting([1, 2, 9, 4])
    assert gate.fixed_probe(first, nxt, table, k=6, eos=9) == ([1, 2, 9], gate.INCOMPAT)
    # an empty table never matches; no table at all (None) always does
    first, nxt, _ = _counting([7, 7, 7, 7])
    assert gate.fixed_probe(first, nxt, [], k=3) == ([7, 7, 7], gate.INCOMPAT)
    first, nxt, _ = _counting([7, 7, 7, 7])
    assert gate.fixed_probe(first, nxt, None, k=3) == ([7, 7, 7], gate.MAXLEN)
    # k = 1: the prompt's logits alone
    first, nxt, calls = _counting([1, 5])
    assert gate.fixed_probe(first, nxt, table, k=1) == ([1], gate.MAXLEN) and calls == []


@pytest.mark.parametrize("seed", range(30))
def test_fixed_probe_same_decision_as_early_exit(seed):
    """Prefix closure: the fixed probe and the gated probe decide alike on every
    prompt; the gated probe's tokens are a prefix of the fixed probe's, which
    always has k tokens unless a stop token came first."""
    g = np.random.default_rng(300 + seed)
    table = [list(g.integers(0, 3, size=g.integers(2, 5))) for _ in range(3)]
    seq = list(g.integers(0, 4, size=14))
    eos = int(g.integers(-1, 4))
    k = int(g.integers(1, 12))
    first, nxt = _scripted(seq)
    qe, ee = gate.probe(first, nxt, table, k=k, eos=eos)
    first, nxt = _scripted(seq)
    qf, ef = gate.fixed_probe(first, nxt, table, k=k, eos=eos)
    assert gate.is_hit(ee) == gate.is_hit(ef)
    if gate.is_hit(ef):
        assert qe == qf and ee == ef
    assert qf[:len(qe)] == qe
    stop = [i for i, y in enumerate(seq[:k]) if y == eos]
    assert len(qf) == (stop[0] + 1 if stop else k)


def test_table_entries_csr():
    assert gate.table_entries(np.array([0, 2, 5]), np.array([4, 5, 6, 7, 8])) == [[4, 5], [6, 7, 8]]


# ---- soft compatibility gate (Appendix C) ----

def _probs_logits(p):
    """logits whose softmax is exactly the distribution p."""
    return np.log(np.asarray(p, np.float64))


def test_top_k_order_ties_and_probabilities():
    z = _probs_logits([0.1, 0.4, 0.4, 0.05, 0.05])
    got = gate.top_k(z, 3)
    assert [a for a, _ in got] == [1, 2, 0]          # equal logits: lower id first
    assert np.allclose([pa for _, pa in got], [0.4, 0.4, 0.1])


def _soft_scene(p_after_i):
    """Scripted probe: token 1 is I; after [I] the next-token distribution is
    p_after_i; after that, DOT forever."""
    first = _probs_logits([0.01] * 1 + [0.9] + [0.01] * 8)    # argmax I (= 1)
    p_dot = [0.02] * 10
    p_dot[DOT] = 0.82

    def nxt(q):
        return _probs_logits(p_after_i) if len(q) == 1 else _probs_logits(p_dot)
    return first, nxt


# after "I": greedy " think" (0.5), then " cannot" (0.2), " can't" (0.15)
P_AFTER_I = [0.02, 0.02, 0.2, 0.15, 0.02, 0.5, 0.02, 0.03, 0.02, 0.02]
SOFT_TABLE = [[I, CANNOT, HELP, DOT], [I, CANT, HELP, DOT], [I, M_SORRY, DOT]]


def test_soft_gate_continues_with_the_most_probable_compatible_alternative():
    first, nxt = _soft_scene(P_AFTER_I)
    # compatible mass 0.2 + 0.15 + 0.02 (" cannot", " can't", "'m sorry") = 0.37 >= 0.1:
    # " cannot", the most probable of them, replaces " think"
    steps = []
    q, ev = gate.soft_probe(first, nxt, SOFT_TABLE, k=6, c=3, K=10, rho=0.1, steps=steps)
    assert q[:2] == [I, CANNOT]
    assert np.isclose(steps[0].mass, 0.37) and steps[0].greedy == THINK and steps[0].appended == CANNOT
    # the probe goes on greedily: DOT after "I cannot" leaves every entry -> third token fails
    assert (q, ev) == ([I, CANNOT, DOT], gate.INCOMPAT)


def test_soft_gate_mass_below_rho_samples():
    first, nxt = _soft_scene(P_AFTER_I)
    assert gate.soft_probe(first, nxt, SOFT_TABLE, k=6, c=3, K=10, rho=0.4) == ([I, THINK], gate.INCOMPAT)


def test_soft_gate_mass_uses_the_full_vocabulary_softmax_within_top_k():
    first, nxt = _soft_scene(P_AFTER_I)
    # top-2 = " think" 0.5, " cannot" 0.2: mass 0.2 (not renormalised to 0.2/0.7 over the top-K)
    assert gate.soft_probe(first, nxt, SOFT_TABLE, k=6, c=3, K=2, rho=0.25)[1] == gate.INCOMPAT
    q, _ = gate.soft_probe(first, nxt, SOFT_TABLE, k=6, c=3, K=2, rho=0.2)
    assert q[:2] == [I, CANNOT]
    # " can't" (rank 3) is outside the top-2 and does not count
    assert gate.soft_probe(first, nxt, [[I, CANT, DOT]], k=6, c=3, K=2, rho=0.01)[1] == gate.INCOMPAT
    assert gate.soft_probe(first, nxt, [[I, CANT, DOT]], k=6, c=3, K=3, rho=0.01)[0][:2] == [I, CANT]


def test_soft_steps_are_only_the_first_c_tokens():
    first, nxt = _soft_scene(P_AFTER_I)
    # the incompatible greedy token is token 2: soft with c >= 2, hard with c = 1
    assert gate.soft_probe(first, nxt, SOFT_TABLE, k=6, c=1, K=10, rho=0.1) == ([I, THINK], gate.INCOMPAT)
    assert gate.soft_probe(first, nxt, SOFT_TABLE, k=6, c=2, K=10, rho=0.1)[0][:2] == [I, CANNOT]


def test_soft_gate_maxlen_after_substitution():
    first, nxt = _soft_scene(P_AFTER_I)
    # a 2-token budget ends right after the substituted token: a hit with the soft probe
    assert gate.soft_probe(first, nxt, SOFT_TABLE, k=2, c=3, K=10, rho=0.1) == ([I, CANNOT], gate.MAXLEN)


@pytest.mark.parametrize("seed", range(30))
def test_soft_gate_reduces_to_the_hard_gate(seed):
    """rho above 1 (no mass can reach it) or K = 1 (the only candidate is the
    failing greedy token) give exactly the hard probe."""
    g = np.random.default_rng(seed)
    V = 6
    table = [list(g.integers(0, V, size=g.integers(2, 5))) for _ in range(4)]
    seqs = g.normal(size=(12, V)) * 2
    first, nxt = seqs[0], (lambda q: seqs[len(q)])
    hard = gate.probe(first, nxt, table, k=8)
    assert gate.soft_probe(first, nxt, table, k=8, c=8, K=V, rho=1.5) == hard
    assert gate.soft_probe(first, nxt, table, k=8, c=8, K=1, rho=0.0) == hard


def test_fixed_length_probe_without_table():
    first, nxt = _scripted([3, 1, 4, 1, 5, 9])
    assert gate.probe(first, nxt, None, k=5) == ([3, 1, 4, 1, 5], gate.MAXLEN)
