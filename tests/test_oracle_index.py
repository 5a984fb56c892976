"""Pins of the oracle's index math (Alg. 1, Alg. 2, Table I) against the paper's
own N=4, B=2 example and Table I at the Sec. V-A setup."""
import os

import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def test_group_formation_matches_paper_example():
    for rank, g, l, K, seq, chunk in [list(map(int, r)) for r in _rows("group_formation_n4_b2.txt")]:
        assert oracle.group_of(4, 2, rank) == (g, l, K)
        L = 1024
        s0, s1, t0, t1 = oracle.seq_partition(L, K, rank)
        assert (s0, s1) == (seq, seq + 1)
        assert (t0, t1) == (chunk * L // K, (chunk + 1) * L // K)


@pytest.mark.parametrize("N,B", [(8, 1), (8, 2), (8, 4), (8, 8), (16, 2), (6, 3), (1, 1)])
def test_groups_partition_the_world(N, B):
    """Every rank is in exactly one group of K contiguous ranks; B groups."""
    K = N // B
    seen = {}
    for r in range(N):
        g, l, k = oracle.group_of(N, B, r)
        assert k == K and 0 <= g < B and 0 <= l < K
        assert r == g * K + l           # contiguous assignment, Sec. IV-A
        seen.setdefault(g, set()).add(l)
    assert sorted(seen) == list(range(B))
    assert all(v == set(range(K)) for v in seen.values())


@pytest.mark.parametrize("N,B,L", [(8, 2, 4096), (4, 2, 64), (8, 1, 512), (8, 8, 32)])
def test_partition_covers_each_sequence_once(N, B, L):
    """Alg. 2: the K ranks of group g tile sequence g with disjoint chunks."""
    K = N // B
    cover = {}
    for r in range(N):
        s0, s1, t0, t1 = oracle.seq_partition(L, K, r)
        assert s1 == s0 + 1 and t1 - t0 == L // K
        cover.setdefault(s0, []).append((t0, t1))
    assert sorted(cover) == list(range(B))
    for chunks in cover.values():
        chunks.sort()
        assert chunks[0][0] == 0 and chunks[-1][1] == L
        assert all(a[1] == b[0] for a, b in zip(chunks, chunks[1:]))


def test_divisibility_and_fallback_errors():
    with pytest.raises(oracle.OracleError):
        oracle.group_of(6, 4, 0)        # N mod B != 0: the assert of Alg. 1
    with pytest.raises(oracle.OracleError):
        oracle.group_of(4, 8, 0)        # B > N: data-parallel fallback, Sec. IV-A
    with pytest.raises(oracle.OracleError):
        oracle.group_of(4, 2, 4)        # rank outside the world
    with pytest.raises(oracle.OracleError):
        oracle.seq_partition(10, 4, 0)  # L not divisible by K


def test_table1_tokens_and_participants():
    """Tokens per GPU of Ulysses (SP=N) and BASP are equal, participants shrink."""
    N, B, S = 8, 2, 16384
    expect = {r[0]: (int(r[1]), int(r[2])) for r in _rows("table1_tokens_n8_b2_s16k.txt")}
    # Ulysses SP=N: every rank holds its N-th chunk of all B sequences.
    ulysses_tokens = B * (S // N)
    # BASP: the rank's group holds one sequence, cut into K chunks.
    K = N // B
    s0, s1, t0, t1 = oracle.seq_partition(S, K, 5)
    basp_tokens = (s1 - s0) * (t1 - t0)
    _, _, k = oracle.group_of(N, B, 5)
    assert (ulysses_tokens, N) == expect["ulysses_sp_n"]
    assert (basp_tokens, k) == expect["basp"]
