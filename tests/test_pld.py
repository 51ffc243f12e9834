"""Prompt-lookup draft matcher (host logic of the PLD loop; no GPU needed).

The reference below is the definition written out: for n from the largest
usable n-gram down to the smallest, the last n tokens are looked for earlier
in the history, and the earliest occurrence that has a continuation gives up
to k drafts (SURVEY's reading c13 of Section 4.2's PLD Configuration)."""
import numpy as np
import pytest

from paper_2604_09752_amd import binding as b


def ref_match(h, nmax, nmin, k):
    h = list(h)
    for n in range(min(nmax, len(h) - 1), nmin - 1, -1):
        suf = h[len(h) - n:]
        for i in range(0, len(h) - n):
            if h[i:i + n] == suf:
                return h[i + n:i + n + k]
    return []


@pytest.mark.parametrize("seed", range(40))
def test_matches_definition_on_random_histories(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 60))
    vocab = int(rng.integers(2, 6))  # small vocabularies: many recurrences
    h = rng.integers(0, vocab, n).astype(np.int32)
    nmax = int(rng.integers(1, 7))
    nmin = int(rng.integers(1, nmax + 1))
    k = int(rng.integers(0, 10))
    got = b.aio_pld_match(h, nmax, nmin, k)
    assert list(got) == ref_match(h, nmax, nmin, k)


def test_planted_three_gram_yields_the_continuation():
    rng = np.random.default_rng(3)
    h = list(rng.integers(100, 1000, 200))
    j = 57
    h += h[j:j + 3]  # the history now ends with the 3-gram at j
    got = b.aio_pld_match(np.array(h, np.int32), 3, 1, 8)
    assert list(got) == h[j + 3:j + 11]


def test_largest_ngram_wins_over_earlier_shorter_match():
    # the 1-gram [9] occurs first at 0, the 2-gram [4, 9] only later at 5
    h = [9, 1, 2, 3, 5, 4, 9, 7, 8, 4, 9]
    assert list(b.aio_pld_match(np.array(h, np.int32), 2, 1, 3)) == [7, 8, 4]
    assert list(b.aio_pld_match(np.array(h, np.int32), 1, 1, 3)) == [1, 2, 3]


def test_no_recurrence_no_drafts_and_k_zero():
    h = np.arange(50, dtype=np.int32)
    assert b.aio_pld_match(h, 6, 1, 8).size == 0
    assert b.aio_pld_match(np.array([1, 1, 1], np.int32), 3, 1, 0).size == 0
    assert b.aio_pld_match(np.array([], np.int32), 3, 1, 4).size == 0


def test_continuation_is_cut_at_the_end_of_the_history():
    h = np.array([5, 6, 7, 5, 6], np.int32)  # [5, 6] recurs, followed by 7, 5, 6
    assert list(b.aio_pld_match(h, 2, 1, 8)) == [7, 5, 6]


def test_rejects_bad_arguments():
    h = np.array([1, 2, 1], np.int32)
    for args in ((3, 0, 2), (1, 2, 2), (3, 1, -1)):
        with pytest.raises(b.AioError) as e:
            b.aio_pld_match(h, *args)
        assert e.value.code == b.AIO_ERANGE
