"""The probe's routing rule (host): the category is the argmax of the label
tokens' logits, H(X) the Shannon entropy (nats) of their softmax, and a
request goes to the small model when it is Code, its context is within the
limit and H(X) <= tau (reading of the paper's Section 3.2 / 3.3 rule)."""
import numpy as np
import pytest

from paper_2604_09752_amd import binding as b


@pytest.mark.parametrize("c", [1, 2, 3, 5, 8])
def test_equal_scores_give_log_c(c):
    _, h, cat = b.aio_probe_route(np.full(c, 1.25), 0, 10)
    assert abs(h - np.log(c)) < 1e-6 and cat == 0  # ties: lowest index


def test_entropy_matches_definition_on_random_scores():
    rng = np.random.default_rng(5)
    for _ in range(50):
        x = rng.normal(0, 3, int(rng.integers(2, 7))).astype(np.float32)
        p = np.exp(x.astype(np.float64) - x.max())
        p /= p.sum()
        ref = float(-(p * np.log(p)).sum())
        _, h, cat = b.aio_probe_route(x, 0, 10)
        assert abs(h - ref) < 1e-5 and cat == int(np.argmax(x))


def test_two_equal_leaders_give_log_two():
    _, h, _ = b.aio_probe_route([5.0, 5.0, -80.0], 0, 10)
    assert abs(h - np.log(2)) < 1e-6


def test_decision_table():
    sure_code = [9.0, 0.0, 0.0]  # H about 2.5e-3
    assert b.aio_probe_route(sure_code, 0, 2048)[0] is True
    assert b.aio_probe_route(sure_code, 0, 2049)[0] is False      # context over the limit
    assert b.aio_probe_route(sure_code, 1, 100)[0] is False       # not the Code category
    unsure = [1.0, 0.5, 0.0]  # H about 1.03 > 0.45
    assert b.aio_probe_route(unsure, 0, 100)[0] is False
    assert b.aio_probe_route(unsure, 0, 100, tau=1.1)[0] is True  # a looser threshold
    # exactly at the threshold is still routed to the small model
    x = np.array([3.0, 0.0], np.float32)
    h = b.aio_probe_route(x, 0, 10)[1]
    assert b.aio_probe_route(x, 0, 10, tau=h)[0] is True


def test_rejects_bad_arguments():
    with pytest.raises(b.AioError):
        b.aio_probe_route([], 0, 10)
    with pytest.raises(b.AioError):
        b.aio_probe_route([1.0, 2.0], 2, 10)
