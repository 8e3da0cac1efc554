"""Pins of the heavy-tail task generator (paper_2609_36314_amd.heavy_tail; Sec. 4.1,
Appendix E.1): labels against the weighted sum written out event by event, a worked
case by hand, the gap law against its truncated Zipf probabilities, the event signs'
balance, and seeding."""
import math

import numpy as np

from paper_2609_36314_amd import heavy_tail as ht


def test_hand_case():
    # +1 at the start and -1 on the last token of 4: y = 4^-0.1 - 1 < 0.
    t = np.array([[ht.PLUS, 0, 0, ht.MINUS]])
    assert ht.labels_of(t)[0] == 0
    # the same events swapped: y = -4^-0.1 + 1 > 0.
    assert ht.labels_of(t[:, ::-1].copy())[0] == 1
    # no events: y = 0, label 0
    assert ht.labels_of(np.zeros((1, 9), dtype=np.uint8))[0] == 0


def test_labels_match_the_sum_event_by_event():
    tok, lab = ht.sample(40, 300, seed=3)
    for row, y in zip(tok, lab):
        s = 0.0
        for k, t in enumerate(row):
            if t != ht.BACKGROUND:
                s += (1.0 if t == ht.PLUS else -1.0) / math.pow(300 - k, ht.GAMMA)
        assert y == int(s > 0)


def _gaps(tok):
    out = []
    for row in tok:
        pos = np.flatnonzero(row)
        out.append(np.diff(np.concatenate([[-1], pos])))
    return np.concatenate(out)


def test_gap_law_is_truncated_zipf():
    tok, _ = ht.sample(64, 20000, seed=4)
    g = _gaps(tok)
    assert g.min() >= 1 and g.max() <= ht.GAP_MAX
    p = ht.gap_pmf()
    n = g.size
    for k in range(1, 31):
        f = np.mean(g == k)
        assert abs(f - p[k - 1]) < 5 * math.sqrt(p[k - 1] * (1 - p[k - 1]) / n), k
    # the tail beyond 100 (the heavy part): probability mass within 5 sigma
    pt = p[100:].sum()
    assert abs(np.mean(g > 100) - pt) < 5 * math.sqrt(pt * (1 - pt) / n)


def test_signs_and_labels_are_balanced_and_seeded():
    tok, lab = ht.sample(2000, 512, seed=5)
    ev = tok[tok != ht.BACKGROUND]
    assert abs(np.mean(ev == ht.PLUS) - 0.5) < 5 * 0.5 / math.sqrt(ev.size)
    assert 0.45 < lab.mean() < 0.55
    t2, l2 = ht.sample(2000, 512, seed=5)
    assert np.array_equal(tok, t2) and np.array_equal(lab, l2)
    assert not np.array_equal(tok, ht.sample(2000, 512, seed=6)[0])
