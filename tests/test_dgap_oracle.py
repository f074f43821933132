"""Pins of the DGAP oracle (oracle/dgap.py) against facts that do not come
from the oracle itself: brute-force orderings, closed forms on hand-made
rows, a library log-sum-exp, invariances and the degenerate weights for
which the detector and corrector have known outputs."""
import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import dgap
from dgap_inputs import DgapWeights, gen_logits, gen_weights


def test_topk_is_the_brute_force_order_with_index_ties():
    r = np.random.default_rng(3)
    for V, k in ((10, 10), (50, 8), (257, 64)):
        z = np.round(r.standard_normal(V) * 2) / 2  # many exact ties
        want = sorted(range(V), key=lambda i: (-z[i], i))[:k]
        assert list(dgap.topk(z, k)) == want


def test_log_sum_exp_matches_a_library_routine():
    z = gen_logits(32768, 1, seed=5)[0].astype(np.float64)
    M, lse, p = dgap.log_softmax_terms(z)
    assert M == z.max()
    assert abs(lse - logsumexp(z)) <= 1e-12 * abs(lse)
    assert abs(p.sum() - 1.0) <= 1e-12


def test_entropy_of_uniform_and_of_a_certain_row():
    V = 4096
    phi = dgap.features(np.zeros(V), 16)
    assert abs(phi[0] - np.log(V)) <= 1e-12 and abs(phi[1] - 1.0) <= 1e-12
    assert abs(phi[3] - 16 / V) <= 1e-15 and abs(phi[5] - 1 / V) <= 1e-15
    assert phi[6] == 0 and phi[7] == 0 and phi[8] == 0 and phi[9] == 0 and phi[10] == 0
    assert abs(phi[11] - np.log(16)) <= 1e-12           # uniform over the top 16
    z = np.zeros(V)
    z[123] = 1000.0                                      # one certain token
    phi = dgap.features(z, 16)
    assert phi[0] < 1e-300 and phi[2] == 0.0 and phi[3] == 1.0 and phi[5] == 1.0
    assert phi[6] == 1000.0 and phi[11] == 0.0


def test_gap_and_dispersion_features_on_an_arithmetic_row():
    # logits 0, 0.5, ..., 9.5: the top 8 are 9.5 .. 6.0, every gap 0.5
    z = np.arange(20) * 0.5
    phi = dgap.features(z, 8)
    assert phi[6] == 0.5 and phi[7] == 0.5 and phi[8] == 0.5 and phi[9] == 0.5
    assert abs(phi[10] - 0.5 * np.sqrt(5.25)) <= 1e-12   # population std of 8 equally spaced values
    assert abs(phi[2] - (9.5 - logsumexp(z))) <= 1e-12


def test_whole_vocabulary_window():
    z = gen_logits(32768, 1, seed=2, kind="flat")[0][:512].astype(np.float64)
    phi = dgap.features(z, z.size)
    assert abs(phi[3] - 1.0) <= 1e-12          # the window holds all the mass
    assert abs(phi[11] - phi[0]) <= 1e-10      # so its entropy is the row's


def test_shift_invariance():
    # softmax, ranks, gaps and margins ignore a common shift of all logits
    z = gen_logits(32768, 1, seed=7)[0].astype(np.float64)
    for k in (16, 128):
        a, b = dgap.features(z, k), dgap.features(z + 37.25, k)
        assert np.allclose(a, b, rtol=1e-9, atol=1e-9)
        assert np.allclose(dgap.candidate_features(z, k), dgap.candidate_features(z + 37.25, k),
                           rtol=1e-9, atol=1e-9)


def test_candidate_features_by_hand():
    z = np.array([1.0, 4.0, 2.0, 4.0, 0.5, 3.0, -1.0, 2.5, 0.0, 3.5])
    xi = dgap.candidate_features(z, 8)
    # order: 4.0 (1), 4.0 (3), 3.5 (9), 3.0 (5), 2.5 (7), 2.0 (2), 1.0 (0), 0.5 (4)
    v = np.array([4.0, 4.0, 3.5, 3.0, 2.5, 2.0, 1.0, 0.5])
    assert list(dgap.topk(z, 8)) == [1, 3, 9, 5, 7, 2, 0, 4]
    assert np.array_equal(xi[:, 0], v - 4.0)
    assert np.allclose(xi[:, 1], v - logsumexp(z), atol=1e-12)
    assert np.allclose(xi[:, 2], np.arange(8) / 7)
    assert np.array_equal(xi[:, 3], [0, 0, 0.5, 0.5, 0.5, 0.5, 1.0, 0.5])
    assert np.array_equal(xi[:, 4], [0, 0.5, 0.5, 0.5, 0.5, 1.0, 0.5, 0])


def _zero_weights(det_out: float, corr_out: float, hd: int = 4, hc: int = 4) -> DgapWeights:
    return DgapWeights(np.zeros((12, hd), np.float32), np.zeros(hd, np.float32), np.zeros(hd, np.float32),
                       det_out, np.zeros((17, hc), np.float32), np.zeros(hc, np.float32),
                       np.zeros(hc, np.float32), corr_out)


def test_detector_and_corrector_with_known_outputs():
    z = gen_logits(32768, 1, seed=1)[0]
    w = _zero_weights(np.log(0.7 / 0.3), 0.25)
    res = dgap.restore(z, 32, w)
    assert abs(res.risk - 0.7) <= 1e-12 and res.corrected
    assert np.array_equal(res.delta, np.full(32, 0.25))
    changed = np.flatnonzero(res.logits != z.astype(np.float64))
    assert np.array_equal(np.sort(changed), np.sort(res.idx))      # only the window moves
    assert np.array_equal(res.logits[res.idx], z[res.idx].astype(np.float64) + 0.25)


def test_bypass_at_or_below_threshold():
    z = gen_logits(32768, 1, seed=4)[0]
    for r in (0.2, 0.6):   # r == tau does not trigger (strict inequality)
        w = _zero_weights(np.log(r / (1 - r)), 5.0)
        res = dgap.restore(z, 64, w)
        assert not res.corrected and np.array_equal(res.logits, z.astype(np.float64))


def test_relu_layer_by_hand():
    # one hidden unit active, one clipped: f = 2 * relu(phi_0 - 1) + 0 * ... - 3
    z = gen_logits(32768, 1, seed=9)[0]
    phi = dgap.features(z, 16)
    w1 = np.zeros((12, 2), np.float32)
    w1[0, 0], w1[0, 1] = 1.0, -1.0
    w = DgapWeights(w1, np.array([-1.0, -1.0], np.float32), np.array([2.0, 5.0], np.float32), -3.0,
                    np.zeros((17, 2), np.float32), np.zeros(2, np.float32), np.zeros(2, np.float32), 0.0)
    s = 2.0 * max(phi[0] - 1.0, 0.0) + 5.0 * max(-phi[0] - 1.0, 0.0) - 3.0
    assert abs(dgap.detector(phi, w) - 1 / (1 + np.exp(-s))) <= 1e-12


def test_permutation_equivariance():
    z = gen_logits(32768, 1, seed=11)[0]
    w = gen_weights(0, det_bias=20.0)
    perm = np.random.default_rng(0).permutation(z.size)
    a = dgap.restore(z, 64, w)
    b = dgap.restore(z[perm], 64, w)
    assert a.corrected and b.corrected
    assert np.allclose(b.logits, a.logits[perm], rtol=0, atol=1e-12)
    assert np.array_equal(perm[b.idx], a.idx)


def test_top8_mass_in_closed_form():
    # 12 logits at log 2 and 20 at 0: the top 8 hold 8 * 2 / (12 * 2 + 20) of
    # the mass, the top 16 hold (12 * 2 + 4) / 44 (a 7- or 9-entry slice, or
    # the top-k slice, gives another number)
    z = np.concatenate([np.full(12, np.log(2.0)), np.zeros(20)])
    phi = dgap.features(z, 16)
    assert abs(phi[4] - 16 / 44) <= 1e-15
    assert abs(phi[3] - 28 / 44) <= 1e-15
    phi8 = dgap.features(z, 8)
    assert abs(phi8[4] - 16 / 44) <= 1e-15 and abs(phi8[3] - 16 / 44) <= 1e-15


def test_smallest_gap_spans_exactly_the_top_eight():
    # leading logits with gaps 1, 1.5, 1, 1.5, 0.8, 1.2, 0.25 between v1..v8,
    # then 0.0625 between v8 and v9: the smallest of the 7 gaps is 0.25; six
    # gaps would give 0.8 and eight 0.0625
    v = np.array([10.0, 9.0, 7.5, 6.5, 5.0, 4.25, 3.0, 2.75, 2.6875])
    z = np.concatenate([v, np.full(23, -4.0)])
    for k in (8, 9, 16):
        assert dgap.features(z, k)[9] == 0.25
    phi = dgap.features(z, 9)
    assert phi[6] == 1.0 and phi[7] == 1.5 and phi[8] == (10.0 - 2.6875) / 8


def test_corrector_by_hand_with_candidate_and_shape_inputs():
    # The 10-logit row of test_candidate_features_by_hand, k = 8: xi is known by
    # hand, and so are phi_6 = v1 - v2 = 0, phi_7 = v2 - v3 = 0.5 and
    # phi_8 = (v1 - v8) / 7 = 0.5.  The corrector input is [xi_k (5), phi (12)],
    # so phi_j sits in row 5 + j of C1.
    z = np.array([1.0, 4.0, 2.0, 4.0, 0.5, 3.0, -1.0, 2.5, 0.0, 3.5])
    v = np.array([4.0, 4.0, 3.5, 3.0, 2.5, 2.0, 1.0, 0.5])
    above = np.array([0, 0, 0.5, 0.5, 0.5, 0.5, 1.0, 0.5])
    rank = np.arange(8) / 7
    c1 = np.zeros((17, 3), np.float32)
    cb1 = np.array([-0.75, 0.5, 2.0], np.float32)
    c2 = np.array([1.5, -2.0, 0.25], np.float32)
    # unit 0: margin above + 2 phi_7 - 0.75     (active where margin > -0.25)
    c1[3, 0], c1[5 + 7, 0] = 1.0, 2.0
    # unit 1: -(v - v1) - 4 phi_8 + 0.5          (active once v1 - v > 1.5)
    c1[0, 1], c1[5 + 8, 1] = -1.0, -4.0
    # unit 2: -4 rank + 3 phi_6 + 2              (active while rank < 0.5)
    c1[2, 2], c1[5 + 6, 2] = -4.0, 3.0
    w = DgapWeights(np.zeros((12, 2), np.float32), np.zeros(2, np.float32), np.zeros(2, np.float32), 20.0,
                    c1, cb1, c2, -0.5)
    h0 = np.maximum(above + 2 * 0.5 - 0.75, 0)
    h1 = np.maximum(-(v - 4.0) - 4 * 0.5 + 0.5, 0)
    h2 = np.maximum(-4 * rank + 3 * 0.0 + 2.0, 0)
    want = 1.5 * h0 - 2.0 * h1 + 0.25 * h2 - 0.5
    res = dgap.restore(z, 8, w)
    assert res.corrected
    assert np.allclose(res.delta, want, rtol=0, atol=1e-12)
    assert np.allclose(res.logits[[1, 3, 9, 5, 7, 2, 0, 4]], v + want, rtol=0, atol=1e-12)
    assert res.logits[6] == -1.0 and res.logits[8] == 0.0
