"""Pins for the retrieval oracle (Sec. 4.2, Eq. retrieval).

* a hand-derived example (tests/golden/retrieval_hand_example.json);
* special cases: exact duplicate pose scores 0 and ranks first, an empty
  admissible set gives count 0, equal scores break ties by smaller j;
* brute force: an exhaustive pure-Python sort agrees with the vectorised
  oracle on random banks.
"""

import json
import math
import os

import numpy as np
import pytest

from oracle import brute, retrieval
from workloads.synth import axis_angle, pose_from


def _pose(centre, tilt_deg, axis=(0.0, 1.0, 0.0)):
    return pose_from(axis_angle(np.array(axis), math.radians(tilt_deg)), np.asarray(centre, float))


def _hand_example(golden_dir):
    with open(os.path.join(golden_dir, "retrieval_hand_example.json")) as f:
        g = json.load(f)
    bank = []
    for j in range(g["n_bank"]):
        e = g["entries"].get(str(j), g["default_entry"])
        bank.append(_pose(e["centre"], e["tilt_deg"]))
    bank = np.asarray(bank, np.float32)
    query = np.eye(4, dtype=np.float32)[None]
    return g, bank, query


@pytest.mark.parametrize("k", [2, 3])
def test_hand_example(golden_dir, k):
    g, bank, query = _hand_example(golden_dir)
    idx, sc, cnt = retrieval.retrieve(bank, query, np.array([g["query_chunk"]]), g["E"], g["w_v"], g["tau_c"],
                                      math.radians(g["tau_v_deg"]), g["delta"], g["first_candidate"], k)
    exp = g["expected"][f"k{k}"]
    assert idx[0].tolist() == exp["idx"]
    assert int(cnt[0]) == exp["count"]
    np.testing.assert_allclose(sc[0, : exp["count"]], exp["score"], atol=g["score_tol"])


def test_duplicate_pose_scores_zero_and_ranks_first():
    rng = np.random.default_rng(0)
    q = _pose([1.0, 2.0, 3.0], 17.0, axis=(0.3, 0.9, 0.1))
    bank = np.stack([_pose(q[:3, 3] + rng.normal(0, 0.3, 3), rng.uniform(0, 20)) for _ in range(20)])
    bank[7] = q
    idx, sc, cnt = retrieval.retrieve(bank.astype(np.float32), q[None].astype(np.float32), np.array([30]),
                                      10.0, 0.5, 1.0, math.radians(45), 3, 0, 3)
    assert idx[0, 0] == 7
    # v is used as stored (fp32, not renormalised): s = w_v (1 - |v|^2), about 1e-8
    vq = q[:3, 2].astype(np.float32).astype(np.float64)
    assert abs(sc[0, 0] - 0.5 * (1.0 - vq @ vq)) < 1e-15
    # an axis-aligned duplicate is exactly zero
    bank[7] = pose_from(np.eye(3), q[:3, 3])
    idx, sc, cnt = retrieval.retrieve(bank.astype(np.float32), bank[7:8].astype(np.float32), np.array([30]),
                                      10.0, 0.5, 1.0, math.radians(45), 3, 0, 3)
    assert idx[0, 0] == 7 and sc[0, 0] == 0.0


def test_empty_admissible_set():
    bank = np.stack([_pose([100.0 + j, 0, 0], 0.0) for j in range(12)]).astype(np.float32)
    idx, sc, cnt = retrieval.retrieve(bank, np.eye(4, dtype=np.float32)[None], np.array([40]),
                                      10.0, 0.5, 0.2, math.radians(45), 3, 0, 4)
    assert cnt[0] == 0
    assert (idx[0] == -1).all()
    assert np.isinf(sc[0]).all()


def test_gap_gate_excludes_recent_chunks():
    bank = np.stack([np.eye(4)] * 10).astype(np.float32)  # every chunk at the query pose
    idx, _, cnt = retrieval.retrieve(bank, np.eye(4, dtype=np.float32)[None], np.array([9]),
                                     1.0, 0.5, 0.1, math.radians(10), 3, 1, 10)
    # admissible: 1 <= j <= 6; all score 0 -> ties by j
    assert cnt[0] == 6
    assert idx[0, :6].tolist() == [1, 2, 3, 4, 5, 6]


def test_tie_break_smaller_index_first():
    p = _pose([0.5, 0.0, 0.0], 10.0)
    bank = np.stack([_pose([50, 0, 0], 0)] * 8)
    bank[5] = p
    bank[2] = p
    idx, sc, cnt = retrieval.retrieve(bank.astype(np.float32), np.eye(4, dtype=np.float32)[None], np.array([20]),
                                      10.0, 0.5, 0.2, math.radians(45), 3, 0, 2)
    assert idx[0].tolist() == [2, 5]
    assert sc[0, 0] == sc[0, 1]


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_agrees(seed):
    rng = np.random.default_rng(100 + seed)
    N = int(rng.integers(5, 80))
    bank = []
    for _ in range(N):
        bank.append(_pose(rng.normal(0, 2.0, 3), rng.uniform(0, 80), axis=rng.normal(size=3)))
    bank = np.asarray(bank, np.float32)
    queries = np.asarray([_pose(rng.normal(0, 2.0, 3), rng.uniform(0, 80), axis=rng.normal(size=3))
                          for _ in range(4)], np.float32)
    qchunk = rng.integers(0, N + 5, size=4).astype(np.int32)
    E, w_v, tau_c, tau_v, delta, fc, k = 5.0, 0.5, 0.6, math.radians(50), 3, 1, 5
    idx, sc, cnt = retrieval.retrieve(bank, queries, qchunk, E, w_v, tau_c, tau_v, delta, fc, k)
    for qi in range(4):
        # the brute force receives the same fp32-rounded parameters as the oracle
        bj, bs = brute.retrieve(bank.astype(np.float64).tolist(), queries[qi].astype(np.float64).tolist(),
                                int(qchunk[qi]), np.float32(E), np.float32(w_v), np.float32(tau_c),
                                np.float32(tau_v), delta, fc, k)
        assert cnt[qi] == len(bj)
        assert idx[qi, : len(bj)].tolist() == bj
        np.testing.assert_allclose(sc[qi, : len(bj)], bs, rtol=0, atol=1e-15)


def test_frame_selection_expands_chunks():
    idx = np.array([[4, 9, -1], [-1, -1, -1]], np.int32)
    sel = retrieval.frame_selection(idx, np.array([2, 0]), 3)
    assert sel[0].tolist() == [12, 13, 14, 27, 28, 29, -1, -1, -1]
    assert (sel[1] == -1).all()


def test_near_ties_hand_built():
    """near_ties counts a tie between the k-th and (k+1)-th admissible scores
    and every gate margin at its threshold. Query chunk n = 10 at the origin
    looking along +z; E = 10, tau_c = 0.25, tau_v = 0 (only exact alignment
    passes, and every entry is exactly aligned: each live entry is an
    alignment margin), Delta = 3, first candidate 1, so j = 1..7 are live.
    j = 1 and j = 2 sit at (+1, 0, 0) and (-1, 0, 0): equal scores 0.1;
    j = 3 at (2.5, 0, 0) has d = 0.25 = tau_c exactly (a distance margin,
    admissible, score 0.25); j = 4..7 are 3 m or more away (d > tau_c)."""
    centres = {0: (0.0, 0.0, 0.0), 1: (1.0, 0.0, 0.0), 2: (-1.0, 0.0, 0.0), 3: (2.5, 0.0, 0.0), 4: (5.0, 0.0, 0.0),
               5: (0.0, 0.0, 3.0), 6: (0.0, 3.0, 0.0), 7: (0.0, -4.0, 0.0), 8: (0.0, 0.0, 0.0), 9: (0.0, 0.0, 0.0)}
    bank = np.asarray([pose_from(np.eye(3), np.asarray(centres[j])) for j in range(10)], np.float32)
    query = np.eye(4, dtype=np.float32)[None]
    args = (bank, query, np.array([10]), 10.0, 0.5, 0.25, 0.0, 3, 1)
    idx, sc, cnt = retrieval.retrieve(*args, 3)
    assert idx[0].tolist() == [1, 2, 3] and cnt[0] == 3
    assert retrieval.near_ties(*args, 1) == (1, 8)  # s_(1) = s_(2) = 0.1
    assert retrieval.near_ties(*args, 2) == (0, 8)  # s_(2) = 0.1 < s_(3) = 0.25
    assert retrieval.near_ties(*args, 3) == (0, 8)  # no (k+1)-th admissible score
