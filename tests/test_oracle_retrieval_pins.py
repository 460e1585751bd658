"""Pins of the retrieval oracle (Section 3.1, Eq. 1-3) against things other
than itself (CPU only): brute-force pixel loops on tiny frames, hand-worked
histograms, intersections and rankings, closed forms of the keyframe rule
(theta limits, piecewise-constant videos), library routines (torch cosine,
numpy stable argsort), and planted mistakes that must break them."""
import numpy as np
import pytest
import torch

from oracle import retrieval as R
from paper_2601_01513_amd import workload as W


def _const_video(colors, h=4, w=5):
    """One frame per entry of `colors` (RGB triples), each frame flat."""
    return np.stack([np.broadcast_to(np.asarray(c, dtype=np.uint8), (h, w, 3)) for c in colors])


def test_histogram_matches_pixel_loop():
    rng = np.random.default_rng(0)
    f = rng.integers(0, 256, size=(3, 5, 7, 3), dtype=np.uint8)
    h = R.frame_histograms(f)
    for i in range(3):
        ref = np.zeros((3, R.BINS), dtype=np.int64)
        for y in range(5):
            for x in range(7):
                for c in range(3):
                    ref[c, int(f[i, y, x, c]) // 4] += 1
        np.testing.assert_array_equal(h[i], ref)
    assert np.all(h.sum(axis=2) == 35)


def test_histogram_hand_worked():
    f = np.array([[[[0, 4, 255], [3, 8, 252]],
                   [[255, 7, 0], [128, 4, 1]]]], dtype=np.uint8)   # one 2x2 frame
    h = R.frame_histograms(f)[0]
    assert h[0, 0] == 2 and h[0, 63] == 1 and h[0, 32] == 1          # R: 0, 3 | 255 | 128
    assert h[1, 1] == 3 and h[1, 2] == 1                               # G: 4, 7, 4 | 8
    assert h[2, 63] == 2 and h[2, 0] == 2                              # B: 255, 252 | 0, 1


def test_intersection_closed_forms():
    same = R.frame_histograms(_const_video([(10, 20, 30), (10, 20, 30)]))
    assert R.histogram_similarity(same[0], same[1], 20) == 1.0
    disjoint = R.frame_histograms(_const_video([(0, 0, 0), (255, 255, 255)]))
    assert R.histogram_similarity(disjoint[0], disjoint[1], 20) == 0.0
    # two channels equal, one different: 2/3
    part = R.frame_histograms(_const_video([(0, 100, 200), (0, 100, 20)]))
    assert R.histogram_similarity(part[0], part[1], 20) == pytest.approx(2.0 / 3.0, abs=1e-15)
    # half the pixels change one channel's bin: 1 - 1/6
    f = _const_video([(40, 40, 40), (40, 40, 40)], h=2, w=2).copy()
    f[1, 0, :, 0] = 200
    h = R.frame_histograms(f)
    assert R.histogram_similarity(h[0], h[1], 4) == pytest.approx(5.0 / 6.0, abs=1e-15)


def test_keyframe_theta_limits_and_scene_cuts():
    video = _const_video([(0, 0, 0)] * 3 + [(200, 10, 10)] * 4 + [(5, 90, 250)] * 2)
    keys, s = R.keyframes(video, 0.5)
    assert keys.tolist() == [0, 3, 7]                      # scene starts
    assert s[0] == -1 and s[1] == 60 and s[3] == 0         # 3 * 20 pixels when equal
    assert R.keyframes(video, 0.0)[0].tolist() == [0]      # nothing is below 0
    assert R.keyframes(video, 1.0001)[0].tolist() == list(range(9))  # everything is below
    assert R.keyframes(video[:1], 0.5)[0].tolist() == [0]
    assert R.keyframes(video[:0], 0.5)[0].tolist() == []


def _wipe_video(n=40):
    """Frame i: the first i of n columns bright, the rest dark (a slow wipe)."""
    v = np.zeros((n, 2, n, 3), dtype=np.uint8)
    for i in range(n):
        v[i, :, :i] = 200
    return v


def test_keyframes_compare_with_the_previous_frame():
    """A slow wipe never crosses theta between neighbours (similarity
    1 - 1/40), although frame 39 keeps only 1/40 of frame 0's histogram."""
    video = _wipe_video()
    keys, s = R.keyframes(video, 0.5)
    assert keys.tolist() == [0]
    assert np.all(s[1:] == 3 * 2 * 39)
    h = R.frame_histograms(video)
    assert R.histogram_similarity(h[0], h[39], 80) == pytest.approx(1.0 / 40.0, abs=1e-15)


def test_generated_video_keyframes_are_its_scene_cuts():
    rc = W.VIDEO_SMALL
    frames = W.make_video(rc, 0)
    keys, _ = R.keyframes(frames, rc.theta)
    rng = W.host_rng(0, "video")
    cuts = np.sort(rng.choice(np.arange(1, rc.n_frames), size=rc.n_scenes - 1, replace=False))
    assert keys.tolist() == [0] + cuts.tolist()


def test_cosine_matches_torch_and_closed_forms():
    rng = np.random.default_rng(1)
    a, b = rng.normal(size=(4, 16)), rng.normal(size=(9, 16))
    ref = torch.nn.functional.cosine_similarity(torch.tensor(a)[:, None], torch.tensor(b)[None],
                                                dim=2).numpy()
    np.testing.assert_allclose(R.cosine_matrix(a, b), ref, rtol=1e-12, atol=1e-12)
    c = R.cosine_matrix([[1.0, 0.0], [0.0, 0.0]], [[3.0, 0.0], [0.0, -2.0], [-1.0, 0.0]])
    np.testing.assert_array_equal(c, [[1.0, 0.0, -1.0], [0.0, 0.0, 0.0]])


def test_top_indices_match_stable_argsort_and_break_ties_low():
    rng = np.random.default_rng(2)
    x = rng.integers(0, 6, size=50).astype(float)          # many ties
    ref = np.argsort(-x, kind="stable")[:7]
    np.testing.assert_array_equal(R.top_indices(x, 7), ref)
    assert R.top_indices(np.array([0.5, 0.9, 0.9, 0.1]), 2).tolist() == [1, 2]
    assert R.top_indices(np.array([0.3]), 3).tolist() == [0]


def test_retrieve_hand_worked():
    # keyframe embeddings along the axes; documents at known angles
    frame_emb = np.eye(3)
    docs = np.array([[1.0, 0.0, 0.0],     # d0: cos 1 with f0
                     [0.8, 0.6, 0.0],     # d1: 0.8 with f0, 0.6 with f1
                     [0.0, 1.0, 0.0],     # d2: 1 with f1
                     [0.0, 0.6, 0.8],     # d3: 0.6 with f1, 0.8 with f2
                     [0.0, 0.0, -1.0]])   # d4: -1 with f2
    top, top_s, T, Ts = R.retrieve(frame_emb, np.array([0, 2]), docs, 2, 3)
    assert top.tolist() == [[0, 1], [3, 0]]    # f2: d3 (0.8), then the 0-ties d0 < d1 < d2
    np.testing.assert_allclose(top_s, [[1.0, 0.8], [0.8, 0.0]], atol=1e-15)
    # T = {0: max(1, 0), 1: 0.8, 3: 0.8} -> T* = [0, 1, 3]
    assert T.tolist() == [0, 1, 3]
    np.testing.assert_allclose(Ts, [1.0, 0.8, 0.8], atol=1e-15)
    top, _, T, Ts = R.retrieve(frame_emb, np.array([1]), docs, 1, 3)
    assert top.tolist() == [[2]] and T.tolist() == [2]    # |T| < K


# --- planted mistakes -------------------------------------------------------------

def test_planted_compare_with_last_keyframe_breaks_drift_pin():
    video = _wipe_video()
    h = R.frame_histograms(video)
    keys, last = [0], 0
    for i in range(1, 40):
        if R.histogram_similarity(h[i], h[last], 80) < 0.5:
            keys.append(i)
            last = i
    assert keys != R.keyframes(video, 0.5)[0].tolist()


def test_planted_bin_shift_breaks_hand_histogram():
    f = np.array([[[[0, 4, 255], [3, 8, 252]], [[255, 7, 0], [128, 4, 1]]]], dtype=np.uint8)
    wrong = np.bincount((f[0, :, :, 1] >> 3).ravel(), minlength=R.BINS)   # 32 bins
    assert not np.array_equal(wrong, R.frame_histograms(f)[0][1])


def test_planted_score_by_last_retrieval_breaks_hand_merge():
    """Scoring a document by its most recent retrieval instead of its best."""
    frame_emb = np.eye(3)
    docs = np.array([[1.0, 0.0, 0.0], [0.0, 0.6, 0.8], [0.8, 0.0, 0.6]])
    # d2: 0.8 with f0, 0.6 with f2; best = 0.8
    top, top_s, T, Ts = R.retrieve(frame_emb, np.array([0, 2]), docs, 2, 3)
    last = {}
    for r in range(top.shape[0]):
        for j, v in zip(top[r], top_s[r]):
            last[int(j)] = float(v)
    assert last[2] != dict(zip(T.tolist(), Ts.tolist()))[2]
