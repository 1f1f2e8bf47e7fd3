"""Placement of the persistent kernels' workgroups among the XCDs
(wavernn_tune / wavernn_set_placement).

CPU: tests/placement_check.cpp, compiled against the library's layout header,
checks the block -> role mapping of every plan shape and candidate.  GPU:
results do not depend on the placement -- every candidate that fits gives
the default placement's samples and final state bit for bit (dense, fused
and block-sparse kernels); the tuner keeps the fastest fitting candidate and
reports the others."""
import os
import subprocess

import numpy as np
import pytest

from paper_1802_08435_amd import synth, wavernn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_placement_roles_on_the_host(tmp_path):
    exe = str(tmp_path / "placement_check")
    subprocess.run(["g++", "-std=c++17", "-Wall", "-I", os.path.join(ROOT, "paper_1802_08435_amd", "csrc"), "-o", exe,
                    os.path.join(ROOT, "tests", "placement_check.cpp")], check=True)
    r = subprocess.run([exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "0 violations" in r.stdout


torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def cuda(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _run(m, T, feat, n_streams=1):
    fin = m.new_state(n_streams)
    out = m.sample(T, cond=None if feat is None else cuda(feat), seed=11, n_streams=n_streams, final=fin)
    m.device_status()
    return out.cpu().numpy(), {k: v.cpu().numpy() for k, v in fin.items() if hasattr(v, "cpu")}


def _fitting(m):
    ok = []
    for i in range(64):
        try:
            m.set_placement(i)
            ok.append(i)
        except wavernn.WaveRNNError:
            pass
    m.set_placement(-1)
    return ok


def _same_everywhere(m, T, feat, cands):
    ref, ref_fin = _run(m, T, feat)
    for i in cands:
        print(f"placement {i}", flush=True)
        m.set_placement(i)
        out, fin = _run(m, T, feat)
        np.testing.assert_array_equal(out, ref, err_msg=f"placement {i}")
        for k in ref_fin:
            np.testing.assert_array_equal(fin[k], ref_fin[k], err_msg=f"placement {i} state {k}")
    m.set_placement(-1)


@pytest.mark.gpu
def test_dense_every_placement_gives_the_same_samples(_gpu):
    w = synth.make_weights(256, seed=3, cond_dim=16)
    m = wavernn.Model(w)
    cands = _fitting(m)
    assert 0 in cands and len(cands) == 64       # 4 heads + 12 units fit any XCD
    feat = synth.features(1, 400, cond_dim=16)
    _same_everywhere(m, 400, feat, cands)
    m.close()


@pytest.mark.gpu
def test_dense896_placements_same_samples(_gpu):
    w = synth.preset("dense896")
    m = wavernn.Model(w)
    cands = _fitting(m)
    assert len(cands) == 64                     # 7 heads and 28 units fit any pair of XCDs
    feat = synth.features(1, 300)
    _same_everywhere(m, 300, feat, [1, 4, 9, 18, 36, 63])
    m.close()


@pytest.mark.gpu
def test_fused_and_block_sparse_placements_same_samples(_gpu):
    wf = synth.make_fused_weights(256, F=2, seed=2, cond_dim=16)
    m = wavernn.Model(wf)
    assert m.path()[0] == "fused"
    _same_everywhere(m, 300, synth.features(1, 300, cond_dim=16), [2, 12, 27, 40, 63])
    m.close()
    ws = synth.make_weights(256, seed=8, cond_dim=16, block=(4, 4), density=0.1)
    m = wavernn.Model(ws, r_format="bsr4x4")
    assert m.path()[0] == "block-sparse"
    cands = _fitting(m)
    _same_everywhere(m, 300, synth.features(1, 300, cond_dim=16), [c for c in cands if c][::5])
    m.close()


@pytest.mark.gpu
def test_tune_keeps_the_fastest_fitting_candidate(_gpu):
    w = synth.make_weights(256, seed=3, cond_dim=16)
    m = wavernn.Model(w)
    feat = synth.features(1, 400, cond_dim=16)
    ref, _ = _run(m, 400, feat)
    grid0 = m.path()[1]
    r = m.tune(n_steps=256, rounds=1)
    us = np.array(r["us_per_step"])
    k = r["chosen"]
    assert 0 <= k < 64 and us[k] > 0 and us[k] == us[us > 0].min()
    assert (us > 0).all()                       # every candidate fits this model
    assert us[0] < 100.0                        # microseconds per step of a short launch, not a failed one
    out, _ = _run(m, 400, feat)
    np.testing.assert_array_equal(out, ref)
    if k % 9:                                   # a placement other than a spread: the grid grew
        assert m.path()[1] > grid0
    m.close()


@pytest.mark.gpu
def test_placement_arguments(_gpu):
    w = synth.make_weights(256, seed=3)
    m = wavernn.Model(w)
    for bad in (-2, 64):
        with pytest.raises(wavernn.WaveRNNError):
            m.set_placement(bad)
    with pytest.raises(wavernn.WaveRNNError):
        m.tune(n_steps=8)
    m.close()
    small = wavernn.Model(synth.make_weights(64, seed=1), dtype="f32")
    assert small.path()[0] == "single-workgroup"
    with pytest.raises(wavernn.WaveRNNError):
        small.set_placement(1)
    assert small.tune(n_steps=64, rounds=1)["chosen"] == -1
    small.close()
