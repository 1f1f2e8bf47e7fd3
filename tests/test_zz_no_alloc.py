"""wavernn_sample_noalloc (the library's per-device workspace, no device
allocation) against wavernn_sample, through the C ABI: samples and final states
bit for bit on every kernel path, on two calls in a row, the second smaller."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_1802_08435_amd import synth, wavernn  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def _both(m, S, T, feat, seed):
    """(samples, final state) of wavernn_sample_noalloc, then of wavernn_sample, same inputs."""
    res = []
    for noalloc in (True, False):
        out = torch.zeros(S, T, dtype=torch.uint16, device="cuda")
        fin = m.new_state(S)
        m.sample(T, cond=feat, seed=seed, n_streams=S, final=fin, out=out, noalloc=noalloc)
        m.device_status()
        res.append((out.cpu().numpy(), {k: v.cpu().numpy() for k, v in fin.items() if k != "t0"}))
    return res


@pytest.mark.parametrize("preset,calls", [
    ("tiny", [(1, 480), (1, 240)]),
    ("dense896", [(1, 2400), (1, 1200)]),
    ("multi4", [(4, 1200), (2, 600)]),
    ("subscale16", [(1, 1600), (1, 800)]),
    ("sparse2048_4x4", [(1, 960), (1, 480)]),
])
def test_noalloc_equals_sample(preset, calls):
    w = synth.preset(preset)
    S0 = max(S for S, _ in calls)
    r_format = {None: "dense", (4, 4): "bsr4x4", (16, 1): "bsr16x1"}[w["block"]]
    m = wavernn.Model(w, dtype="bf16" if w["bf16"] else "f32", r_format=r_format, max_streams=S0)
    print(f"noalloc {preset}: path {m.path(S0)}", flush=True)
    for k, (S, T) in enumerate(calls):
        feat = None if w.get("Wc") is None else torch.from_numpy(synth.features(S, T, per_stream_seed=S > 1)).cuda()
        (a, fa), (b, fb) = _both(m, S, T, feat, seed=3 + k)
        np.testing.assert_array_equal(a, b)
        for key in fa:
            np.testing.assert_array_equal(fa[key], fb[key])
        assert len(np.unique(a)) > 50, "degenerate output"
    m.close()


def test_noalloc_rejects_a_call_above_the_workspace():
    """A call whose per-frame table exceeds the 16 MiB workspace fails before any launch."""
    w = synth.preset("dense896")
    m = wavernn.Model(w)
    feat = torch.zeros(1, 2000, 64, device="cuda")     # 2000 frames x 2688 rows x 4 B = 21.5 MB
    out = torch.zeros(1, 240, dtype=torch.uint16, device="cuda")
    with pytest.raises(wavernn.WaveRNNError, match="workspace"):
        m.sample(240, cond=feat, out=out, noalloc=True)
    m.sample(240, cond=feat, out=out)                 # the allocating entry point serves it
    m.device_status()
    m.close()
