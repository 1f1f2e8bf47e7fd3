"""Subscale calls run in pieces of their schedule (wavernn_sample_steps,
Sec. 4: an utterance generated over several calls, e.g. streamed), through the
C ABI.

Bar: bit-exact.  Running the steps [0, K) of a call's schedule in several
calls, each handing its state to the next and reading the samples of earlier
steps from the utterance buffer, makes the samples and final state of one
wavernn_sample call bit for bit, for lockstep rows, for the paper's order with
a future horizon, and with the conditioning CNN; pieces of one step, pieces
that end inside the ramp-up or ramp-down of the lagged lanes, and two
utterances per call are covered.  One call is pinned to the oracle elsewhere
(the subscale and CNN parity tests), so pieces equal to it are pinned too.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_1802_08435_amd import synth, wavernn  # noqa: E402


def cuda(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.cpu().numpy()


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)


def subscale_model(kind, H=128, B=4, seed=1):
    w = synth.make_weights(H, seed=seed, cond_dim=16, B=B, ctx_dim=64 if kind != "cnn" else 128)
    if kind == "horizon":
        w["F"] = 4
    if kind == "cnn":
        w["F"] = 130
        w["cnn"] = synth.make_cnn_weights(B, Rc=128, Cc=128, Dx=128, layers=10, seed=seed + 10)
    return w


def run_in_pieces(m, S, N, feat, seed, bounds):
    out = torch.zeros(S, N, dtype=torch.uint16, device="cuda")
    st = m.new_state(S)
    for a, b in zip(bounds, bounds[1:]):
        print(f"  steps [{a}, {b})", flush=True)
        m.sample_steps(out, a, b - a, cond=cuda(feat), seed=seed, init=st if a > 0 else None, final=st)
    m.device_status()
    return host(out), {k: host(v) for k, v in st.items() if k != "t0"}


@pytest.mark.parametrize("kind,B,S", [("lockstep", 4, 2), ("horizon", 4, 2), ("horizon", 16, 1), ("cnn", 4, 2)])
def test_pieces_of_the_schedule_equal_one_call(kind, B, S):
    N = B * 150
    w = subscale_model(kind, B=B)
    feat = synth.features(S, N, cond_dim=16, per_stream_seed=True)
    m = wavernn.Model(w, max_streams=S)
    assert m.path(S)[0] == "batched"
    fin = m.new_state(S)
    whole = host(m.sample(N, cond=cuda(feat), seed=3, n_streams=S, final=fin))
    m.device_status()
    fin = {k: host(v) for k, v in fin.items() if k != "t0"}
    K = m.schedule_steps(N)
    F = int(w.get("F", -1))
    assert K == N // B + ((B - 1) * (F + 1) if F >= 0 else 0)
    rng = np.random.default_rng(B + S)
    # a one-step piece, a piece ending in the ramp-up (lane B - 1 not started), the rest in uneven parts
    inner = sorted({1, 2, max(3, min(K - 3, (B - 1) * (F + 1) // 2 if F >= 0 else K // 3)),
                    *rng.integers(4, K - 1, size=3).tolist()})
    bounds = [0, *[b for b in inner if 0 < b < K], K]
    print(f"  {kind}: B = {B}, S = {S}, {K} steps, bounds {bounds}", flush=True)
    out, st = run_in_pieces(m, S, N, feat, 3, bounds)
    np.testing.assert_array_equal(out, whole)
    for k in ("h", "c", "f"):
        np.testing.assert_array_equal(st[k], fin[k], err_msg=k)
    assert len(np.unique(whole)) > 50
    m.close()


def test_step_calls_check_their_arguments():
    w = subscale_model("horizon")
    m = wavernn.Model(w)
    N = 4 * 40
    K = m.schedule_steps(N)
    out = torch.zeros(1, N, dtype=torch.uint16, device="cuda")
    feat = cuda(synth.features(1, N, cond_dim=16))
    for step0, n in ((-1, 1), (0, K + 1), (K, 1)):
        with pytest.raises(wavernn.WaveRNNError) as e:
            m.sample_steps(out, step0, n, cond=feat)
        assert e.value.status == wavernn.E_INVALID
    with pytest.raises(wavernn.WaveRNNError) as e:   # a later piece needs the state it starts from
        m.sample_steps(out, 5, 1, cond=feat)
    assert e.value.status == wavernn.E_INVALID
    m.sample_steps(out, K, 0, cond=feat)              # nothing to run
    assert m.schedule_steps(N + 1) == -1
    m.device_status()
    m.close()
    dense = wavernn.Model(synth.make_weights(128, seed=2, cond_dim=0))
    assert dense.schedule_steps(N) == -1
    with pytest.raises(wavernn.WaveRNNError) as e:
        dense.sample_steps(torch.zeros(1, N, dtype=torch.uint16, device="cuda"), 0, 1)
    assert e.value.status == wavernn.E_UNSUPPORTED
    dense.close()
    # the window context refills its rings by lane (B a power of two) when a call resumes
    w3 = synth.make_weights(128, seed=4, cond_dim=0, B=24, ctx_dim=64)
    m3 = wavernn.Model(w3)
    out3 = torch.zeros(1, 24 * 30, dtype=torch.uint16, device="cuda")
    st = m3.new_state()
    m3.sample_steps(out3, 0, 10, final=st)
    with pytest.raises(wavernn.WaveRNNError) as e:
        m3.sample_steps(out3, 10, 5, init=st, final=st)
    assert e.value.status == wavernn.E_UNSUPPORTED
    m3.device_status()
    m3.close()


@pytest.mark.parametrize("name", ["subscale16_h4", "subscale16_cnn"])
def test_benchmarked_subscale_call_in_pieces(name):
    """The benchmarked calls (WaveRNN-896, B = 16, 24,000 samples; future
    horizon 4, or F = 223 with the paper's CNN) run as five calls of their
    schedule make the one call's samples and state bit for bit."""
    w = synth.preset(name)
    N = w["samples"]
    feat = synth.features(1, N)
    m = wavernn.Model(w)
    fin = m.new_state()
    whole = host(m.sample(N, cond=cuda(feat), seed=11, final=fin))
    m.device_status()
    fin = {k: host(v) for k, v in fin.items() if k != "t0"}
    K = m.schedule_steps(N)
    bounds = [0, K // 7, K // 3, K // 2 + 1, K - 40, K]
    print(f"  {name}: {K} steps, bounds {bounds}", flush=True)
    out, st = run_in_pieces(m, 1, N, feat, 11, bounds)
    np.testing.assert_array_equal(out, whole)
    for k in ("h", "c", "f"):
        np.testing.assert_array_equal(st[k], fin[k], err_msg=k)
    m.close()
