"""Pins of the CPU oracle against things other than itself (CPU only).

Every pin here is a closed form, a special case that reduces to a library
routine (numpy's Philox, libm's exp/tanh in double, torch's bf16 cast), a
saturated-gate case whose result follows from Eq. 2 by inspection, or an
invariant that Eq. 2 / Eq. 4 imply.  A plausible slip in the oracle (gate order,
reset placement, a transposed R, a dropped bias or conditioning term, the I*
mask, the coarse/fine split, Philox counter layout, subscale masking) fails at
least one of them; ``test_oracle_mutants.py`` checks that claim.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O

N = 256


def zero_model(H=2, Dc=0, Dx=0, B=1, frame_len=120):
    Hh = H // 2
    d = dict(H=H, B=B, frame_len=frame_len,
             R=np.zeros((3, H, H), np.float32), I=np.zeros((3, H, 3), np.float32),
             b=np.zeros((3, H), np.float32),
             O1=np.zeros((Hh, Hh), np.float32), b1=np.zeros(Hh, np.float32),
             O2=np.zeros((N, Hh), np.float32), b2=np.zeros(N, np.float32),
             O3=np.zeros((Hh, Hh), np.float32), b3=np.zeros(Hh, np.float32),
             O4=np.zeros((N, Hh), np.float32), b4=np.zeros(N, np.float32),
             Wc=np.zeros((3 * H, Dc), np.float32) if Dc else None,
             Wx=np.zeros((3 * H, Dx), np.float32) if Dx else None)
    return d


def W(d):
    return O.Weights.from_dict(d)


def _counter_minus_one(t, stream):
    """The 256-bit little-endian counter (t, stream, 0, 0) minus one."""
    v = (t + (stream << 64) - 1) % 2**256
    return np.array([(v >> (64 * k)) & (2**64 - 1) for k in range(4)], dtype=np.uint64)


def numpy_uniforms(seed, stream, t):
    """Uniforms from numpy's independent Philox4x64-10 (it advances the counter
    before producing a block, so start one below)."""
    from numpy.random import Philox
    raw = Philox(key=seed, counter=_counter_minus_one(t, stream)).random_raw(4)
    return (int(raw[0]) >> 40) / 2.0**24, (int(raw[1]) >> 40) / 2.0**24


# ----------------------------------------------------------------------------- RNG

@pytest.mark.parametrize("seed,stream,t", [(1, 0, 1), (1, 0, 5), (7, 3, 123456), (2**63 + 5, 63, 2**40),
                                           (0, 1, 0), (1, 15, 1499)])
def test_philox_matches_numpy(seed, stream, t):
    from numpy.random import Philox
    ref = Philox(key=seed, counter=_counter_minus_one(t, stream)).random_raw(4)
    got = O.philox4x64_10([t, stream, 0, 0], [seed, 0])
    assert [int(x) for x in got] == [int(x) for x in ref]
    uc, uf = O.uniforms(seed, stream, t)
    assert (uc, uf) == numpy_uniforms(seed, stream, t)


# ------------------------------------------------------------------- elementary fns

def _ulp32(x):
    x = abs(float(x))
    return float(np.spacing(np.float32(x))) if x > 0 else float(np.spacing(np.float32(0)))


def test_exp_accuracy_and_specials():
    ys = np.concatenate([np.linspace(-86, 88, 60001), np.linspace(-1, 1, 20001),
                         np.array([0.5 * math.log(2) * k for k in range(-120, 120)])]).astype(np.float32)
    worst = 0.0
    for y in ys:
        got = O.exp(float(y))
        ref = math.exp(float(y))
        worst = max(worst, abs(got - ref) / _ulp32(ref))
    assert worst <= 2.0, worst
    assert O.exp(0.0) == 1.0
    assert O.exp(-87.0) == 0.0 and O.exp(-1000.0) == 0.0
    assert math.isinf(O.exp(89.0))


def test_sigmoid_tanh_accuracy():
    xs = np.concatenate([np.linspace(-85, 85, 40001), np.linspace(-2, 2, 20001)]).astype(np.float32)
    ws, wt_abs, wt_rel = 0.0, 0.0, 0.0
    for x in xs:
        x = float(x)
        s = O.sigmoid(x)
        ref = 1.0 / (1.0 + math.exp(-x))
        ws = max(ws, abs(s - ref) / _ulp32(ref))
        t = O.tanh(x)
        tr = math.tanh(x)
        wt_abs = max(wt_abs, abs(t - tr))
        if abs(x) >= 0.5:
            wt_rel = max(wt_rel, abs(t - tr) / _ulp32(tr))
        assert O.tanh(-x) == -t
    assert ws <= 4.0, ws
    assert wt_abs <= 4 * 2.0**-24, wt_abs
    assert wt_rel <= 4.0, wt_rel
    assert O.sigmoid(0.0) == 0.5 and O.tanh(0.0) == 0.0
    assert O.sigmoid(100.0) == 1.0 and O.sigmoid(-100.0) == 0.0


def test_scale_is_correctly_rounded():
    for v in range(256):
        exact = Fraction(2 * v - 255, 255)
        got = Fraction(O.scale(v))
        f = np.float32(float(exact))
        cands = [Fraction(float(np.nextafter(f, np.float32(-2)))), Fraction(float(f)),
                 Fraction(float(np.nextafter(f, np.float32(2))))]
        best = min(cands, key=lambda c: (abs(c - exact), c))
        assert got == best, v
    assert O.scale(0) == -1.0 and O.scale(255) == 1.0


def test_bf16_round_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    a = rng.standard_normal(100000).astype(np.float32) * 3
    # exact ties between two bf16 neighbours, both parities
    ties = (np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32)
    a = np.concatenate([a, ties, -ties, np.array([0.0, -0.0, 1e-40, 3e38], np.float32)])
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(O.bf16_round(a).view(np.uint32), ref.view(np.uint32))


# ------------------------------------------------------------------------- sampling

def test_draw_uniform_logits_is_floor_256u():
    z = np.zeros(N, np.float32)
    rng = np.random.default_rng(1)
    for q in list(rng.integers(0, 2**24, 3000)) + [0, 1, 2**24 - 1, 2**23, 65536 * 7]:
        u = q / 2.0**24
        assert O.draw(z, u) == math.floor(256 * u)


def test_draw_point_mass_and_zero_probability_classes():
    z = np.full(N, -1000.0, np.float32)
    z[77] = 3.0
    for u in (0.0, 0.3, 1 - 2**-24):
        assert O.draw(z, u) == 77
    # logits far above exp's range: the max shift keeps the weights finite
    z = np.full(N, 100.0, np.float32)
    z[200] = 200.0
    for u in (0.0, 0.5, 1 - 2**-24):
        assert O.draw(z, u) == 200
    # classes with zero weight are never drawn, even at the ends of [0, 1)
    z = np.full(N, -200.0, np.float32)
    z[10:20] = 0.0
    for u in (0.0, 1e-7, 0.5, 1 - 2**-24):
        k = O.draw(z, u)
        assert 10 <= k < 20


def test_draw_block_of_equal_classes_among_zero_probability_ones():
    """Logits +100 on the four classes 37..40 and -200 elsewhere (max shift and
    252 zero-probability classes): the running sums are 0 .. 0, 1, 2, 3, 4, so
    the class is 37 + floor(4 U) exactly, at both ends of [0, 1) too."""
    z = np.full(N, -200.0, np.float32)
    z[37:41] = 100.0
    for q in [0, 1, 2**22 - 1, 2**22, 2**23 + 5, 3 * 2**22, 2**24 - 1]:
        u = q / 2.0**24
        assert O.draw(z, u) == 37 + math.floor(4 * u)


def test_draw_distribution_chi_square():
    from scipy import stats
    rng = np.random.default_rng(5)
    z = (rng.standard_normal(N) * 2).astype(np.float32)
    p = np.exp(z.astype(np.float64) - z.max())
    p /= p.sum()
    n = 100000
    us = rng.integers(0, 2**24, n) / 2.0**24
    counts = np.bincount([O.draw(z, float(u)) for u in us], minlength=N)
    exp_c = p * n
    big = exp_c >= 5
    obs = np.append(counts[big], counts[~big].sum())
    ex = np.append(exp_c[big], exp_c[~big].sum())
    assert stats.chisquare(obs, ex).pvalue > 1e-4


# ---------------------------------------------------------------- closed-form runs

def test_zero_model_samples_are_floor_256u_and_nll_is_2ln256():
    d = zero_model(H=4)
    T = 500
    r = O.run(W(d), 1, T, seed=9)
    for t in range(T):
        uc, uf = numpy_uniforms(9, 0, t)
        assert r["out"][0, t] == 256 * math.floor(256 * uc) + math.floor(256 * uf), t
    tgt = np.random.default_rng(3).integers(0, 65536, (2, 300)).astype(np.uint16)
    r = O.run(W(d), 2, 300, target=tgt, nll=True, logits=True)
    assert np.all(r["zc"] == 0) and np.all(r["zf"] == 0)
    np.testing.assert_allclose(r["nll"], 2 * math.log(256), rtol=0, atol=1e-12)


def _point_mass_nll(hot):
    """-log P of class k under logits 40 at class ``hot`` and 0 elsewhere
    (closed form): log(1 + 255 e^-40) for the hot class, 40 more for any other."""
    base = math.log1p(255.0 * math.exp(-40.0))
    return lambda k: base if k == hot else 40.0 + base


def test_nll_and_samples_at_point_mass_logits():
    """Zero weights except the head biases: h stays 0 (u = r = 1/2, e = 0), so the
    logits are exactly b2 and b4 (Eq. 2 with relu(0) = 0).  b2 puts 40 on class
    c* = 3, b4 on f* = 200.  Free-running draws are (c*, f*) at every step, and
    the NLL of a target (c, f) is the closed form of each softmax: coarse and
    fine terms differ, so a coarse/fine mix-up changes the value."""
    d = zero_model(H=4)
    d["b2"][3] = 40.0
    d["b4"][200] = 40.0
    r = O.run(W(d), 1, 64, seed=5)
    assert np.all(r["out"] == 256 * 3 + 200)
    tgt = np.array([[256 * 3 + 200, 256 * 200 + 3, 256 * 3 + 7, 256 * 9 + 200, 0, 65535]], np.uint16)
    t = O.run(W(d), 1, tgt.shape[1], target=tgt, nll=True, logits=True)
    assert np.all(t["zc"][0] == d["b2"]) and np.all(t["zf"][0] == d["b4"])
    pc, pf = _point_mass_nll(3), _point_mass_nll(200)
    for k, u in enumerate(tgt[0]):
        want = pc(int(u) >> 8) + pf(int(u) & 255)
        assert abs(t["nll"][0, k] - want) <= 1e-12 * max(1.0, want), (k, t["nll"][0, k], want)


def test_nll_at_unequal_coarse_and_fine_distributions():
    """Two different non-uniform softmaxes with closed-form probabilities: the
    coarse logits are 2 on the 16 classes 32..47 and 0 elsewhere, the fine
    logits ln 3 on the 64 even classes below 128 and 0 elsewhere.  So
    P(c) = e^2 / (16 e^2 + 240) or 1 / (16 e^2 + 240), and
    P(f) = 3 / 448 or 1 / 448.  Sampled free-running, the class frequencies
    follow the same probabilities (binomial bound)."""
    d = zero_model(H=4)
    d["b2"][32:48] = 2.0
    d["b4"][0:128:2] = np.float32(math.log(3.0))
    zc2 = float(np.float32(2.0))
    l3 = float(np.float32(math.log(3.0)))
    Zc = 16 * math.exp(zc2) + 240
    Zf = 64 * math.exp(l3) + 192
    pc = lambda c: (math.exp(zc2) if 32 <= c < 48 else 1.0) / Zc
    pf = lambda f: (math.exp(l3) if (f < 128 and f % 2 == 0) else 1.0) / Zf
    rng = np.random.default_rng(8)
    tgt = rng.integers(0, 65536, (2, 400)).astype(np.uint16)
    tgt[0, :4] = [256 * 40 + 2, 256 * 2 + 40, 256 * 130 + 130, 256 * 47 + 127]
    t = O.run(W(d), 2, 400, target=tgt, nll=True)
    for s in range(2):
        for k in range(400):
            c, f = int(tgt[s, k]) >> 8, int(tgt[s, k]) & 255
            want = -math.log(pc(c)) - math.log(pf(f))
            assert abs(t["nll"][s, k] - want) <= 1e-12 * want, (s, k)
    r = O.run(W(d), 1, 20000, seed=3)["out"][0].astype(np.int64)
    n = len(r)
    for frac, p in ((np.mean((r >> 8 >= 32) & (r >> 8 < 48)), 16 * math.exp(zc2) / Zc),
                    (np.mean(((r & 255) < 128) & ((r & 255) % 2 == 0)), 64 * math.exp(l3) / Zf)):
        assert abs(frac - p) < 5 * math.sqrt(p * (1 - p) / n), (frac, p)


def test_zero_model_streams_use_their_own_philox_stream():
    d = zero_model(H=2)
    r = O.run(W(d), 5, 40, seed=3)
    for s in range(5):
        for t in range(40):
            uc, uf = numpy_uniforms(3, s, t)
            assert r["out"][s, t] == 256 * math.floor(256 * uc) + math.floor(256 * uf)


def test_update_gate_saturated_at_one_keeps_state():
    """u = sigma(100) rounds to exactly 1, so h_t = h_{t-1} (Eq. 2) whatever R, I, b_e."""
    rng = np.random.default_rng(0)
    d = zero_model(H=4)
    d["R"] = rng.standard_normal((3, 4, 4)).astype(np.float32) * 0.1
    d["R"][0] = 0
    d["I"] = rng.standard_normal((3, 4, 3)).astype(np.float32) * 0.1
    d["I"][0] = 0
    d["b"][0] = 100.0      # u
    d["b"][1] = -100.0     # r (so a u/r mix-up gives u = 0)
    d["b"][2] = 0.7
    h0 = np.array([[0.3, -0.7, 0.2, 0.9]], np.float32)
    r = O.run(W(d), 1, 7, seed=2, h0=h0)
    np.testing.assert_array_equal(r["h"], h0)


def _hand_heads(d):
    d["O1"][:] = 2.0
    d["b1"][:] = 0.1
    d["O2"][:, 0] = (np.arange(N) - 128) / 64.0
    d["b2"][:] = 0.01 * (np.arange(N) % 7)
    d["O3"][:] = -1.5
    d["b3"][:] = 0.3
    d["O4"][:, 0] = ((np.arange(N) % 13) - 6) / 8.0
    d["b4"][:] = 0.0


def _heads_ref(d, y_c, y_f):
    o1 = max(2.0 * y_c + 0.1, 0.0)
    o3 = max(-1.5 * y_f + 0.3, 0.0)
    zc = d["O2"][:, 0].astype(np.float64) * o1 + d["b2"]
    zf = d["O4"][:, 0].astype(np.float64) * o3 + d["b4"]
    return zc, zf


def test_hand_case_input_mask_and_heads():
    """u = r = 0: h = e = tanh(I*_e x + b_e).  The coarse unit must ignore its I*
    column 2 (set to 5 here); the fine unit sees c_t.  Heads by hand."""
    d = zero_model(H=2)
    d["b"][0] = -100.0
    d["b"][1] = -100.0
    d["b"][2] = [0.1, -0.2]
    d["I"][2, 0] = [0.5, -0.25, 5.0]
    d["I"][2, 1] = [0.5, -0.25, 0.75]
    _hand_heads(d)
    tgt = np.array([[200 * 256 + 17]], np.uint16)
    r = O.run(W(d), 1, 1, target=tgt, logits=True)
    x0, x1, x2 = 1 / 255, -1.0, 145 / 255
    e0 = math.tanh(0.5 * x0 - 0.25 * x1 + 0.1)
    e1 = math.tanh(0.5 * x0 - 0.25 * x1 + 0.75 * x2 - 0.2)
    np.testing.assert_allclose(r["h"][0], [e0, e1], rtol=2e-7, atol=1e-7)
    zc, zf = _heads_ref(d, e0, e1)
    np.testing.assert_allclose(r["zc"][0, 0], zc, rtol=1e-6, atol=1e-6)
    np.testing.assert_allclose(r["zf"][0, 0], zf, rtol=1e-6, atol=1e-6)


def test_hand_case_reset_gate_placement_and_R_orientation():
    """u = 0, r = (0.5, 0): e_i = tanh(r_i (R_e h)_i + b_e_i) with a non-symmetric R_e."""
    d = zero_model(H=2)
    d["b"][0] = -100.0
    d["b"][1] = [0.0, -100.0]
    d["b"][2] = [0.1, -0.2]
    d["R"][2] = [[1.0, 2.0], [3.0, 4.0]]
    d["I"][:, 0, 2] = 5.0      # masked, ignored
    _hand_heads(d)
    h0 = np.array([[0.3, -0.7]], np.float32)
    tgt = np.array([[0x8000]], np.uint16)
    r = O.run(W(d), 1, 1, target=tgt, h0=h0, logits=True)
    g = [0.3 * 1.0 + -0.7 * 2.0, 0.3 * 3.0 + -0.7 * 4.0]
    e = [math.tanh(0.5 * g[0] + 0.1), math.tanh(0.0 * g[1] - 0.2)]
    np.testing.assert_allclose(r["h"][0], e, rtol=2e-7, atol=1e-7)
    zc, zf = _heads_ref(d, e[0], e[1])
    np.testing.assert_allclose(r["zc"][0, 0], zc, rtol=1e-6, atol=1e-6)


def test_hand_case_update_gate_interpolates():
    """u = 0.5 exactly (zero pre-activation), r = 1 (b_r = 100), R = 0:
    h_t = 0.5 h_{t-1} + 0.5 tanh(b_e + I_e x); two steps by hand."""
    d = zero_model(H=2)
    d["b"][1] = 100.0
    d["b"][2] = [0.4, -0.3]
    d["I"][2, :, 1] = 0.2          # f_{t-1} column
    h0 = np.array([[0.8, -0.6]], np.float32)
    tgt = np.array([[0x1234, 0xff00]], np.uint16)
    r = O.run(W(d), 1, 2, target=tgt, h0=h0)
    h = np.array([0.8, -0.6])
    for t, fprev in enumerate([0, 0x34]):
        x1 = (2 * fprev - 255) / 255
        e = np.tanh(np.array([0.4, -0.3]) + 0.2 * x1)
        h = 0.5 * h + 0.5 * e
    np.testing.assert_allclose(r["h"][0], h, rtol=1e-6, atol=1e-7)


def test_hand_case_conditioning_frames():
    """u = 0, r = 1, R = I = 0: h_t = tanh(W_cond,e . feat[floor(t/3)] + b_e).
    Only the e rows of W_cond are nonzero."""
    d = zero_model(H=2, Dc=2, frame_len=3)
    d["b"][0] = -100.0
    d["b"][1] = 100.0
    d["b"][2] = [0.05, -0.05]
    d["Wc"][4] = [0.5, -0.5]
    d["Wc"][5] = [1.0, 0.25]
    feat = np.array([[[0.2, 0.4], [-0.6, 0.1], [1.0, 1.0]]], np.float32)
    tgt = np.zeros((1, 8), np.uint16)
    hs = []
    for T in range(1, 9):
        hs.append(O.run(W(d), 1, T, feat=feat, target=tgt[:, :T])["h"][0].copy())
    for t in range(8):
        fr = feat[0, min(t // 3, 2)].astype(np.float64)
        ref = [math.tanh(0.5 * fr[0] - 0.5 * fr[1] + 0.05), math.tanh(fr[0] + 0.25 * fr[1] - 0.05)]
        np.testing.assert_allclose(hs[t], ref, rtol=1e-6, atol=1e-7)


# ------------------------------------------------------------------------ invariants

def _random_tiny(H=16, Dc=0, seed=0):
    from paper_1802_08435_amd import synth
    return synth.make_weights(H, seed=seed, cond_dim=Dc)


def test_coarse_logits_do_not_depend_on_current_coarse_byte():
    d = _random_tiny()
    rng = np.random.default_rng(8)
    a = rng.integers(0, 65536, (1, 120)).astype(np.uint16)
    b = a.copy()
    b[0, 50] = (int(b[0, 50]) + 256 * 77) % 65536       # change only c_50
    ra = O.run(W(d), 1, 120, target=a, logits=True)
    rb = O.run(W(d), 1, 120, target=b, logits=True)
    np.testing.assert_array_equal(ra["zc"][0, :51], rb["zc"][0, :51])
    np.testing.assert_array_equal(ra["zf"][0, :50], rb["zf"][0, :50])
    assert not np.array_equal(ra["zf"][0, 50], rb["zf"][0, 50])
    assert not np.array_equal(ra["zc"][0, 51], rb["zc"][0, 51])


def test_softmax_of_logits_sums_to_one():
    d = _random_tiny()
    r = O.run(W(d), 1, 200, logits=True)
    for z in (r["zc"][0], r["zf"][0]):
        w = np.array([[O.exp(float(v - row.max())) for v in row] for row in z[:20]], np.float64)
        p = w / w.sum(axis=1, keepdims=True)
        np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-12)
        assert np.all(w.max(axis=1) == 1.0)


def test_chunked_sampling_equals_one_call():
    d = _random_tiny(Dc=8)
    from paper_1802_08435_amd import synth
    feat = synth.features(2, 1300, cond_dim=8)
    full = O.run(W(d), 2, 1300, feat=feat, seed=4)
    a = O.run(W(d), 2, 700, feat=feat, seed=4)
    b = O.run(W(d), 2, 600, feat=feat, seed=4, h0=a["h"], c0=a["c"], f0=a["f"], t0=700)
    np.testing.assert_array_equal(np.concatenate([a["out"], b["out"]], axis=1), full["out"])
    np.testing.assert_array_equal(b["h"], full["h"])


def test_subscale_without_context_is_interleaved_plain_streams():
    """Eq. 4 fold/unfold: with W_ctx = 0, lane s of a B = 16 subscale run is a
    plain run on Philox stream s, and the output interleaves the lanes."""
    d = _random_tiny(H=16)
    ds = dict(d, B=16, Wx=np.zeros((48, 256), np.float32))
    T = 16 * 60
    sub = O.run(W(ds), 1, T, seed=6)["out"][0]
    plain = O.run(W(d), 16, 60, seed=6)["out"]
    np.testing.assert_array_equal(sub.reshape(60, 16).T, plain)


@pytest.mark.parametrize("j", [0, 5, 15])
def test_subscale_context_masks_samples_of_the_current_row(j):
    """Only context pair j is wired (W_ctx columns 2j, 2j+1).  Lane s at row i
    sees sample 16i+s-1-j only if it was made in an earlier row, i.e. j >= s."""
    d = _random_tiny(H=16)
    T = 16 * 12
    base = dict(d, B=16, Wx=np.zeros((48, 256), np.float32))
    wired = dict(base, Wx=base["Wx"].copy())
    wired["Wx"][:, 2 * j:2 * j + 2] = 0.8
    a = O.run(W(base), 1, T, seed=2)["out"][0].reshape(12, 16)
    b = O.run(W(wired), 1, T, seed=2)["out"][0].reshape(12, 16)
    for s in range(16):
        if j >= s:
            assert not np.array_equal(a[:, s], b[:, s]), s
        else:
            np.testing.assert_array_equal(a[:, s], b[:, s])


def _horizon_model(B, F, Dx, H=8):
    d = _random_tiny(H=H)
    return W(dict(d, B=B, F=F, Wx=np.zeros((3 * H, Dx), np.float32)))


def _pairs(seq, idx):
    """Expected context: (c, f) scaled of seq[q] for each q, zeros for None."""
    out = []
    for q in idx:
        out += [0.0, 0.0] if q is None else [O.scale(int(seq[q]) >> 8), O.scale(int(seq[q]) & 255)]
    return np.array(out, np.float32)


@pytest.mark.parametrize("B,F,Dx,s,i,idx", [
    # Sec. 4.1-4.2 by hand: the context of sample 4i + s holds the previous sub-tensors
    # z < s up to position i + F; the window is Dx/4 samples before n, then Dx/4 after.
    (4, 1, 8, 2, 1, [5, 4, None, 8]),            # n = 6: 5 (z1), 4 (z0); 7 is z3 > s; 8 = (k2, z0), k <= 2
    (4, 1, 8, 0, 2, [None, None, None, None]),   # n = 8: sub-tensor 0 sees no other sub-tensor
    (4, 1, 8, 3, 1, [6, 5, 8, 9]),               # n = 7: future 8, 9 of z0, z1 at k = 2 <= 2
    (4, 1, 8, 3, 2, [10, 9, 12, 13]),            # n = 11: future 12, 13 at k = 3 <= i + F = 3
    (4, 0, 8, 3, 2, [10, 9, None, None]),        # F = 0: k = 3 > 2 is beyond the horizon
    (4, 1, 8, 1, 0, [0, None, None, None]),      # n = 1: q = -1 does not exist
    (4, 1, 8, 2, 3, [13, 12, None, None]),       # n = 14: 15 is z3; 16 is past the end (N = 16)
    (4, 1, 16, 1, 2, [8, None, None, None, None, None, 12, None]),   # n = 9: own past 5 and own future 13 unseen
])
def test_subscale_horizon_context_hand_cases(B, F, Dx, s, i, idx):
    w = _horizon_model(B, F, Dx)
    seq = (np.arange(16) * 4099 + 77) % 65536
    np.testing.assert_array_equal(O.subscale_context(w, seq.astype(np.uint16), s, i), _pairs(seq, idx))


def test_subscale_horizon_without_context_is_interleaved_plain_streams():
    """With W_ctx = 0 the order of generation does not matter: the horizon-F
    run equals the lockstep run and B interleaved plain streams."""
    d = _random_tiny(H=16)
    Wx = np.zeros((48, 256), np.float32)
    lag = O.run(W(dict(d, B=16, F=3, Wx=Wx)), 1, 16 * 40, seed=6)["out"][0]
    lock = O.run(W(dict(d, B=16, Wx=Wx)), 1, 16 * 40, seed=6)["out"][0]
    plain = O.run(W(d), 16, 40, seed=6)["out"]
    np.testing.assert_array_equal(lag, lock)
    np.testing.assert_array_equal(lag.reshape(40, 16).T, plain)


@pytest.mark.parametrize("F", [0, 1, 3])
def test_subscale_horizon_dependencies_precede_in_the_lagged_schedule(F):
    """Brute force on a tiny model: change one target sample q = B k + z and see
    which teacher-forced logits move.  Under the batched schedule of Sec. 4.2
    sub-tensor s runs position i at step i + s (F + 1 + A), with the context
    formed A >= 0 steps ahead: every sample of its own sub-tensor a logit
    depends on is made at an earlier step, every sample of another sub-tensor
    at least A + 1 steps earlier, for A = 0 and A = 1, and some sample of an
    earlier sub-tensor from the logit's future (within F, so only for F > 0:
    with F = 0 every sample an earlier sub-tensor has made up to position i
    precedes B i + s in time) must matter."""
    B, N, H, Dx = 4, 48, 8, 16
    d = _random_tiny(H=H)
    rng = np.random.default_rng(5)
    Wx = (rng.standard_normal((3 * H, Dx)) * 0.6).astype(np.float32)
    w = W(dict(d, B=B, F=F, Wx=Wx))
    tgt = rng.integers(0, 65536, size=(1, N)).astype(np.uint16)
    base = O.run(w, 1, N, target=tgt, logits=True)
    step = lambda n, A: n // B + (n % B) * (F + 1 + A)
    future_dep = False
    for q in range(N):
        t2 = tgt.copy()
        t2[0, q] ^= 0x8181
        r = O.run(w, 1, N, target=t2, logits=True)
        moved = (np.abs(r["zc"][0] - base["zc"][0]).max(axis=1) > 0) | (np.abs(r["zf"][0] - base["zf"][0]).max(axis=1) > 0)
        for n in np.flatnonzero(moved):
            if n == q:
                continue            # its own fine logits see its own coarse byte
            for A in (0, 1):
                gap = 1 if q % B == n % B else A + 1
                assert step(q, A) <= step(n, A) - gap, (q, n, A)
            future_dep |= q > n
    assert future_dep == (F > 0)


def test_pruned_blocks_equal_dense_with_zeroed_blocks():
    """Sparse WaveRNN (Sec. 3): pruned weights are exactly zero, so the dense
    oracle on the masked matrix is the sparse model.  Zeroing one more block
    changes only the gates it feeds."""
    from paper_1802_08435_amd import synth
    d = synth.make_weights(32, seed=1, block=(4, 4), density=0.25)
    m = d["mask"]
    assert m.shape == (3, 8, 8) and int(m.sum()) == 3 * 16
    full = np.repeat(np.repeat(m, 4, axis=1), 4, axis=2)
    assert np.all(d["R"][full == 0] == 0) and np.all(d["R"][full == 1] != 0)
    r = O.run(W(d), 1, 300, seed=1)
    assert r["out"].shape == (1, 300)


def test_wavernn896_parameter_count_matches_the_paper():
    """Sec. 2.1: WaveRNN-896 has about 3M parameters, and streaming them for
    each of 24,000 samples at 4 bytes each is about 288 GB.  The shapes read
    from Eq. 2 (R 3H x H, O1/O3 Hh x Hh, O2/O4 256 x Hh) must give that count."""
    from paper_1802_08435_amd import synth
    w = synth.preset("dense896")
    n = sum(w[k].size for k in ("R", "O1", "O2", "O3", "O4"))
    assert n == 3 * 896 * 896 + 2 * 448 * 448 + 2 * 256 * 448
    assert abs(n - 3e6) / 3e6 < 0.02
    assert abs(n * 24e3 * 4 / 1e9 - 288) / 288 < 0.02


# ------------------------------------------------- Fused Subscale WaveRNN 2x (Sec. 4.4)

def fused_model(H=8, F=2, seed=0, scale=1.0):
    Q = H // 4
    rng = np.random.default_rng(seed)
    g = lambda *s: (scale * rng.normal(0, 1.0 / math.sqrt(s[-1]), s)).astype(np.float32)
    return dict(H=H, F=F, R=g(3, H, H), I=g(3, H, 6), b=g(3, H, 1)[..., 0] * 0.3,
                O1=g(4, Q, Q), b1=g(4, Q, 1)[..., 0] * 0.3, O2=g(4, 2, 16, Q), b2=g(4, 2, 16, 1)[..., 0] * 0.3)


def fused_zero_model(H=8, F=2):
    d = fused_model(H, F)
    return {k: (np.zeros_like(v) if isinstance(v, np.ndarray) else v) for k, v in d.items()}


def numpy_words(seed, stream, t):
    from numpy.random import Philox
    return [int(x) >> 40 for x in Philox(key=seed, counter=_counter_minus_one(t, stream)).random_raw(4)]


def test_fused_zero_model_nibbles_are_floor_16u_and_nll_is_4ln16():
    """All weights zero: every nibble softmax is uniform, so sample 2 i + s of
    utterance u is built from floor(16 U) of the four Philox words of
    counter (i, 2 u + s) (coarse high, coarse low, fine high, fine low), and
    each sample costs 4 ln 16 nats."""
    d = fused_zero_model()
    S, N = 2, 60
    r = O.fused_run(d, S, N, seed=11)
    for u in range(S):
        for n in range(N):
            i, s = divmod(n, 2)
            w = numpy_words(11, 2 * u + s, i)
            nib = [math.floor(16 * (x / 2.0**24)) for x in w]
            assert r["out"][u, n] == 256 * (16 * nib[0] + nib[1]) + 16 * nib[2] + nib[3], (u, n)
    tgt = np.random.default_rng(2).integers(0, 65536, (S, N)).astype(np.uint16)
    t = O.fused_run(d, S, N, target=tgt)
    assert np.all(t["zc"] == 0) and np.all(t["zf"] == 0)
    np.testing.assert_allclose(t["nll"], 4 * math.log(16), rtol=0, atol=1e-12)


def test_fused_nll_at_point_mass_nibbles():
    """Fused model with zero weights except the nibble biases b2: the state stays
    0, so each nibble's logits are exactly its bias row.  Head k = 2 level + s
    puts 40 on high nibble (1 + k) and on low nibble (14 - 3k).  Free-running,
    every byte is that pair; the NLL of a target is the sum over the four
    nibbles of the point-mass closed form (log(1 + 15 e^-40), 40 more off the
    hot nibble), which a high/low or coarse/fine mix-up changes."""
    d = fused_zero_model(H=8, F=2)
    hot = {}
    for k in range(4):
        hot[(k, 0)], hot[(k, 1)] = 1 + k, 14 - 3 * k
        d["b2"][k, 0, hot[(k, 0)]] = 40.0
        d["b2"][k, 1, hot[(k, 1)]] = 40.0
    S, N = 1, 40
    r = O.fused_run(d, S, N, seed=2)
    for n in range(N):
        s = n % 2
        c, f = int(r["out"][0, n]) >> 8, int(r["out"][0, n]) & 255
        assert (c >> 4, c & 15, f >> 4, f & 15) == (hot[(s, 0)], hot[(s, 1)], hot[(2 + s, 0)], hot[(2 + s, 1)]), n
    base = math.log1p(15.0 * math.exp(-40.0))
    pm = lambda k, part, v: base if v == hot[(k, part)] else 40.0 + base
    rng = np.random.default_rng(6)
    tgt = rng.integers(0, 65536, (S, N)).astype(np.uint16)
    tgt[0, 0] = 256 * (16 * hot[(0, 0)] + hot[(0, 1)]) + 16 * hot[(2, 0)] + hot[(2, 1)]
    tgt[0, 1] = 256 * (16 * hot[(1, 1)] + hot[(1, 0)]) + 16 * hot[(3, 0)] + hot[(3, 1)]
    t = O.fused_run(d, S, N, target=tgt)
    for n in range(N):
        s = n % 2
        c, f = int(tgt[0, n]) >> 8, int(tgt[0, n]) & 255
        want = pm(s, 0, c >> 4) + pm(s, 1, c & 15) + pm(2 + s, 0, f >> 4) + pm(2 + s, 1, f & 15)
        assert abs(t["nll"][0, n] - want) <= 1e-12 * max(1.0, want), (n, t["nll"][0, n], want)


@pytest.mark.parametrize("s", [0, 1])
def test_fused_state_reduces_to_the_plain_oracle(s):
    """With the input columns of the other sub-tensor zero (and c_s,t kept
    from the other fine quarter), the fused state is the plain WaveRNN's
    state driven by sub-tensor s alone: sub-tensor 0 from step 0, idle (its
    last sample repeated) for the last F + 1 steps; sub-tensor 1 idle on
    silence (128, 0) for the first F + 1 steps.  The plain oracle is pinned
    on its own; this fixes the fused schedule, input layout and masks."""
    H, F, N = 8, 2, 40
    Q, rows = H // 4, N // 2
    rng = np.random.default_rng(5 + s)
    d = fused_model(H, F, seed=7 + s)
    Ip = rng.normal(0, 0.7, (3, H, 3)).astype(np.float32)     # plain columns c_{t-1}, f_{t-1}, c_t
    # the plain model's fine half is [2Q, 4Q); the fine quarter of the other
    # sub-tensor must not see c_t
    Ip[:, (3 * Q if s == 0 else 2 * Q):(4 * Q if s == 0 else 3 * Q), 2] = 0.0
    If = rng.normal(0, 0.7, (3, H, 6)).astype(np.float32)
    own, other = ((0, 1, 4), (2, 3, 5)) if s == 0 else ((2, 3, 5), (0, 1, 4))
    for k in range(3):
        If[:, :, own[k]] = Ip[:, :, k]
        If[:, :, other[k]] = 0.0
    If[:, :2 * Q, own[2]] = 5.0                                 # coarse units ignore c_t (mask)
    If[:, (2 * Q if s == 0 else 3 * Q):(3 * Q if s == 0 else 4 * Q), other[2]] = 5.0   # own fine quarter ignores the other c_t
    assert np.abs(If[:, :, own[2]]).max() > 0
    d["I"] = If
    tgt = rng.integers(0, 65536, (1, N)).astype(np.uint16)
    fused = O.fused_run(d, 1, N, target=tgt)
    seq = tgt[0, s::2]
    if s == 0:
        plain_t = np.concatenate([seq, np.full(F + 1, seq[-1], np.uint16)])
    else:
        plain_t = np.concatenate([np.full(F + 1, 128 * 256, np.uint16), seq])
    p = zero_model(H=H)
    p.update(R=d["R"], I=Ip, b=d["b"])
    plain = O.run(W(p), 1, rows + F + 1, target=plain_t[None, :])
    np.testing.assert_array_equal(fused["h"][0], plain["h"][0])


@pytest.mark.parametrize("k", [0, 1, 2, 3])
def test_fused_heads_read_their_own_quarter(k):
    """Head k = 2 level + s reads quarter k of the state and feeds the two
    nibbles of byte (level) of sub-tensor s.  h is pinned by the gates
    (u = 0, r = 0: h = tanh(b_e)), positive on quarter k only, and head j
    turns a positive input into a near point mass on nibbles (3 + j, 12 - j);
    every other head sees zeros and draws uniform nibbles."""
    H, Q, N = 8, 2, 400
    d = fused_zero_model(H)
    d["b"][0] = -100.0
    d["b"][1] = -100.0
    d["b"][2] = -2.0
    d["b"][2, k * Q:(k + 1) * Q] = 2.0
    for j in range(4):
        d["O1"][j] = np.eye(Q, dtype=np.float32)
        d["O2"][j, 0, 3 + j] = 40.0
        d["O2"][j, 1, 12 - j] = 40.0
    r = O.fused_run(d, 1, N, seed=4)
    level, s = divmod(k, 2)
    byte = (r["out"][0, s::2] >> (8 if level == 0 else 0)) & 255
    assert np.all(byte == 16 * (3 + k) + (12 - k))
    other = (r["out"][0, (1 - s)::2] >> (8 if level == 0 else 0)) & 255
    assert np.mean(other == 16 * (3 + k) + (12 - k)) < 0.05


@pytest.mark.parametrize("F", [0, 2])
def test_fused_dependencies_follow_the_fused_order(F):
    """Brute force on a tiny model (teacher-forced; change one sample, see
    which logits move).  Position i of sub-tensor s is made at step
    tau = i + s (F + 1).  Coarse logits of a sample depend exactly on the
    samples made at earlier steps; fine logits also on the sample's own
    coarse byte, and on nothing else of its own step.  Hence sub-tensor 1 at
    position i sees sub-tensor 0 up to position i + F, not i + F + 1."""
    H, N = 8, 24
    d = fused_model(H, F, seed=21, scale=2.0)
    rng = np.random.default_rng(9)
    tgt = rng.integers(0, 65536, (1, N)).astype(np.uint16)
    base = O.fused_run(d, 1, N, target=tgt)
    tau = lambda n: n // 2 + (n % 2) * (F + 1)
    for n in range(N):
        t2 = tgt.copy()
        t2[0, n] ^= 0x8181                                   # both bytes change
        r = O.fused_run(d, 1, N, target=t2)
        dc = np.abs(r["zc"][0] - base["zc"][0]).max(axis=1) > 0
        df = np.abs(r["zf"][0] - base["zf"][0]).max(axis=1) > 0
        for m in range(N):
            assert dc[m] == (tau(n) < tau(m)), (n, m, "coarse")
            assert df[m] == (tau(n) < tau(m) or n == m), (n, m, "fine")
    # the horizon, read off the schedule the test just checked
    assert all(tau(2 * (i + F)) < tau(2 * i + 1) <= tau(2 * (i + F + 1)) for i in range(N // 2 - F - 1))


# ------------------------------- subscale conditioning network (Sec. 4.1, 5): masked dilated CNN

def cnn_model(B=4, Rc=6, Cc=5, Dx=3, layers=10, seed=0):
    rng = np.random.default_rng(seed)
    g = lambda *s: rng.normal(0, 1.0 / math.sqrt(s[-1]), s).astype(np.float32)
    return dict(B=B, layers=layers, Win=g(Rc, 2 * B), bin=g(Rc, 1)[:, 0], Wc=g(layers, Cc, 3, Rc),
                bc=np.full((layers, Cc), 0.5, np.float32), Wo=g(layers, Rc, Cc), bo=g(layers, Rc, 1)[..., 0],
                Wp=g(Dx, Rc), bp=g(Dx, 1)[:, 0])


@pytest.mark.parametrize("layers", [1, 2, 5, 10])
def test_cnn_shift_layers_sum_the_future_rows(layers):
    """One channel carried through: input c of sub-tensor 0 (positive), every
    layer adds r at the row 2d ahead (tap 2, weight 1; relu passes positives),
    so with dilations 1, 2, 4, 8, 16 the output of row k is the sum of x over
    rows k, k + 2, ..., k + 2 (2^layers - 1) (rows past the end are zero)."""
    B, Rc, Cc, Dx, rows = 2, 1, 1, 1, 80
    m = dict(B=B, layers=layers, Win=np.zeros((Rc, 2 * B), np.float32), bin=np.zeros(Rc, np.float32),
             Wc=np.zeros((layers, Cc, 3, Rc), np.float32), bc=np.zeros((layers, Cc), np.float32),
             Wo=np.ones((layers, Rc, Cc), np.float32), bo=np.zeros((layers, Rc), np.float32),
             Wp=np.ones((Dx, Rc), np.float32), bp=np.zeros(Dx, np.float32))
    m["Win"][0, 0] = 1.0                                         # c of sub-tensor 0
    m["Wc"][:, 0, 2, 0] = 1.0                                    # the tap 2d ahead
    rng = np.random.default_rng(layers)
    seq = rng.integers(128 * 256, 65536, rows * B).astype(np.uint16)   # c >= 128: scaled c > 0
    out = O.ctx_cnn(m, seq, 1)[:, 0]
    xc = np.array([O.scale(int(v) >> 8) for v in seq[0::B]], np.float64)
    span = 2 * (2 ** min(layers, 5) - 1) if layers <= 5 else None
    for k in range(rows):
        if layers <= 5:
            want = sum(xc[k + j] for j in range(0, span + 1, 2) if k + j < rows)
        else:   # layers 6..10 repeat the dilations: offsets are sums of two such sets
            offs = [a + b for a in range(0, 63, 2) for b in range(0, 2 * (2 ** (layers - 5) - 1) + 1, 2)]
            want = sum(xc[k + j] for j in offs if k + j < rows)
        assert abs(out[k] - want) <= 1e-5 * max(1.0, abs(want)), (layers, k, out[k], want)


def test_cnn_sees_only_previous_sub_tensors_within_124_rows_ahead():
    """Brute force: change one sample (row k, sub-tensor z); the conditioning
    of sub-tensor s moves exactly at rows k - 124 .. k when z < s, nowhere
    when z >= s (the mask over sub-tensors, the future taps, ten layers)."""
    m = cnn_model()
    B, rows, s = 4, 150, 2
    rng = np.random.default_rng(4)
    seq = rng.integers(0, 65536, rows * B).astype(np.uint16)
    base = O.ctx_cnn(m, seq, s)
    for k, z in [(0, 0), (60, 1), (149, 0), (130, 1), (70, 2), (70, 3)]:
        q = seq.copy()
        q[B * k + z] ^= 0x8080
        moved = np.flatnonzero(np.abs(O.ctx_cnn(m, q, s) - base).max(axis=1) > 0)
        want = np.arange(max(0, k - 124), k + 1) if z < s else np.array([], int)
        np.testing.assert_array_equal(moved, want, err_msg=f"k={k} z={z}")


def test_cnn_first_sub_tensor_sees_nothing():
    m = cnn_model()
    seq = np.random.default_rng(5).integers(0, 65536, 4 * 40).astype(np.uint16)
    out = O.ctx_cnn(m, seq, 0)
    zero = O.ctx_cnn(m, np.full_like(seq, 128 * 256), 0)
    np.testing.assert_array_equal(out, zero)


def _cnn_subscale(B=3, H=8, Dx=4, layers=2, seed=11):
    """A tiny subscale WaveRNN (head biases positive, so the heads' relus pass)
    conditioned by a tiny CNN (reach 2 + 4 = 6 rows)."""
    rng = np.random.default_rng(seed)
    d = zero_model(H=H, Dx=Dx, B=B)
    for k in ("R", "I", "b", "O1", "O2", "b2", "O3", "O4", "b4", "Wx"):
        d[k] = (rng.normal(0, 1.5, d[k].shape) / math.sqrt(max(1, d[k].shape[-1]))).astype(np.float32)
    d["b1"][:] = 1.0
    d["b3"][:] = 1.0
    d["F"] = 6
    d["cnn"] = cnn_model(B=B, Rc=5, Cc=4, Dx=Dx, layers=layers, seed=seed + 1)
    return d


def test_cnn_conditioned_subscale_dependencies():
    """Brute force on the CNN-conditioned Subscale WaveRNN (teacher-forced):
    change one sample (sub-tensor z, row k) and see which logits move.  Those
    of sub-tensor s at position i move exactly when z < s and the change
    reaches s's conditioning at some row j <= i (the CNN's own dependencies,
    pinned above: rows k - 6 .. k here; earlier rows reach position i through
    the state: Fig. 3's unbounded past, future horizon tied to the CNN's
    receptive field), or z = s and k < i (its own past); the fine logits also
    at k = i (the sample's own coarse byte).  Nothing else: not the sample's
    own future, not a later sub-tensor."""
    d = _cnn_subscale()
    B, rows = 3, 12
    N = B * rows
    rng = np.random.default_rng(2)
    tgt = rng.integers(0, 65536, (1, N)).astype(np.uint16)
    base = O.run(W(d), 1, N, target=tgt, logits=True)
    cb = [O.ctx_cnn(d["cnn"], tgt[0], s_) for s_ in range(B)]
    for q in range(N):
        t = tgt.copy()
        t[0, q] ^= 0x8181
        r = O.run(W(d), 1, N, target=t, logits=True)
        k, z = divmod(q, B)
        first = [np.flatnonzero(np.abs(O.ctx_cnn(d["cnn"], t[0], s_) - cb[s_]).max(axis=1) > 0) for s_ in range(B)]
        for n in range(N):
            i, s_ = divmod(n, B)
            dep = (z < s_ and len(first[s_]) > 0 and first[s_].min() <= i) or (z == s_ and k < i)
            mc = np.abs(r["zc"][0, n] - base["zc"][0, n]).max() > 0
            mf = np.abs(r["zf"][0, n] - base["zf"][0, n]).max() > 0
            assert mc == dep, ("coarse", q, n)
            assert mf == (dep or q == n), ("fine", q, n)


def test_cnn_with_zero_output_is_the_plain_subscale_model():
    """A CNN whose output layer is zero gives every sub-tensor a zero context:
    the run equals the same subscale model without context, which is the
    interleaving of plain per-sub-tensor streams (pinned separately)."""
    d = _cnn_subscale()
    d["cnn"]["Wp"][:] = 0.0
    d["cnn"]["bp"][:] = 0.0
    plain = {k: v for k, v in d.items() if k not in ("cnn", "Wx")}
    a = O.run(W(d), 2, 36, seed=4, nll=True)
    b = O.run(W(plain), 2, 36, seed=4, nll=True)
    np.testing.assert_array_equal(a["out"], b["out"])
    np.testing.assert_array_equal(a["h"], b["h"])


def test_cnn_relu_clips_a_negative_layer():
    """The shift network of one layer with bias -10 on the convolution: every
    pre-activation is below zero (|x| <= 1), relu gives 0, and the residual
    passes the input row through unchanged."""
    B, rows = 2, 30
    m = dict(B=B, layers=1, Win=np.zeros((1, 2 * B), np.float32), bin=np.zeros(1, np.float32),
             Wc=np.zeros((1, 1, 3, 1), np.float32), bc=np.full((1, 1), -10.0, np.float32),
             Wo=np.ones((1, 1, 1), np.float32), bo=np.zeros((1, 1), np.float32),
             Wp=np.ones((1, 1), np.float32), bp=np.zeros(1, np.float32))
    m["Win"][0, 0] = 1.0
    m["Wc"][0, 0, 2, 0] = 1.0
    seq = np.random.default_rng(8).integers(0, 65536, rows * B).astype(np.uint16)
    out = O.ctx_cnn(m, seq, 1)[:, 0]
    np.testing.assert_array_equal(out, np.array([O.scale(int(v) >> 8) for v in seq[0::B]], np.float32))


def test_lane_subset_equals_the_full_teacher_forced_run():
    """With a target the subscale lanes are independent: a run over lanes
    [2, 4) reproduces those lanes of the full run bit for bit, lockstep and
    with a horizon (the test path that replays long subscale calls)."""
    for F in (-1, 1):
        d = zero_model(H=4, Dx=8, B=5)
        rng = np.random.default_rng(9)
        for k in ("R", "I", "b", "O1", "O2", "O3", "O4", "Wx"):
            d[k] = rng.normal(0, 0.7, d[k].shape).astype(np.float32)
        d["F"] = F
        tgt = rng.integers(0, 65536, (2, 40)).astype(np.uint16)
        full = O.run(W(d), 2, 40, target=tgt, logits=True, nll=True)
        part = O.run_lanes(W(d), 2, 40, tgt, (2, 4))
        for s_ in range(5):
            idx = np.arange(s_, 40, 5)
            if 2 <= s_ < 4:
                np.testing.assert_array_equal(part["zc"][:, idx], full["zc"][:, idx])
                np.testing.assert_array_equal(part["nll"][:, idx], full["nll"][:, idx])
            else:
                assert not part["zc"][:, idx].any()
