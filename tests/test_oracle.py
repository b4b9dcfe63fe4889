"""Pins for the CPU oracle: it is checked against what the paper and the
mathematics fix, never against itself.

  * closed forms: H H^T = K I, FWHT(FWHT(x)) = K x, FWHT(e_j) = row j of H;
  * a library routine: scipy's Sylvester Hadamard matrix and a dense product;
  * identities the paper states: (XR)(R^-1 W) = XW (Fig. 2(a)) and
    (X diag(s)^-1)(diag(s) W) = XW (Section 2.2), in binary64;
  * the single-spike worked example of Eq. 4 and the multi-spike form of
    Appendix A.1 (exact with epsilon = 0);
  * hand-worked fixtures under tests/golden/;
  * special cases that reduce to textbook routines (plain per-token RTN,
    naive Runtime Smooth of Eq. 1-3, an integer GEMM when s = 1);
  * brute-force integer triple loops for the grouped partial sums.
"""
import json
import os

import numpy as np
import pytest
import scipy.linalg

import synth
from oracle import rrs_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- Hadamard / FWHT

@pytest.mark.parametrize("K", [1, 2, 4, 8, 64, 512, 1024])
def test_hadamard_is_sylvester(K):
    np.testing.assert_array_equal(O.hadamard(K), scipy.linalg.hadamard(K).astype(np.float64))


@pytest.mark.parametrize("K", [2, 16, 512, 2048])
def test_hadamard_orthogonal(K):
    H = O.hadamard(K)
    np.testing.assert_array_equal(H @ H.T, K * np.eye(K))


@pytest.mark.parametrize("K", [4096, 8192, 16384])
def test_fwht_rows_orthogonal_large(K):
    # Rows of H_K obtained as FWHT(e_j) for sampled j: pairwise products = K I.
    rng = np.random.default_rng(K)
    idx = rng.choice(K, 24, replace=False)
    E = np.zeros((len(idx), K))
    E[np.arange(len(idx)), idx] = 1.0
    rows = O.fwht(E, "fp64")
    assert set(np.unique(rows)) <= {-1.0, 1.0}
    np.testing.assert_array_equal(rows @ rows.T, K * np.eye(len(idx)))
    # Sylvester entry: H[i, j] = (-1)^popcount(i & j).
    j = np.arange(K)
    for r, i in zip(rows, idx):
        pc = np.array([bin(int(i) & int(t)).count("1") for t in j])
        np.testing.assert_array_equal(r, (-1.0) ** pc)


@pytest.mark.parametrize("K", [2, 8, 128, 1024])
def test_fwht_equals_dense_product(K):
    rng = np.random.default_rng(K + 1)
    x = rng.integers(-1000, 1000, size=(5, K)).astype(np.float64)
    H = scipy.linalg.hadamard(K).astype(np.float64)
    np.testing.assert_array_equal(O.fwht(x, "fp64"), x @ H)
    # Column form (axis 0) used for the weights: H W.
    w = rng.integers(-1000, 1000, size=(K, 3)).astype(np.float64)
    np.testing.assert_array_equal(O.fwht(w, "fp64", axis=0), H @ w)


@pytest.mark.parametrize("K", [512, 4096])
def test_fwht_involution(K):
    rng = np.random.default_rng(3)
    x = rng.integers(-2000, 2000, size=(4, K)).astype(np.float64)
    np.testing.assert_array_equal(O.fwht(O.fwht(x, "fp64"), "fp64"), K * x)


def test_fwht_fp16_inputs_exact_in_fp64():
    # fp16 inputs need at most 53 significant bits after 13 stages (K <= 8192).
    K = 8192
    x = synth.activations(synth.custom("t", 4, K, 16, 128, 7, n_chan=8, n_spike=4))
    y64 = O.fwht(x, "fp64")
    # Exact rational check through integers: scale by 2^24 (fp16 quantum).
    xi = (x.astype(np.float64) * 2 ** 24).astype(np.int64)
    yi = xi.copy()
    h = 1
    while h < K:
        v = yi.reshape(4, K // (2 * h), 2, h)
        a = v[:, :, 0, :].copy()
        b = v[:, :, 1, :].copy()
        v[:, :, 0, :] = a + b
        v[:, :, 1, :] = a - b
        h *= 2
    np.testing.assert_array_equal(y64 * 2 ** 24, yi.astype(np.float64))


def test_fwht_fp32_within_rounding_bound():
    K = 4096
    x = synth.activations(synth.custom("t", 8, K, 16, 128, 11, n_chan=40, n_spike=10,
                                       spike_mag=(100, 500)))
    y32 = O.fwht(x, "fp32").astype(np.float64)
    y64 = O.fwht(x, "fp64")
    # Each stage adds one rounding of relative size <= 2^-24 to every partial sum.
    bound = np.log2(K) * 2.0 ** -24 * np.abs(x.astype(np.float64)).sum(axis=1, keepdims=True)
    assert np.all(np.abs(y32 - y64) <= bound)


def test_fwht_basis_vectors():
    K = 256
    H = scipy.linalg.hadamard(K)
    for j in (0, 1, 77, 255):
        e = np.zeros(K)
        e[j] = 1
        np.testing.assert_array_equal(O.fwht(e, "fp64"), H[j])


# ---------------------------------------------------------------- identities

def test_rotation_equivalence_fp64():
    # (X R)(R^-1 W) = X W with R = H/sqrt(K) orthogonal (Fig. 2(a), Section 2.3).
    w = synth.custom("t", 32, 1024, 48, 128, 5, n_chan=10, n_spike=5)
    X = synth.activations(w).astype(np.float64)
    W = synth.weights(w).astype(np.float64)
    K = X.shape[1]
    lhs = (O.fwht(X, "fp64") @ O.fwht(W, "fp64", axis=0)) / K
    ref = X @ W
    assert np.max(np.abs(lhs - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_smoothing_equivalence_fp64():
    # (X diag(s)^-1)(diag(s) W) = X W with s expanded from the group scales
    # (Section 2.2 identity; Eq. 3 with block-constant s).
    w = synth.custom("t", 32, 512, 40, 64, 6, n_chan=6, n_spike=3)
    X = synth.activations(w)
    W = synth.weights(w).astype(np.float64)
    y = O.fwht(X, "fp64")
    u = O.fwht(W, "fp64", axis=0)
    s, _ = O.group_scales(O.channel_max(y), 64, "fp64")
    sk = np.repeat(s, 64)
    lhs = (y / sk[None, :]) @ (sk[:, None] * u)
    ref = y @ u
    assert np.max(np.abs(lhs - ref)) <= 1e-12 * np.max(np.abs(ref))


# ---------------------------------------------------------------- Eq. 4 and Appendix A.1

@pytest.mark.parametrize("K,i,O_", [(512, 3, 200.0), (4096, 1234, -377.5), (8192, 8191, 1e3)])
def test_eq4_single_spike(K, i, O_):
    t = np.zeros((1, K))
    t[0, i] = O_
    rot = O.fwht(t, "fp64")
    # every entry is c_{i,j} O: magnitude |O| unnormalized, |O|/sqrt(K) normalized
    np.testing.assert_array_equal(np.abs(rot), np.full((1, K), abs(O_)))
    np.testing.assert_array_equal(rot[0], O_ * scipy.linalg.hadamard(K)[i])
    norm = rot / np.sqrt(K)
    np.testing.assert_allclose(np.abs(norm), abs(O_) / np.sqrt(K), rtol=1e-15)
    # consistent smoothing scales: every group scale is |O|, every code is +-7
    act = O.rotate_smooth_quant(t.astype(np.float16), 128, mode="fp32")
    assert np.all(act.s == np.float32(abs(O_)))
    np.testing.assert_array_equal(act.q[0], (7 * np.sign(rot[0])).astype(np.int8))


def test_appendix_multi_spike():
    # t_rot = (1/sqrt(K)) [sum_d s_{i_d, j} O_{i_d}]_j, exact for epsilon = 0.
    K = 1024
    H = scipy.linalg.hadamard(K).astype(np.float64)
    idx = [5, 100, 900]
    Os = [300.0, -250.0, 120.0]
    t = np.zeros(K)
    for i, o in zip(idx, Os):
        t[i] = o
    expect = sum(o * H[i] for i, o in zip(idx, Os))
    np.testing.assert_array_equal(O.fwht(t, "fp64"), expect)


def test_eq4_with_noise_bound():
    # With epsilon != 0: | |t_rot,j| - |O| | <= ||eps||_1 (unnormalized form).
    K = 2048
    rng = np.random.default_rng(9)
    t = rng.standard_normal(K) * 0.01
    t[17] = 500.0
    eps = t.copy()
    eps[17] = 0
    rot = O.fwht(t, "fp64")
    assert np.all(np.abs(np.abs(rot) - 500.0) <= np.abs(eps).sum() + 1e-9)


# ---------------------------------------------------------------- quantizer

def test_rtn_golden():
    gold = _load("rtn_int4.json")
    assert O.QMAX == gold["qmax"]
    for case in gold["cases"]:
        x = np.array([case["x"]], dtype=np.float16)
        K = x.shape[1]
        for mode in ("fp32", "fp64"):
            act = O.rotate_smooth_quant(x, K, mode=mode, rotate=False, smooth=False)
            np.testing.assert_array_equal(act.q[0], np.array(case["codes"], np.int8))
            assert float(act.alpha[0]) == pytest.approx(case["alpha"], rel=1e-7)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_codes_range_and_argmax(seed):
    w = synth.WORKLOADS["tiny"]
    X = synth.activations(w, seed)
    act = O.rotate_smooth_quant(X, w.g)
    assert act.q.min() >= -7 and act.q.max() <= 7
    # the element that attains a_i lands on +-7
    M, K = X.shape
    sm = np.abs(act.y) * np.repeat(act.r, w.g)[None, :]
    jmax = np.argmax(sm, axis=1)
    assert np.all(np.abs(act.q[np.arange(M), jmax]) == 7)
    # packing round trip
    np.testing.assert_array_equal(O.unpack_int4(act.packed), act.q)


@pytest.mark.parametrize("seed", [1, 4])
def test_rtn_error_bound(seed):
    # |z_ij - q_ij alpha_i| <= alpha_i / 2 (+ rounding of the scale chain),
    # z = y_ij / s_b the smoothed activation (Eq. 2, Section 2.1).
    w = synth.WORKLOADS["tiny"]
    X = synth.activations(w, seed)
    act = O.rotate_smooth_quant(X, w.g, mode="fp64")
    z = act.y / np.repeat(act.s, w.g)[None, :]
    err = np.abs(z - act.q * act.alpha[:, None])
    assert np.all(err <= act.alpha[:, None] * (0.5 + 1e-12))


def test_worked_example_k4():
    gold = _load("rrs_worked_k4.json")
    X = np.array(gold["X"], dtype=np.float16)
    W = np.array(gold["W"], dtype=np.float16)
    g = gold["g"]
    Y, act, wq, P = O.linear(X, W, g)
    np.testing.assert_array_equal(act.y, np.array(gold["y"], np.float32))
    np.testing.assert_array_equal(act.c, np.array(gold["c"], np.float32))
    np.testing.assert_array_equal(act.s, np.array(gold["s"], np.float32))
    np.testing.assert_array_equal(act.q, np.array(gold["codes_x"], np.int8))
    np.testing.assert_array_equal(
        act.packed, np.array([[int(h, 16) for h in r] for r in gold["packed_x_hex"]], np.uint8))
    np.testing.assert_array_equal(wq.u, np.array(gold["u"], np.float32))
    np.testing.assert_array_equal(wq.b, np.array(gold["b"], np.float32))
    np.testing.assert_array_equal(wq.q, np.array(gold["codes_w"], np.int8))
    np.testing.assert_array_equal(
        wq.packed, np.array([[int(h, 16) for h in r] for r in gold["packed_w_hex"]], np.uint8))
    np.testing.assert_array_equal(P, np.array(gold["P"], np.int64))
    num, den = gold["alpha_fraction"]
    assert np.all(act.alpha == np.float32(num) / np.float32(den))
    for n, (bn, bd) in enumerate(gold["beta_fraction"]):
        assert wq.beta[n] == np.float32(bn) / np.float32(bd)
    sP = np.array(gold["sum_sP"], np.float64)
    expect = (sP * act.alpha.astype(np.float64)[:, None]
              * wq.beta.astype(np.float64)[None, :] / gold["K"]).astype(np.float32)
    np.testing.assert_array_equal(Y, expect)
    # and the RRS output approximates the exact product
    np.testing.assert_allclose(Y, np.array(gold["XW"], np.float64), rtol=0.15)


# ---------------------------------------------------------------- special cases

def _ties(v):
    return np.abs(np.abs(v - np.floor(v)) - 0.5) < 1e-6


def test_special_case_plain_per_token_rtn():
    # rotation off, one group spanning K: Runtime Smooth degenerates to one
    # uniform scale, so the codes are plain per-token RTN of X (Section 2.1).
    w = synth.custom("t", 24, 512, 8, 512, 21, n_chan=4, n_spike=3)
    X = synth.activations(w)
    act = O.rotate_smooth_quant(X, 512, mode="fp32", rotate=False)
    x = X.astype(np.float64)
    v = 7 * x / np.abs(x).max(axis=1, keepdims=True)
    ref = np.clip(np.rint(v), -7, 7)
    ok = ~_ties(v)
    np.testing.assert_array_equal(act.q[ok], ref[ok])
    assert ok.mean() > 0.99


def test_special_case_naive_runtime_smooth():
    # rotation off, g = 1: Eq. 1-3 exactly. s_j = max_i |X_ij| (Eq. 1),
    # X_hat = Quantize(X / s) per token (Eq. 2), Y = sum_j X_hat_j W_hat_j s_j (Eq. 3).
    w = synth.custom("t", 6, 16, 5, 1, 22, n_chan=2, n_spike=1)
    X = synth.activations(w)
    W = synth.weights(w)
    act = O.rotate_smooth_quant(X, 1, mode="fp64", rotate=False)
    wq = O.prepare_weight(W, mode="fp64", rotate=False)
    x = X.astype(np.float64)
    np.testing.assert_array_equal(act.s, np.abs(x).max(axis=0))
    z = x / np.abs(x).max(axis=0)[None, :]
    v = 7 * z / np.abs(z).max(axis=1, keepdims=True)
    ok = ~_ties(v)
    np.testing.assert_array_equal(act.q[ok], np.clip(np.rint(v), -7, 7)[ok])
    P = O.group_partials(act.q, wq.q, 1)
    Y = O.output(P, act.s, act.alpha, wq.beta, norm=1)
    M, K = x.shape
    N = W.shape[1]
    ref = np.zeros((M, N))
    for i in range(M):
        for n in range(N):
            acc = 0.0
            for j in range(K):
                acc += (act.q[i, j] * act.alpha[i]) * (wq.q[j, n] * wq.beta[n]) * act.s[j]
            ref[i, n] = acc
    np.testing.assert_allclose(Y, ref, rtol=1e-6, atol=1e-9)


def test_special_case_unit_scales_is_integer_gemm():
    # s = 1 (smoothing off): per-token A4W4 after rotation, the QuaRot scheme
    # (Section 2.3); Y = alpha_i beta_n / K * sum_j q_ij w_jn.
    w = synth.custom("t", 10, 512, 12, 128, 23, n_chan=4, n_spike=2)
    X = synth.activations(w)
    W = synth.weights(w)
    act = O.rotate_smooth_quant(X, 128, smooth=False)
    wq = O.prepare_weight(W)
    P = O.group_partials(act.q, wq.q, 128)
    Y = O.output(P, act.s, act.alpha, wq.beta, norm=512)
    full = act.q.astype(np.int64) @ wq.q.astype(np.int64)
    ref = (full * act.alpha.astype(np.float64)[:, None] * wq.beta.astype(np.float64)[None, :]
           / 512).astype(np.float32)
    np.testing.assert_array_equal(Y, ref)


def test_partials_bruteforce():
    rng = np.random.default_rng(31)
    M, K, N, g = 3, 16, 4, 4
    qx = rng.integers(-7, 8, size=(M, K)).astype(np.int8)
    qw = rng.integers(-7, 8, size=(K, N)).astype(np.int8)
    P = O.group_partials(qx, qw, g)
    for b in range(K // g):
        for i in range(M):
            for n in range(N):
                acc = 0
                for j in range(b * g, (b + 1) * g):
                    acc += int(qx[i, j]) * int(qw[j, n])
                assert P[b, i, n] == acc


def test_partials_extremes_fit_int32():
    g = 512
    qx = np.full((1, g), -7, np.int8)
    qw = np.full((g, 1), -7, np.int8)
    assert O.group_partials(qx, qw, g)[0, 0, 0] == 49 * g


def test_zero_groups_rows_columns():
    # s_b = 0 => r_b = 0 and codes 0; a_i = 0 => alpha_i = 0; b_n = 0 => codes 0.
    K = 512
    X = np.zeros((3, K), np.float16)
    X[1, :] = 1.0   # rotates to [K, 0, 0, ...]: only channel 0 is nonzero
    act = O.rotate_smooth_quant(X, 128)
    assert act.s[0] == K and np.all(act.s[1:] == 0) and np.all(act.r[1:] == 0)
    assert act.alpha[0] == 0 and act.alpha[2] == 0
    assert np.all(act.q[0] == 0) and np.all(act.q[2] == 0)
    assert act.q[1, 0] == 7 and np.all(act.q[1, 1:] == 0)
    W = np.zeros((K, 2), np.float16)
    wq = O.prepare_weight(W)
    assert np.all(wq.q == 0) and np.all(wq.beta == 0)


def test_permutation_preserves_product():
    # Reordering channels of activations and weight rows alike leaves the
    # product unchanged (Fig. 4 step (1)).
    w = synth.custom("t", 8, 512, 6, 128, 24, n_chan=4, n_spike=2)
    X = synth.activations(w)
    W = synth.weights(w)
    perm = synth.permutation(512, 5)
    a0 = O.rotate_smooth_quant(X, 128, mode="fp64")
    a1 = O.rotate_smooth_quant(X, 128, perm=perm, mode="fp64")
    u0 = O.prepare_weight(W, mode="fp64").u
    u1 = O.prepare_weight(W, perm=perm, mode="fp64").u
    np.testing.assert_allclose(a1.y @ u1, a0.y @ u0, rtol=1e-12)
    np.testing.assert_array_equal(a1.c, a0.c[perm])
    ident = np.arange(512, dtype=np.int32)
    a2 = O.rotate_smooth_quant(X, 128, perm=ident)
    a3 = O.rotate_smooth_quant(X, 128)
    np.testing.assert_array_equal(a2.q, a3.q)


def test_fp32_mode_matches_fp64_away_from_ties():
    w = synth.WORKLOADS["tiny"]
    X = synth.activations(w)
    a32 = O.rotate_smooth_quant(X, w.g, mode="fp32")
    a64 = O.rotate_smooth_quant(X, w.g, mode="fp64")
    far = np.abs(np.abs(a64.v - np.floor(a64.v)) - 0.5) > 1e-4
    np.testing.assert_array_equal(a32.q[far], a64.q[far])


def test_diagnostics():
    t = np.array([[1.0, 1.0, 1.0, 1.0], [4.0, 0.0, 0.0, 0.0]])
    np.testing.assert_allclose(O.smoothness_rms(t), [1.0, 2.0])
    np.testing.assert_allclose(O.smoothness_l2(t), [0.5, 1.0])
    assert O.victim_measure(np.ones(8)) == pytest.approx(1.0)


def _variant_errors(w):
    # Relative Frobenius error of each variant's output against the fp64
    # product X W, all four variants quantizing the same inputs.
    X = synth.activations(w)
    W = synth.weights(w)
    ref = O.fp64_reference(X, W)
    out = {}
    for name, rot, sm in (("rrs", True, True), ("rs", False, True),
                          ("quarot", True, False), ("none", False, False)):
        act = O.rotate_smooth_quant(X, w.g, rotate=rot, smooth=sm)
        wq = O.prepare_weight(W, rotate=rot)
        P = O.group_partials(act.q, wq.q, w.g)
        Y = O.output(P, act.s, act.alpha, wq.beta, norm=w.K if rot else 1)
        out[name] = float(np.linalg.norm(Y - ref) / np.linalg.norm(ref))
    return out


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_ablation_ordering_spikes(seed):
    # Section 3.2 and the ablation of Section 4: Runtime Smooth alone is hurt by
    # a few huge spike tokens (they inflate the channel maxima, which then
    # crush every other token's values), while the rotation spreads each spike
    # over all channels. On spike data both rotated variants must clearly beat
    # both unrotated ones, and Runtime Smooth alone must be the worst.
    w = synth.custom("s", 128, 2048, 128, 128, seed, n_chan=0, n_spike=20,
                     spike_mag=(100, 500))
    e = _variant_errors(w)
    assert e["rs"] > 1.5 * e["rrs"], e
    assert e["none"] > 1.1 * e["quarot"], e
    assert e["rs"] > e["none"], e
    assert e["rrs"] < 1.05 * e["quarot"], e


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_ablation_ordering_channels_and_spikes(seed):
    # Channel-wise outliers plus spikes (the mix Section 3 describes): RRS must
    # beat both Runtime Smooth alone and no treatment at all.
    w = synth.custom("b", 128, 2048, 128, 128, seed, n_chan=20, chan_factor=(20, 100),
                     n_spike=20, spike_mag=(100, 500))
    e = _variant_errors(w)
    assert e["rrs"] < 0.8 * e["rs"], e
    assert e["rrs"] < 0.85 * e["none"], e
    assert e["rrs"] < 1.05 * e["quarot"], e


def test_fwht_fp32_canonical_stage_order():
    # The binary32 rounding order is a reading the oracle and the kernels share
    # (stages h = 1, 2, 4, ...), not something the paper fixes. Check the
    # vectorised oracle against that definition executed one scalar butterfly
    # at a time, on data where the reverse order rounds differently (so the
    # check has teeth).
    K = 64
    rng = np.random.default_rng(77)
    x = (rng.standard_normal(K) * np.exp(rng.uniform(-8, 8, K))).astype(np.float16)

    def scalar_fwht(order):
        y = [np.float32(v) for v in x]
        for h in order:
            for p in range(K):
                if p & h == 0:
                    a, b = y[p], y[p + h]
                    y[p], y[p + h] = np.float32(a + b), np.float32(a - b)
        return np.array(y, np.float32)

    fwd = scalar_fwht([1 << i for i in range(6)])
    rev = scalar_fwht([1 << i for i in reversed(range(6))])
    assert not np.array_equal(fwd, rev)
    np.testing.assert_array_equal(O.fwht(x[None, :], "fp32")[0], fwd)


# ---------------------------------------------------------------- efficiency baselines
# (per-channel and sub-channel A4W4 of Section 4.5, Fig. 6)

def _rtn_row_fp32(row, qmax=7):
    """Textbook symmetric RTN of one block in binary32 scalar steps."""
    m = np.float32(0)
    for x in row:
        m = max(m, np.float32(abs(np.float32(x))))
    inv = np.float32(0) if m == 0 else np.float32(np.float32(qmax) / m)
    codes = [int(np.clip(np.rint(np.float32(np.float32(x) * inv)), -qmax, qmax)) for x in row]
    return m, codes


def test_sub_channel_brute_force_tiny():
    rng = np.random.default_rng(3)
    X = (rng.standard_normal((3, 16)) * 4).astype(np.float16)
    X[1, 5] = 0  # exercise a zero code
    X[2, 8:12] = 0  # an all-zero group: scale 0, codes 0
    q = O.sub_channel_quant(X, 4, rotate=False)
    for i in range(3):
        for b in range(4):
            m, codes = _rtn_row_fp32(X[i, 4 * b:4 * b + 4])
            assert q.m[i, b] == m
            assert q.scale[i, b] == np.float32(m / np.float32(7))
            assert list(q.q[i, 4 * b:4 * b + 4]) == codes


def test_sub_channel_one_group_is_per_token_rtn():
    # g = K leaves one group per row: the same codes and scales as per-token
    # quantization without smoothing (the per-channel A4W4 activation quantizer)
    w = synth.custom("sc", 5, 512, 16, 128, 21, n_chan=4, n_spike=2)
    X = synth.activations(w)
    sub = O.sub_channel_quant(X, 512)
    per = O.rotate_smooth_quant(X, 128, smooth=False)
    np.testing.assert_array_equal(sub.q, per.q)
    np.testing.assert_array_equal(sub.scale[:, 0], per.alpha)


def test_sub_channel_block_extremes_and_reconstruction():
    w = synth.custom("sc", 7, 1024, 16, 64, 22, n_chan=10, n_spike=5)
    q = O.sub_channel_quant(synth.activations(w), 64)
    blocks = q.q.reshape(7, 16, 64).astype(np.int32)
    assert np.abs(blocks).max() <= 7
    ymax = np.abs(q.y.reshape(7, 16, 64)).argmax(axis=2)
    hit = np.take_along_axis(np.abs(blocks), ymax[:, :, None], axis=2)[:, :, 0]
    assert np.all(hit[q.m > 0] == 7)
    recon = blocks * q.scale[:, :, None].astype(np.float64)
    err = np.abs(recon - q.y.reshape(7, 16, 64).astype(np.float64))
    assert np.all(err <= q.scale[:, :, None] * (0.5 + 1e-5) + 1e-30)


def test_sub_channel_weight_matches_columns():
    # weights are quantized per output channel and group: column n of W is
    # sub-channel quantized like a token row of its transpose
    rng = np.random.default_rng(9)
    W = (rng.standard_normal((256, 6)) * 0.02).astype(np.float16)
    wq = O.sub_channel_weight(W, 64)
    ref = O.sub_channel_quant(np.ascontiguousarray(W.T), 64)
    np.testing.assert_array_equal(wq.q, ref.q)
    np.testing.assert_array_equal(wq.scale, ref.scale)
    assert wq.packed.shape == (6, 128)


def test_output_sub_channel_brute_force_and_reduction():
    rng = np.random.default_rng(4)
    M, N, G = 3, 5, 4
    P = rng.integers(-3000, 3000, size=(G, M, N))
    a = rng.uniform(0.1, 2, (M, G)).astype(np.float32)
    b = rng.uniform(0.1, 2, (N, G)).astype(np.float32)
    Y = O.output_sub_channel(P, a, b, norm=8)
    for i in range(M):
        for n in range(N):
            ref = sum(float(a[i, k]) * float(b[n, k]) * int(P[k, i, n]) for k in range(G)) / 8
            assert Y[i, n] == np.float32(ref)
    # equal scales across groups: the per-channel output with s = 1
    alpha = rng.uniform(0.1, 2, M).astype(np.float32)
    beta = rng.uniform(0.1, 2, N).astype(np.float32)
    Ysub = O.output_sub_channel(P, np.repeat(alpha[:, None], G, 1), np.repeat(beta[:, None], G, 1), 8)
    Yper = O.output(P, np.ones(G, np.float32), alpha, beta, 8)
    np.testing.assert_array_equal(Ysub, Yper)


# ---------------------------------------------------------------- runtime reorder

def test_reorder_golden():
    gold = _load("reorder_worked.json")
    for case in gold["cases"]:
        X = np.array(case["X"], dtype=np.float16)
        g, block, rot = case["g"], case["block"], case["rotate"]
        act, order, perm = O.rotate_smooth_quant_reorder(X, g, block, rotate=rot)
        np.testing.assert_array_equal(order, case["order"])
        if "perm" in case:
            np.testing.assert_array_equal(perm, case["perm"])
        if "y" in case:
            np.testing.assert_array_equal(act.y, np.array(case["y"], np.float32))
        np.testing.assert_array_equal(act.s, np.array(case["s"], np.float32))
        np.testing.assert_array_equal(act.q, np.array(case["codes_x"], np.int8))
        num, den = case["alpha_fraction"]
        assert np.all(act.alpha == np.float32(num) / np.float32(den))
        if "W" in case:
            W = np.array(case["W"], dtype=np.float16)
            Y, act2, wq, P, order2 = O.linear_reorder(X, W, g, block, rotate=rot)
            np.testing.assert_array_equal(order2, case["order"])
            np.testing.assert_array_equal(wq.q, np.array(case["codes_w"], np.int8))
            np.testing.assert_array_equal(P, np.array(case["P"], np.int64))
            sP = np.array(case["sum_sP"], np.float64)
            expect = (sP * act2.alpha.astype(np.float64)[:, None]
                      * wq.beta.astype(np.float64)[None, :] / case["K"]).astype(np.float32)
            np.testing.assert_array_equal(Y, expect)


@pytest.mark.parametrize("block", [1, 32])
def test_reorder_sorted_and_largest_first(block):
    # After the reorder the block keys never increase along K, so the first
    # group holds the largest channel maximum and the group scales never
    # increase; the reordered columns are the original ones moved.
    w = synth.custom("r", 64, 1024, 8, 128, 31, n_chan=12, chan_factor=(5, 60), n_spike=3)
    X = synth.activations(w)
    act, order, perm = O.rotate_smooth_quant_reorder(X, 128, block)
    y = O.fwht(X)
    c = O.channel_max(y)
    np.testing.assert_array_equal(np.sort(perm), np.arange(1024))
    np.testing.assert_array_equal(act.y, y[:, perm])
    keys = act.c.reshape(-1, block).max(axis=1)
    assert np.all(np.diff(keys) <= 0)
    assert act.s[0] == c.max()
    assert np.all(np.diff(act.s) <= 0)


@pytest.mark.parametrize("block", [1, 32])
def test_reorder_equal_keys_keep_index_order(block):
    # Every block of `block` channels is one base block scaled by 1, 2 or 4
    # (exact in fp16), so the keys take three values and most of them tie:
    # the order is the blocks of scale 4, then 2, then 1, each run in
    # increasing block index (Fig. 4 step (1) with equal keys in index order).
    rng = np.random.default_rng(5)
    nb = 1024 // block
    base = rng.uniform(-1, 1, size=(6, block))
    scale = rng.choice([1.0, 2.0, 4.0], size=nb)
    X = np.concatenate([base * c for c in scale], axis=1).astype(np.float16)
    _, order, _ = O.rotate_smooth_quant_reorder(X, 128, block, rotate=False)
    expect = np.concatenate([np.flatnonzero(scale == c) for c in (4.0, 2.0, 1.0)])
    np.testing.assert_array_equal(order, expect)


def test_reorder_sum_of_scales_is_minimal_brute_force():
    # Cutting the sorted blocks into consecutive groups minimises the sum of
    # the group maxima over every assignment of blocks to positions: checked
    # against all 8! orders of a tiny case (no rotation, 16 channels in blocks
    # of 2, groups of g = 4 channels = 2 blocks, so 4 groups).
    import itertools
    rng = np.random.default_rng(5)
    X = rng.uniform(-4, 4, size=(3, 16)).astype(np.float16)
    block, g = 2, 4
    act, order, perm = O.rotate_smooth_quant_reorder(X, g, block, rotate=False)
    c = O.channel_max(np.array(X, np.float32))
    keys = c.reshape(8, 2).max(axis=1)
    best = min(sum(max(keys[p[2 * b]], keys[p[2 * b + 1]]) for b in range(4))
               for p in itertools.permutations(range(8)))
    assert float(act.s.sum()) == pytest.approx(float(best), rel=0, abs=0)


def test_reorder_ties_keep_index_order():
    # Zero input: every key is 0, so the order is the identity. Duplicated
    # blocks (no rotation): equal keys stay in increasing block index.
    X = np.zeros((4, 512), np.float16)
    _, order, _ = O.rotate_smooth_quant_reorder(X, 128, 32)
    np.testing.assert_array_equal(order, np.arange(16))
    rng = np.random.default_rng(9)
    base = rng.uniform(-1, 1, size=(5, 32)).astype(np.float16)
    scale = np.array([1, 3, 1, 2, 3, 1, 2, 2, 1, 3, 3, 1, 2, 1, 2, 3], np.float16)
    X = np.concatenate([base * s for s in scale], axis=1)
    _, order, _ = O.rotate_smooth_quant_reorder(X, 128, 32, rotate=False)
    expect = sorted(range(16), key=lambda B: (-float(scale[B]), B))
    np.testing.assert_array_equal(order, expect)


def test_reorder_invariant_to_input_block_order():
    # Without rotation, moving X's column blocks around gives the same sorted
    # operand: codes and scales are identical, only the reported order moves.
    rng = np.random.default_rng(2)
    # block B scaled by 1.25^B: keys far apart, so no two are equal
    X = (rng.normal(0, 1, size=(32, 1024))
         * np.repeat(1.25 ** rng.permutation(32), 32)[None, :]).astype(np.float16)
    Q = rng.permutation(32)
    Xq = X[:, O.block_order_to_perm(Q, 32)]
    a0, o0, _ = O.rotate_smooth_quant_reorder(X, 128, 32, rotate=False)
    a1, o1, _ = O.rotate_smooth_quant_reorder(Xq, 128, 32, rotate=False)
    keys = O.channel_max(np.array(X, np.float32)).reshape(32, 32).max(axis=1)
    assert len(np.unique(keys)) == 32  # distinct keys: the sorted operand is unique
    np.testing.assert_array_equal(a1.q, a0.q)
    np.testing.assert_array_equal(a1.s, a0.s)
    np.testing.assert_array_equal(a1.alpha, a0.alpha)
    np.testing.assert_array_equal(Q[o1], o0)


def test_reorder_one_group_changes_nothing():
    # With one group over all of K the grouping cannot change: the output is
    # bit-identical to the layer without reorder (the integer sum is the same
    # set of products).
    w = synth.custom("o", 16, 512, 24, 512, 43, n_chan=6, n_spike=2)
    X, W = synth.activations(w), synth.weights(w)
    Y0, *_ = O.linear(X, W, 512)
    Y1, *_ = O.linear_reorder(X, W, 512, 32)
    np.testing.assert_array_equal(Y1, Y0)


def test_reorder_block_equal_to_group_moves_whole_groups():
    # Blocks as large as a group move whole groups: the same scales, the same
    # partials, summed in another order.
    w = synth.custom("q", 16, 1024, 24, 128, 44, n_chan=6, n_spike=2)
    X, W = synth.activations(w), synth.weights(w)
    Y0, a0, _, P0 = O.linear(X, W, 128)
    Y1, a1, _, P1, order = O.linear_reorder(X, W, 128, 128)
    np.testing.assert_array_equal(a1.s, a0.s[order])
    np.testing.assert_array_equal(P1, P0[order])
    np.testing.assert_allclose(Y1, Y0, rtol=1e-6, atol=0)


def test_reorder_weight_rows_move_with_channels():
    # Per-output-channel weight scales do not depend on the row order, so the
    # reordered weight codes are the unreordered codes with rows moved: the
    # GEMM may gather rows of weights prepared once, without the reorder.
    w = synth.custom("w", 4, 1024, 40, 128, 45)
    W = synth.weights(w)
    perm = O.block_order_to_perm(np.random.default_rng(3).permutation(32), 32)
    w0 = O.prepare_weight(W)
    w1 = O.prepare_weight(W, perm)
    np.testing.assert_array_equal(w1.q, w0.q[perm])
    np.testing.assert_array_equal(w1.beta, w0.beta)


def test_reorder_groups_outlier_channels_together():
    # What Fig. 4 step (1) is for: outlier channels scattered over every group
    # inflate every group's scale; after the reorder they share one group and
    # the other channels keep small scales, which lowers the error of
    # Runtime Smooth (no rotation) on this channel-outlier input.
    rng = np.random.default_rng(7)
    M, K, N, g = 64, 512, 32, 128
    X = rng.normal(0, 1, size=(M, K))
    X[:, [5, 133, 261, 389]] *= 80.0  # one outlier channel in each group
    X = X.astype(np.float16)
    W = rng.normal(0, 1, size=(K, N))
    W[[5, 133, 261, 389], :] /= 80.0  # outliers do not dominate the product
    W = W.astype(np.float16)
    ref = O.fp64_reference(X, W)

    def err(Y):
        return float(np.linalg.norm(Y - ref) / np.linalg.norm(ref))

    act = O.rotate_smooth_quant(X, g, rotate=False)
    wq = O.prepare_weight(W, rotate=False)
    Y0 = O.output(O.group_partials(act.q, wq.q, g), act.s, act.alpha, wq.beta, 1)
    Y1, act1, *_ = O.linear_reorder(X, W, g, 1, rotate=False)
    assert act1.s[1] < act.s.min() / 10
    assert err(Y1) < 0.7 * err(Y0), (err(Y1), err(Y0))


# ---------------------------------------------------------------- rounding-bound magnitudes
#
# output_abs_terms / output_sub_channel_abs_terms give T, the magnitude that the
# elementwise output tolerance scales: the binary32 sum over the G group terms
# of Eq. 3 (rescaled per block, Fig. 4 step (3)) rounds by at most about
# G * 2^-24 * T in any order. The pins below fix T by hand-worked values, a
# scalar brute force on mixed signs (so a dropped absolute value shows), the
# 1 / norm factor (norm = K and norm = 1), the triangle inequality with equality
# when every term has one sign, and the rounding bound itself over random
# summation orders.

def _dyadic(rng, shape, lo, hi, denom=8):
    """Random multiples of 1/denom in [lo, hi], never 0: exact in binary32/64."""
    v = rng.integers(int(lo * denom), int(hi * denom) + 1, size=shape).astype(np.float64)
    v[v == 0] = 1.0
    return v / denom


def test_output_abs_terms_hand_worked():
    # One output, two groups: P = (3, -5), s = (2, -0.5) (a negative s only
    # tests the absolute value), alpha = -0.5, beta = 4, norm = 8:
    # sum_b |s_b P_b| = 6 + 2.5 = 8.5 and T = 0.5 * 4 / 8 * 8.5 = 2.125.
    P = np.array([3, -5]).reshape(2, 1, 1)
    T = O.output_abs_terms(P, np.array([2.0, -0.5]), np.array([-0.5]), np.array([4.0]), 8)
    assert T.shape == (1, 1) and T[0, 0] == 2.125
    # norm = 1 gives 8 times that, and the signed output is 0.5 * 4 / 8 * (6 + 2.5).
    T1 = O.output_abs_terms(P, np.array([2.0, -0.5]), np.array([-0.5]), np.array([4.0]), 1)
    assert T1[0, 0] == 17.0
    Y = O.output(P, np.array([2.0, 0.5]), np.array([0.5]), np.array([4.0]), 8)
    assert Y[0, 0] == np.float32(0.25 * (6 - 2.5))


@pytest.mark.parametrize("norm", [1, 512])
def test_output_abs_terms_brute_force_mixed_signs(norm):
    rng = np.random.default_rng(71 + norm)
    G, M, N = 4, 3, 5
    P = rng.integers(-6000, 6001, size=(G, M, N))
    s = _dyadic(rng, G, -4, 4)
    alpha = _dyadic(rng, M, -3, 3)
    beta = _dyadic(rng, N, -3, 3)
    T = O.output_abs_terms(P, s, alpha, beta, norm)
    for i in range(M):
        for n in range(N):
            acc = 0.0
            for b in range(G):
                acc += abs(float(s[b]) * int(P[b, i, n]))
            # every value is dyadic with few bits: all of this is exact in binary64
            assert T[i, n] == abs(float(alpha[i])) * abs(float(beta[n])) * acc / norm


def test_output_abs_terms_triangle_and_equality():
    rng = np.random.default_rng(72)
    G, M, N, K = 8, 4, 6, 4096
    P = rng.integers(-6000, 6001, size=(G, M, N))
    s = rng.uniform(0.01, 30, G).astype(np.float32)
    alpha = rng.uniform(0.001, 2, M).astype(np.float32)
    beta = rng.uniform(0.001, 0.1, N).astype(np.float32)
    T = O.output_abs_terms(P, s, alpha, beta, K)
    Y = O.output(P, s, alpha, beta, K).astype(np.float64)
    # |Y| <= T up to the final binary32 rounding of Y
    assert np.all(np.abs(Y) <= T * (1 + 2.0 ** -23))
    # one sign in every term: T = |Y| (up to that rounding); a T that kept a
    # factor K (a dropped 1 / norm) or summed before the absolute value fails
    Pp = np.abs(P)
    Tp = O.output_abs_terms(Pp, s, alpha, beta, K)
    Yp = O.output(Pp, s, alpha, beta, K).astype(np.float64)
    np.testing.assert_allclose(Tp, Yp, rtol=2.0 ** -23, atol=0)
    Tn = O.output_abs_terms(-Pp, s, alpha, beta, K)
    np.testing.assert_allclose(Tn, -O.output(-Pp, s, alpha, beta, K).astype(np.float64),
                               rtol=2.0 ** -23, atol=0)
    # one group: T = |Y| whatever the sign
    T1 = O.output_abs_terms(P[:1], s[:1], alpha, beta, K)
    Y1 = O.output(P[:1], s[:1], alpha, beta, K).astype(np.float64)
    np.testing.assert_allclose(T1, np.abs(Y1), rtol=2.0 ** -23, atol=0)


def test_output_abs_terms_bounds_binary32_sums_in_any_order():
    # The use the tests make of T: a binary32 evaluation of sum_b s_b P_b in any
    # order, scaled by fl(alpha beta / K), differs from the binary64 value by at
    # most (G + 3) 2^-24 T. Outputs here cancel strongly (mixed-sign partials),
    # which is where the bound, not the relative 1e-2, is what matters.
    rng = np.random.default_rng(73)
    G, M, N, K = 32, 6, 40, 4096
    P = rng.integers(-3000, 3001, size=(G, M, N))
    s = rng.uniform(0.5, 40, G).astype(np.float32)
    alpha = rng.uniform(0.01, 3, M).astype(np.float32)
    beta = rng.uniform(0.001, 0.05, N).astype(np.float32)
    T = O.output_abs_terms(P, s, alpha, beta, K)
    exact = (np.tensordot(s.astype(np.float64), P.astype(np.float64), axes=(0, 0))
             * alpha.astype(np.float64)[:, None] * beta.astype(np.float64)[None, :] / K)
    f = np.float32
    worst = 0.0
    for trial in range(12):
        order = rng.permutation(G)
        acc = np.zeros((M, N), np.float32)
        for b in order:
            acc = (acc + (f(s[b]) * P[b].astype(np.float32)).astype(np.float32)).astype(np.float32)
        scale = ((alpha[:, None] * beta[None, :]).astype(np.float32) * f(1.0 / K)).astype(np.float32)
        y = (acc * scale).astype(np.float32).astype(np.float64)
        err = np.abs(y - exact)
        assert np.all(err <= (G + 3) * 2.0 ** -24 * T)
        worst = max(worst, float((err / T).max()))
    # and the bound is not vacuous: the observed error reaches a visible part of it
    assert worst > 2.0 ** -24


def test_output_sub_channel_abs_terms_hand_worked_and_brute_force():
    # Hand-worked: one output, two groups, P = (3, -5), token scales (0.5, -2),
    # channel scales (-4, 0.25), norm = 8:
    # |0.5 * -4 * 3| + |-2 * 0.25 * -5| = 6 + 2.5 = 8.5, T = 8.5 / 8.
    P = np.array([3, -5]).reshape(2, 1, 1)
    a = np.array([[0.5, -2.0]])
    b = np.array([[-4.0, 0.25]])
    assert O.output_sub_channel_abs_terms(P, a, b, 8)[0, 0] == 8.5 / 8
    assert O.output_sub_channel_abs_terms(P, a, b, 1)[0, 0] == 8.5
    # Brute force on mixed signs, dyadic values (exact), norm = K and 1.
    rng = np.random.default_rng(74)
    G, M, N = 3, 4, 5
    P = rng.integers(-6000, 6001, size=(G, M, N))
    a = _dyadic(rng, (M, G), -3, 3)
    b = _dyadic(rng, (N, G), -3, 3)
    for norm in (1, 256):
        T = O.output_sub_channel_abs_terms(P, a, b, norm)
        for i in range(M):
            for n in range(N):
                acc = 0.0
                for k in range(G):
                    acc += abs(float(a[i, k]) * float(b[n, k]) * int(P[k, i, n]))
                assert T[i, n] == acc / norm
    # one sign per term: T equals |Y|; equal scales across groups: the
    # per-channel magnitude
    Pp = np.abs(P)
    ap, bp = np.abs(a), np.abs(b)
    np.testing.assert_allclose(O.output_sub_channel_abs_terms(Pp, ap, bp, 8),
                               O.output_sub_channel(Pp, ap, bp, 8).astype(np.float64),
                               rtol=2.0 ** -23, atol=0)
    alpha = _dyadic(rng, M, -2, 2)
    beta = _dyadic(rng, N, -2, 2)
    np.testing.assert_array_equal(
        O.output_sub_channel_abs_terms(P, np.repeat(alpha[:, None], G, 1),
                                       np.repeat(beta[:, None], G, 1), 8),
        O.output_abs_terms(P, np.ones(G), alpha, beta, 8))
