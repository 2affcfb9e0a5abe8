"""Pins of the oracle's attention, softmax(t q k^T) v with Algorithm 2's
softmax (Sec. III-C) between two products. The products are numpy float64
matrix products (a library primitive; products of bfloat16 values are exact in
float64), so the pins check the composition against things fixed without it:
a single key gives v back exactly; all-equal scores give the plain mean of the
allowed values of v (the causal prefix); the per-row numerators and sums
reproduce the (separately pinned) softmax oracle; in EXACT mode the result is
the textbook float64 attention within the rounding the path states; the QuAKE
modes stay within their pinned error range of it; and planted mistakes in the
composition (mask, transposition, normalisation) fail these pins."""
import inspect
import textwrap

import numpy as np
import pytest

from paper_2412_00408_amd import synth


def _np(t):
    return synth.bits(t)


def _f64(bits16, dt="bf16"):
    import oracle
    return oracle.decode(np.ascontiguousarray(bits16).reshape(-1), dt).astype(
        np.float64).reshape(bits16.shape)


def _inputs(h, s, seed, ldv=None, pad=0.0, dt="bf16"):
    q, k, vt = synth.attention_inputs(h, s, seed, ldv=ldv, pad=pad, dt=dt)
    return _np(q), _np(k), _np(vt)


def _textbook(q, k, vt, t, causal, dt="bf16"):
    """float64 softmax(t q k^T) v with the standard exponential; also
    sum_k p_k |v_k| / sum_k p_k and sum_k |v_k| / sum_k p_k (allowed keys)."""
    s_len = q.shape[1]
    sc = np.matmul(_f64(q, dt), np.transpose(_f64(k, dt), (0, 2, 1))) * t
    allowed = np.ones((s_len, s_len), bool)
    if causal:
        allowed = ~np.triu(allowed, 1)
        sc[:, ~allowed] = -np.inf
    sc -= sc.max(axis=2, keepdims=True)
    p = np.exp(sc)
    va = np.abs(_f64(vt, dt)[:, :, :s_len])
    ref = np.matmul(p, np.transpose(_f64(vt, dt)[:, :, :s_len], (0, 2, 1))) / p.sum(axis=2, keepdims=True)
    pv = np.matmul(p, np.transpose(va, (0, 2, 1))) / p.sum(axis=2, keepdims=True)
    sv = np.matmul(allowed.astype(np.float64)[None], np.transpose(va, (0, 2, 1))) / p.sum(
        axis=2, keepdims=True)
    return ref, pv, sv


# unit roundoff u of the format, and the absolute rounding floor of a value
# below its normal range (binary16 probabilities can be subnormal)
U = {"bf16": 2.0 ** -8, "f16": 2.0 ** -11}
FLOOR = {"bf16": 2.0 ** -134, "f16": 2.0 ** -25}


def _bound(ref, pv, sv, dt, rel):
    return U[dt] * np.abs(ref) + (U[dt] + 2.0 ** -12 + rel) * pv + FLOOR[dt] * (sv + 1)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("causal", [True, False])
def test_single_key_returns_v(oracle, mode, causal, dt):
    q, k, vt = _inputs(3, 1, 40, dt=dt)
    o = oracle.attention(q, k, vt, mode, 0.125, causal, dt=dt)
    assert np.array_equal(o, np.transpose(vt, (0, 2, 1)))


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("causal", [True, False])
def test_equal_scores_give_the_mean_of_v(oracle, mode, causal, dt):
    h, s = 2, 37
    _, k, vt = _inputs(h, s, 41, dt=dt)
    q = np.zeros((h, s, 64), np.uint16)                 # every score is 0: p = 1 exactly
    o = _f64(oracle.attention(q, k, vt, mode, 0.125, causal, dt=dt), dt)
    v = np.transpose(_f64(vt, dt), (0, 2, 1))
    if causal:
        mean = np.cumsum(v, axis=1) / np.arange(1, s + 1)[None, :, None]
    else:
        mean = np.broadcast_to(v.mean(axis=1, keepdims=True), v.shape)
    want = _f64(oracle.round_to(mean.reshape(-1), dt).reshape(mean.shape), dt)
    assert np.array_equal(o, want)


def test_causal_first_query_sees_only_key_zero(oracle):
    q, k, vt = _inputs(4, 29, 42)
    o = oracle.attention(q, k, vt, 2, 0.125, True)
    assert np.array_equal(o[:, 0, :], vt[:, :, 0])


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_numerators_reproduce_the_softmax_oracle(oracle, mode):
    s = (np.random.default_rng(43).standard_normal((64, 77)) * 6).astype(np.float32)
    s[5, 30:] = -np.inf
    s[9, :] = -np.inf
    p, sums = oracle.softmax_numerators(s, mode, 0.37)
    with np.errstate(invalid="ignore", divide="ignore"):
        y = np.where(sums[:, None] > 0, p / sums[:, None], 0.0).astype(np.float32)
    assert np.array_equal(y, oracle.softmax(s, "f32", mode, 0.37))
    assert np.all(p[9] == 0) and sums[9] == 0


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("causal", [True, False])
def test_exact_mode_is_textbook_attention(oracle, causal, dt):
    q, k, vt = _inputs(3, 45, 44, dt=dt)
    o = _f64(oracle.attention(q, k, vt, 0, 0.125, causal, dt=dt), dt)
    ref, pv, sv = _textbook(q, k, vt, 0.125, causal, dt)
    # output rounding and probability rounding (unit roundoff u of the format
    # each, plus the subnormal floor of binary16 probabilities), the binary32
    # scores and exponent argument (far below 2^-12 relative here)
    assert np.all(np.abs(o - ref) <= _bound(ref, pv, sv, dt, 0.0))


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("mode,err", [(1, 0.0299), (2, 0.00342), (3, 0.00173)])
def test_quake_modes_within_their_error_range(oracle, mode, err, dt):
    # every exponential is within its mode's relative error range (pinned with
    # the scalar oracle: QuAKE1 2.99 %, QuAKE2 0.342 %, minimax 0.173 %), so
    # sum_j p_j v_j / sum_j p_j moves by at most (1 + err) / (1 - err) - 1,
    # below 2.2 err, times sum_j p_j |v_j| / sum_j p_j
    q, k, vt = _inputs(2, 64, 45, dt=dt)
    o = _f64(oracle.attention(q, k, vt, mode, 0.125, True, dt=dt), dt)
    ref, pv, sv = _textbook(q, k, vt, 0.125, True, dt)
    assert np.all(np.abs(o - ref) <= _bound(ref, pv, sv, dt, 2.2 * err))


def test_padding_of_vt_is_ignored(oracle):
    q, k, vt = _inputs(2, 21, 46, ldv=32, pad=float("nan"))
    o = oracle.attention(q, k, vt, 2, 0.125, False)
    assert np.array_equal(o, oracle.attention(q, k, np.ascontiguousarray(vt[:, :, :21]), 2,
                                              0.125, False))


MUTANTS = {
    "probabilities_always_bfloat16": (
        'pb = decode(round_to(p.astype(np.float64).reshape(-1), dt), dt).astype(np.float64)',
        'pb = decode(round_to(p.astype(np.float64).reshape(-1), "bf16"), "bf16").astype(np.float64)'),
    "causal_mask_includes_diagonal": ("np.arange(s_len)[None, :] > np.asarray(rows)[:, None]",
                                      "np.arange(s_len)[None, :] >= np.asarray(rows)[:, None]"),
    "v_not_transposed": ("o = np.matmul(pb.reshape(h, nr, s_len), np.transpose(vd, (0, 2, 1)))",
                         "o = np.matmul(pb.reshape(h, nr, s_len), vd.reshape(h, s_len, d))"),
    "keys_transposed_as_queries": ("scores = np.matmul(qd, np.transpose(kd, (0, 2, 1)))",
                                   "scores = np.matmul(kd, np.transpose(qd, (0, 2, 1)))"),
    "no_normalisation": ("o = np.where(sums.reshape(h, nr, 1) > 0, o / sums.reshape(h, nr, 1), 0.0)",
                         "o = np.where(sums.reshape(h, nr, 1) > 0, o, 0.0)"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_attention_mutant(oracle, name):
    src = "\n".join(textwrap.dedent(inspect.getsource(f)) for f in (
        oracle.attention, oracle._attention_heads, oracle._attention_core))
    old, new = MUTANTS[name]
    assert old in src, name
    ns = dict(vars(oracle))
    exec(compile(src.replace(old, new), "<mutant %s>" % name, "exec"), ns)
    mut = ns["attention"]
    caught = []
    for causal, dt in ((True, "bf16"), (False, "bf16"), (True, "f16")):
        q, k, vt = _inputs(2, 37, 47, dt=dt)
        try:
            o = _f64(mut(q, k, vt, 0, 0.125, causal, dt=dt), dt)
        except ValueError:
            caught.append(True)
            continue
        ref, pv, sv = _textbook(q, k, vt, 0.125, causal, dt)
        caught.append(not np.all(np.abs(o - ref) <= _bound(ref, pv, sv, dt, 0.0)))
    assert any(caught), name


@pytest.mark.parametrize("dt", ["bf16", "f16"])
@pytest.mark.parametrize("causal", [True, False])
def test_sampled_rows_are_the_rows_of_the_full_result(oracle, causal, dt):
    """attention_rows (queries taken one by one against all keys, the causal
    mask at each query's own index) gives the rows of attention itself; the
    float64 products may sum in another order, which moves a rounded output
    by one ulp at most, and rarely."""
    q, k, vt = _inputs(3, 200, 48, ldv=205, pad=float("nan"), dt=dt)
    full = oracle.attention(q, k, vt, 2, 0.125, causal, dt=dt)
    rows = [0, 1, 31, 32, 33, 100, 198, 199]
    part = oracle.attention_rows(q, k, vt, rows, 2, 0.125, causal, dt=dt)
    a, b = _f64(part, dt), _f64(full[:, rows], dt)
    ulp = np.ldexp(1.0, (np.floor(np.log2(np.maximum(np.abs(b), 2.0 ** -126))) -
                         (7 if dt == "bf16" else 10)).astype(int))
    assert np.all(np.abs(a - b) <= ulp)
    assert np.mean(a == b) >= 0.99
    with pytest.raises(ValueError):
        oracle.attention_rows(q, k, vt, [200], 2, 0.125, causal, dt=dt)
