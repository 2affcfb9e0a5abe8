"""GPU parity of quake_attention (both products on the matrix cores, the
softmax of Algorithm 2 between them, all in one kernel) against the oracle's
attention on the same seeded bfloat16 q, k and transposed v.

Tolerance per output element (derived, written here). The GPU sums the 64
products of a score in binary32 in its own order, the oracle rounds the exact
sum once: |dS| <= 65 * 2^-24 * sum_i |q_i k_i| =: ds per score, and the row max
moves by at most the same. An exponential of (s - m) t changes by a relative
1.5 t (|ds| + |dm|) at most (QuAKE's piecewise slope is at most 1.44 times
e^x's; EXACT's v_exp_f32 adds 2^-23), so each probability moves by at most
rp = 3 t ds_max + 2^-22 before its rounding to bfloat16, which can then land on
the neighbouring value (one bfloat16 ulp, at most 2^-7 relative). The second
product and the row sum add (seq + 4) 2^-24 relative in binary32, and each side
rounds the result once to bfloat16:
  |gpu - ref| <= ulp_bf16(ref) + (2^-7 + 2.2 rp + (seq + 4) 2^-24) * pv
with pv = sum_k p_k |v_k| / sum_k p_k (textbook probabilities, times 1.1 to
cover QuAKE's <= 3 % error). Further, at least 99 % of the elements must be
within one bfloat16 ulp of the oracle (probability roundings rarely flip).
Cases: every mode, causal and not, one to several 32-query tiles, a ragged
last tile, ragged key blocks, each one-pass workgroup size (4 waves up to 512
keys, 8 up to 1024) with its longest sequence, longer ones (the two-pass
kernel, from 1025 keys, with one or two 32-query groups per tile, including
last tiles whose second group lies partly or wholly past the sequence), a
single key, padded v^T rows whose padding is NaN, and the full 96-head x 512
workload in the launch configuration the benchmark times, compared element by
element."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import THREADS, host_bits, say
from paper_2412_00408_amd import synth

pytestmark = pytest.mark.gpu

T = 0.125


@pytest.fixture(scope="module")
def q():
    assert torch.cuda.is_available(), "GPU tests need cuda:0"
    from paper_2412_00408_amd import quake
    return quake


def _ulp(v, dt="bf16"):
    a = np.abs(v)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    if dt == "bf16":
        return np.where(a >= 2.0 ** -126, np.ldexp(1.0, (e - 7).astype(int)), 2.0 ** -133)
    return np.where(a >= 2.0 ** -14, np.ldexp(1.0, (e - 10).astype(int)), 2.0 ** -24)


def _dec(b, dt="bf16"):
    return oracle.decode(np.ascontiguousarray(b).reshape(-1), dt).astype(np.float64).reshape(b.shape)


def _bound(qb, kb, vtb, seq, causal, ref, dt="bf16"):
    out = np.empty(ref.shape)
    for h0 in range(0, ref.shape[0], 4):
        sl = slice(h0, h0 + 4)
        out[sl] = _bound_heads(qb[sl], kb[sl], vtb[sl], seq, causal, ref[sl], dt)
    return out


def _bound_heads(qb, kb, vtb, seq, causal, ref, dt):
    qd, kd = _dec(qb, dt), _dec(kb, dt)
    vd = _dec(vtb, dt)[:, :, :seq]
    sc = np.matmul(qd, np.transpose(kd, (0, 2, 1)))
    sa = np.matmul(np.abs(qd), np.transpose(np.abs(kd), (0, 2, 1)))
    if causal:
        mask = np.triu(np.ones((seq, seq), bool), 1)
        sc[:, mask] = -np.inf
        sa[:, mask] = 0.0
    ds_max = 65 * 2.0 ** -24 * sa.max(axis=2, keepdims=True)
    rp = 3 * T * ds_max + 2.0 ** -22
    p = np.exp(T * (sc - sc.max(axis=2, keepdims=True)))
    pv = 1.1 * np.matmul(p, np.transpose(np.abs(vd), (0, 2, 1))) / p.sum(axis=2, keepdims=True)
    if dt == "bf16":
        return _ulp(ref, dt) + (2.0 ** -7 + 2.2 * rp + (seq + 4) * 2.0 ** -24) * pv
    # binary16: a probability flip is one binary16 ulp (2^-10 relative, or
    # 2^-24 absolute for subnormal probabilities), on any key
    allowed = np.ones((seq, seq)) if not causal else np.tril(np.ones((seq, seq)))
    sv = np.matmul(allowed[None], np.transpose(np.abs(vd), (0, 2, 1))) / p.sum(axis=2, keepdims=True)
    return (_ulp(ref, dt) + (2.0 ** -10 + 2.2 * rp + (seq + 4) * 2.0 ** -24) * pv
            + 2.0 ** -24 * sv)


def _bound_rows(qb, kb, vtb, rows, causal, ref, dt="bf16"):
    """_bound_heads for the queries `rows` only (one head at a time is enough
    for the long sequences this serves)."""
    seq = kb.shape[1]
    rows = np.asarray(rows)
    qd, kd = _dec(np.ascontiguousarray(qb[:, rows]), dt), _dec(kb, dt)
    vd = _dec(vtb, dt)[:, :, :seq]
    sc = np.matmul(qd, np.transpose(kd, (0, 2, 1)))
    sa = np.matmul(np.abs(qd), np.transpose(np.abs(kd), (0, 2, 1)))
    allowed = np.ones((rows.size, seq), bool)
    if causal:
        allowed = np.arange(seq)[None, :] <= rows[:, None]
        sc[:, ~allowed] = -np.inf
        sa[:, ~allowed] = 0.0
    ds_max = 65 * 2.0 ** -24 * sa.max(axis=2, keepdims=True)
    rp = 3 * T * ds_max + 2.0 ** -22
    p = np.exp(T * (sc - sc.max(axis=2, keepdims=True)))
    pv = 1.1 * np.matmul(p, np.transpose(np.abs(vd), (0, 2, 1))) / p.sum(axis=2, keepdims=True)
    if dt == "bf16":
        return _ulp(ref, dt) + (2.0 ** -7 + 2.2 * rp + (seq + 4) * 2.0 ** -24) * pv
    sv = np.matmul(allowed[None].astype(np.float64), np.transpose(np.abs(vd), (0, 2, 1))) / \
        p.sum(axis=2, keepdims=True)
    return (_ulp(ref, dt) + (2.0 ** -10 + 2.2 * rp + (seq + 4) * 2.0 ** -24) * pv
            + 2.0 ** -24 * sv)


def _check_against(g_bits, r_bits, bound, name, dt="bf16"):
    g, r = _dec(g_bits, dt), _dec(r_bits, dt)
    assert not np.isnan(g).any(), "%s: unwritten or NaN outputs" % name
    err = np.abs(g - r)
    bad = ~(err <= bound)
    i = int(np.argmax((err - bound).reshape(-1)))
    assert not bad.any(), "%s: %d of %d outside the bound, worst at %d: gpu %r ref %r bound %r" % (
        name, int(bad.sum()), bad.size, i, g.reshape(-1)[i], r.reshape(-1)[i], bound.reshape(-1)[i])
    assert np.mean(err <= _ulp(r, dt)) >= 0.99, "%s: fewer than 99 %% within one ulp" % name


def _run(q, heads, seq, mode, causal, seed, ldv=None, pad=0.0, dt="bf16"):
    say("attention %s heads=%d seq=%d ldv=%s mode=%d causal=%d seed=%d" % (
        dt, heads, seq, ldv, mode, causal, seed))
    qc, kc, vtc = synth.attention_inputs(heads, seq, seed, ldv=ldv, pad=pad, dt=dt)
    qg, kg, vtg = qc.to("cuda:0"), kc.to("cuda:0"), vtc.to("cuda:0")
    o = torch.full((heads, seq, 64), float("nan"), dtype=qc.dtype, device="cuda:0")
    if ldv is not None and ldv != seq:
        vt_view = vtg[:, :, :seq]
    else:
        vt_view = vtg
    q.quake_attention(qg, kg, vt_view, o, mode=mode, t=T, causal=causal)
    torch.cuda.synchronize()
    qb, kb, vtb = host_bits(qc), host_bits(kc), host_bits(vtc)
    ref = oracle.attention(qb, kb, vtb, mode, T, causal, threads=THREADS, dt=dt)
    return host_bits(o), ref, (qb, kb, vtb)


def _check(g_bits, r_bits, ins, seq, causal, name, dt="bf16"):
    g, r = _dec(g_bits, dt), _dec(r_bits, dt)
    assert not np.isnan(g).any(), "%s: unwritten or NaN outputs" % name
    bound = _bound(*ins, seq, causal, r, dt)
    err = np.abs(g - r)
    bad = ~(err <= bound)
    i = int(np.argmax((err - bound).reshape(-1)))
    assert not bad.any(), "%s: %d of %d outside the bound, worst at %d: gpu %r ref %r bound %r" % (
        name, int(bad.sum()), bad.size, i, g.reshape(-1)[i], r.reshape(-1)[i], bound.reshape(-1)[i])
    within1 = np.mean(err <= _ulp(r, dt))
    assert within1 >= 0.99, "%s: only %.4f within one ulp" % (name, within1)
    return err


SHAPES = [(2, 64), (3, 40), (2, 96), (1, 512), (2, 33), (5, 8)]
# one pass with 8 waves (513 to 1024 keys)
LONG_SHAPES = [(2, 513), (1, 777), (1, 1000), (2, 1024)]
# past 1024 keys the two-pass kernel (scores computed twice, never stored)
TWO_PASS_SHAPES = [(1, 1025), (1, 1500), (2, 2048), (1, 2049), (1, 4096)]


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("heads,seq", SHAPES)
def test_attention_matches_oracle(q, mode, causal, heads, seq):
    g, r, ins = _run(q, heads, seq, mode, causal, 60 + seq)
    _check(g, r, ins, seq, causal, "h%d s%d m%d c%d" % (heads, seq, mode, causal))


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("heads,seq", LONG_SHAPES)
def test_long_sequences_match_oracle(q, mode, causal, heads, seq):
    g, r, ins = _run(q, heads, seq, mode, causal, 70 + seq)
    _check(g, r, ins, seq, causal, "long h%d s%d m%d c%d" % (heads, seq, mode, causal))


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("heads,seq", TWO_PASS_SHAPES)
def test_two_pass_sequences_match_oracle(q, mode, causal, heads, seq):
    g, r, ins = _run(q, heads, seq, mode, causal, 75 + seq)
    _check(g, r, ins, seq, causal, "two-pass h%d s%d m%d c%d" % (heads, seq, mode, causal))


def _two_group_heads(seq, causal):
    """The fewest heads for which the two-pass kernel takes tiles of two
    32-query groups: 512 such tiles of 64 queries without the mask, 1024 with
    it (below that it takes one group per tile)."""
    tiles = -(-seq // 64)
    return -(-(1024 if causal else 512) // tiles)


# ragged tails where the last tile's second group is partly (1130) or wholly
# (1100, 1056) past s, and a key block past the last full one (2049)
TWO_GROUP_SEQS = [1130, 1056, 2049]


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("causal", [True, False])
def test_two_group_two_pass_matches_oracle(q, mode, causal):
    heads = _two_group_heads(1100, causal)
    g, r, ins = _run(q, heads, 1100, mode, causal, 85)
    _check(g, r, ins, 1100, causal, "two-group h%d s1100 m%d c%d" % (heads, mode, causal))


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("seq", TWO_GROUP_SEQS)
def test_two_group_ragged_tails_match_oracle(q, causal, seq):
    heads = _two_group_heads(seq, causal)
    g, r, ins = _run(q, heads, seq, 2, causal, 86 + seq)
    _check(g, r, ins, seq, causal, "two-group h%d s%d c%d" % (heads, seq, causal))


@pytest.mark.parametrize("ldv", [1103, 1104])
@pytest.mark.parametrize("causal", [True, False])
def test_two_group_padded_vt_rows(q, causal, ldv):
    heads = _two_group_heads(1100, causal)
    g, r, ins = _run(q, heads, 1100, 2, causal, 87, ldv=ldv, pad=float("nan"))
    _check(g, r, ins, 1100, causal, "two-group padded h%d ldv%d c%d" % (heads, ldv, causal))


@pytest.mark.parametrize("mode", [0, 2])
@pytest.mark.parametrize("causal", [True, False])
def test_two_group_binary16_matches_oracle(q, mode, causal):
    heads = _two_group_heads(1100, causal)
    g, r, ins = _run(q, heads, 1100, mode, causal, 88, dt="f16")
    _check(g, r, ins, 1100, causal, "two-group f16 h%d m%d c%d" % (heads, mode, causal), dt="f16")


@pytest.mark.parametrize("causal", [True, False])
def test_two_group_and_one_group_give_the_same_bits(q, causal):
    """Enough heads of 1100 keys for two-group tiles; each head alone (too few
    tiles for two groups) runs as one-group tiles. Per query the arithmetic
    is the same, so the outputs must agree bit for bit."""
    heads = _two_group_heads(1100, causal)
    say("attention two-group vs one-group heads=%d causal=%d" % (heads, causal))
    qc, kc, vtc = synth.attention_inputs(heads, 1100, 89)
    qg, kg, vtg = qc.to("cuda:0"), kc.to("cuda:0"), vtc.to("cuda:0")
    whole = q.quake_attention(qg, kg, vtg, mode=2, t=T, causal=causal)
    for hd in (0, heads // 2, heads - 1):
        one = q.quake_attention(qg[hd:hd + 1].contiguous(), kg[hd:hd + 1].contiguous(),
                                vtg[hd:hd + 1].contiguous(), mode=2, t=T, causal=causal)
        assert torch.equal(one[0].view(torch.int16), whole[hd].view(torch.int16)), hd


@pytest.mark.parametrize("seq,ldv", [(777, 781), (777, 784), (1111, 1115), (2100, 2103),
                                     (2100, 2104)])
@pytest.mark.parametrize("causal", [True, False])
def test_long_sequence_padded_vt_rows(q, causal, seq, ldv):
    g, r, ins = _run(q, 1, seq, 2, causal, 71, ldv=ldv, pad=float("nan"))
    _check(g, r, ins, seq, causal, "long padded s%d ldv%d" % (seq, ldv))


@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("heads,seq", [(2, 64), (3, 40), (1, 512), (2, 1000), (1, 1024),
                                       (1, 2049)])
def test_binary16_matches_oracle(q, mode, causal, heads, seq):
    g, r, ins = _run(q, heads, seq, mode, causal, 80 + seq, dt="f16")
    _check(g, r, ins, seq, causal, "f16 h%d s%d m%d c%d" % (heads, seq, mode, causal), "f16")


def test_binary16_full_workload(q):
    g, r, ins = _run(q, 96, 512, 2, True, 81, dt="f16")
    _check(g, r, ins, 512, True, "f16 full", "f16")


@pytest.mark.parametrize("mode", [0, 2])
def test_single_key_returns_v(q, mode):
    g, r, ins = _run(q, 4, 1, mode, False, 61)
    assert np.array_equal(g.reshape(4, 64), ins[2].reshape(4, 64))


@pytest.mark.parametrize("ldv", [208, 203])     # vector rows; element-wise rows
@pytest.mark.parametrize("causal", [True, False])
def test_padded_vt_rows_with_nan_padding(q, causal, ldv):
    g, r, ins = _run(q, 3, 200, 2, causal, 62, ldv=ldv, pad=float("nan"))
    _check(g, r, ins, 200, causal, "padded")


@pytest.mark.parametrize("seq", [64, 40])                  # whole key blocks; a ragged last one
@pytest.mark.parametrize("ldv", [1 << 24, (1 << 24) + 8])   # rows read as 16-byte vectors with
def test_vt_row_stride_at_the_lane_offset_limit(q, ldv, seq):  # the largest 32-bit lane offsets; past it
    """v^T rows 2^24 elements apart (2 GiB per head), NaN in the padding: the
    widest stride whose byte offsets within a 64-row block fit 32 bits, and the
    next one, which takes the element-wise path."""
    qc, kc, vtc = synth.attention_inputs(1, seq, 67 + seq)
    say("attention bf16 heads=1 seq=%d ldv=%d (2 GiB v^T)" % (seq, ldv))
    big = torch.full((1, 64, ldv), float("nan"), dtype=torch.bfloat16, device="cuda:0")
    big[:, :, :seq] = vtc.to("cuda:0")
    o = q.quake_attention(qc.to("cuda:0"), kc.to("cuda:0"), big[:, :, :seq], mode=2, t=T,
                          causal=True)
    torch.cuda.synchronize()
    del big
    ins = (host_bits(qc), host_bits(kc), host_bits(vtc))
    ref = oracle.attention(*ins, 2, T, True, threads=THREADS)
    _check(host_bits(o.cpu()), ref, ins, seq, True, "ldv %d seq %d" % (ldv, seq))


@pytest.mark.parametrize("causal", [True, False])
def test_longest_sequence_on_sampled_queries(q, causal):
    """131072 keys, the longest sequence accepted (one head, QuAKE2, two
    passes): queries across the sequence (both ends, query-tile and key-block
    edges, the middle) against the oracle's outputs for those queries."""
    seq = 131072
    say("attention bf16 heads=1 seq=%d causal=%d (sampled queries)" % (seq, causal))
    qc, kc, vtc = synth.attention_inputs(1, seq, 77)
    o = q.quake_attention(qc.to("cuda:0"), kc.to("cuda:0"), vtc.to("cuda:0"), mode=2, t=T,
                          causal=causal)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 31, 32, 1023, 1024, 65535, 65536, 99999, 131039, 131040, 131071])
    ins = (host_bits(qc), host_bits(kc), host_bits(vtc))
    got = np.ascontiguousarray(host_bits(o.cpu())[:, rows])
    ref = oracle.attention_rows(*ins, rows, 2, T, causal, threads=THREADS)
    _check_against(got, ref, _bound_rows(*ins, rows, causal, _dec(ref)),
                   "longest causal %d" % causal)


def test_full_workload_causal_quake2(q):
    """96 heads x 512 keys, the configuration the benchmark times."""
    g, r, ins = _run(q, 96, 512, 2, True, 63)
    _check(g, r, ins, 512, True, "full")


def test_bench_config_1024_keys_causal_quake2(q):
    """64 heads x 1024 keys, the eight-wave one-pass configuration the benchmark times."""
    g, r, ins = _run(q, 64, 1024, 2, True, 92)
    _check(g, r, ins, 1024, True, "64x1024 causal")


def test_bench_config_2048_keys_noncausal_quake2(q):
    """32 heads x 2048 keys without the mask, the two-pass configuration the benchmark times."""
    g, r, ins = _run(q, 32, 2048, 2, False, 93)
    _check(g, r, ins, 2048, False, "32x2048 non-causal")


def test_full_workload_noncausal_exact(q):
    g, r, ins = _run(q, 96, 512, 0, False, 64)
    _check(g, r, ins, 512, False, "full exact")


def test_deterministic_and_zero_sizes(q):
    qc, kc, vtc = synth.attention_inputs(8, 128, 65)
    qg, kg, vtg = qc.to("cuda:0"), kc.to("cuda:0"), vtc.to("cuda:0")
    a = q.quake_attention(qg, kg, vtg, mode=2, t=T)
    b = q.quake_attention(qg, kg, vtg, mode=2, t=T)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    e = torch.empty((0, 128, 64), dtype=torch.bfloat16, device="cuda:0")
    et = torch.empty((0, 64, 128), dtype=torch.bfloat16, device="cuda:0")
    assert q.quake_attention(e, e, et, mode=2).shape == (0, 128, 64)


def test_bad_arguments_raise(q):
    qc, kc, vtc = synth.attention_inputs(2, 64, 66)
    qg, kg, vtg = qc.to("cuda:0"), kc.to("cuda:0"), vtc.to("cuda:0")
    with pytest.raises(q.QuakeError):
        q.quake_attention(qg, kg, vtg, t=-1.0)
    with pytest.raises(q.QuakeError):
        q.quake_attention(qg.float(), kg.float(), vtg.float())
    with pytest.raises(ValueError):
        q.quake_attention(qg, kg, vtg, o=qg)            # output over an input
    big = torch.zeros((1, 131073, 64), dtype=torch.bfloat16, device="cuda:0")
    with pytest.raises(q.QuakeError):                     # longer than 131072 keys
        q.quake_attention(big, big, torch.zeros((1, 64, 131073), dtype=torch.bfloat16,
                                                device="cuda:0"))


def test_two_streams_at_once(q):
    """Two launches in flight on two streams (no shared state in the kernel)."""
    a = [x.to("cuda:0") for x in synth.attention_inputs(8, 512, 90)]
    b = [x.to("cuda:0") for x in synth.attention_inputs(16, 256, 91)]
    ref_a = q.quake_attention(*a, mode=2, t=T)
    ref_b = q.quake_attention(*b, mode=1, t=T, causal=False)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    outs_a, outs_b = [], []
    for _ in range(4):
        with torch.cuda.stream(s1):
            outs_a.append(q.quake_attention(*a, mode=2, t=T))
        with torch.cuda.stream(s2):
            outs_b.append(q.quake_attention(*b, mode=1, t=T, causal=False))
    torch.cuda.synchronize()
    for oa, ob in zip(outs_a, outs_b):
        assert torch.equal(oa.view(torch.int16), ref_a.view(torch.int16))
        assert torch.equal(ob.view(torch.int16), ref_b.view(torch.int16))
