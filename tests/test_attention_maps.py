"""Index maps of the fused attention kernel (csrc/attention.hip), restated and
checked on the CPU: the LDS slot maps of the K and V^T staging are bijective,
every slot read back is the slot written for the same (row, chunk), and no
16-byte access of the writes or the operand reads has a bank conflict, whether
the LDS serves 8 lanes per clock over 32 four-byte banks or 16 lanes over 64;
the probabilities reach the second product's B operand in the key order its A
operand (V^T) uses; the tile order is a bijection onto (head, query tile); the
live-block count per wave matches the blocks the wave owns (4 or 8 waves);
and the waves' share of the output tile covers it once."""
import itertools

import pytest


def kswz(r):
    return (r & 7) ^ ((r >> 3) & 1)


def vswz(d):
    return ((d >> 1) ^ (d >> 2)) & 3


def k_store(lane, j):               # load j of a K block: row 8j + lane/8, chunk lane%8
    r, c = 8 * j + (lane >> 3), lane & 7
    return (r, c), 8 * r + (c ^ kswz(r))


def k_read(lane, ks):               # A operand: key lane%32, dims 16ks + 8(lane/32) ..
    fr, h = lane & 31, lane >> 5
    c = 2 * ks + h
    return (fr, c), 8 * fr + (c ^ kswz(fr))


def v_store(lane, j):               # load j of a V^T block: dim 16j + lane/4, keys 8(lane%4) ..
    d, c = 16 * j + (lane >> 2), lane & 3
    return (d, c), 4 * d + (c ^ vswz(d))


def v_read(lane, ks, db):           # A operand: dim 32db + lane%32, keys 16ks + 8(lane/32) ..
    fr, h = lane & 31, lane >> 5
    d, c = 32 * db + fr, 2 * ks + h
    return (d, c), 4 * d + (c ^ vswz(d))


def _accesses():
    return {
        "k_store": [[k_store(l, j) for l in range(64)] for j in range(4)],
        "k_read": [[k_read(l, ks) for l in range(64)] for ks in range(4)],
        "v_store": [[v_store(l, j) for l in range(64)] for j in range(4)],
        "v_read": [[v_read(l, ks, db) for l in range(64)] for ks in range(2) for db in range(2)],
    }


@pytest.mark.parametrize("name", ["k_store", "k_read", "v_store", "v_read"])
def test_slot_maps_are_bijective_and_consistent(name):
    acc = _accesses()[name]
    slots = [s for ins in acc for _, s in ins]
    assert sorted(slots) == list(range(256))            # 4 KB = 256 slots, each once
    where = {}
    for ins in _accesses()[name.split("_")[0] + "_store"]:
        for key, s in ins:
            where[key] = s
    for ins in acc:                                      # a (row, chunk) lives in one slot
        for key, s in ins:
            assert where[key] == s


@pytest.mark.parametrize("lanes,banks", [(8, 32), (16, 64)])
@pytest.mark.parametrize("name", ["k_store", "k_read", "v_store", "v_read"])
def test_no_bank_conflicts(name, lanes, banks):
    for ins in _accesses()[name]:
        for g0 in range(0, 64, lanes):
            used = [(4 * s + b) % banks for _, s in ins[g0:g0 + lanes] for b in range(4)]
            assert len(used) == len(set(used)), (name, g0)


def permlane32_swap(a, b):
    """v_permlane32_swap: lanes 32-63 of the first operand trade places with
    lanes 0-31 of the second; returns (new first, new second)."""
    r0 = a[:32] + b[:32]
    r1 = a[32:] + b[32:]
    return r0, r1


def test_probabilities_reach_the_b_operand_in_key_order():
    # the S^T accumulator: lane l, register r holds key 8(r/4) + 4(l/32) + r%4 of the block
    acc = [[8 * (r // 4) + 4 * (l // 32) + r % 4 for r in range(16)] for l in range(64)]
    for ks in range(2):
        # dword pairs of groups 2ks and 2ks+1 (keys as pairs of bfloat16)
        g = [[(acc[l][4 * gi], acc[l][4 * gi + 1]) for l in range(64)] for gi in range(4)]
        g2 = [[(acc[l][4 * gi + 2], acc[l][4 * gi + 3]) for l in range(64)] for gi in range(4)]
        s0 = permlane32_swap(g[2 * ks], g[2 * ks + 1])
        s1 = permlane32_swap(g2[2 * ks], g2[2 * ks + 1])
        for l in range(64):
            operand = [*s0[0][l], *s1[0][l], *s0[1][l], *s1[1][l]]
            h = l // 32
            assert operand == [16 * ks + 8 * h + j for j in range(8)], (ks, l, operand)


@pytest.mark.parametrize("heads,qblocks", [(1, 1), (3, 16), (8, 1), (8, 16), (96, 16),
                                           (97, 3), (104, 2)])
def test_tile_order_is_a_bijection(heads, qblocks):
    seen = set()
    for b in range(heads * qblocks):
        if heads % 8 == 0:
            h8 = heads // 8
            x, slot = b & 7, b >> 3
            bh, qb = x * h8 + slot % h8, qblocks - 1 - slot // h8
        else:
            bh, qb = b // qblocks, qblocks - 1 - b % qblocks
        assert 0 <= bh < heads and 0 <= qb < qblocks
        seen.add((bh, qb))
    assert len(seen) == heads * qblocks


def _waves(seq):
    """Waves of the one-pass workgroup (four key blocks of 32 per wave), 0 for two passes."""
    return 4 if seq <= 512 else 8 if seq <= 1024 else 0


@pytest.mark.parametrize("seq,causal", itertools.product(
    [1, 31, 32, 33, 200, 511, 512, 513, 1000, 1024, 1025, 2047, 2048, 2049, 3000], [True, False]))
def test_live_blocks_per_wave(seq, causal):
    kblocks = (seq + 31) // 32
    w_count = _waves(seq) or 4
    for qb in range((seq + 31) // 32):
        nkb = min(kblocks, qb + 1) if causal else kblocks
        owned = 0
        for wave in range(w_count):
            nlive = max(0, int((nkb - wave + w_count - 1) / w_count))   # C++ division truncates
            blocks = [w_count * i + wave for i in range(nkb) if w_count * i + wave < nkb]
            assert nlive == len(blocks) and blocks == [w_count * i + wave for i in range(nlive)]
            if _waves(seq):
                assert nlive <= 4                  # the one-pass kernel holds four blocks per wave
            owned += nlive
        assert owned == nkb


@pytest.mark.parametrize("waves", [4, 8])
def test_output_rows_cover_the_tile_once(waves):
    """attn_finish: wave w sums accumulator rows R w .. R w + R - 1 (R = 32 / W);
    row j = 16 db + r of lane l is dim 32 db + 8 (r / 4) + 4 (l / 32) + r mod 4 of
    query l mod 32; stores are runs of 4 consecutive dims, 8-byte aligned."""
    rr = 32 // waves
    run = 4
    seen = set()
    for w in range(waves):
        for lane in range(64):
            for i0 in range(0, rr, run):
                dims = []
                for i in range(i0, i0 + run):
                    j = rr * w + i
                    db, r = j >> 4, j & 15
                    dims.append(32 * db + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3))
                assert dims == list(range(dims[0], dims[0] + run))
                assert (2 * dims[0]) % (2 * run) == 0          # byte offset in the row
                for d in dims:
                    seen.add((lane & 31, d))
    assert len(seen) == 32 * 64 and seen == {(qq, d) for qq in range(32) for d in range(64)}
