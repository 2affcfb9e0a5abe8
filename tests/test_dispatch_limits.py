"""The softmax kernels' row-length limits as the source defines them, checked
against the limits the C header documents and the boundaries the GPU tests
exercise (CPU only; reads the sources, runs nothing)."""
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = open(os.path.join(ROOT, "paper_2412_00408_amd", "csrc", "softmax.hip")).read()
HDR = open(os.path.join(ROOT, "include", "quake.h")).read()


def _int(pattern):
    return int(re.search(pattern, SRC).group(1))


def _shape():
    m = re.search(r"struct ResShape \{(.*?)\};", SRC, re.S).group(1)
    f = {k: (int(a), int(b)) for k, a, b in re.findall(r"(NK2|NK1|NL1) = \(DT == F32\) \? (\d+) : (\d+);", m)}
    return f


def test_resident_capacity_matches_the_header():
    block = _int(r"constexpr int kResBlock = (\d+);")
    s = _shape()
    f32 = (s["NK1"][0] + s["NL1"][0]) * block * 4
    b16 = (s["NK1"][1] + s["NL1"][1]) * block * 8
    assert (f32, b16) == (129024, 131072)
    text = " ".join(" ".join(l.strip().lstrip("*") for l in HDR.splitlines()).split())
    assert "up to 129024 (binary32) or 131072 (16-bit) elements" in text


def test_resident_lds_and_register_shapes_fit():
    block = _int(r"constexpr int kResBlock = (\d+);")
    s = _shape()
    for i, v in ((0, 4), (1, 8)):
        lds = s["NL1"][i] * block * v * 4 + (block // 64) * (4 + 8)
        assert lds <= 160 * 1024
        # the register shapes nest: two workgroups per CU, then one, then LDS
        assert s["NK2"][i] < s["NK1"][i]


def test_gpu_tests_cover_each_resident_shape_boundary():
    src = open(os.path.join(ROOT, "tests", "test_gpu_softmax.py")).read()
    cols = re.search(r"RESIDENT_COLS = \{(.*?)\}\n", src, re.S).group(1)
    f32 = [int(c) for c in re.search(r'"f32": \[([^\]]*)\]', cols).group(1).split(",")]
    bf = [int(c) for c in re.search(r'"bf16": \[([^\]]*)\]', cols).group(1).split(",")]
    block = _int(r"constexpr int kResBlock = (\d+);")
    s = _shape()
    for lst, i, v in ((f32, 0, 4), (bf, 1, 8)):
        for n in (s["NK2"][i], s["NK1"][i], s["NK1"][i] + s["NL1"][i]):
            last = n * block * v
            assert last in lst and last + v in lst, (v, last)


def test_split_chunk_is_the_documented_16384():
    assert _int(r"constexpr int64_t kChunkElems = (\d+);") == 16384
    assert "ceil(cols / 16384)" in HDR
