"""The benchmark's multiply-add counts (the flop figure of its roofline) equal
the multiply-adds that the generated sweep code performs per edge and channel.

The table generator is built and run here (g++, no GPU); the operations of
each group's per-edge contraction are counted in its output (every fused multiply-add and
every plain product) and compared with bench.fma_counts, which derives the
same figures from the plan's coupling records."""
import os
import shutil
import subprocess

import pytest

import bench
from paper_2609_35099_amd import e3mi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_35099_amd", "csrc")

VARIANTS = [
    ("8x0e+8x1o", 2, 2, "V_x01_s2_o2"),
    ("32x0e+32x1o+32x2e", 2, 2, "V_x012_s2_o2"),
    ("64x0e+64x1o", 3, 3, "V_x01_s3_o3"),
    ("128x0e+128x1o+128x2e", 3, 3, "V_x012_s3_o3"),
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, "V_x0123_s3_o3"),
    ("128x1o+128x0e+128x3o+128x2e", 3, 3, "V_x1032_s3_o3"),
]


@pytest.fixture(scope="module")
def generated(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("needs g++")
    d = tmp_path_factory.mktemp("gen")
    exe = str(d / "e3gen")
    subprocess.run(["g++", "-O1", "-std=c++17", "-o", exe, os.path.join(CSRC, "gen.cpp"),
                    os.path.join(CSRC, "builder.cpp")], check=True)
    subprocess.run([exe, str(d)], check=True)
    return (d / "variants.inc").read_text()


def _edge_ops(text, tag, kind):
    """Multiply-adds in the per-edge contraction of every group of one kind
    (FG: forward, BG: backward) of a variant."""
    total, g = 0, 0
    while f"struct {tag}::{kind}<{g}>" in text:
        i = text.index(f"struct {tag}::{kind}<{g}>")
        body = text[i:text.index("\n};", i)]
        body = body[body.index("static void edge("):]
        nxt = body.find("__device__", 1)  # the next member function (edge3) is not counted
        body = body if nxt < 0 else body[:nxt]
        total += body.count("e3fma(") + body.count(" * ")
        g += 1
    assert g > 0, (tag, kind)
    return total


@pytest.mark.parametrize("irreps,lsh,lout,tag", VARIANTS)
def test_bench_counts_equal_generated_code(generated, irreps, lsh, lout, tag):
    fwd, bwd = bench.fma_counts(e3mi.Plan(irreps, lsh, lout))
    assert fwd == _edge_ops(generated, tag, "FG")
    assert bwd == _edge_ops(generated, tag, "BG")


def test_backward_routes_cheaper_than_the_plain_order():
    """The per-path orders never cost more than the single order they replaced
    (two per entry, one per coupling coefficient, one per output row, two per
    harmonic row)."""
    plan = e3mi.Plan("128x0e+128x1o+128x2e+128x3o", 3, 3)
    i0, i1, _, val = plan.records()
    pairs = len(set(zip(i0.tolist(), i1.tolist())))
    s2 = sum(2 * int(p[1]) + 1 for p in plan.paths())
    plain = 2 * pairs + len(val) + plan.D_out + 2 * s2
    assert plain == 2161
    assert bench.fma_counts(plan)[1] < plain
