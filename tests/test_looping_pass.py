"""The kernel-looping compiler pass (Sec. 3) on a toy kernel-call IR
(paper_2410_23668_amd/looping, C++), CPU only.

Pinned to the paper's worked examples (Sec. 3.3, Fig. 8 (a)-(d): usage
properties, LiveAfter, collapsed call, buffers and stores, in
tests/golden/looping_examples.json); the lattice join checked against an
independent reading of Fig. 6b on every pair and triple; every rewritten
program run by an interpreter next to the original, with every live output
bit-identical (the rewrite is semantics-preserving, Sec. 3.2) and every
on-chip intermediate left unwritten; two planted mistakes (a missing double
buffer, a chain without the uniqueness condition) must change an output;
2000 seeded random programs."""
import json
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "tests", "cpu", "looping_examples.cpp"),
       os.path.join(ROOT, "paper_2410_23668_amd", "looping", "kl_looping.cpp")]
INC = os.path.join(ROOT, "paper_2410_23668_amd", "looping")
GOLD = json.load(open(os.path.join(ROOT, "tests", "golden", "looping_examples.json")))


@pytest.fixture(scope="module")
def out(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("looping") / "looping_examples")
    subprocess.run([gxx, "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-I", INC,
                    "-o", exe] + SRC, check=True)
    r = subprocess.run([exe, "--fuzz", "2000"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    lines = [json.loads(l) for l in r.stdout.splitlines() if l.strip()]
    res = {"examples": {l["example"]: l for l in lines if "example" in l}}
    for l in lines:
        if "example" not in l:
            res.update(l)
    return res


@pytest.mark.parametrize("name", ["a", "b", "c", "d"])
def test_paper_examples(out, name):
    want = GOLD["examples"][name]
    got = out["examples"][name]
    assert got["calls_after"] == 1 and got["equivalent"] and got["untouched"]
    (loop,) = got["loops"]
    assert sorted(loop["live_after"]) == sorted(want["live_after"])
    assert loop["props"] == want["props"]
    assert loop["call"] == want["call"]
    assert loop["buffers"] == want["buffers"]
    assert loop["stores_each_iteration"] == want["stores_each_iteration"]
    assert loop["stores_at_end"] == want["stores_at_end"]
    # grouped exactly where Eq. 3 says: Live, or neither Local nor Const
    for p, P in loop["props"].items():
        grouped = "Live" in P or ("Local" not in P and "Const" not in P)
        assert (p in loop["grouped"]) == grouped, (p, P)


def test_decoder_layers_collapse_into_one_looped_call(out):
    # weights grouped over the layers, the hidden state chained on chip, the
    # per-layer caches grouped and stored every layer, the shared table Const
    for name, y in (("decoder", "{Local,Out}"), ("decoder_dump_hidden", "{Local,Live,Out}")):
        got = out["examples"][name]
        assert got["calls_before"] == 4 and got["calls_after"] == 1
        assert got["equivalent"] and got["untouched"]
        (loop,) = got["loops"]
        assert loop["props"] == {"wa": "{In}", "wb": "{In}", "cs": "{Const,In}",
                                 "x": "{In,Local}", "y": y, "kv": "{In,Live,Out}"}
        assert loop["call"][2] == ["cs"] and loop["call"][3] == ["x0"]
        assert loop["call"][5] == ["kv0", "kv1", "kv2", "kv3"]
        if name == "decoder":   # (rule 10: the last hidden state once, at the end)
            assert loop["call"][4] == ["x4"] and loop["stores_at_end"] == ["y"]
        else:                   # (rule 8: every layer's output stored)
            assert loop["call"][4] == ["x1", "x2", "x3", "x4"]
            assert loop["stores_each_iteration"] == ["y"]


def test_cases_that_must_not_chain_or_match(out):
    ex = out["examples"]
    # the same output every call: {Const} joined with {Out} is the top
    assert ex["same_output"]["calls_after"] == 2 and ex["same_output"]["loops"] == []
    # writes covering half of the next call's reads; an intermediate named
    # again two calls later; an intermediate re-read by a later call of the
    # list: grouped, never Local
    for name in ("half_write", "ping_pong", "reread_chain"):
        (loop,) = ex[name]["loops"]
        assert loop["buffers"] == [] and all("Local" not in P for P in loop["props"].values())
        assert ex[name]["equivalent"]


def test_greedy_driver_collapses_each_run(out):
    m = out["examples"]["mixed"]
    assert m["calls_before"] == 6 and m["calls_after"] == 3 and m["equivalent"]
    assert [(l["kernel"], l["first"], l["count"]) for l in m["loops"]] == [
        ("kernel_c", 0, 3), ("kernel_b", 4, 2)]


def test_lattice_join_matches_the_figure(out):
    assert out["lattice_mismatches"] == 0


def test_planted_mistakes_change_an_output(out):
    assert out["planted_single_buffer_detected"]
    assert out["planted_chain_without_uniqueness_detected"]


def test_random_programs_keep_their_outputs(out):
    assert out["fuzz_programs"] == 2000 and out["fuzz_failures"] == 0
    # the random programs reach every kind of rewrite
    assert out["looped_kernels"] > 1000 and out["buffers"] > 300
    assert out["double_buffers"] > 100
    assert out["stores_each_iteration"] > 100 and out["stores_at_end"] > 100
