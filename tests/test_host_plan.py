"""The library's host code (registry, planner, round executor) compiled for
the CPU against a stub HIP runtime, with AddressSanitizer, and driven
through whole inference rounds of every workload. The stub's kernel
launchers check that every pointer range each kernel would read or write
lies inside one live allocation, and that any two launches (or weight
copies) that are not ordered by stream order, events or graph edges touch
no common bytes unless both only read them. Multi-stream plans, graph
rounds built from the launch dependencies (and as one chain), the
weight-swap schedule and split-K are all exercised. No GPU is needed."""

import json
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
STUB = os.path.join(ROOT, "tests", "hoststub")
LIB = os.path.join(ROOT, "_build", "libgemel_host.so")
CSRC = os.path.join(ROOT, "paper_2201_07705_amd", "csrc")


@pytest.fixture(scope="module")
def hostlib():
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    cmd = ["g++", "-std=c++17", "-g", "-O1", "-fsanitize=address",
           "-fno-omit-frame-pointer", "-fPIC", "-shared", f"-I{STUB}",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
           os.path.join(CSRC, "registry.cpp"), os.path.join(CSRC, "plan.cpp"),
           os.path.join(STUB, "hoststub.cpp"), "-o", LIB + f".{os.getpid()}"]
    subprocess.check_call(cmd)
    # atomic: parallel test workers may build and load it at the same time
    os.replace(LIB + f".{os.getpid()}", LIB)
    return LIB


def drive(lib, name, kw, opts, rounds=2):
    asan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"],
                                   text=True).strip()
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0")
    r = subprocess.run(["python", os.path.join(STUB, "drive.py"), lib, name,
                        json.dumps(kw), json.dumps(opts), str(rounds)],
                       capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stderr[-3000:]
    return json.loads(r.stdout.strip().splitlines()[-1])


CASES = [
    ("tiny2", {}, {}),
    ("resnet18x2", {}, {}),
    ("resnet18x2", {"res": 64, "frames": 3},
     {"OPT_STREAMS": 4, "OPT_USE_GRAPH": 0}),
    ("resnet18x2", {"res": 64, "frames": 3}, {"OPT_SPLIT_MERGED": 1}),
    ("r50x2_vgg16x2", {"res": 64, "frames": 2},
     {"OPT_STREAMS": 4, "OPT_USE_GRAPH": 0}),
    ("r50x2_vgg16x2", {}, {}),
    ("yolov3x3", {"res": 96, "frames": 2},
     {"OPT_STREAMS": 8, "OPT_USE_GRAPH": 0}),
    ("yolov3x3", {"res": 96, "frames": 2}, {}),
    ("yolov3x3", {"res": 96, "frames": 2},
     {"OPT_STREAMS": 8, "OPT_FORK_US": 0}),
    ("r50x2_vgg16x2", {"res": 64, "frames": 2},
     {"OPT_STREAMS": 8, "OPT_FORK_US": 0, "OPT_GRAPH_DAG": 1,
      "OPT_AUTOTUNE": 0}),
    ("r50x2_vgg16x2", {"res": 64, "frames": 2}, {"ROUNDS": 14}),
    ("r50x2_vgg16x2", {"res": 64, "frames": 2},
     {"OPT_CONV_SPLITS": 4, "OPT_STREAMS": 8, "OPT_FORK_US": 0,
      "OPT_SPLITK_FUSED": 2}),
    ("r50x2_vgg16x2", {"res": 64, "frames": 2},
     {"OPT_CONV_SPLITS": 4, "OPT_STREAMS": 8, "OPT_FORK_US": 0,
      "OPT_SPLITK_FUSED": 0}),
    ("yolov3x3", {"res": 96, "frames": 2}, {"OPT_TUNE": 0}),
    ("mix8_budget40", {"res": 32, "frames": 2}, {}),
    ("variants", {"res": 32, "frames": 2}, {}),
    ("mix8_budget40", {"res": 32, "frames": 2},
     {"OPT_SWAP_SLOT_BYTES": 1 << 20, "OPT_SWAP_SLOTS": 2,
      "OPT_STREAMS": 3, "OPT_USE_GRAPH": 0}),
]


@pytest.mark.parametrize("name,kw,opts", CASES,
                         ids=[f"{c[0]}-{i}" for i, c in enumerate(CASES)])
def test_every_kernel_access_in_bounds(hostlib, name, kw, opts):
    opts = dict(opts)
    rounds = opts.pop("ROUNDS", 2)
    out = drive(hostlib, name, kw, opts, rounds)
    assert out["status"] == [0] * rounds, out["error"]
    assert out["selftest"] == 1
    assert out["hazards"] == 0, out["last"]
    assert out["violations"] == 0, out["last"]
    assert out["launches"] >= out["plan_launches"] > 0
    if name == "mix8_budget40":
        assert out["streamed"] > 0


def test_all_groups_merged_still_batches_across_models(hostlib):
    """With every candidate group merged, groups hold several appearances of
    one model that depend on each other (repeated blocks); the plan batches
    the k-th appearance of each model together and splits only nodes on a
    dependency cycle, so it has fewer launches than running every member
    separately."""
    merged = drive(hostlib, "variants", {"res": 32, "frames": 2}, {}, 1)
    split = drive(hostlib, "variants", {"res": 32, "frames": 2},
                  {"OPT_SPLIT_MERGED": 1}, 1)
    for out in (merged, split):
        assert out["status"] == [0] and out["violations"] == 0 and out["hazards"] == 0, out
    assert merged["plan_launches"] < split["plan_launches"]
