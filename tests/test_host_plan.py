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
           os.path.join(CSRC, "batching.cpp"), os.path.join(STUB, "hoststub.cpp"), "-o", LIB + f".{os.getpid()}"]
    subprocess.check_call(cmd)
    # atomic: parallel test workers may build and load it at the same time
    os.replace(LIB + f".{os.getpid()}", LIB)
    return LIB


def drive(lib, name, kw, opts, rounds=2, scenario=None):
    asan = subprocess.check_output(["gcc", "-print-file-name=libasan.so"],
                                   text=True).strip()
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0")
    r = subprocess.run(["python", os.path.join(STUB, "drive.py"), lib, name,
                        json.dumps(kw), json.dumps(opts), str(rounds),
                        json.dumps(scenario or {})],
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
    # small staging slots: many segments per round, slots reused in a round
    ("mix8_budget40", {"res": 32, "frames": 1},
     {"OPT_SWAP_SLOT_BYTES": 1 << 20, "OPT_SWAP_SLOTS": 2}),
    ("variants", {"res": 32, "frames": 2}, {}),
    ("many", {"n": 18, "dtype": "bf16"}, {}),
    ("many", {"n": 18, "dtype": "f32"}, {"OPT_STREAMS": 4, "OPT_USE_GRAPH": 0}),
    ("chain", {"route": True}, {}),
    # grouped launches of ragged segments, fused split-K (one arrival
    # counter per output tile of every segment)
    ("grouped", {"case": 1}, {"OPT_GROUP_UNMERGED": 1, "OPT_CONV_TILE": 12,
                              "OPT_CONV_SPLITS": 3, "OPT_SPLITK_FUSED": 2}),
    ("grouped", {"case": 0}, {"OPT_GROUP_UNMERGED": 1, "OPT_CONV_TILE": 9,
                              "OPT_CONV_SPLITS": 3, "OPT_SPLITK_FUSED": 2}),
    ("yolov3x3", {"res": 96, "frames": 2},
     {"OPT_GROUP_UNMERGED": 1, "OPT_CONV_SPLITS": 3, "OPT_SPLITK_FUSED": 2,
      "OPT_STREAMS": 8, "OPT_FORK_US": 0}),
    ("r50x2_vgg16x2", {"res": 64, "frames": 2},
     {"OPT_GROUP_UNMERGED": 1, "OPT_CONV_SPLITS": 3, "OPT_SPLITK_FUSED": 0}),
    ("chain", {"route": True}, {"OPT_CONV_SPLITS": 3, "OPT_SPLITK_FUSED": 0}),
    ("chain", {"route": False}, {"OPT_CONV_SPLITS": 2, "OPT_SPLITK_FUSED": 2}),
]


def _case_args(case):
    name, kw, opts = case
    opts = dict(opts)
    rounds = opts.pop("ROUNDS", 2)
    return name, kw, opts, rounds


@pytest.fixture(scope="module")
def case_results(hostlib, request):
    """Without pytest-xdist (one process runs every test), drive the
    selected cases below at once, six subprocesses at a time; the tests
    then read their results. Under xdist each test drives its own case."""
    if os.environ.get("PYTEST_XDIST_WORKER"):
        return {}
    selected = sorted({item.callspec.params["idx"] for item in request.session.items
                       if item.originalname == "test_every_kernel_access_in_bounds"})
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=6) as ex:
        futs = {i: ex.submit(drive, hostlib, *_case_args(CASES[i])) for i in selected}
        out = {}
        for i, f in futs.items():
            try:
                out[i] = f.result()
            except Exception:     # the test drives the case again and reports
                pass
    return out


@pytest.mark.parametrize("idx", range(len(CASES)),
                         ids=[f"{c[0]}-{i}" for i, c in enumerate(CASES)])
def test_every_kernel_access_in_bounds(hostlib, case_results, idx):
    name, kw, opts, rounds = _case_args(CASES[idx])
    out = case_results.get(idx) or drive(hostlib, name, kw, opts, rounds)
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


def test_conv_launches_prefetch_the_next_conv_weights(hostlib):
    """In a round that moves more bytes than the memory-side cache holds (2x
    ResNet-50 + 2x VGG-16 at 224 px: about 2.1 GB), a conv launch names the
    weights of the next conv launch on its stream as its prefetch region,
    checked like every other access (a live allocation, in bounds); with
    OPT_PREFETCH 0 none does, nor in a round that fits the cache (2x
    ResNet-18, 4 frames each: about 176 MB) unless OPT_PREFETCH is 2."""
    on = drive(hostlib, "r50x2_vgg16x2", {}, {}, 1)
    off = drive(hostlib, "r50x2_vgg16x2", {}, {"OPT_PREFETCH": 0}, 1)
    small = drive(hostlib, "resnet18x2", {}, {}, 1)
    forced = drive(hostlib, "resnet18x2", {}, {"OPT_PREFETCH": 2}, 1)
    for out in (on, off, small, forced):
        assert out["status"] == [0] and out["violations"] == 0 and out["hazards"] == 0, out["last"]
    assert on["prefetches"] > 0 and off["prefetches"] == 0 and small["prefetches"] == 0
    assert on["plan_prefetches"] > 0 and off["plan_prefetches"] == 0 and small["plan_prefetches"] == 0
    assert forced["plan_prefetches"] > 0
    assert on["launches"] == off["launches"]


ESTATE, EDEVICE = -7, -6


@pytest.mark.parametrize("name,kw,opts", [
    ("r50x2_vgg16x2", {"res": 64, "frames": 2}, {}),
    ("r50x2_vgg16x2", {"res": 64, "frames": 2}, {"OPT_USE_GRAPH": 0}),
    ("yolov3x3", {"res": 96, "frames": 2}, {"OPT_STREAMS": 8, "OPT_FORK_US": 0}),
])
def test_rounds_on_alternating_streams_are_ordered(hostlib, name, kw, opts):
    """Rounds share the plan's arena, split-K regions and counters: a round
    on another stream than the previous one waits for it, so no two
    launches of different rounds touch common bytes unordered."""
    out = drive(hostlib, name, kw, opts, 5, {"streams": [0, 1, 1, 0, 2]})
    assert out["status"] == [0] * 5, out["error"]
    assert out["hazards"] == 0 and out["violations"] == 0, out["last"]


@pytest.mark.parametrize("opts", [{}, {"OPT_AUTOTUNE": 0},
                                  {"OPT_USE_GRAPH": 0}, {"OPT_STREAMS": 1}])
def test_captured_round_uses_the_callers_stream_only(hostlib, opts):
    """While the caller's stream is being captured, a round whose plan and
    weights exist enqueues every launch on that stream alone: no worker
    stream, event, allocation or synchronisation (the stub flags each),
    in a valid order (the ordering check covers the captured launches),
    and as many launches as the plan has."""
    out = drive(hostlib, "r50x2_vgg16x2", {"res": 64, "frames": 2}, opts, 3,
                {"capture": [1]})
    assert out["status"] == [0, 0, 0], out["error"]
    assert out["hazards"] == 0 and out["violations"] == 0, out["last"]
    assert out["round_launches"][1] == out["plan_launches"]


def test_capture_before_the_first_round_is_refused(hostlib):
    """A first round needs allocations and synchronous copies (weight
    placement, plan): under capture it is refused with ESTATE before any
    of them, and the next round outside capture still works."""
    out = drive(hostlib, "resnet18x2", {"res": 64, "frames": 2}, {}, 2,
                {"capture": [0]})
    assert out["status"] == [ESTATE, 0], out["error"]
    assert out["violations"] == 0 and out["hazards"] == 0, out["last"]
    assert out["round_launches"][0] == 0


def test_captured_round_that_streams_weights_is_refused(hostlib):
    out = drive(hostlib, "mix8_budget40", {"res": 32, "frames": 2}, {}, 2,
                {"capture": [1]})
    assert out["status"] == [0, ESTATE], out["error"]
    assert out["violations"] == 0 and out["hazards"] == 0, out["last"]


@pytest.mark.parametrize("at,opts,streams", [
    (1, {}, [0, 0, 0, 1]),                      # before the first launch
    (7, {}, [0, 0, 0, 1]),
    (20, {"OPT_STREAMS": 1}, [0, 0, 0, 1]),
    (3, {}, [0, 0, 1, 2]),                      # next round on another stream
    (20, {}, [0, 0, 1, 2]),
])
def test_copy_failure_part_way_leaves_rounds_ordered(hostlib, at, opts,
                                                     streams):
    """A weight copy that fails after launches (and the fork to worker
    streams) were enqueued: the round returns EDEVICE, its partial work is
    joined back to the caller's stream, and the next rounds, on the same
    and on other streams (also the round right after the failure), are
    ordered after it (no hazard)."""
    out = drive(hostlib, "mix8_budget40", {"res": 32, "frames": 2},
                dict(opts, OPT_SWAP_SLOT_BYTES=1 << 20, OPT_SWAP_SLOTS=2), 4,
                {"fail": {"1": at}, "streams": streams})
    assert out["status"] == [0, EDEVICE, 0, 0], out["error"]
    assert out["hazards"] == 0 and out["violations"] == 0, out["last"]


ENOMEM = -2


@pytest.mark.parametrize("name,kw,opts", [
    ("resnet18x2", {"res": 64, "frames": 2}, {}),
    # a weight budget: staging slots and pinned host copies as well
    ("resnet18x2", {"res": 64, "frames": 2},
     {"OPT_WEIGHT_BUDGET": 12000000, "OPT_SWAP_SLOT_BYTES": 1 << 20,
      "OPT_SWAP_SLOTS": 2}),
])
def test_allocation_failures_report_enomem_and_leak_nothing(hostlib, name,
                                                            kw, opts):
    """The n-th device or pinned allocation of the first round fails, for
    every n the round makes: the round reports ENOMEM (or, when the failed
    allocation was the scratch of plan-time tuning, succeeds untuned), the
    next round succeeds, nothing is left half-enqueued, and the destroyed
    context holds no memory."""
    base = drive(hostlib, name, kw, opts, 1)
    assert base["status"] == [0] and base["leaked"] == 0
    A = base["allocs"]
    assert A >= 3
    # every allocation when there are few; else the first and last ones
    # (weight pool, staging, plan buffers) and a sample of the pinned copies
    ns = sorted(set(range(1, A + 1)) if A <= 24 else
                set(range(1, 6)) | set(range(A - 7, A + 1)) |
                {A // 4, A // 2, 3 * A // 4})
    out = drive(hostlib, name, kw, opts, 2,
                {"each": [{"fail_alloc": {"0": n}} for n in ns]})
    assert out["violations"] == 0 and out["hazards"] == 0, out["last"]
    seen_enomem = 0
    for n, r in zip(ns, out["runs"]):
        assert r["status"][0] in (0, ENOMEM), (n, r["error"])
        assert r["status"][1] == 0, (n, r["error"])
        assert r["leaked"] == 0, n
        seen_enomem += r["status"][0] == ENOMEM
    assert seen_enomem >= 3


EBUDGET = -5


@pytest.mark.parametrize("name,kw,opts", [
    ("resnet18x2", {"res": 64, "frames": 2}, {}),
    ("yolov3x3", {"res": 96, "frames": 2}, {}),
    ("r50x2_vgg16x2", {"res": 64, "frames": 2},
     {"OPT_CONV_SPLITS": 3, "OPT_SPLITK_FUSED": 2}),
])
def test_noalloc_rounds_allocate_nothing_and_use_one_stream(hostlib, name, kw,
                                                           opts):
    """gemel_infer_noalloc after a normal round: no device allocation, every
    access inside the static scratch or other live buffers, no hazard with
    the normal rounds before and after it, and (under capture) only the
    caller's stream, with no synchronisation."""
    # the captured round comes last: captured work runs only when its graph
    # is replayed, which the caller orders against other rounds
    out = drive(hostlib, name, kw, opts, 5,
                {"noalloc": [1, 2, 4], "capture": [4], "streams": [0, 0, 1, 1, 1]})
    assert out["status"] == [0] * 5, out["error"]
    assert out["hazards"] == 0 and out["violations"] == 0, out["last"]
    assert out["round_allocs"][1] == out["round_allocs"][2] == 0
    assert out["round_allocs"][4] == 0


def test_noalloc_refuses_unplaced_weights_and_oversized_rounds(hostlib):
    out = drive(hostlib, "resnet18x2", {"res": 64, "frames": 2}, {}, 2,
                {"noalloc": [0, 1]})
    assert out["status"] == [ESTATE, ESTATE], out["error"]
    assert out["round_launches"] == [0, 0]
    # full-size VGG-16 activations exceed the static scratch
    out = drive(hostlib, "r50x2_vgg16x2", {}, {}, 2, {"noalloc": [1]})
    assert out["status"] == [0, EBUDGET], out["error"]
    assert "static scratch" in out["error"]
    assert out["round_launches"][1] == 0 and out["round_allocs"][1] == 0


@pytest.mark.parametrize("name,kw,per_round", [
    ("mix8_budget40", {"res": 32, "frames": 1}, 1),
    ("mix8_budget40", {"res": 32, "frames": 1}, 2),
    ("r50x2_vgg16x2", {"res": 32, "frames": 1}, 1),
])
def test_weight_cache_rounds_follow_the_swap_oracle(hostlib, name, kw,
                                                    per_round):
    """Time-shared rounds over subsets of the models, in the library's
    sharing-aware load order, two cycles, with the weight cache: every
    round's loaded, evicted and cached bytes equal the swap oracle's
    (oracle/swap.py), the load order equals the oracle's, and every access
    stays in bounds and ordered."""
    from oracle import swap as S
    from swapcase import schedule
    from workloads import configs
    wl = configs.get(name, **kw)
    sc = schedule(wl, per_round)
    rounds, order, need = sc.rounds, sc.order, sc.need
    sizes, users, pm = sc.sizes, sc.users, sc.per_model
    cycle = rounds[:len(rounds) // 2]
    opts = {"OPT_SWAP_CACHE": 1, "OPT_WEIGHT_BUDGET": sc.budget}
    out = drive(hostlib, name, kw, opts, len(rounds), {"rounds": rounds})
    assert out["status"] == [0] * len(rounds), out["error"]
    assert out["cache_capacity"] >= need
    assert out["hazards"] == 0 and out["violations"] == 0, out["last"]
    assert out["load_order"] == order
    want = S.simulate(sizes, users, pm, out["cache_capacity"], rounds)
    got = out["cache"]
    assert [w[:3] for w in want] == [tuple(g) for g in got], (want, got)
    # the second cycle reloads less than the first (shared layers stay)
    first = sum(w[0] for w in want[:len(cycle)])
    second = sum(w[0] for w in want[len(cycle):])
    assert 0 < second <= first


def test_profile_batches_runs_every_batch_and_frees_its_buffers(hostlib):
    """gemel_profile_batches on the CPU stub: one plan per (model, batch),
    every launch in bounds and ordered, a full nondecreasing cost table
    (the stub's event clock reads 0.001 ms per pair), no plan kept, and the
    rounds after it still run; the context frees everything at the end."""
    out = drive(hostlib, "r50x2_vgg16x2", {"res": 32, "frames": 1}, {}, 2,
                {"profile": [3, 2]})
    prof = out["profile"]
    assert prof["status"] == 0, prof["error"]
    assert prof["plans_after"] == 0          # plans dropped
    assert prof["table"] == [0.001 * 1.0] * len(prof["table"]) or \
        all(abs(x - 0.001) < 1e-6 for x in prof["table"])
    assert len(prof["table"]) == 4 * 3
    assert out["status"] == [0, 0], out["error"]
    assert out["hazards"] == 0 and out["violations"] == 0, out["last"]
    assert out["leaked"] == 0
