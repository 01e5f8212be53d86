"""C ABI tests that need no GPU: the library loads, exports every function
include/gemel.h declares, validates arguments before touching the device,
accounts bytes of merged and unmerged weights, and rejects merges of layers
that are not architecturally identical (Section 4.1)."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2201_07705_amd import gemel as G
from workloads import configs, zoo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    txt = open(os.path.join(ROOT, "include", "gemel.h")).read()
    return sorted(set(re.findall(r"\b(gemel_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_function():
    lib = G.lib()
    declared = header_functions()
    assert set(declared) == set(G.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_header_compiles_as_c_and_cxx():
    import subprocess
    h = os.path.join(ROOT, "include", "gemel.h")
    for lang in ("c", "c++"):
        r = subprocess.run(["gcc", "-fsyntax-only", "-Wall", "-Werror", "-x",
                            lang, h], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_library_is_newer_than_its_sources():
    import glob
    lib = os.path.join(ROOT, "paper_2201_07705_amd", "libgemel.so")
    srcs = glob.glob(os.path.join(ROOT, "paper_2201_07705_amd", "csrc", "*")) \
        + [os.path.join(ROOT, "include", "gemel.h")]
    newest = max(os.path.getmtime(p) for p in srcs)
    assert os.path.getmtime(lib) >= newest, "libgemel.so is stale: rebuild"


def test_kernels_use_no_scratch_memory():
    """Every HIP kernel of the build keeps its state in registers and LDS:
    no per-lane scratch (a by-value argument block indexed with a computed
    segment number, or a register spill, would put it there and cost an
    order of magnitude in memory traffic)."""
    import json
    from paper_2201_07705_amd import build as B
    assert os.path.getmtime(B.RESOURCES) >= os.path.getmtime(B.LIB) - 60
    res = json.load(open(B.RESOURCES))
    assert len(res) >= 30
    bad = {k: v for k, v in res.items() if v.get("scratchsize", 0)}
    assert not bad, bad


def test_header_enums_match_binding():
    txt = open(os.path.join(ROOT, "include", "gemel.h")).read()
    for name, val in [("GEMEL_EBUDGET", G.EBUDGET), ("GEMEL_OP_CONCAT", 5),
                      ("GEMEL_Q_GRAPH_REPLAYS", G.Q_GRAPH_REPLAYS),
                      ("GEMEL_OPT_WEIGHT_BUDGET", G.OPT_WEIGHT_BUDGET)]:
        m = re.search(rf"{name}\s*=\s*(-?\d+)", txt)
        assert m and int(m.group(1)) == val, name
    # every query key and option of the header, by name, in the binding
    for prefix in ("Q", "OPT"):
        found = re.findall(rf"GEMEL_{prefix}_(\w+)\s*=\s*(\d+)", txt)
        assert found
        for name, val in found:
            assert getattr(G, f"{prefix}_{name}") == int(val), name
    # kernel families: the binding's names in GEMEL_K_* order
    fams = dict((int(v), n) for n, v in
                re.findall(r"GEMEL_K_(\w+)\s*=\s*(\d+)", txt))
    count = fams.pop(max(fams))
    assert count == "COUNT" and len(G.KERNEL_FAMILIES) == len(fams)
    for i, n in fams.items():
        assert G.KERNEL_FAMILIES[i] == n.lower(), (i, n)
    assert ctypes.sizeof(G.LayerDesc) == 4 * 14 + 8 * 6 + 8


def _ctx(dtype="bf16"):
    return G.Context(0, dtype, 0)


def _tiny_params():
    return configs.tiny2().params(0)


def test_create_rejects_bad_arguments():
    h = ctypes.c_void_p()
    assert G.lib().gemel_create(None, 0, 1, 0) == G.EINVAL
    assert G.lib().gemel_create(ctypes.byref(h), -1, 1, 0) == G.EINVAL
    assert G.lib().gemel_create(ctypes.byref(h), 0, 7, 0) == G.EINVAL
    assert b"dtype" in G.lib().gemel_last_error(None)
    assert G.lib().gemel_destroy(None) == G.OK


def test_register_merge_and_accounting():
    w = configs.resnet18x2()
    c = _ctx()
    ids = [c.register_model(m.layers, w.params(i), m.in_chw)
           for i, m in enumerate(w.models)]
    assert ids == [0, 1]
    un = c.query(G.Q_UNMERGED_BYTES)
    assert c.query(G.Q_MERGED_BYTES) == un
    c.merge(w.groups)
    merged = c.query(G.Q_MERGED_BYTES)
    # one copy per merged layer: the second model only adds its FC head
    fc_b = 80 * 512 * 2 + 2 * 80 * 4
    r18 = w.models[0].layers
    # stored bytes of one ResNet-18 in kernel layout: bf16 weights with the
    # stem's 3 input channels padded to 8, plus fp32 scale and shift
    own = 0
    for l in r18:
        if l["op"] == "conv":
            cin_p = -(-l["cin"] // 8) * 8
            own += l["cout"] * l["kh"] * l["kw"] * cin_p * 2 + l["cout"] * 8
        elif l["op"] == "fc":
            own += l["cout"] * l["cin"] * 2 + l["cout"] * 8
    assert merged == own + fc_b
    # replacing the map with nothing unmerges
    c.merge([])
    assert c.query(G.Q_MERGED_BYTES) == un
    assert c.query(G.Q_N_MODELS) == 2
    assert c.n_outputs(0) == 1 and c.output_shape(1, 0, 4) == (4, 80)
    c.close()


def test_merge_rejects_non_identical_layers_without_state_change():
    w = configs.resnet18x2()
    c = _ctx()
    for i, m in enumerate(w.models):
        c.register_model(m.layers, w.params(i), m.in_chw)
    c.merge(w.groups[:3])
    before = c.query(G.Q_MERGED_BYTES)
    names = [l["name"] for l in w.models[0].layers]
    a = names.index("layer1.0.conv1")     # 64 -> 64, 3x3
    b = names.index("layer2.0.conv1")     # 64 -> 128, 3x3, stride 2
    with pytest.raises(G.GemelError) as e:
        c.merge([[(0, a), (1, b)]])
    assert e.value.code == G.ENOTMERGEABLE
    assert c.query(G.Q_MERGED_BYTES) == before
    # FC heads 512->1000 and 512->80 differ in cout
    with pytest.raises(G.GemelError) as e:
        c.merge([[(0, len(names) - 1), (1, len(names) - 1)]])
    assert e.value.code == G.ENOTMERGEABLE
    # a layer in two groups, unknown model, bad layer index
    for bad in ([[(0, a), (1, a)], [(0, a), (1, b)]], [[(0, a), (5, a)]],
                [[(0, a), (1, 999)]]):
        with pytest.raises(G.GemelError) as e:
            c.merge(bad)
        assert e.value.code == G.EINVAL
    assert c.query(G.Q_MERGED_BYTES) == before
    c.close()


def test_identity_ignores_weights_and_spatial_size():
    # same conv in a 32x32 and a 64x64 model: architecturally identical
    lay = zoo.tiny()
    p0 = configs.tiny2().params(0)
    p1 = configs.tiny2().params(1)
    c = _ctx()
    c.register_model(lay, p0, (3, 32, 32))
    c.register_model(lay, p1, (3, 64, 64))
    c.merge([[(0, 0), (1, 0)], [(0, 1), (1, 1)]])
    c.close()


def _desc_error(layers, params, in_chw=(3, 8, 8)):
    c = _ctx()
    with pytest.raises(G.GemelError) as e:
        c.register_model(layers, params, in_chw)
    assert c.query(G.Q_N_MODELS) == 0
    c.close()
    return e.value.code


def test_register_validation():
    lay = zoo.tiny()
    p = _tiny_params()
    bad = [dict(l) for l in lay]
    bad[1]["cin"] = 15
    assert _desc_error(bad, p) == G.ESHAPE
    bad = [dict(l) for l in lay]
    bad[1]["src0"] = 3
    assert _desc_error(bad, p) == G.EINVAL
    bad = [dict(l) for l in lay]
    bad[4]["cin"] = 31
    assert _desc_error(bad, p) == G.ESHAPE
    bad = [dict(l, out=False) for l in lay]
    assert _desc_error(bad, p) == G.EINVAL
    pm = list(p)
    pm[0] = None
    assert _desc_error(lay, pm) == G.EINVAL          # conv without weights
    big = [dict(lay[0], kh=9, kw=9, pad=0)] + [dict(l) for l in lay[1:]]
    pb = list(p)
    pb[0] = {"w": np.zeros((16, 3, 9, 9), np.float32), "b": None, "bn": None}
    assert _desc_error(big, pb, (3, 8, 8)) == G.ESHAPE   # window > input
    cat = [dict(lay[0], out=True),
           dict(lay[0], name="cat", op="concat", src0=0, src1=-1, cin=16,
                cout=19, act="none", bias=False, out=True)]
    assert _desc_error(cat, [p[0], None]) == G.ESHAPE  # 3-channel concat input


def test_infer_validates_before_device():
    c = _ctx()
    lay = zoo.tiny()
    c.register_model(lay, _tiny_params(), (3, 32, 32))
    assert c.infer_raw([0], [0], [1], [0], 0) == G.EINVAL       # null frames
    assert c.infer_raw([3], [1], [1], [1], 0) == G.EINVAL       # bad id
    assert c.infer_raw([0], [1], [-1], [1], 0) == G.EINVAL      # negative n
    assert c.infer_raw([0], [1], [1], [0], 0) == G.EINVAL       # null output
    st = c.infer_raw([0], [1], [0], [0], 0)                     # 0 frames
    assert st == G.OK
    with pytest.raises(G.GemelError):
        c.set_option(G.OPT_SWAP_SLOTS, 1)
    with pytest.raises(G.GemelError):
        c.query(99)
    c.close()
