"""CPU-side checks of the C ABI (no GPU compute): libhq.so loads, exports
every function include/hq.h declares, validates arguments before touching the
device, and its host Rice-k rule equals the oracle's formula."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hq.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hq_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import build, hq as H
    if not os.path.exists(build.LIB):
        build.build()
    return H


def test_library_exports_every_declared_symbol(hq):
    L = hq.lib()
    names = declared_functions()
    assert "hq_plan" in names and "hq_encode" in names and "hq_dequant_gemm_int8" in names
    for n in names:
        assert hasattr(L, n), n
    assert set(hq.EXPORTED) <= set(names)


def test_status_strings(hq):
    L = hq.lib()
    assert L.hq_status_string(0) == b"ok"
    assert L.hq_status_string(-7).startswith(b"no calibration")


def test_plan_argument_errors_are_synchronous(hq):
    L = hq.lib()
    h = C.c_void_p()
    info = hq.PlanInfo()
    o = hq.Options(0, 0, 0, 0, 0, 0, 1, 0, 20.0)
    # tile not a power of two / smaller than the lattice / cols not divisible
    assert L.hq_plan(96, 0, 4.0, 0, -1, 4096, C.byref(o), C.byref(h), C.byref(info)) == -1
    assert L.hq_plan(4, 0, 4.0, 0, -1, 4096, C.byref(o), C.byref(h), C.byref(info)) == -1
    assert L.hq_plan(128, 0, 4.0, 0, -1, 4000, C.byref(o), C.byref(h), C.byref(info)) == -1
    assert L.hq_plan(128, 7, 4.0, 0, -1, 4096, C.byref(o), C.byref(h), C.byref(info)) == -1
    assert L.hq_plan(128, 0, 4.0, 0, 16, 4096, C.byref(o), C.byref(h), C.byref(info)) == -1
    # valid for the method, not built here: tiles past 2048; long tiles, or
    # sub-streams of 1024 / 2048 symbols, with a KV option (rotation, dither,
    # fp16 norms); sub-stream lengths other than 512, 1024 and 2048
    assert L.hq_plan(4096, 0, 4.0, 0, -1, 8192, C.byref(o), C.byref(h), C.byref(info)) == -2
    for rot, dith, nd in ((1, 0, 0), (0, 1, 0), (0, 0, 2)):
        ok = hq.Options(rot, dith, 0, 0, nd, 0, 1, 0, 20.0)
        assert L.hq_plan(256, 0, 4.0, 0, -1, 4096, C.byref(ok), C.byref(h), C.byref(info)) == -2
        for S in (1024, 2048):
            ok = hq.Options(rot, dith, 0, 0, nd, S, 1, 0, 20.0)
            assert L.hq_plan(128, 0, 4.0, 0, -1, 4096, C.byref(ok), C.byref(h), C.byref(info)) == -2
    for S in (256, 4096):
        o2 = hq.Options(0, 0, 0, 0, 0, S, 1, 0, 20.0)
        assert L.hq_plan(128, 0, 4.0, 0, -1, 8192, C.byref(o2), C.byref(h), C.byref(info)) == -2
    # a sub-stream length that neither holds whole tiles nor divides one
    o3 = hq.Options(0, 0, 0, 0, 0, 768, 1, 0, 20.0)
    assert L.hq_plan(1024, 0, 4.0, 0, -1, 6144, C.byref(o3), C.byref(h), C.byref(info)) == -1
    # null output handle
    assert L.hq_plan(128, 0, 4.0, 0, -1, 4096, C.byref(o), None, None) == -1


def test_encode_decode_argument_errors(hq):
    L = hq.lib()
    s = hq.StreamStruct()
    assert L.hq_encode(None, None, 0, 0, 0, C.byref(s), 0, None) == -1
    assert L.hq_decode(None, C.byref(s), 0, 0, None, 0, 0, None) == -1
    assert L.hq_dequant_gemm_int8(None, None, 0, None, 0, None, 0, None, 0, None) == -1


@pytest.mark.parametrize("count", [512, 384, 256, 128, 1])
def test_host_rice_kstar_equals_oracle(hq, count):
    # the kernels evaluate k* through integer thresholds precomputed on the
    # host; they must agree with the paper's formula at every sum.
    L = hq.lib()
    sums = list(range(0, 70000)) + list(np.unique(np.geomspace(70000, 2**31, 3000).astype(np.int64)))
    for s in sums:
        assert L.hq_rice_kstar(count, int(s)) == O.rice_k_auto(count, int(s)), (count, s)


def test_library_calibration_matches_oracle_operating_points(hq):
    # App. B: both sides invert a realized-rate curve measured on iid Gaussian
    # tiles; the library's table (its own encoder, torch samples) and the
    # oracle's bisection (its own encoder, numpy samples) must agree.
    import json
    pts = json.load(open(os.path.join(ROOT, "tests", "golden", "operating_points.json")))["points"]
    for p in pts:
        lat = hq.LATTICES[p["lattice"]]
        snr = hq.hq_calibrated_snr(lat, -1, p["bps"])
        assert abs(snr - p["snr_db"]) < 0.05, (p, snr)
    # fixed-k curves exist too, and bps below their 1 + k floor is rejected
    assert hq.hq_calibrated_snr(hq.HQ_E8, 2, 4.0) > 0
    with pytest.raises(hq.HQError):
        hq.hq_calibrated_snr(hq.HQ_E8, 3, 2.0)


def test_group_argument_errors_are_synchronous(hq):
    L = hq.lib()
    assert L.hq_encode_group(None, None, 0, None, None, None, 0, None) == 0  # nothing to do
    assert L.hq_encode_group(None, None, 0, None, None, None, 2, None) == -1
    assert L.hq_encode_group(None, None, 0, None, None, None, -1, None) == -1
    assert L.hq_decode_group(None, None, None, 0, None, 0, None) == 0
    assert L.hq_decode_group(None, None, None, 0, None, 3, None) == -1
    assert L.hq_decode_group(None, None, None, 7, None, 0, None) == -1  # bad output type


def test_fused_entry_points_reject_null_plans(hq):
    # argument errors come back before any device work (no GPU needed)
    L = hq.lib()
    assert L.hq_gemv_workspace_bytes(None) == 0
    assert L.hq_attention_workspace_bytes(None, 1, 8, 64) == 0
    assert L.hq_decode_gemv(None, None, 0, 1, None, 0, None, 0, None, 0, None) == -1
    assert L.hq_decode_attention(None, None, None, None, None, 0, 1, 8, C.c_float(0.1), None, 1, 16,
                                 None, None, None, 0, 0, None, 0, None, 0, None) == -1


def test_long_tile_plans_keep_the_heap_intact(hq):
    # Regression: the rotation sign mask was built over the whole tile into a
    # four-word buffer, so a 256..2048-tile plan wrote past it.  glibc's heap
    # checks (MALLOC_CHECK_=3) abort a process whose heap was overrun; plans
    # of every long tile are made in a child process with them on (without a
    # GPU hq_plan returns HQ_ERR_HIP after its host work, which is the part
    # under test).
    import subprocess
    import sys
    code = (
        "import ctypes as C, sys\n"
        f"sys.path.insert(0, {ROOT!r})\n"
        "from paper_2606_23406_amd import hq\n"
        "L = hq.lib()\n"
        "for t in (256, 512, 1024, 2048, 2048, 1024):\n"
        "    o = hq.Options(0, 0, 0, 0, 0, 0, 1, 0, 20.0)\n"
        "    h = C.c_void_p(); info = hq.PlanInfo()\n"
        "    rc = L.hq_plan(t, 0, 4.0, 0, -1, 8192, C.byref(o), C.byref(h), C.byref(info))\n"
        "    assert rc in (0, -5), rc\n"
        "    if rc == 0: L.hq_plan_destroy(h)\n"
        "    junk = [bytearray(64) for _ in range(2000)]\n"
        "print('heap ok')\n")
    env = dict(os.environ, MALLOC_CHECK_="3", HIP_VISIBLE_DEVICES=os.environ.get("HIP_VISIBLE_DEVICES", ""))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and "heap ok" in r.stdout, r.stdout + r.stderr
