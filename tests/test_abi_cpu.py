"""The C ABI without a GPU: the library loads, exports every function the
header declares, and reports argument errors before touching a device."""
import os
import re

import numpy as np
import pytest

from paper_2103_03231_amd import binding as b
from paper_2103_03231_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "donerf.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(donerf_\w+)\s*\(", src)))


def test_header_declarations_are_exported():
    names = _declared()
    assert set(names) == set(b.EXPORTS)
    L = b.lib()
    for n in names:
        assert hasattr(L, n), n


@pytest.mark.parametrize("B", [64, 128, 192, 256])
def test_weight_count_matches_blob(B):
    assert b.donerf_weight_count(B) == inputs.n_weights(B) == inputs.make_weights(B, 0).size
    pos = inputs.n_weights(B, "positions")
    assert b.donerf_weight_count(B, b.DEPTH_POSITIONS) == pos == inputs.make_weights(B, 0, "positions").size
    assert pos - inputs.n_weights(B) == 256 * (6 + 3 * B - 90)
    assert b.donerf_weight_count(0) == 0
    assert b.donerf_weight_count(B, 2) == 0


def test_status_strings():
    for s in (0, -1, -2, -3, -4, -5, -6, -7):
        assert b.donerf_status_str(s) and b.donerf_status_str(s) != "unknown status"
    assert b.donerf_status_str(-99) == "unknown status"


W128 = inputs.make_weights(128, 0)


@pytest.mark.parametrize("kw,status", [
    ({"near": 0.0}, b.E_INVALID_ARG),
    ({"near": 5.0, "far": 5.0}, b.E_INVALID_ARG),
    ({"fov_x_deg": 180.0}, b.E_INVALID_ARG),
    ({"radius": -1.0}, b.E_INVALID_ARG),
    ({"n_max": 0}, b.E_INVALID_ARG),
    ({"n_max": 17}, b.E_INVALID_ARG),
    ({"precision": 7}, b.E_INVALID_ARG),
    ({"select": 3}, b.E_INVALID_ARG),
    ({"depth_input": 2}, b.E_INVALID_ARG),
    ({"far": float("inf")}, b.E_NONFINITE),
    ({"centre": (0.0, float("nan"), 0.0)}, b.E_NONFINITE),
    ({"n_bins": 100}, b.E_UNSUPPORTED),
    ({"n_bins": 32}, b.E_UNSUPPORTED),
])
def test_create_rejects_bad_config(kw, status):
    with pytest.raises(b.DonerfError) as e:
        b.donerf_create(b.Config(**kw), W128)
    assert e.value.status == status
    assert b.donerf_last_error()


def test_create_rejects_bad_weights():
    with pytest.raises(b.DonerfError) as e:
        b.donerf_create(b.Config(), W128[:-1])
    assert e.value.status == b.E_SIZE
    # the positions input needs the wider first layer
    with pytest.raises(b.DonerfError) as e:
        b.donerf_create(b.Config(depth_input=b.DEPTH_POSITIONS), W128)
    assert e.value.status == b.E_SIZE
    w = W128.copy()
    w[12345] = np.inf
    with pytest.raises(b.DonerfError) as e:
        b.donerf_create(b.Config(), w)
    assert e.value.status == b.E_NONFINITE
    with pytest.raises(b.DonerfError) as e:
        b.donerf_create(b.Config(), None)
    assert e.value.status == b.E_INVALID_ARG


def test_calls_on_null_handle():
    poses = inputs.make_poses([0])
    for fn in (lambda: b.donerf_render(None, poses, 1, 4, 4, 4, 1),
               lambda: b.donerf_render_static_scratch(None, poses, 1, 4, 4, 4, 1),
               lambda: b.donerf_render_debug(None, poses, 1, 4, 4, 4, 1),
               lambda: b.donerf_debug_topn(None, 1, 4, 4, 1),
               lambda: b.donerf_targets(None, 1, 1, 4, 4, 5, 5, 1),
               lambda: b.donerf_debug_bins(None, 128),
               lambda: b.donerf_debug_mfma_peak(None, 1, 1, 1),
               lambda: b.donerf_set_stream(None, 0)):
        with pytest.raises(b.DonerfError) as e:
            fn()
        assert e.value.status == b.E_INVALID_ARG
    b.donerf_destroy(None)


def test_create_without_gpu_reports_device_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(b.DonerfError) as e:
        b.donerf_create(b.Config(), W128)
    assert e.value.status == b.E_DEVICE


def test_missing_library_fails_loudly():
    """Without the built library every entry point raises; nothing falls
    back to another implementation.  Run in a fresh interpreter, since the
    module keeps the library it loaded."""
    import subprocess
    import sys
    code = ("from paper_2103_03231_amd import binding as b, inputs\n"
            "b.LIB_PATH = '/nonexistent/libdonerf.so'\n"
            "for f in (lambda: b.donerf_weight_count(128),\n"
            "          lambda: b.Renderer(b.Config(n_bins=128, n_max=4), inputs.make_weights(128, 0))):\n"
            "    try:\n"
            "        f()\n"
            "    except b.DonerfLibraryMissing:\n"
            "        continue\n"
            "    raise SystemExit('no error')\n"
            "print('raised')\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "raised" in r.stdout, r.stderr[-2000:]
