"""The C ABI without a GPU: the library loads and exports every function that
include/mita.h declares; the header-only validation passes its host test."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mita.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|size_t|const char \*)\s*\*?\s*(mita_\w+)\s*\(", text, re.M)))


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ("mita_forward", "mita_landmarks", "mita_topk", "mita_attend", "mita_scores", "mita_gather",
              "mita_route", "mita_workspace_size", "mita_check"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2602_01219_amd import mita
    if not os.path.exists(mita.LIB_PATH):
        pytest.skip("libmita.so not built")
    lib = mita.load_library()
    for n in _declared():
        assert hasattr(lib, n), n
    assert set(_declared()) <= set(mita.EXPORTED) | {"mita_status_string", "mita_last_error"}


def test_host_validation_without_gpu():
    from paper_2602_01219_amd import mita, synth
    if not os.path.exists(mita.LIB_PATH):
        pytest.skip("libmita.so not built")
    import dataclasses
    cfg = mita.Config.from_workload(synth.WORKLOADS["dense_pred_bf16"])
    assert mita.check(cfg) == mita.MITA_OK
    assert mita.check(dataclasses.replace(cfg, d=96)) == mita.MITA_ERR_UNSUPPORTED
    assert mita.check(dataclasses.replace(cfg, k=0)) == mita.MITA_ERR_INVALID_ARG
    assert mita.workspace_size(cfg) > 0
    assert mita.workspace_size(cfg, mita.WS_TOPK) == 0


@pytest.mark.parametrize("sanitize", [False, True], ids=["plain", "asan_ubsan"])
def test_check_header_host_program(tmp_path, sanitize):
    """The header-only validation, workspace layout, selection plan and LDS
    dispatch rule, built with g++ (host code only), plainly and under
    AddressSanitizer + UndefinedBehaviorSanitizer."""
    exe = tmp_path / "test_check"
    src = os.path.join(ROOT, "tests", "host", "test_check.cpp")
    flags = ["-std=c++17", "-O1", "-Wall", "-g"]
    if sanitize:
        flags += ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    r = subprocess.run(["g++", *flags, "-I", os.path.join(ROOT, "include"), src, "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "host checks ok" in r.stdout
