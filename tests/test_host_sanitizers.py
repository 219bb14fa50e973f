"""The host-side bookkeeping under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The host-only library (validation, chunk plans, cost model, arena with every placement and
eviction policy, queueing) is rebuilt with both sanitizers, every report fatal, and driven by
tests/host_sanitize_driver.cpp through valid, malformed and random inputs of the workloads'
layouts. A canary program with a planted heap overflow checks that the toolchain's sanitizer
really reports under the same flags."""
import os
import subprocess

import pytest

import synth
import paper_2306_03622_amd as tp
from paper_2306_03622_amd import build as tp_build

HERE = os.path.dirname(os.path.abspath(__file__))
INCLUDE = os.path.join(os.path.dirname(HERE), "include")


def _write_models(path, models):
    with open(path, "w") as f:
        for m in models:
            d = tp.ModelDesc.of(m)
            f.write(f"model {d.desc.arch} {d.desc.dtype} {' '.join(str(v) for v in d.desc.dims)} {m.total_bytes} "
                    f"{len(d.tensors)}\n")
            for i in range(len(d.tensors)):
                t = d._arr[i]
                f.write(f"t {t.layer} {t.role} {t.offset} {t.bytes} {' '.join(str(t.shape[k]) for k in range(4))}\n")


def _compile(src, out, *extra):
    r = subprocess.run(["g++", "-O1", "-std=c++17", *tp_build.SANITIZE, f"-I{INCLUDE}", src, *extra, "-o", out],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


@pytest.mark.slow
def test_sanitizers_report_a_planted_overflow(tmp_path):
    src = tmp_path / "canary.cpp"
    src.write_text("#include <vector>\nint main(int c, char**) { std::vector<int> v(4); return v.data()[3 + c]; }\n")
    _compile(str(src), str(tmp_path / "canary"))
    r = subprocess.run([str(tmp_path / "canary")], capture_output=True, text=True)
    assert r.returncode != 0 and "AddressSanitizer" in r.stderr


@pytest.mark.slow
def test_host_library_under_sanitizers(tmp_path):
    lib = tp_build.build_host(str(tmp_path / "libtorpor_host_san.so"), sanitize=True)
    exe = str(tmp_path / "driver")
    _compile(os.path.join(HERE, "host_sanitize_driver.cpp"), exe, lib, f"-Wl,-rpath,{tmp_path}")
    models = [synth.config_model(c, 0) for c in (1, 2, 3, 4)] + [
        synth.bert(seed=1, layers=2, d=128, heads=2, ffn=264, seq=64, vocab=100, maxpos=64),
        synth.resnet50(seed=3, classes=10, image=96),
        synth.mlp(3, 200, "bf16", "gelu", seed=7)]
    _write_models(tmp_path / "models.txt", models)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, str(tmp_path / "models.txt")], capture_output=True, text=True, env=env, timeout=600)
    print(r.stdout, r.stderr[-4000:])
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "Sanitizer" not in r.stderr
    assert ", 0 failed" in r.stdout
