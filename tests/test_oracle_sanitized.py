"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(host code only; test infrastructure): tests/c/oracle_sanitized.c runs every
oracle entry point -- downsample, bbox, correspondence for several anchor
sets and K, transport and reconstruction in float32 and bfloat16, the host
schedule, UniPC, the coverage schedule -- on a workload's position maps,
and must finish without a sanitizer report.  Orthographic (tiny sphere) and
pinhole (Hunyuan-shaped) rigs."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import synth
from synth.configs import C1, C2

from conftest import latent_maps

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if not shutil.which("gcc"):
        pytest.skip("gcc is not available")
    out = str(tmp_path_factory.mktemp("san") / "oracle_sanitized")
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-ffp-contract=off",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(ROOT, "tests", "c", "oracle_sanitized.c"),
           "-lm", "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "sanitize" in r.stderr and "cannot find" in r.stderr:
        pytest.skip("the sanitizer runtimes are not installed")
    assert r.returncode == 0, r.stderr
    return out


@pytest.mark.parametrize("w", [C1, C2], ids=lambda w: w.name)
def test_oracle_under_sanitizers(driver, tmp_path, w):
    P = np.ascontiguousarray(latent_maps(w.name), np.float32)
    B, N, H, W = P.shape[:4]
    cams = synth.batch_cameras(w)
    files = {
        "pos.bin": P,
        "model.bin": np.broadcast_to(cams["model"], (B, N)).astype(np.int32),
        "R.bin": np.broadcast_to(cams["R"], (B, N, 3, 3)).astype(np.float32),
        "t.bin": np.broadcast_to(cams["t"], (B, N, 3)).astype(np.float32),
        "k.bin": np.stack([np.broadcast_to(cams[n], (B, N)) for n in ("fx", "fy", "cx", "cy")], -1).astype(np.float32),
        "hi.bin": P.reshape(B * N, H, W, 3),   # the downsample runs on the latent maps themselves
    }
    for name, arr in files.items():
        np.ascontiguousarray(arr).tofile(str(tmp_path / name))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([driver, str(tmp_path), str(B), str(N), str(H), str(W), str(B * N), str(H), str(W)],
                       capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "oracle under sanitizers: ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
