"""The C ABI from C: tests/capi/fig1_capi.c uses only include/ngpu_lm.h, the
HIP runtime and libngpu_lm.so (no Python binding, no torch).

CPU: the header compiles as C11 with warnings as errors and the program links
against the library.  GPU: the program builds, uploads and queries the worked
example of Section 2.1 (Figure 1, hand-derived values in
tests/golden/fig1_trigram.json), follows its sentence with plain fused steps at
lambda = 0, and gets NGPU_E_INVALID_ARG for a negative batch size.
"""

import json
import os
import shutil
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIBDIR = os.path.join(ROOT, "paper_2505_22857_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _compile(out):
    if shutil.which("gcc") is None or not os.path.isdir(os.path.join(ROCM, "include", "hip")):
        pytest.skip("gcc or the HIP headers are not available")
    if not os.path.exists(os.path.join(LIBDIR, "libngpu_lm.so")):
        pytest.skip("libngpu_lm.so is not built")
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           os.path.join(HERE, "capi", "fig1_capi.c"), "-o", out,
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-L", LIBDIR, "-lngpu_lm",
           "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-Wl,-rpath," + LIBDIR]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]


def _fig1_list_file(path):
    with open(os.path.join(HERE, "golden", "fig1_trigram.json")) as f:
        fx = json.load(f)
    N, ngr = fx["max_order"], fx["ngrams"]
    tokens = np.full((len(ngr), N), -1, np.int32)
    for i, g in enumerate(ngr):
        tokens[i, :len(g[0])] = g[0]
    with open(path, "wb") as f:
        f.write(np.array([len(fx["vocab"]), N], np.int32).tobytes())
        f.write(np.array([len(ngr)], np.int64).tobytes())
        f.write(np.array([np.nan], np.float32).tobytes())
        f.write(np.array([0], np.uint32).tobytes())
        f.write(np.array([len(g[0]) for g in ngr], np.int32).tobytes())
        f.write(tokens.tobytes())
        f.write(np.array([g[1] for g in ngr], np.float32).tobytes())
        f.write(np.array([g[2] for g in ngr], np.float32).tobytes())
    return fx


def test_header_compiles_as_c_and_links(tmp_path):
    _compile(str(tmp_path / "fig1_capi"))


@pytest.mark.gpu
def test_worked_example_through_the_c_abi(tmp_path):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    exe = str(tmp_path / "fig1_capi")
    _compile(exe)
    fx = _fig1_list_file(str(tmp_path / "fig1.list"))
    sent = fx["sentence"]
    print("[case] C ABI worked example", flush=True)
    r = subprocess.run([exe, str(tmp_path / "fig1.list")], input="\n".join(map(str, sent["tokens"])) + "\n",
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-3000:]
    rows, steps, err, bad = {}, [], None, None
    for line in r.stdout.splitlines():
        w = line.split()
        if w[0] == "state":
            rows.setdefault(int(w[1]), {})[int(w[3])] = (float(w[5]), int(w[7]))
        elif w[0] == "step":
            steps.append((int(w[3]), int(w[5])))
        elif w[0] == "error":
            err = int(w[1])
        elif w[0] == "bad":
            bad = int(w[2])
    assert r.stdout.strip().endswith("ok")
    assert len(rows) == len(fx["state_contexts"])
    for s, row in fx["rows"].items():
        got = rows[int(s)]
        np.testing.assert_allclose([got[v][0] for v in range(len(row["scores"]))], row["scores"], atol=1e-6)
        assert [got[v][1] for v in range(len(row["next"]))] == row["next"]
    assert [t for t, _ in steps] == sent["tokens"]
    assert [s for _, s in steps] == sent["states"]
    assert bad == 0
    assert err == -1          # NGPU_E_INVALID_ARG
