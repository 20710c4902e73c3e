"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

* libfa's client code: tests/host_sanitize.cpp with the library's host source
  (the kernel launchers are left unresolved: the check never launches one)
  encodes random slot vectors and decodes their residues at N = 2^10 .. 2^16.
* The oracle's C core: a build with both sanitizers, loaded by a child
  process with the AddressSanitizer runtime preloaded, runs key generation,
  encryption, a rotation and a diagonal block product; its ciphertexts must
  equal the regular build's word for word.
"""
import os
import subprocess
import sys

import numpy as np
import pytest

from oracle import ckks

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/lib/llvm/bin/clang++"
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0", "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _asan_runtime():
    r = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not installed")
def test_client_encode_decode_under_sanitizers(tmp_path):
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2608_21131_amd", "csrc")]
    flags = ["--offload-host-only", "-c", "-O1", "-g", "-std=c++17", "-ffp-contract=off", "-fno-omit-frame-pointer",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
    objs = []
    for src in (os.path.join(ROOT, "paper_2608_21131_amd", "csrc", "fa_host.cpp"),
                os.path.join(ROOT, "tests", "host_sanitize.cpp")):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        r = subprocess.run([HIPCC, *flags, *inc, src, "-o", obj], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        objs.append(obj)
    exe = str(tmp_path / "host_sanitize")
    r = subprocess.run([CLANG, "-fsanitize=address,undefined", *objs, "-L/opt/rocm/lib", "-lamdhip64",
                        "-Wl,--unresolved-symbols=ignore-all", "-Wl,-rpath,/opt/rocm/lib", "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    sets = [(10, 3), (13, 3), (15, 8), (16, 12)]
    inp = "".join(f"{logn} {L} " + " ".join(str(q) for q in ckks.Params(logn=logn, L=L, K=1).q) + "\n"
                  for logn, L in sets)
    r = subprocess.run([exe], input=inp, capture_output=True, text=True, timeout=600,
                       env=dict(os.environ, **SAN_ENV))
    assert r.returncode == 0, r.stdout + r.stderr
    assert [ln.split()[:3] for ln in r.stdout.splitlines()] == [["ok", str(a), str(b)] for a, b in sets]


CHILD = r"""
import sys
import numpy as np
sys.path.insert(0, sys.argv[1])
from oracle import ckks
from paper_2608_21131_amd import gen
par = ckks.Params(logn=10, L=3, K=1)
orc = ckks.Oracle(par)
s = gen.ternary_secret(gen.rng(3, gen.STREAM_SECRET), par.n)
B, d = 4, 16
keys = {}
for r in ckks.steps_for_bsgs(d, B):
    a = gen.uniform_residues(gen.rng(3, gen.STREAM_KEY_A, r), par.primes, par.dnum, par.n)
    e = gen.rounded_gaussian(gen.rng(3, gen.STREAM_KEY_E, r), (par.dnum, par.n))
    keys[r] = orc.keygen(s, r, a, e)
q = gen.gaussian_unit_rows(gen.rng(3, gen.STREAM_QUERY), 1, d)[0]
ea = gen.uniform_residues(gen.rng(3, gen.STREAM_ENC_A), par.q, 1, par.n)[0]
ee = gen.rounded_gaussian(gen.rng(3, gen.STREAM_ENC_E), par.n)
ct = orc.encrypt(ckks.encode(ckks.replicate(q, par.slots), par.n, 40), ea, ee, s)
X = gen.gaussian_unit_rows(gen.rng(3, gen.STREAM_DB), 100, d)
pts = np.stack([ckks.to_residues(c, par.q) for c in ckks.layout_b_coeffs(X, par, d, B)])
out = orc.bsgs_block(orc.baby_rotations(ct, B, keys), pts.reshape(d // B, B, par.L, par.n), B, d // B, keys)
np.save(sys.argv[2], np.stack([ct, orc.rotate(ct, 1, keys[1]), out]))
"""


@pytest.mark.skipif(_asan_runtime() is None, reason="gcc's AddressSanitizer runtime not installed")
def test_oracle_core_under_sanitizers(tmp_path):
    so = str(tmp_path / "liboracle_san.so")
    r = subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-shared", "-fPIC", "-fno-omit-frame-pointer",
                        "-fsanitize=address,undefined", "-o", so, os.path.join(ROOT, "oracle", "ckks_oracle.c")],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    outs = []
    for lib, preload in ((so, _asan_runtime()), ("", None)):
        path = str(tmp_path / ("san.npy" if lib else "plain.npy"))
        env = dict(os.environ, **SAN_ENV, FA_ORACLE_LIB=lib, OMP_NUM_THREADS="4")
        if preload:
            env["LD_PRELOAD"] = preload
        r = subprocess.run([sys.executable, "-c", CHILD, ROOT, path], capture_output=True, text=True, env=env,
                           timeout=600)
        assert r.returncode == 0, r.stderr[-4000:]
        outs.append(np.load(path))
    assert np.array_equal(outs[0], outs[1])
