"""The host code of the C ABI under AddressSanitizer and UBSan, on the CPU.

A g++ sanitizer build of the host side (``build_sanitized``; the kernel
object is the ordinary one, no GPU code is instrumented) runs the CPU ABI
tests and a seeded fuzz of malformed partition inputs in a child process
with the sanitizer runtimes preloaded.  Any report aborts the child.  No
kernel is launched."""
import os
import subprocess
import sys

import pytest

from conftest import ROOT

FUZZ = r'''
import ctypes
import sys
import numpy as np
sys.path.insert(0, sys.argv[1])
ctypes.CDLL(None)["__asan_init"]   # the preloaded AddressSanitizer runtime is live
from paper_2206_00057_amd import digest as D
assert D.LIB_PATH.endswith("libdigest_host_sanitized.so"), D.LIB_PATH
rng = np.random.default_rng(0)
created = rejected = 0
for trial in range(400):
    n = int(rng.integers(1, 60))
    n_own = int(rng.integers(0, n + 1))
    owned = np.sort(rng.choice(n, n_own, replace=False)).astype(np.int64)
    deg = rng.integers(0, 6, n_own)
    indptr = np.zeros(n_own + 1, np.int64)
    np.cumsum(deg, out=indptr[1:])
    nnz = int(indptr[-1])
    indices = rng.integers(0, n, nnz).astype(np.int64)
    mine = np.zeros(n, bool)
    mine[owned] = True
    halo = np.unique(indices[~mine[indices]]) if nnz else np.zeros(0, np.int64)
    values = rng.random(nnz).astype(np.float32)
    widths = [int(rng.integers(1, 9)) for _ in range(int(rng.integers(2, 4)))]
    kind = trial % 8
    if kind == 1 and nnz:
        indices[rng.integers(nnz)] = n + int(rng.integers(0, 5))   # id out of range
    if kind == 2 and nnz:
        indices[rng.integers(nnz)] = -1
    if kind == 3 and n_own > 1:
        indptr[1], indptr[2] = indptr[2] + 3, indptr[1]          # not monotone
    if kind == 4 and len(halo):
        halo = np.concatenate([halo, halo[:1]])                  # repeated halo id
    if kind == 5 and n_own:
        halo = np.concatenate([halo, owned[:1]])                 # owned id in the halo
    if kind == 6:
        widths[0] = 0
    if kind == 7 and nnz and len(halo):
        halo = halo[1:]                                          # column neither owned nor halo
    try:
        h = D.digest_partition_create(n, indptr, indices, values, owned, halo, widths)
    except D.DigestError:
        rejected += 1
        continue
    created += 1
    D.digest_partition_export_maps(h)
    D.digest_partition_export_transpose(h)
    for layer in range(1, len(widths)):
        D.digest_partition_plan(h, layer)
    D.digest_profile_model(h, D.MODEL_GCN)
    D.digest_profile_model(h, D.MODEL_GAT)
assert created >= 50 and rejected >= 200, (created, rejected)
print("fuzz", created, "created", rejected, "rejected")
'''


@pytest.mark.timeout(600)
def test_host_code_clean_under_asan_and_ubsan(tmp_path):
    from paper_2206_00057_amd import build_sanitized
    lib = build_sanitized.build()
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": build_sanitized.runtime_preload(),
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "DIGEST_LIBRARY": lib,
    })
    script = tmp_path / "fuzz.py"
    script.write_text(FUZZ)
    fuzz = subprocess.run([sys.executable, str(script), ROOT], env=env, cwd=ROOT,
                          stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert fuzz.returncode == 0, fuzz.stdout[-4000:]
    assert "ERROR: AddressSanitizer" not in fuzz.stdout and "runtime error" not in fuzz.stdout
    abi = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi_cpu.py")], env=env, cwd=ROOT,
                         stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert abi.returncode == 0, abi.stdout[-4000:]
    assert "ERROR: AddressSanitizer" not in abi.stdout and "runtime error" not in abi.stdout
