"""The oracle rebuilt with AddressSanitizer and UndefinedBehaviorSanitizer
(gcc, CPU only): a child process with the sanitizer runtime preloaded runs
compositions (both orders, the epsilon filter's planted mistakes, three
inputs), scores, posteriors, scatters and the in-arc index over the test
workloads with that build; any out-of-bounds access, use after free or
undefined behaviour ends it with an error, and every result must equal the
plain build's, bit for bit."""
import hashlib
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CASES = r"""
import hashlib, json, sys
import numpy as np
sys.path.insert(0, ROOT)
import oracle
from paper_2110_02848_amd import synth


def digest(r):
    h = hashlib.sha256()
    for k in sorted(r):
        v = r[k]
        if isinstance(v, np.ndarray):
            h.update(k.encode())
            h.update(np.ascontiguousarray(v).tobytes())
        elif isinstance(v, (int, float)):
            h.update(f"{k}={v!r}".encode())
    return h.hexdigest()


out = {}
for seed in range(4):
    A, B = synth.workload("random-64", seed)
    for order in (oracle.ORDER_PAPER, oracle.ORDER_FORWARD):
        out[f"r64-{seed}-{order}"] = digest(oracle.compose(A, B, order))
A, B = synth.workload("random-1000", 1)
out["r1000"] = digest(oracle.compose(A, B, oracle.ORDER_FORWARD))
A, B = synth.workload("lexicon-T100-W1000", 0)
C = oracle.compose(A, B, oracle.ORDER_PAPER)
out["lex"] = digest(C)
sc = oracle.score(C)
out["lex-score"] = digest({"alpha": sc["alpha"], "beta": sc["beta"], "total": sc["total"]})
post = oracle.posterior(C, sc["alpha"], sc["beta"], sc["total"])
out["lex-post"] = digest({"p": post})
out["lex-scatter"] = digest({"a": oracle.scatter(post, C["arc_a"], len(A["src"])),
                             "b": oracle.scatter(post, C["arc_b"], len(B["src"]))})
for seed in range(24):
    rng = np.random.default_rng([505, seed])
    A = synth.tiny_random(rng, 1 + seed % 5, 4, 3, 0.35, n_start=1 + seed % 2)
    B = synth.tiny_random(rng, 1 + (seed // 5) % 5, 4, 3, 0.35)
    D = synth.tiny_random(rng, 1 + seed % 4, 4, 3, 0.35)
    out[f"tiny-{seed}"] = digest(oracle.compose(A, B, oracle.ORDER_PAPER, seed % 7))
    out[f"tiny3-{seed}"] = digest(oracle.compose3(A, B, D, seed % 5))
A, B, D, _ = synth.emissions_lexicon_grammar("grammar-T40-W300-G6", 0)
out["grammar"] = digest(oracle.compose3(A, B, D))
for V in (0, 1, 7):
    dst = np.arange(3 * V, dtype=np.int32) % max(V, 1)
    off, arcs = oracle.in_csr(V, dst[: 3 * V] if V else dst[:0])
    out[f"incsr-{V}"] = digest({"off": off, "arcs": arcs})
G = synth.random_dag(3, 2000, hubs=2, hub_degree=300)
sc = oracle.score(G)
out["dag"] = digest({"alpha": sc["alpha"], "beta": sc["beta"], "total": sc["total"]})
print(json.dumps(out))
"""


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = p.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(900)
def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = str(tmp_path / "liboracle_sanitized.so")
    cmd = ["gcc", "-O1", "-g", "-std=gnu11", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-fast-math", "-ffp-contract=off", "-o", lib, *oracle.sources(), "-lm"]
    subprocess.run(cmd, check=True)
    env = dict(os.environ, FSTC_ORACLE_LIB=lib, LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    child = subprocess.run([sys.executable, "-c", CASES.replace("ROOT", repr(ROOT), 1)],
                           env=env, capture_output=True, text=True, timeout=800)
    assert child.returncode == 0, child.stderr[-4000:]
    assert "runtime error" not in child.stderr, child.stderr[-4000:]
    got = json.loads(child.stdout.strip().splitlines()[-1])
    # the same cases with the plain build, in this process
    plain = subprocess.run([sys.executable, "-c", CASES.replace("ROOT", repr(ROOT), 1)],
                           capture_output=True, text=True, timeout=800,
                           env={k: v for k, v in os.environ.items() if k != "FSTC_ORACLE_LIB"})
    assert plain.returncode == 0, plain.stderr[-2000:]
    ref = json.loads(plain.stdout.strip().splitlines()[-1])
    assert got.keys() == ref.keys()
    bad = [k for k in ref if got[k] != ref[k]]
    assert not bad, bad
