"""The pins of the oracle's Python parts (the omission test of section 5.4 and the content identity
of section 5.3) must catch plausible mistakes.  Each case plants one mistake in a copy of the
oracle package (on the CPU) and runs the pin tests against that copy; every mutant must make them
fail."""

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")
PINS = {"identity.py": ["tests/test_oracle_identity.py"], "omission.py": ["tests/test_oracle_omission.py"]}

# (file, name, [(old, new), ...]); every `old` must occur in the file.
MUTANTS = [
    ("identity.py", "leaves of 512 bytes", [("LEAF = 1024", "LEAF = 512")]),
    ("identity.py", "fan-in of 8", [("FANIN = 16", "FANIN = 8")]),
    ("identity.py", "leaf prefix 0x01", [('sha256(b"\\x00" + data[i:i + LEAF])', 'sha256(b"\\x01" + data[i:i + LEAF])')]),
    ("identity.py", "node prefix 0x00", [('sha256(b"\\x01" + b"".join', 'sha256(b"\\x00" + b"".join')]),
    ("identity.py", "empty tensor hashed without its prefix", [('return [sha256(b"\\x00")]', 'return [sha256(b"")]')]),
    ("identity.py", "dtype length prefix dropped", [('struct.pack("<I", len(dtype)) + dtype', 'dtype')]),
    ("identity.py", "dimensions as u32", [('struct.pack("<Q", int(d)) for d in shape', 'struct.pack("<I", int(d)) for d in shape')]),
    ("identity.py", "byte length left out of the record", [('return out + struct.pack("<Q", len(data)) + root', 'return out + root')]),
    ("identity.py", "records in reverse name order", [("for n, dt, shape, d in tensors)", "for n, dt, shape, d in tensors), reverse=True)")]),
    ("identity.py", "configuration fields unsorted", [("cfg = sorted((bytes(k), bytes(v)) for k, v in config)", "cfg = [(bytes(k), bytes(v)) for k, v in config]")]),
    ("omission.py", "projection keeps the withheld dimensions", [("if names is None or n in names]", "if names is None or n not in names]")]),
    ("omission.py", "variant keeps the old value too", [("[(n, v) for n, v in desc if n != name] + [(name, value)]", "[(n, v) for n, v in desc] + [(name, value)]")]),
    ("omission.py", "keys compared byte by byte", [("(ka == kb).all(axis=1)", "(ka == kb).any(axis=1)")]),
    ("omission.py", "per-request counts shifted", [("same = np.concatenate([[0], np.cumsum(", "same = np.concatenate([np.cumsum(")]),
    ("omission.py", "declared change ignored", [('"omission": (coll > 0) & changes[None, :]', '"omission": (coll > 0)')]),
    ("omission.py", "variant projected before it is varied", [("project(vary(d, dim, case.variants[dim]), names)", "vary(project(d, names), dim, case.variants[dim])")]),
]


def _build_and_run(fname, name, edits, tmp):
    d = os.path.join(tmp, name.replace(" ", "_"))
    pkg = os.path.join(d, "oracle")
    shutil.copytree(ORACLE, pkg, ignore=shutil.ignore_patterns("__pycache__", "*.tmp"))
    path = os.path.join(pkg, fname)
    src = open(path).read()
    for old, new in edits:
        assert old in src, f"{name}: pattern not found: {old!r}"
        src = src.replace(old, new, 1)
    open(path, "w").write(src)
    # the copy comes first on the path (cwd); the repository root stays importable after it
    env = dict(os.environ, PYTHONPATH=os.pathsep.join([d, ROOT]), PKV_ORACLE_LIB=os.path.join(pkg, "liboracle.so"))
    pins = [os.path.join(ROOT, p) for p in PINS[fname]]
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "--import-mode=append",
                        "--rootdir", ROOT,
                        "-m", "not gpu"] + pins, cwd=d, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout[-400:]


def test_every_planted_mistake_in_the_python_oracle_fails_the_pins():
    with tempfile.TemporaryDirectory() as tmp:
        with cf.ThreadPoolExecutor(max_workers=4) as ex:
            futs = {name: ex.submit(_build_and_run, f, name, edits, tmp) for f, name, edits in MUTANTS}
            results = {name: f.result() for name, f in futs.items()}
    survivors = [name for name, (rc, _out) in results.items() if rc == 0]
    assert not survivors, f"mutants not caught by the pins: {survivors}"


def test_the_unmutated_copy_passes_the_pins():
    # the harness itself: the same copy without a planted mistake must pass
    with tempfile.TemporaryDirectory() as tmp:
        rc, out = _build_and_run("identity.py", "unmutated identity", [], tmp)
        assert rc == 0, out
        rc, out = _build_and_run("omission.py", "unmutated omission", [], tmp)
        assert rc == 0, out
