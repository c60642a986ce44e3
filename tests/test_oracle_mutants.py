"""The oracle's pins must catch plausible mistakes.  Each case plants one mistake in a copy of the
oracle's C source (on the CPU), builds it, and runs the pin tests against that build; every
mutant must make them fail."""

import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCE = os.path.join(ROOT, "oracle", "pkv_oracle.c")
PINS = ["tests/test_oracle_sha256.py", "tests/test_oracle_encoding.py", "tests/test_oracle_chain.py",
        "tests/test_oracle_index.py", "tests/test_contract_oracle.py", "tests/test_oracle_budget.py"]

# (name, [(old, new), ...]); every `old` must occur in the source.
MUTANTS = [
    ("Sigma1 rotation", [("rotr(x, 6) ^ rotr(x, 11) ^ rotr(x, 25)", "rotr(x, 6) ^ rotr(x, 11) ^ rotr(x, 24)")]),
    ("Ch operands swapped", [("return (x & y) ^ (~x & z);", "return (x & z) ^ (~x & y);")]),
    ("Maj term dropped", [("return (x & y) ^ (x & z) ^ (y & z);", "return (x & y) ^ (x & z);")]),
    ("sigma0 shift", [("rotr(x, 7) ^ rotr(x, 18) ^ (x >> 3)", "rotr(x, 7) ^ rotr(x, 18) ^ (x >> 2)")]),
    ("schedule index", [("w[t - 7] + small_sigma0(w[t - 15])", "w[t - 6] + small_sigma0(w[t - 15])")]),
    ("round constants from square roots", [("k[t] = (uint32_t)integer_root(n, 3);",
                                             "k[t] = (uint32_t)integer_root(n >> 32, 2);")]),
    ("bit length little-endian", [("tail[tail_len - 1 - i] = (uint8_t)(bits >> (8 * i));",
                                   "tail[tail_len - 8 + i] = (uint8_t)(bits >> (8 * i));")]),
    ("core dimension order", [('{"model_id", "adapter_id",', '{"adapter_id", "model_id",')]),
    ("length prefix big-endian", [("p[0] = (uint8_t)v; p[1] = (uint8_t)(v >> 8); p[2] = (uint8_t)(v >> 16); "
                                   "p[3] = (uint8_t)(v >> 24);",
                                   "p[3] = (uint8_t)v; p[2] = (uint8_t)(v >> 8); p[1] = (uint8_t)(v >> 16); "
                                   "p[0] = (uint8_t)(v >> 24);")]),
    ("further dimensions sorted descending", [("return name_cmp(a, b) < 0;", "return name_cmp(a, b) > 0;")]),
    ("value length prefix left out", [
        ("len += 4 + (uint64_t)f[i].name_len + 4 + (uint64_t)f[i].value_len;",
         "len += 4 + (uint64_t)f[i].name_len + (uint64_t)f[i].value_len;"),
        ("put_u32le(p, x->value_len); p += 4;", "")]),
    ("chain seed is the digest", [("memset(prev, 0, 16);", "memcpy(prev, digest, 16);")]),
    ("digest only in the first block", [("memcpy(msg + 16, digest, 16);",
                                         "if (i == 0) memcpy(msg + 16, digest, 16); else memset(msg + 16, 0, 16);")]),
    ("tokens big-endian", [("msg[32 + 4 * q] = (uint8_t)t;", "msg[32 + 4 * q] = (uint8_t)(t >> 24);"),
                           ("msg[32 + 4 * q + 3] = (uint8_t)(t >> 24);", "msg[32 + 4 * q + 3] = (uint8_t)t;")]),
    ("last complete block dropped", [("key_off[r + 1] = key_off[r] + len / block;",
                                      "key_off[r + 1] = key_off[r] + (len > 0 ? (len - 1) / block : 0);"),
                                     ("int64_t n = len / block;", "int64_t n = len > 0 ? (len - 1) / block : 0;")]),
    ("truncation keeps the rightmost half", [("memcpy(out, full, 16);", "memcpy(out, full + 16, 16);")]),
    ("lookup counts the first miss", [("while (h < n && contains(t, keys + 16 * (key_off[r] + h))) ++h;",
                                       "while (h < n && contains(t, keys + 16 * (key_off[r] + h))) ++h;\n"
                                       "        if (h < n) ++h;")]),
    ("largest location wins", [("return (x->loc > y->loc) - (x->loc < y->loc);",
                                "return (x->loc < y->loc) - (x->loc > y->loc);")]),
    ("present keys inserted again", [("if (contains(t, s[i].key)) continue;", "")]),
    ("capacity off by one", [("if (t->size + n_new > t->capacity)", "if (t->size + n_new >= t->capacity)")]),
    ("capacity counts every candidate", [("if (t->size + n_new > t->capacity)", "if (t->size + ns > t->capacity)")]),
    ("hit lengths ignored by the store", [("hits[r] < 0 ? 0 : hits[r]", "0")]),
    ("eviction cut one generation late", [("uint64_t cut = (uint64_t)ep[budget] + 1;",
                                           "uint64_t cut = (uint64_t)ep[budget];")]),
    ("touching store leaves present keys", [("if (p >= 0) t->e[p].epoch = epoch;", "if (p >= 0) (void)0;")]),
    ("touching lookup skips the first hit", [("for (int64_t j = 0; j < hits[r]; ++j) t->e[find",
                                              "for (int64_t j = 1; j < hits[r]; ++j) t->e[find")]),
]


def _build_and_run(name, edits, tmp):
    src = open(SOURCE).read()
    for old, new in edits:
        assert old in src, f"{name}: pattern not found: {old!r}"
        src = src.replace(old, new)
    d = os.path.join(tmp, name.replace(" ", "_"))
    os.makedirs(d)
    c_path = os.path.join(d, "pkv_oracle.c")
    open(c_path, "w").write(src)
    so = os.path.join(d, "liboracle.so")
    subprocess.run(["gcc", "-std=c11", "-O1", "-fPIC", "-shared", "-I", os.path.join(ROOT, "oracle"), "-o", so,
                    c_path, "-lpthread"], check=True, capture_output=True)
    env = dict(os.environ, PKV_ORACLE_LIB=so)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"] + PINS,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode


def test_every_planted_mistake_fails_the_pins():
    with tempfile.TemporaryDirectory() as tmp:
        with cf.ThreadPoolExecutor(max_workers=4) as ex:
            futs = {name: ex.submit(_build_and_run, name, edits, tmp) for name, edits in MUTANTS}
            survivors = [name for name, f in futs.items() if f.result() == 0]
    assert not survivors, f"mutants not caught by the pins: {survivors}"
