"""Automatic prefix caching, host side (no GPU).

* Pins for the oracle (oracle/prefix_cache.py), worked out by hand from its
  definition: the page granularity, the rule that one prompt token is always
  left to compute, that a page is only found under its whole prefix, that a
  decode step or a fork ends a sequence's contributions, and that known
  prefixes outlive their sequences.
* Parity of the library's sequence table (paper_2411_03519_amd/csrc/kv_pool.cpp,
  the code behind metro_seq_open_cached) with the oracle: random scripts of
  opens, cached opens, prefills, decode steps, forks and closes are replayed
  through both, and every cached open must take over exactly the number of
  tokens the oracle gives.  The C++ side runs as a small host program built
  with g++ (tests/kvpool_test.cpp, "replay" mode).
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle.prefix_cache import OraclePrefixCache


def test_oracle_page_granularity_and_last_token():
    c = OraclePrefixCache()
    c.open(1)
    a = list(range(100, 140))          # 40 tokens: pages [0,16) and [16,32) are known
    c.prefill(1, a)
    assert c.open_cached(2, a) == 32
    assert c.open_cached(3, a[:35] + [7, 7]) == 32
    assert c.open_cached(4, a[:31] + [7, 7, 7]) == 16
    assert c.open_cached(5, a[:33]) == 32
    assert c.open_cached(6, a[:32]) == 16   # one token is always left to compute
    assert c.open_cached(7, a[:17]) == 16
    assert c.open_cached(8, a[:16]) == 0
    assert c.open_cached(9, []) == 0


def test_oracle_whole_prefix_must_match():
    c = OraclePrefixCache()
    c.open(1)
    a = list(range(64))
    c.prefill(1, a)
    b = list(a)
    b[0] = 999                          # second page equal, first not: nothing
    assert c.open_cached(2, b) == 0
    b = list(a)
    b[40] = 999                         # third page differs: two pages
    assert c.open_cached(3, b) == 32


def test_oracle_decode_and_fork_end_contributions():
    c = OraclePrefixCache()
    c.open(1)
    c.prefill(1, list(range(20)))
    c.decode(1)
    c.prefill(1, list(range(20, 40)))   # after a decode step: not known
    assert c.open_cached(2, list(range(41))) == 16
    c.open(3)
    c.fork(3)
    c.prefill(3, list(range(500, 540)))
    assert c.open_cached(4, list(range(500, 541))) == 0


def test_oracle_prefixes_outlive_sequences_and_chain_through_hits():
    c = OraclePrefixCache()
    c.open(1)
    c.prefill(1, list(range(32)))
    c.close(1)
    assert c.open_cached(2, list(range(40))) == 32
    # the hit sequence continues; its new pages extend the known prefixes
    c.prefill(2, list(range(32, 70)))
    c.close(2)
    assert c.open_cached(3, list(range(70)) + [1]) == 64


def random_script(seed, n_ops=400):
    """Operations over prompts drawn from a few families that share leading
    tokens, as agents' prompts share instructions and persona text."""
    rng = np.random.default_rng(seed)
    fams = [rng.integers(0, 50, 200).tolist() for _ in range(3)]
    ops, live, nid = [], {}, 1

    def prompt():
        f = fams[rng.integers(0, 3)]
        k = int(rng.integers(0, 120))
        return f[:k] + rng.integers(0, 3, int(rng.integers(1, 40))).tolist()

    for _ in range(n_ops):
        r = rng.random()
        if not live or r < 0.3:
            p = prompt()
            ops.append(("c", nid, p))
            live[nid] = True
            nid += 1
        elif r < 0.38:
            ops.append(("o", nid))
            live[nid] = True
            nid += 1
        elif r < 0.6:
            sid = list(live)[rng.integers(0, len(live))]
            ops.append(("p", sid, rng.integers(0, 3, int(rng.integers(1, 40))).tolist()))
        elif r < 0.7:
            sid = list(live)[rng.integers(0, len(live))]
            ops.append(("d", sid))
        elif r < 0.75:
            sid = list(live)[rng.integers(0, len(live))]
            ops.append(("f", nid, sid))
            live[nid] = True
            nid += 1
        else:
            sid = list(live)[rng.integers(0, len(live))]
            ops.append(("x", sid))
            del live[sid]
    return ops


def run_oracle(ops):
    c = OraclePrefixCache()
    lens, out, script = {}, [], []
    for op in ops:
        if op[0] in "pdx" and op[1] not in lens:
            continue   # a fork of an empty sequence was dropped
        if op[0] == "f" and op[2] not in lens:
            continue
        if op[0] == "c":
            _, sid, p = op
            if len(p) == 0:
                continue
            k = c.open_cached(sid, p)
            lens[sid] = k
            out.append((sid, k))
            script.append(f"c {sid} {len(p)} " + " ".join(map(str, p)))
            # the request's prefill of the rest of its prompt
            rest = p[k:]
            c.prefill(sid, rest)
            lens[sid] += len(rest)
            script.append(f"p {sid} {len(rest)} " + " ".join(map(str, rest)))
        elif op[0] == "o":
            c.open(op[1])
            lens[op[1]] = 0
            script.append(f"o {op[1]}")
        elif op[0] == "p":
            c.prefill(op[1], op[2])
            lens[op[1]] += len(op[2])
            script.append(f"p {op[1]} {len(op[2])} " + " ".join(map(str, op[2])))
        elif op[0] == "d":
            if lens[op[1]] == 0:
                continue
            c.decode(op[1])
            lens[op[1]] += 1
            script.append(f"d {op[1]}")
        elif op[0] == "f":
            _, new, src = op
            n = lens[src]
            if n == 0:
                continue
            c.fork(new)
            lens[new] = n
            script.append(f"f {new} {src} {n}")
        elif op[0] == "x":
            c.close(op[1])
            del lens[op[1]]
            script.append(f"x {op[1]}")
    return out, "\n".join(script) + "\n"


@pytest.fixture(scope="module")
def kvpool_exe(repo_root, tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("kvp") / "kvpool_test")
    subprocess.run([gxx, "-std=c++17", "-O1", os.path.join(repo_root, "tests", "kvpool_test.cpp"),
                    os.path.join(repo_root, "paper_2411_03519_amd", "csrc", "kv_pool.cpp"), "-o", exe], check=True)
    return exe


@pytest.mark.parametrize("seed", range(6))
def test_sequence_table_matches_oracle(kvpool_exe, seed):
    ops = random_script(seed)
    want, script = run_oracle(ops)
    r = subprocess.run([kvpool_exe, "replay"], input=script, capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    got = [tuple(int(v) for v in line.split()[1:]) for line in r.stdout.splitlines() if line.startswith("c ")]
    assert got == want
    assert sum(k for _, k in want) > 0   # the scripts do exercise hits
