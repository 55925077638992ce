"""The union-find walks of tg_mask_rois (csrc/unionfind.h) on the CPU: the header is
compiled with g++ (under AddressSanitizer and UndefinedBehaviorSanitizer) into a small
driver (uf_harness.cpp). Consistent forests give the connected components, each rooted at
its smallest index; arrays that break the walks' invariant (a cycle, a link upwards or below zero, a link reported by a racing writer that
is not smaller) end the walk with a failure after a bounded number of reads instead of
looping."""
import os
import shutil
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2404_09267_amd", "csrc")


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    exe = str(tmp_path_factory.mktemp("uf") / "uf_harness")
    subprocess.run([gxx, "-std=c++17", "-O1", "-Wall", "-Werror", "-g", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-I", CSRC,
                    os.path.join(HERE, "uf_harness.cpp"), "-o", exe], check=True)

    def run(lines):
        out = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True,
                             text=True, timeout=60, check=True).stdout
        return [list(map(int, ln.split())) for ln in out.strip().splitlines()]

    return run


def _arr(a):
    return f"{len(a)} " + " ".join(map(str, a))


def _walk(a, i):
    """Root of i by following the links; -1 if a link on the way is not smaller (or is
    negative) before a node that points to itself."""
    while True:
        p = a[i]
        if p == i:
            return i
        if p < 0 or p > i:
            return -1
        i = p


def _components(n, edges):
    """Smallest index of each node's connected component (breadth-first search)."""
    adj = [[] for _ in range(n)]
    for a, b in edges:
        adj[a].append(b)
        adj[b].append(a)
    low = [-1] * n
    for s in range(n):
        if low[s] >= 0:
            continue
        stack, seen = [s], [s]
        low[s] = s
        while stack:
            u = stack.pop()
            for v in adj[u]:
                if low[v] < 0:
                    low[v] = s
                    stack.append(v)
                    seen.append(v)
    return low


def test_cycles_and_bad_links_fail(harness):
    cases = [
        ([1, 0], 0), ([1, 0], 1),                    # two-cycle
        ([0, 0, 1, 6, 3, 4, 5, 6], 7),               # chain 7..3 with 3 -> 6 upwards
        ([0, 0, 1, 2, 3, 4, 5, 6], 7),               # a valid chain, for contrast
        ([0, -3, 1], 2),                             # negative link
        ([0, 5], 1),                                 # link past the array
        ([2, 0, 2], 1),                              # upward link one step away
        ([0, 1, 2, 3], 3),                           # a root
    ]
    got = harness([f"F {_arr(a)} {i}" for a, i in cases])
    for (a, i), (root, reads) in zip(cases, got):
        assert root == _walk(a, i), (a, i, root)
        assert reads <= 2 * len(a) + 2
    assert [g[0] for g in got] == [-1, -1, -1, 0, -1, -1, -1, 3]


def test_unite_on_broken_arrays_fails(harness):
    cases = ["U 2 1 0 0 1",                 # two-cycle
             "U 4 0 3 1 2 3 0",             # 1 -> 3 upwards
             "U 3 0 -1 2 1 2",              # negative
             "X 3 0 1 2 1 2 7",             # the replaced link is reported past b
             "X 3 0 1 2 1 2 -5",            # ... or negative
             "X 4 0 1 2 3 2 3 1",           # ... or a smaller root: retried from there
             "U 4 0 1 2 3 3 1"]             # a plain unite
    got = harness(cases)
    assert [g[0] for g in got] == [0, 0, 0, 0, 0, 1, 1]
    for g in got:
        assert g[1] <= 40
    # the plain unite links the larger root under the smaller
    assert got[-1][2:] == [0, 1, 2, 1]
    # after the planted retry, 3 and 2 are joined under 1, 0 alone
    arr = got[-2][2:]
    assert _walk(arr, 3) == _walk(arr, 2) and _walk(arr, 0) == 0


def test_random_forests_give_components(harness):
    rng = np.random.default_rng(11)
    lines, want = [], []
    for trial in range(60):
        n = int(rng.integers(1, 300))
        m = int(rng.integers(0, 2 * n))
        edges = [(int(a), int(b)) for a, b in rng.integers(0, n, size=(m, 2))]
        lines.append(f"E {n} {m} " + " ".join(f"{a} {b}" for a, b in edges))
        want.append((n, _components(n, edges)))
    for (n, low), g in zip(want, harness(lines)):
        assert g[0] == 1
        roots, arr = g[1:1 + n], g[1 + n:]
        assert roots == low  # every set rooted at its smallest index
        assert all(0 <= arr[i] <= i for i in range(n))  # links never point upwards
        assert all(low[arr[i]] == low[i] for i in range(n))  # links stay in their set


def test_random_arrays_walk_like_the_definition(harness):
    """Arbitrary arrays, most of them broken: the find equals following the links (or
    -1), and its reads stay bounded by the array's size."""
    rng = np.random.default_rng(12)
    lines, cases = [], []
    for trial in range(300):
        n = int(rng.integers(1, 40))
        a = rng.integers(-2, n + 3, size=n)
        keep = rng.random(n) < 0.7  # mostly downward links, some anything
        a = np.where(keep, [int(rng.integers(0, i + 1)) for i in range(n)], a).tolist()
        i = int(rng.integers(0, n))
        lines.append(f"F {_arr(a)} {i}")
        cases.append((a, i))
    for (a, i), (root, reads) in zip(cases, harness(lines)):
        assert root == _walk(a, i)
        assert reads <= 2 * len(a) + 2
