"""The transposed-route position used by the backward's dQ kernel.

The dK/dV kernel stores dS per entry of the transposed route (key block i ->
the query blocks that select it); the dQ kernel walks the forward route and
finds the entry of a pair (query block j selects key block i) in closed form,
route_user_rank in csrc/bf1_route.h.  A wrong position would make the dQ
kernel read another pair's dS, so the closed form is checked here on the CPU,
compiled with the host compiler, against the oracle's own transposed table
(§3.1, Eq. 1, read column-wise) for every pair of several routes.
"""

import os
import shutil
import subprocess

import pytest

from oracle import bf1_oracle as orc

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "..", "paper_2608_20427_amd", "csrc")

PROGRAM = r"""
#include <cstdio>
#include <cstdint>
#include "bf1_route.h"
int main() {
    long long L, i, j;
    while (std::scanf("%lld %lld %lld", &L, &i, &j) == 3)
        std::printf("%lld\n", (long long)bf1::route_user_rank(L, i, j));
    return 0;
}
"""


@pytest.fixture(scope="module")
def rank_exe(tmp_path_factory):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    d = tmp_path_factory.mktemp("rank")
    src, exe = d / "rank.cpp", d / "rank"
    src.write_text(PROGRAM)
    subprocess.run([cxx, "-O1", "-std=c++17", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    return str(exe)


@pytest.mark.parametrize("n,b,L", [(64, 64, 2), (4096, 64, 2), (32768, 64, 2), (32768, 128, 2),
                                   (5000, 64, 0), (5000, 64, 1), (9000, 64, 3), (20000, 64, 5),
                                   (70000, 128, 8)])
def test_route_user_rank_matches_oracle_transpose(rank_exe, n, b, L):
    rp_t, ci_t = orc.csr_transposed(n, b, L)
    NB = len(rp_t) - 1
    pairs = [(i, j) for j in range(NB) for i in orc.route(j, L)]
    inp = "".join(f"{L} {i} {j}\n" for i, j in pairs)
    out = subprocess.run([rank_exe], input=inp, capture_output=True, text=True, check=True).stdout.split()
    assert len(out) == len(pairs)
    for (i, j), r in zip(pairs, out):
        r = int(r)
        users = ci_t[rp_t[i]:rp_t[i + 1]]
        assert 0 <= r < len(users) and users[r] == j, (n, b, L, i, j, r)
