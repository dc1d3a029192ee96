"""The task order of the k-center in rounds, checked on the host.

`decode_task` in rounds.hip maps a queue position to a task (select,
candidate block pair, greedy, or fold tile of one request and round). The
persistent kernel is deadlock-free and its completion counts are exact only
if, in every macro-round, each task of each request appears exactly once
and each task's dependencies (Sec. 3.4: a round's select needs the previous
round's folds; candidates need the select; the greedy needs the candidates;
the folds need the greedy) sit at smaller queue positions. This test
compiles the function's own text with the host compiler and checks both on
batches of several shapes.
"""
import os
import re
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2607_27952_amd", "csrc", "rounds.hip")
HDR = os.path.join(ROOT, "paper_2607_27952_amd", "csrc", "last_internal.h")


def _constant(text, name):
    m = re.search(r"constexpr int %s = (\d+);" % name, text)
    assert m, name
    return int(m.group(1))


@pytest.fixture(scope="module")
def decoder(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    src = open(SRC).read()
    hdr = open(HDR).read()
    sub = _constant(hdr, "kRoundCands") // 32
    k_ct = sub * (sub + 1) // 2   # 32 x 32 block pairs of the candidate Gram, one task each
    f_rows = _constant(hdr, "kRoundFoldRows")
    a = src.index("template <typename Ft>\n__device__ __forceinline__ int64_t decode_task")
    b = src.index("\n}\n", a) + 3
    fn = src[a:b].replace("__device__ __forceinline__ ", "")
    prog = (
        "#include <cstdint>\n#include <cstdio>\n#include <vector>\n"
        f"static const int kCT = {k_ct};\n" + fn + r"""
int main() {
  int R, M;
  if (scanf("%d %d", &R, &M) != 2) return 1;
  std::vector<int64_t> ft(R + 1, 0);
  for (int i = 0; i < R; ++i) { long t; if (scanf("%ld", &t) != 1) return 1; ft[i + 1] = ft[i] + t; }
  auto fta = [&](int64_t i) -> int64_t { return ft[i]; };
  int64_t Q = 0;
  for (int i = 0; i < R; ++i) Q += 2 + kCT + (ft[i + 1] - ft[i]);
  for (int64_t m = 0; m < M; ++m)
    for (int64_t u = 0; u < Q; ++u) {
      int kind = 0, r = 0, sub = 0;
      const int64_t tq = decode_task(u, (int64_t)R, fta, kind, r, sub);
      printf("%ld %ld %d %d %ld %d\n", (long)m, (long)u, kind, r, (long)(m + tq), sub);
    }
  return 0;
}
""")
    d = tmp_path_factory.mktemp("decode")
    cpp, exe = d / "decode.cpp", d / "decode"
    cpp.write_text(prog)
    subprocess.run([gxx, "-O1", "-std=c++17", "-o", str(exe), str(cpp)], check=True)
    return str(exe), k_ct, f_rows


CASES = [
    [85, 183, 295],          # three small requests, both halves
    [150],                   # one request: no second half
    [1, 1],                  # one-token requests
    [0, 512, 0, 700, 3],     # empty requests
    [16384] * 8,             # the video batch
    [32768, 32768],          # the long-video batch
]


@pytest.mark.parametrize("N", CASES + ["ragged128", "ragged33"], ids=str)
def test_decode_order(decoder, N):
    exe, k_ct, f_rows = decoder
    rng = np.random.default_rng(7)
    if N == "ragged128":
        N = list(rng.integers(256, 16385, 128))
    elif N == "ragged33":
        N = list(rng.integers(0, 3000, 33))
    R, M = len(N), 4
    tiles = [(int(n) + f_rows - 1) // f_rows for n in N]
    out = subprocess.run([exe], input=f"{R} {M} " + " ".join(map(str, tiles)), capture_output=True, text=True,
                         check=True).stdout
    rows = np.array([list(map(int, line.split())) for line in out.split("\n") if line], np.int64)
    Q = sum(2 + k_ct + t for t in tiles)
    assert len(rows) == M * Q
    RA = (R + 1) // 2
    pos = {}
    for m in range(M):
        got = [tuple(x) for x in rows[rows[:, 0] == m][:, 2:]]
        assert len(set(got)) == Q, "a task listed twice in one macro-round"
        want = set()
        for r in range(R):
            for kind, count in ((0, 1), (1, k_ct), (2, 1), (3, tiles[r])):
                n = m - 1 if (kind == 3 and r >= RA) else m   # the second half folds a round behind
                want.update((kind, r, n, s) for s in range(count))
        assert set(got) == want
        for u, key in enumerate(got):
            if key[2] >= 0:
                pos[key] = m * Q + u
    for (kind, r, n, s), p in pos.items():
        if kind == 0:
            deps = [(3, r, n - 1, t) for t in range(tiles[r])] if n > 0 else []
        elif kind == 1:
            deps = [(0, r, n, 0)]
        elif kind == 2:
            deps = [(1, r, n, t) for t in range(k_ct)]
        else:
            deps = [(2, r, n, 0)]
        for dep in deps:
            assert dep in pos and pos[dep] < p, f"{(kind, r, n, s)} listed before its dependency {dep}"
