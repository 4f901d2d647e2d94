"""Host-only checks of the work-item schedule (csrc/schedule.h).

The kernel's deadlock freedom rests on two properties of the ordered item
list: every item appears exactly once, and every item an item waits for
comes earlier in the list (statistics of a request < its decide < its pass-2
items < its pick).  A small C++ driver compiled with g++ enumerates the list
for many shapes and these tests check both properties."""

import os
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_26004_amd", "csrc")

DRIVER = r"""
#include <cstdio>
#include <cstdlib>
#include "schedule.h"
using namespace asym;
int main(int argc, char** argv) {
  const int B = atoi(argv[1]), K = atoi(argv[2]), S = atoi(argv[3]), G = atoi(argv[4]);
  const int ee = argc > 5 ? atoi(argv[5]) : 0;
  const int p2 = argc > 6 ? atoi(argv[6]) : 1;
  Sched sc;
  if (!sched_build(B, K, S, G, sc, ee, p2)) { printf("FAIL build\n"); return 1; }
  printf("T %d %d %d %d\n", sc.total, sc.L1, sc.L2, sc.L3);
  for (int i = 0; i < sc.total; ++i) {
    const Item it = sched_item(sc, K, S, i);
    printf("%d %d %d\n", it.type, it.req, it.sub);
  }
  const Item past = sched_item(sc, K, S, sc.total);
  printf("P %d\n", past.type);
  return 0;
}
"""


@pytest.fixture(scope="module")
def driver():
    d = tempfile.mkdtemp(prefix="asym_sched_")
    src = os.path.join(d, "drv.cpp")
    exe = os.path.join(d, "drv")
    with open(src, "w") as f:
        f.write(DRIVER)
    subprocess.run(["g++", "-O1", "-std=c++17", "-I", CSRC, src, "-o", exe], check=True)
    return exe


def enumerate_items(exe, B, K, S, G, ee=0, p2=1):
    out = subprocess.run([exe, str(B), str(K), str(S), str(G), str(ee), str(p2)], check=True,
                         capture_output=True, text=True).stdout.split("\n")
    head = out[0].split()
    assert head[0] == "T"
    total = int(head[1])
    items = [tuple(map(int, ln.split())) for ln in out[1:1 + total]]
    assert out[1 + total] == "P -1"          # past the end: no item
    return items


SHAPES = [(1, 0, 1, 1), (1, 4, 4, 512), (8, 5, 8, 1024), (32, 8, 10, 1024),
          (128, 6, 10, 1024), (512, 8, 16, 1024), (3, 63, 2, 7), (200, 1, 1, 3),
          (7, 2, 30, 2048), (128, 6, 19, 256)]


@pytest.mark.parametrize("p2", [1, 2, 4])
@pytest.mark.parametrize("B,K,S,G", SHAPES)
def test_every_item_once_and_dependencies_first(driver, B, K, S, G, p2):
    """Pass 2 runs as p2 items per chunk (sub = chunk * p2 + part)."""
    items = enumerate_items(driver, B, K, S, G, 0, p2)
    S2 = S * p2
    stats, decide, pass2, pick = {}, {}, {}, {}
    for idx, (ty, req, sub) in enumerate(items):
        assert 0 <= req < B
        if ty == 0:
            assert 0 <= sub < (K + 1) * S
            assert (req, sub) not in stats
            stats[(req, sub)] = idx
        elif ty == 1:
            assert req not in decide
            decide[req] = idx
        elif ty == 2:
            assert 0 <= sub < S2 and (req, sub) not in pass2
            pass2[(req, sub)] = idx
        elif ty == 3:
            assert req not in pick
            pick[req] = idx
        else:
            pytest.fail(f"unknown item type {ty}")
    assert len(stats) == B * (K + 1) * S
    assert len(decide) == len(pick) == B and len(pass2) == B * S2
    for r in range(B):
        last_stat = max(stats[(r, s)] for s in range((K + 1) * S))
        assert decide[r] > last_stat
        for m in range(S2):
            assert pass2[(r, m)] > decide[r]
        assert pick[r] > max(pass2[(r, m)] for m in range(S2))


def test_lags_cover_the_items_in_flight(driver):
    # away from the end of the list (where no statistics items are left to
    # put in between), the decide item of a request comes at least G items
    # after its last statistics item, so with G workgroups it rarely waits
    B, K, S, G = 128, 6, 10, 1024
    items = enumerate_items(driver, B, K, S, G)
    n_stats = B * (K + 1) * S
    last_stat = {}
    seen = 0
    for idx, (ty, req, sub) in enumerate(items):
        if ty == 0:
            last_stat[req] = idx
            seen += 1
        elif ty == 1 and seen < n_stats:
            assert idx - last_stat[req] >= G, (req, idx, last_stat[req])


GROUP_DRIVER = r"""
#include <cstdio>
#include <cstdlib>
#include "schedule.h"
int main(int argc, char** argv) {
  const int n = atoi(argv[1]);
  for (int s = 0; s < n; ++s) printf("%d\n", asym::xcd_grouped(s, n));
  return 0;
}
"""


def test_xcd_grouped_renumbering(tmp_path):
    """A bijection on [0, n) that gives the items one XCD runs (sub, sub + 8,
    ...) consecutive positions, so a row's chunks share few XCDs."""
    src = tmp_path / "g.cpp"
    exe = tmp_path / "g"
    src.write_text(GROUP_DRIVER)
    subprocess.run(["g++", "-O1", "-std=c++17", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    for n in (1, 5, 7, 8, 9, 70, 71, 135, 512):
        p = [int(x) for x in subprocess.run([str(exe), str(n)], check=True, capture_output=True,
                                            text=True).stdout.split()]
        assert sorted(p) == list(range(n))
        for s in range(n - 8):
            assert p[s + 8] == p[s] + 1


EE_SHAPES = [(1, 1, 1, 1, 1), (128, 6, 10, 1024, 2), (128, 6, 10, 1024, 1), (32, 8, 10, 1024, 3),
             (512, 8, 16, 1024, 2), (7, 2, 30, 2048, 2), (200, 3, 1, 3, 1), (5, 63, 2, 7, 60)]


@pytest.mark.parametrize("p2", [1, 4])
@pytest.mark.parametrize("B,K,S,G,ee", EE_SHAPES)
def test_early_exit_order(driver, B, K, S, G, ee, p2):
    """With early exit the first ee rows of a request are read, then its
    verdict, then the other rows (skipped after a sure rejection); every
    item appears once and each comes after all items it waits for."""
    items = enumerate_items(driver, B, K, S, G, ee, p2)
    S2 = S * p2
    n1 = ee * S
    stats, verdict, decide, pass2, pick = {}, {}, {}, {}, {}
    for idx, (ty, req, sub) in enumerate(items):
        assert 0 <= req < B
        if ty in (0, 5):
            assert (sub < n1) == (ty == 0)
            assert 0 <= sub < (K + 1) * S and (req, sub) not in stats
            stats[(req, sub)] = idx
        elif ty == 4:
            assert req not in verdict
            verdict[req] = idx
        elif ty == 1:
            decide[req] = idx
        elif ty == 2:
            pass2[(req, sub)] = idx
        elif ty == 3:
            pick[req] = idx
        else:
            pytest.fail(f"unknown item type {ty}")
    assert len(stats) == B * (K + 1) * S and len(verdict) == len(decide) == len(pick) == B
    for r in range(B):
        assert verdict[r] > max(stats[(r, s)] for s in range(n1))
        assert min(stats[(r, s)] for s in range(n1, (K + 1) * S)) > verdict[r]
        assert decide[r] > max(stats[(r, s)] for s in range((K + 1) * S))
        assert len([m for m in range(S2) if (r, m) in pass2]) == S2
        assert min(pass2[(r, m)] for m in range(S2)) > decide[r]
        assert pick[r] > max(pass2[(r, m)] for m in range(S2))


def test_early_exit_off_when_no_second_group(driver):
    # ee >= K + 1 leaves nothing to skip: the plain schedule
    assert enumerate_items(driver, 4, 2, 3, 64, 3) == enumerate_items(driver, 4, 2, 3, 64, 0)
