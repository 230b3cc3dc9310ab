"""The host suffix's fork-join pool (csrc/host_pool.h): every index of a run
is executed exactly once, also when runs of different sizes follow each other
on an oversubscribed pool, where a thread that missed the end of one run may
wake during the next.  Built with g++ from the header alone and run on the CPU."""
import os
import shutil
import subprocess

import pytest

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2608_14586_amd", "csrc")

DRIVER = r'''
#include <cstdio>
#include "host_pool.h"
int main(int argc, char** argv) {
  const int threads = atoi(argv[1]), runs = atoi(argv[2]);
  vla::host::Pool p(threads);
  const int sizes[] = {3, 70, 17, 1, 64, 2, 129};
  for (int r = 0; r < runs; ++r) {
    const int n = sizes[r % 7];
    std::vector<std::atomic<int>> hits(n);
    for (auto& h : hits) h = 0;
    p.run(n, [&](int i) { hits[i].fetch_add(1); });
    for (int i = 0; i < n; ++i)
      if (hits[i].load() != 1) { std::printf("run %d index %d ran %d times\n", r, i, hits[i].load()); return 1; }
  }
  std::printf("ok %d\n", runs);
  return 0;
}
'''


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_pool_runs_every_index_once(tmp_path):
    src = tmp_path / "pool_driver.cpp"
    src.write_text("#include <atomic>\n#include <cstdlib>\n" + DRIVER)
    exe = tmp_path / "pool_driver"
    subprocess.run(["g++", "-O2", "-std=c++17", "-pthread", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    # four times as many threads as CPUs: preemption inside a claim is common
    threads = 4 * len(os.sched_getaffinity(0))
    r = subprocess.run([str(exe), str(threads), "30000"], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0 and r.stdout.strip() == "ok 30000", r.stdout + r.stderr
