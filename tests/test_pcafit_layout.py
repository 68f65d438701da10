"""Host check of the PCA fit's workspace layout (no GPU): the regions the fit
carves from the caller's workspace are aligned, disjoint, in order and large
enough, and the eigenvector array holds all n columns (the eigensolver may use
its columns as scratch). Compiles a small C++ program against the layout
header with the host compiler."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_37842_amd", "csrc")

PROGRAM = r"""
#include <cstdio>
#include <vector>
#include "pcafit_layout.h"
using eogp::fit_layout;
int main() {
  const long long cases[][3] = {{10, 4, 0}, {10, 9, 1000}, {2048, 1024, 123457},
                                {10000, 8192, 1 << 20}, {1, 1, 7}, {4096, 64, 333}};
  int bad = 0;
  for (const auto& c : cases) {
    const long long n = c[0], k = c[1];
    const size_t sb = (size_t)c[2];
    const eogp::FitLayout L = fit_layout(n, k, sb);
    struct R { size_t off, need; const char* name; };
    const std::vector<R> regs = {{L.ints, 16, "ints"}, {L.solver, sb, "solver"},
                                 {L.g, (size_t)(n * n * 8), "G"}, {L.w, (size_t)(n * 8), "W"},
                                 {L.v, (size_t)(n * n * 8), "V"}, {L.vs, (size_t)(n * k * 8), "Vs"}};
    for (size_t i = 0; i < regs.size(); ++i) {
      const size_t end = (i + 1 < regs.size()) ? regs[i + 1].off : L.total;
      if (regs[i].off % 256) { std::printf("%s misaligned\n", regs[i].name); ++bad; }
      if (end < regs[i].off || end - regs[i].off < regs[i].need) {
        std::printf("n=%lld k=%lld: %s has %zu bytes, needs %zu\n", n, k, regs[i].name,
                    end - regs[i].off, regs[i].need);
        ++bad;
      }
    }
    if (regs[0].off != 0) { std::printf("layout does not start at 0\n"); ++bad; }
  }
  std::printf("%s\n", bad ? "FAIL" : "OK");
  return bad ? 1 : 0;
}
"""


def test_pca_fit_workspace_layout(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    src = tmp_path / "layout.cpp"
    src.write_text(PROGRAM)
    exe = tmp_path / "layout"
    subprocess.run([cxx, "-std=c++17", "-O1", f"-I{CSRC}", str(src), "-o", str(exe)], check=True,
                   capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True)
    assert res.returncode == 0 and res.stdout.strip().endswith("OK"), res.stdout
