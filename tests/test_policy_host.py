"""Host-side checks of the closed-form helpers that the device kernels share with the host (csrc/policy.h),
compiled with g++ into a small program (no GPU).

paged_pool_row maps a position to its row of a paged pool (Section 3.1's paged engine: a block table per
sequence).  The cases here are the ones whose arithmetic could overflow or read outside the table: a block
number whose row does not fit in int32, positions past the table, freed (negative) entries, the largest
block size the ABI accepts."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_01483_amd", "csrc")

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")

DRIVER = r"""
#include <stdio.h>
#include <stdint.h>
#include "policy.h"
using murmur::paged_pool_row;
static int fails = 0;
#define EXPECT(got, want) do { long long g_ = (got), w_ = (want); \
    if (g_ != w_) { printf("line %d: got %lld want %lld\n", __LINE__, g_, w_); ++fails; } } while (0)
int main() {
    const int32_t table[4] = {3, -1, 0x7fffffff, 1 << 27};
    // ordinary rows: block 0 -> physical block 3
    EXPECT(paged_pool_row(table, 4, 4, 0), 48);
    EXPECT(paged_pool_row(table, 4, 4, 15), 63);
    // a freed block and a position past the table
    EXPECT(paged_pool_row(table, 4, 4, 16), -1);
    EXPECT(paged_pool_row(table, 4, 4, 64), -1);
    EXPECT(paged_pool_row(table, 2, 4, 40), -1);
    // block numbers whose row exceeds 2^31 - 1: no wrap-around into the pool
    EXPECT(paged_pool_row(table, 4, 4, 32), -1);          // 0x7fffffff * 16
    EXPECT(paged_pool_row(table, 4, 4, 48), -1);          // 2^27 * 16 = 2^31
    EXPECT(paged_pool_row(table, 4, 3, 24), (1LL << 30)); // 2^27 * 8 = 2^30 fits
    // block size 1 and the largest block size (2^20)
    EXPECT(paged_pool_row(table, 4, 0, 0), 3);
    EXPECT(paged_pool_row(table, 4, 0, 2), 0x7fffffff);
    EXPECT(paged_pool_row(table, 4, 20, 5), 3LL * (1 << 20) + 5);
    const int32_t small[1] = {2047};
    EXPECT(paged_pool_row(small, 1, 20, (1 << 20) - 1), 2047LL * (1 << 20) + (1 << 20) - 1);
    const int32_t big[1] = {2048};
    EXPECT(paged_pool_row(big, 1, 20, 0), -1);            // 2048 * 2^20 = 2^31
    printf(fails ? "FAILED\n" : "paged rows: ok\n");
    return fails != 0;
}
"""


def test_paged_pool_row(tmp_path):
    src = tmp_path / "paged_rows.cpp"
    src.write_text(DRIVER)
    exe = str(tmp_path / "paged_rows")
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", f"-I{CSRC}", str(src), "-o", exe], check=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert res.returncode == 0 and "paged rows: ok" in res.stdout, res.stdout + res.stderr
