"""The oracle's C converter (oracle/convert.c) built with the host
AddressSanitizer and UndefinedBehaviorSanitizer (gcc; nothing here touches
the GPU) runs clean over special values, a stride through all 2^32 fp32
patterns and misaligned, ragged buffers, and agrees bit for bit with the
unsanitized build the tests use."""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import convert

DRIVER = r"""
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

uint16_t oracle_trunc16_one(float x);
void oracle_trunc16(const float* x, uint16_t* out, int64_t n);
void oracle_trunc16_range(uint32_t first, int64_t count, uint16_t* out);

int main(void) {
  uint64_t h = 1469598103934665603ull;   /* FNV-1a over every output */
  const int64_t stride = 4099;            /* blocks of 16384 consecutive patterns, 4099 blocks apart */
  uint16_t* out = malloc(1 << 16);
  for (uint64_t u = 0; u < (1ull << 32); u += stride * 16384) {
    const int64_t cnt = 16384;
    oracle_trunc16_range((uint32_t)u, cnt, out);
    for (int64_t i = 0; i < cnt; ++i) { h ^= out[i]; h *= 1099511628211ull; }
  }
  /* misaligned, ragged buffers: n = 0 .. 67 starting 1 float into an allocation of exactly n + 1 */
  for (int64_t n = 0; n < 68; ++n) {
    float* x = malloc(sizeof(float) * (size_t)(n + 1));
    uint16_t* o = malloc(sizeof(uint16_t) * (size_t)(n + 1));
    for (int64_t i = 0; i <= n; ++i) { uint32_t b = 0x9E3779B9u * (uint32_t)(i + 7 * n); memcpy(&x[i], &b, 4); }
    oracle_trunc16(x + 1, o + 1, n);
    for (int64_t i = 1; i <= n; ++i) { h ^= o[i]; h *= 1099511628211ull; }
    free(x);
    free(o);
  }
  free(out);
  printf("%016llx\n", (unsigned long long)h);
  return 0;
}
"""


def _build(tmp, sanitize):
    drv = os.path.join(tmp, "driver.c")
    with open(drv, "w") as f:
        f.write(DRIVER)
    exe = os.path.join(tmp, "san" if sanitize else "plain")
    flags = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"] \
        if sanitize else []
    subprocess.run(["gcc", "-O1", "-std=c99", "-fno-fast-math", "-ffp-contract=off", *flags, convert.SRC, drv,
                    "-o", exe, "-lm"], check=True, capture_output=True, text=True)
    return exe


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_converter_clean_under_asan_and_ubsan(tmp_path):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    san = subprocess.run([_build(str(tmp_path), True)], capture_output=True, text=True, env=env, timeout=600)
    assert san.returncode == 0, san.stderr[-2000:]
    assert "runtime error" not in san.stderr and "AddressSanitizer" not in san.stderr, san.stderr[-2000:]
    plain = subprocess.run([_build(str(tmp_path), False)], capture_output=True, text=True, timeout=600)
    assert plain.returncode == 0 and plain.stdout == san.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_sanitized_walk_matches_the_library(tmp_path):
    """The unsanitized driver's hash equals one computed from the library the
    tests load, over the same inputs (the driver hashes what it computed)."""
    plain = subprocess.run([_build(str(tmp_path), False)], capture_output=True, text=True, timeout=600)
    h = np.uint64(1469598103934665603)
    prime = np.uint64(1099511628211)
    with np.errstate(over="ignore"):
        for u in range(0, 1 << 32, 4099 * 16384):
            out = convert.truncate_bf16_bits(
                (np.arange(16384, dtype=np.uint64) + np.uint64(u)).astype(np.uint32).view(np.float32))
            for v in out.astype(np.uint64):
                h = (h ^ v) * prime
        for n in range(68):
            b = (np.uint32(0x9E3779B9) * (np.arange(n + 1, dtype=np.uint32) + np.uint32(7 * n))).astype(np.uint32)
            out = convert.truncate_bf16_bits(b[1:].view(np.float32))
            for v in out.astype(np.uint64):
                h = (h ^ v) * prime
    assert plain.stdout.strip() == f"{int(h):016x}"
