"""Static checks of the compiled 4-wave 16-bit GEMM loop (CPU only: hipcc
cross-compiles the two whole-tile translation units to gfx950 assembly).

The loop issues its 16 x 16 x 32 MFMAs as inline assembly on accumulators tied
to AGPR quadruples, so the compiler inserts none of the wait states an MFMA's
accumulators need; the source keeps them itself. These tests check, in every
4-wave kernel, what that relies on:
  - no instruction between the loop's MFMAs touches an accumulator register
    (no v_accvgpr copies, no spills to scratch inside the loop);
  - every MFMA reads its accumulator from the registers it writes;
  - at least 19 wait states (s_nop) separate the last MFMA from the first read
    of a result, and the zeroing of the accumulators from the first MFMA;
    every accumulator an MFMA uses was zeroed.
"""

import concurrent.futures
import os
import re
import subprocess

import pytest

from paper_1603_04467_amd import build as B

pytestmark = pytest.mark.timeout(600)

MFMA = "v_mfma_f32_16x16x32_bf16"


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    out = tmp_path_factory.mktemp("isa")

    def compile_asm(src):
        path = os.path.join(out, src + ".s")
        cmd = [B._hipcc(), *B.FLAGS, *B.SOURCE_FLAGS.get(src, []), "--cuda-device-only", "-S",
               os.path.join(B.CSRC, src), "-o", path]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return open(path).read()

    with concurrent.futures.ThreadPoolExecutor(2) as ex:
        texts = list(ex.map(compile_asm, ["gemm_bf16.hip", "gemm_bf16_tn.hip"]))
    found = {}
    for text in texts:
        for m in re.finditer(r"^(_Z\S*gemm_bf16_256\S*Li2ELi2E\S*):", text, re.M):
            name = m.group(1)
            end = text.index(".Lfunc_end", m.end())
            body = []
            for line in text[m.end():end].splitlines():
                s = line.split(";")[0].strip()
                if s and not s.startswith(".") and not s.endswith(":"):
                    body.append(s)
            found[name] = body
    assert len(found) >= 12, sorted(found)
    return found


def _agprs(operand):
    m = re.fullmatch(r"a\[(\d+):(\d+)\]", operand)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.fullmatch(r"a(\d+)", operand)
    return {int(m.group(1))} if m else set()


def _wait_states(lines):
    n = 0
    for s in lines:
        m = re.match(r"s_nop\s+(\d+)", s)
        if m:
            n += int(m.group(1)) + 1
    return n


def test_loop_has_no_accumulator_copies(kernels):
    for name, body in kernels.items():
        idx = [i for i, s in enumerate(body) if s.startswith(MFMA)]
        assert len(idx) >= 256, (name, len(idx))
        inner = body[idx[0]:idx[-1] + 1]
        bad = [s for s in inner if s.startswith("v_accvgpr") or "scratch_" in s]
        assert not bad, (name, bad[:5])


def test_mfma_accumulator_is_tied(kernels):
    for name, body in kernels.items():
        for s in body:
            if s.startswith(MFMA):
                ops = [o.strip() for o in s[len(MFMA):].split(",")]
                assert ops[0] == ops[3] and ops[0].startswith("a["), (name, s)


def test_wait_states_around_the_mfmas(kernels):
    for name, body in kernels.items():
        idx = [i for i, s in enumerate(body) if s.startswith(MFMA)]
        first, last = idx[0], idx[-1]
        # first read of an MFMA result after the loop
        reads = [i for i in range(last + 1, len(body)) if body[i].startswith("v_accvgpr_read")]
        assert reads, name
        assert _wait_states(body[last + 1:reads[0]]) >= 19, (name, body[last + 1:reads[0]])
        # last accumulator write (v_accvgpr_write or _mov) before the first MFMA
        writes = [i for i in range(first) if body[i].startswith(("v_accvgpr_write", "v_accvgpr_mov"))]
        assert writes, name
        assert _wait_states(body[writes[-1] + 1:first]) >= 19, name
        # every accumulator the MFMAs use was zeroed before the first MFMA
        zeroed = set()
        for i in writes:
            zeroed |= _agprs(body[i].split()[1].rstrip(","))
        used = set()
        for i in idx:
            used |= _agprs(body[i][len(MFMA):].split(",")[0].strip())
        assert used <= zeroed, (name, sorted(used - zeroed)[:8])
