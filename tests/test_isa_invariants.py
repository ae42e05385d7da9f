"""Properties of the generated gfx950 assembly that the attention kernel relies on.

The K/V copies are issued as inline assembly that loads M0 with the LDS destination and then
issues global_load_lds_dwordx4.  That is only safe if the compiler keeps no value of its own in
M0 across those statements, so every M0 write in the kernels must be one of these copies.

The copy ring is only as deep as the explicit vmcnt waits allow: a vector-memory wait that the
compiler inserts inside the stage loop (for a load it sees as still outstanding there) drains
every copy in flight.  The kernel's own waits touch vmcnt only; the compiler's waits inside the
compute appear as waits on vmcnt and lgkmcnt together, so none may exist.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2606_18954_amd", "csrc", "seg_attn.hip")
HIPCC = "/opt/rocm/bin/hipcc"


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / "seg_attn.s"
    from paper_2606_18954_amd import build_lib     # compile exactly as the library build does
    flags = [f for f in build_lib.CFLAGS if f != "-fPIC"]
    cmd = [HIPCC, *flags, "-x", "hip", "-S", "--cuda-device-only", SRC, "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    return out.read_text()


def _kernels(text):
    parts = re.split(r"^(_ZN2ga\w*k_seg_attn\w*):", text, flags=re.M)
    return {parts[i]: parts[i + 1].split("s_endpgm")[0] for i in range(1, len(parts) - 1, 2)}


def test_every_m0_write_feeds_a_direct_to_lds_copy(asm):
    ks = _kernels(asm)
    # {D 64, 128} x ({bf16, f32} x {decode, causal} + bf16 decode at three workgroups per CU)
    assert len(ks) == 10
    for name, body in ks.items():
        lines = [l.strip() for l in body.splitlines()
                 if l.strip() and not l.strip().startswith(";") and not l.strip().startswith(".")]
        copies = 0
        for i, l in enumerate(lines):
            if re.search(r"\bm0\b", l):
                assert re.match(r"s_mov_b32 m0, (s\d+|vcc_lo|vcc_hi)$", l), (name, l)
                assert lines[i + 1].startswith("global_load_lds_dwordx4"), (name, lines[i + 1])
                copies += 1
        assert copies >= 1, name
        assert sum(l.startswith("global_load_lds_dwordx4") for l in lines) == copies, name


def test_kernels_do_not_spill(asm):
    found = 0
    parts = re.split(r"^(_ZN2ga\w*k_seg_attn\w*):", asm, flags=re.M)
    for name, body in zip(parts[1::2], parts[2::2]):
        m = re.search(r"ScratchSize:\s+(\d+)", body)
        assert m, name
        assert int(m.group(1)) == 0, name
        found += 1
    assert found == 10


def test_wide_inline_stores_are_followed_by_wait_states(asm):
    """A global store of more than 64 bits reads its data VGPRs a cycle after issue; the
    compiler's hazard recognizer does not see stores written as inline assembly, so each of
    them must carry its own s_nop (a VALU write of the data registers right after such a store
    has corrupted stored partial rows)."""
    found = 0
    for name, body in _kernels(asm).items():
        lines = [l.strip() for l in body.splitlines() if l.strip() and not l.strip().startswith(";")]
        for i, l in enumerate(lines):
            if re.match(r"global_store_dwordx[34] .*\bsc1\b", l):
                assert lines[i + 1].startswith("s_nop"), (name, l, lines[i + 1])
                found += 1
    assert found > 0


def test_no_compiler_vector_memory_waits_in_the_compute(asm):
    for name, body in _kernels(asm).items():
        mixed = [w for w in re.findall(r"s_waitcnt vmcnt\((\d+)\)(?: expcnt\(\d+\))? lgkmcnt\((\d+)\)", body)
                 if int(w[0]) < 63 and int(w[1]) < 15]     # (63, 15) is "wait for nothing"
        assert not mixed, (name, mixed[:3])

