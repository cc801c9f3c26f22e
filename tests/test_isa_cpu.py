"""Properties of the gfx950 assembly the kernels compile to, checked on the
CPU (hipcc cross-compiles; nothing runs on a GPU).

Buffer instructions range-check their vector and immediate offsets against
the descriptor's extent but not the scalar offset operand. Every kernel
builds its descriptors over one head's (or one buffer's) extent and must
keep the scalar offset at 0, so that a partial last block, and a corrupt
block index in a caller's list, cannot reach memory outside that extent."""
import os
import re

import pytest

from paper_2607_03612_amd import build

SOURCES = ["attn.hip", "pool.hip", "select.hip", "cosine.hip", "nmse.hip"]
# buffer_<op> [vdata,] vaddr|off, s[a:b], soffset [offen] [offset:N] [lds] ...
BUFFER = re.compile(r"^\s*(buffer_\w+)\s+(.*)$")


def _buffer_soffsets(asm):
    found = []
    for line in asm.splitlines():
        m = BUFFER.match(line)
        if not m or m.group(1).startswith(("buffer_wbl2", "buffer_inv", "buffer_wbinvl1")):
            continue
        ops = [x.strip() for x in m.group(2).split(",")]
        rsrc = next(i for i, x in enumerate(ops) if re.match(r"s\[\d+:\d+\]", x))
        found.append((m.group(1), ops[rsrc + 1].split()[0], line.strip()))
    return found


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    d = tmp_path_factory.mktemp("asm")
    return {s: open(build.device_asm(s, str(d / (s + ".s")))).read() for s in SOURCES}


def test_no_buffer_instruction_uses_a_scalar_offset(asm):
    total = 0
    for src, text in asm.items():
        for op, soff, line in _buffer_soffsets(text):
            total += 1
            assert soff == "0", f"{src}: {line} (scalar offset {soff} escapes the range check)"
    # the attention kernels stage every K/V tile with buffer-to-LDS loads
    assert total > 100


def test_tile_loads_are_buffer_to_lds_with_descriptor_offsets(asm):
    lds = [x for x in _buffer_soffsets(asm["attn.hip"]) if x[2].endswith(" lds") or " lds" in x[2]]
    assert len(lds) >= 64
    offsets = {int(m.group(1)) for _, _, line in lds for m in [re.search(r"offset:(\d+)", line)] if m}
    # the four 1 KB row groups of a half tile sit in the immediate offset
    assert offsets <= {1024, 2048, 3072}


def test_planted_scalar_offset_is_reported():
    text = "\tbuffer_load_dwordx4 v231, s[24:27], s8 offen lds\n" \
           "\tbuffer_store_dwordx4 v[6:9], v18, s[0:3], 0 offen\n"
    got = [(op, soff) for op, soff, _ in _buffer_soffsets(text)]
    assert got == [("buffer_load_dwordx4", "s8"), ("buffer_store_dwordx4", "0")]


def _kernel_body(text, substr):
    names = [m.group(1) for m in re.finditer(r"^(\S+):\s*;\s*@\S+", text, re.M) if substr in m.group(1)]
    assert len(names) == 1, (substr, names)
    start = text.index(names[0] + ":")
    return text[start:text.index(".Lfunc_end", start)]


def test_sparse_attention_kernels_use_no_scratch(asm):
    # the list and strided walks fit in the registers of two waves per SIMD:
    # no spill stores or reloads anywhere in them
    for mode in ("ILi0E", "ILi2E"):
        body = _kernel_body(asm["attn.hip"], "attn_bf16_kernel" + mode)
        assert "scratch_" not in body, mode


def test_dense_kernel_loop_has_one_barrier_per_step_and_no_scratch(asm):
    # the shared-tile dense walk: its loop (the block that branches back to
    # the loop header) holds four half-tile steps, each one barrier and two
    # buffer-to-LDS loads per wave, and no scratch access, whose wait would
    # also wait for the tile loads in flight
    body = _kernel_body(asm["attn.hip"], "attn_bf16_dense_kernel")
    header = re.search(r"^(\.LBB\d+_\d+):\s*;\s*=>This Inner Loop Header", body, re.M).group(1)
    start = body.index(header + ":")
    end = body.index(header, start + len(header) + 1)  # the branch back to the header
    loop = body[start:end]
    assert loop.count("s_barrier") == 4
    assert len(re.findall(r"buffer_load_dwordx4 .* lds", loop)) == 8
    assert "scratch_" not in loop
    assert len(re.findall(r"v_mfma_f32_32x32x16_bf16", loop)) == 64
