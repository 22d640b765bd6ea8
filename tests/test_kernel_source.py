"""Rules that the hand-written device assembly keeps, checked on the source
text of the kernels (no GPU needed).

* An LDS DMA (buffer_load ... lds) reads its LDS destination from M0, and on
  the gfx9 family it needs one wait state after an SALU write of M0: every
  instruction of an inline-assembly block that writes M0 and is followed by
  another instruction must be followed by an s_nop.
* No packed fp32 arithmetic is written by hand (the build also turns the
  compiler's own use of it off).
"""
import pathlib
import re

CSRC = pathlib.Path(__file__).resolve().parents[1] / "paper_2608_17379_amd" / "csrc"
SOURCES = sorted(list(CSRC.glob("*.hip")) + list(CSRC.glob("*.hpp")))


def asm_blocks(text):
    """The instruction lists of the asm statements in `text`."""
    blocks = []
    for m in re.finditer(r"\basm\s+volatile\s*\(", text):
        # The template is the run of adjacent string literals that opens the
        # statement.
        pos = m.end()
        parts = []
        while True:
            lit = re.match(r'\s*"((?:[^"\\]|\\.)*)"', text[pos:])
            if not lit:
                break
            parts.append(lit.group(1))
            pos += lit.end()
        insts = [i.strip() for i in "".join(parts).replace("\\n", "\n").replace("\\t", "").split("\n")]
        blocks.append([i for i in insts if i])
    return blocks


def writes_m0(inst):
    op, _, rest = inst.partition(" ")
    return op.startswith("s_") and rest.split(",")[0].strip() == "m0"


def test_sources_found():
    assert any(p.suffix == ".hip" for p in SOURCES)
    assert any(asm_blocks(p.read_text()) for p in SOURCES)


def test_m0_write_is_followed_by_a_wait_state():
    checked = 0
    for p in SOURCES:
        for block in asm_blocks(p.read_text()):
            for i, inst in enumerate(block[:-1]):
                if writes_m0(inst):
                    nxt = block[i + 1]
                    # Restoring M0 at the end of a block is followed by no DMA
                    # of the block; a write followed by a DMA needs the nop.
                    if "lds" in " ".join(block[i + 1:]).split():
                        assert nxt.startswith("s_nop"), (p.name, block)
                        checked += 1
    assert checked > 0


def test_block_parser_on_a_known_block():
    text = 'asm volatile(\n "s_mov_b32 m0, %1\\n\\t"\n "s_nop 0\\n\\t"\n "buffer_load_dwordx4 %2, %3, 0 offen lds"\n : : );'
    assert asm_blocks(text) == [["s_mov_b32 m0, %1", "s_nop 0", "buffer_load_dwordx4 %2, %3, 0 offen lds"]]
    assert writes_m0("s_mov_b32 m0, %1") and writes_m0("s_add_u32 m0, m0, 0x400")
    assert not writes_m0("s_mov_b32 %0, m0")


def test_no_handwritten_packed_fp32():
    names = ["v_pk_" + op + "_f32" for op in ("add", "mul", "fma")]
    for p in SOURCES:
        text = p.read_text()
        for n in names:
            assert n not in text, (p.name, n)
