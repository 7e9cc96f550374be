"""The wide kernel's jump tables in the built device code (CPU only: reads the
gfx950 code object of the library's own build with llvm-objdump).

The one-word-per-lane replay jumps with s_swappc_b64 to table + 68 i for an
action byte i, so every table must hold exactly 256 leaves of 68 bytes: eight
8-byte VOP3 updates in the order of i's bits (v_fma_f32 where bit e is set,
v_mul_f32 otherwise) and an s_setpc_b64 return; the offsets the prologue adds
to s_getpc_b64 must be the distances to the table and to the clearing routine,
and every step multiplies the byte by 68.  Any other layout would send a wave
into the wrong code, so the layout is checked here, before any device run."""
import os
import re
import subprocess

from paper_2207_07736_amd import build

LEAF_BYTES = 68


def _disassemble(tmp_path):
    obj = build.device_object(str(tmp_path / "dev.o"))
    objdump = os.path.join(os.path.dirname(os.path.realpath(build.HIPCC)), "..", "llvm", "bin", "llvm-objdump")
    text = subprocess.run([objdump, "-d", obj], capture_output=True, text=True, check=True).stdout
    labels, ins = {}, []
    for ln in text.splitlines():
        m = re.match(r"^([0-9a-f]+) <(\S+)>:", ln)
        if m:
            labels[m.group(2)] = int(m.group(1), 16)
            continue
        m = re.match(r"^\s+(\S.*?)\s*// ([0-9A-F]+): ([0-9A-F ]+)$", ln)
        if m:
            ins.append((int(m.group(2), 16), m.group(1), 4 * len(m.group(3).split())))
    return labels, ins


def test_jump_tables_have_the_layout_the_replay_jumps_into(tmp_path):
    labels, ins = _disassemble(tmp_path)
    at = {a: i for i, (a, _, _) in enumerate(ins)}
    tables = {k[len("Ljtab"):]: v for k, v in labels.items() if k.startswith("Ljtab")}
    assert tables, "no jump table in the built library"
    for uid, base in tables.items():
        for lab, reg, target in (("Ljbase0_", "s36", base), ("Ljbase1_", "s38", labels["Ljclr" + uid])):
            start = labels[lab + uid]
            m = re.match(rf"s_add_u32 {reg}, {reg}, (0x[0-9a-f]+|\d+)$", ins[at[start]][1])
            assert m and start + int(m.group(1), 0) == target, (uid, lab, ins[at[start]])
        k = at[base]
        for leaf in range(256):
            assert ins[k][0] == base + LEAF_BYTES * leaf, (uid, leaf)
            for e in range(8):
                _, text, size = ins[k]
                want = "v_fma_f32 " if (leaf >> e) & 1 else "v_mul_f32_e64 "
                assert text.startswith(want) and size == 8, (uid, leaf, e, text, size)
                k += 1
            assert ins[k][1] == "s_setpc_b64 s[44:45]" and ins[k][2] == 4, (uid, leaf, ins[k])
            k += 1
    # within each replay block (from its prologue to its end label): every index
    # multiply is by 68, and there are as many calls as its steps and stubs make
    for uid in tables:
        lo, hi = labels["Ljbase0_" + uid], labels["Ljend" + uid]
        body = [t for a, t, _ in ins if lo <= a < hi]
        muls = {t for t in body if t.startswith("s_mul_i32 ")}
        assert muls == {f"s_mul_i32 s40, s40, {LEAF_BYTES:#x}"}, (uid, muls)
        calls = [t for t in body if t.startswith("s_swappc_b64 s[44:45], ")]
        assert len(calls) == 4 * 32, (uid, len(calls))
