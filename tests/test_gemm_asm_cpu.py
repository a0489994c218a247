"""Static check of the tiled GEMM's built device code (CPU only).

The tiled GEMM loads its A fragments with inline-asm global loads and waits
for them with explicit ``s_waitcnt vmcnt(n)`` statements, because the
compiler would otherwise wait for the direct-to-LDS weight copies and the A
loads together. The compiler does not track those loads, so nothing but the
hand-written counts guarantees that an A register is not read (or
overwritten) while its load is in flight. This test compiles
``csrc/k_gemm.hip`` to gfx950 assembly with the library's own flags and
checks, for every ``gemm_tiled_bf16`` instantiation, that each A load is
covered by a wait before any instruction names one of its registers: on the
path into the main loop, around the loop (the next iteration) and out of it
into the last stage. Loads complete in issue order for ``vmcnt``, so a wait
``vmcnt(n)`` covers a load once at least n later vector-memory operations
have been issued.
"""

from __future__ import annotations

import os
import re
import subprocess
import tempfile

import pytest

from paper_2606_18600_amd import build

KERNEL = r"_ZN7stage_k12_GLOBAL__N_115gemm_tiled_bf16\w+"


def _device_asm() -> str:
    try:
        cc = build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k_gemm.s")
        cmd = [cc, *build.HIPCC_FLAGS, "-x", "hip", "--cuda-device-only", "-S",
               os.path.join(build.SRC, "k_gemm.hip"), "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        with open(out) as f:
            return f.read()


@pytest.fixture(scope="module")
def asm() -> str:
    return _device_asm()


def _regs(text: str) -> set[int]:
    out: set[int] = set()
    for m in re.finditer(r"\bv\[(\d+):(\d+)\]", text):
        out |= set(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\bv(\d+)\b", text):
        out.add(int(m.group(1)))
    return out


def _instrs(lines: list[str]) -> list[str]:
    out = []
    for line in lines:
        t = line.split(";")[0].strip()
        if t and not t.endswith(":") and not t.startswith("."):
            out.append(t)
    return out


def _is_vmem(t: str) -> bool:
    return t.startswith(("global_load", "buffer_load", "global_store", "buffer_store"))


def _is_a_load(t: str) -> bool:
    return t.startswith("global_load_dwordx4") and "lds" not in t


def _first_touch_before_wait(after: list[str], dest: set[int]) -> str | None:
    """The first instruction in ``after`` that names a register of ``dest``
    before a wait covers the load, or None if a wait comes first."""
    later = 0
    for t in after:
        m = re.match(r"s_waitcnt\b.*\bvmcnt\((\d+)\)", t)
        if m and later >= int(m.group(1)):
            return None
        if _is_vmem(t):
            later += 1
        if _regs(t) & dest:
            return t
    return "end of kernel without a covering wait"


def check_function(body: str) -> tuple[int, list[str]]:
    """(A loads checked, violations) for one kernel's assembly body."""
    lines = body.split("\n")
    heads = [i for i, l in enumerate(lines) if "Inner Loop Header" in l]
    assert heads, "no main loop found"
    h = heads[0]
    label = lines[h].split(":")[0].strip()
    ends = [i for i, l in enumerate(lines) if i > h and re.search(r"s_cbranch_\w+\s+" + re.escape(label) + r"\b", l)]
    assert ends, "no loop back-edge found"
    e = ends[0]
    pre, loop, post = _instrs(lines[:h]), _instrs(lines[h:e + 1]), _instrs(lines[e + 1:])
    checked, bad = 0, []
    for i, t in enumerate(pre):
        if _is_a_load(t):
            checked += 1
            r = _first_touch_before_wait(pre[i + 1:] + loop, _regs(t.split(",")[0]))
            if r:
                bad.append(f"prologue {t} -> {r}")
            r = _first_touch_before_wait(pre[i + 1:] + post, _regs(t.split(",")[0]))
            if r:
                bad.append(f"prologue (loop skipped) {t} -> {r}")
    for i, t in enumerate(loop):
        if _is_a_load(t):
            checked += 1
            dest = _regs(t.split(",")[0])
            r = _first_touch_before_wait(loop[i + 1:] + loop, dest)
            if r:
                bad.append(f"loop {t} -> {r}")
            r = _first_touch_before_wait(loop[i + 1:] + post, dest)
            if r:
                bad.append(f"loop exit {t} -> {r}")
    return checked, bad


def _functions(text: str) -> list[tuple[str, str]]:
    return re.findall(r"\n(" + KERNEL + r"):(.*?)s_endpgm", text, re.S)


def test_every_tiled_instantiation_waits_before_using_a_registers(asm):
    funcs = _functions(asm)
    # 256-, 192- and 128-row tilings with their epilogues, each with the A
    # loads one and two stages ahead
    assert len(funcs) >= 20, [n for n, _ in funcs]
    for name, body in funcs:
        checked, bad = check_function(body)
        assert checked > 0, f"{name}: no inline-asm A loads found"
        assert not bad, f"{name}:\n" + "\n".join(bad)


def test_main_loop_does_not_drain_all_loads(asm):
    """The loop's waits leave the next stage's A loads in flight (a
    ``vmcnt(0)`` inside the loop would serialize them)."""
    for name, body in _functions(asm):
        lines = body.split("\n")
        h = [i for i, l in enumerate(lines) if "Inner Loop Header" in l][0]
        label = lines[h].split(":")[0].strip()
        e = [i for i, l in enumerate(lines)
             if i > h and re.search(r"s_cbranch_\w+\s+" + re.escape(label) + r"\b", l)][0]
        waits = [int(m.group(1)) for l in lines[h:e + 1]
                 for m in [re.search(r"s_waitcnt\b.*\bvmcnt\((\d+)\)", l)] if m]
        assert waits and min(waits) > 0, f"{name}: loop waits {waits}"


def test_checker_flags_a_weakened_wait(asm):
    """The check itself: raising one wait count in the loop of a copy of the
    assembly text must be reported."""
    # a one-stage-ahead instantiation (template flag DEEP = false, "Lb0E" in
    # the mangled name), whose first A wait is the one that covers the load
    name, body = [f for f in _functions(asm) if "Lb0E" in f[0]][0]
    h = body.index("Inner Loop Header")
    m = re.search(r"s_waitcnt vmcnt\((\d+)\)", body[h:])
    assert m
    j = h + m.start()
    weakened = body[:j] + "s_waitcnt vmcnt(40)" + body[j + len(m.group(0)):]
    _, bad = check_function(weakened)
    assert bad
