"""Properties of the gfx950 code the compiler emits for the bf16 conv kernels.

The operand pipeline of conv_bf16_k and wgrad_tr_bf16_k keeps several K-steps
of DMA loads (buffer loads that write LDS) in flight and orders them with its
own partial vmcnt waits and a barrier.  Two source patterns make the compiler
add a full `s_waitcnt vmcnt(0)` after that barrier, which empties the pipeline
at every step without changing any result: a second LDS object in the kernel
(the statistics' merge area), and the LDS transpose-read builtin.  The kernels
avoid both; these tests compile the source to assembly and check that the main
loops carry no such wait, and that the transpose reads issued as inline asm
(which the compiler does not count) leave their destination registers alone
until the kernel's own lgkmcnt wait.

The fp32 weight-gradient tile kernel stages its tiles in batches of eight
loads per thread; with a conditional load and the BN fold right behind each,
the compiler sent them out one round trip at a time.  The kernel issues a
batch's loads first; a test checks that every instance still does.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2203_06638_amd import build as B

pytestmark = pytest.mark.skipif(shutil.which("hipcc") is None, reason="needs hipcc")


def compile_asm(tmp_path_factory, name):
    out = str(tmp_path_factory.mktemp("asm") / (name + ".s"))
    src = os.path.join(B.CSRC, name + ".hip")
    r = subprocess.run(["hipcc"] + B.COMMON + ["--cuda-device-only", "-S", src, "-o", out],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read()


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    return compile_asm(tmp_path_factory, "conv_bf16")


def functions(s, prefix):
    """{mangled name: [instruction lines]} for the kernels whose names start with prefix."""
    out = {}
    for m in re.finditer(r"^(%s\S*):" % re.escape(prefix), s, re.M):
        end = s.index(".Lfunc_end", m.end())
        out[m.group(1)] = [l.strip() for l in s[m.end():end].split("\n")
                           if l.strip() and not l.strip().startswith(";")]
    return out


def waits_after_barriers(body, first_read):
    """For every barrier followed (before any other LDS read) by a read that
    first_read(i) accepts: the s_waitcnt lines between the two."""
    res = []
    for i, l in enumerate(body):
        if l != "s_barrier":
            continue
        for j in range(i + 1, min(i + 40, len(body))):
            if body[j].startswith("ds_read"):
                if first_read(j):
                    res.append([x for x in body[i + 1:j] if x.startswith("s_waitcnt")])
                break
    return res


def test_conv_main_loops_keep_partial_waits(asm):
    fns = {k: v for k, v in functions(asm, "_ZN3lpp11conv_bf16_k").items()
           if re.search(r"ELb1ELi\d+EE", k)}   # DMA instances (template argument DMA = true)
    assert len(fns) >= 12                        # six tile shapes, with and without statistics
    for name, body in fns.items():
        # the main loop's fragment reads: 16-row blocks of 64-byte rows, 1 KB apart
        loops = waits_after_barriers(body, lambda j: body[j].startswith("ds_read_b128") and "offset" not in body[j]
                                     and body[j + 1].startswith("ds_read_b128") and body[j + 1].endswith("offset:1024"))
        assert loops, name
        for w in loops:
            assert not any("vmcnt(0)" in x for x in w), (name, w)


def regs(text):
    out = set()
    for r in re.findall(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b", text):
        out |= {int(r[2])} if r[2] else set(range(int(r[0]), int(r[1]) + 1))
    return out


def test_wgrad_transpose_reads(asm):
    fns = functions(asm, "_ZN3lpp15wgrad_tr_bf16_k")
    assert len(fns) == 3                          # 256-, 128- and 64-channel tiles
    for name, body in fns.items():
        loops = waits_after_barriers(body, lambda j: body[j].startswith("ds_read_b64_tr_b16"))
        assert loops, name
        for w in loops:
            assert not any("vmcnt(0)" in x for x in w), (name, w)
        # every path from the reads to the MFMAs: the loop's blocks in layout
        # order from the barrier on, then from the loop's first block back to
        # it (a superset of each path); no instruction may touch a register an
        # issued read has yet to fill, until the lgkmcnt(0) wait
        labels = [(i, l) for i, l in enumerate(body) if l.startswith(".LBB")]
        loop = [i for i, l in labels if "Loop" in l]
        after = [i for i, _ in labels if i > max(loop)]
        end = after[0] if after else len(body)
        ib = [i for i, l in enumerate(body) if l == "s_barrier" and i > min(loop)][0]
        seq = body[ib:end] + body[min(loop):ib]
        inflight, waited = set(), False
        for l in seq:
            if l.startswith("ds_read_b64_tr_b16"):
                m = re.match(r"ds_read_b64_tr_b16 v\[(\d+):(\d+)\], v(\d+)", l)
                assert int(m.group(3)) not in inflight, (name, l)
                inflight |= set(range(int(m.group(1)), int(m.group(2)) + 1))
                continue
            if l.startswith("s_waitcnt") and "lgkmcnt(0)" in l and inflight:
                waited = True
                break
            if l.startswith(".") or l.startswith("s_") or " " not in l:
                continue
            assert not (regs(l.split(" ", 1)[1]) & inflight), (name, l)
        assert waited, name


def test_fp32_wgrad_staging_loads_in_flight(tmp_path_factory):
    fns = functions(compile_asm(tmp_path_factory, "conv_f32"), "_ZN3lpp19conv_wgrad_tile_f32")
    assert len(fns) >= 12
    for name, body in fns.items():
        # loads (G) and full vmcnt waits (V) in program order
        seq = "".join("G" if l.startswith(("global_load", "flat_load", "buffer_load")) else "V" for l in body
                      if l.startswith(("global_load", "flat_load", "buffer_load"))
                      or (l.startswith("s_waitcnt") and "vmcnt(0)" in l))
        # the first staging batch: eight loads before the first full wait,
        # and nowhere a run of single loads each followed by one
        assert seq.find("V") >= 8, (name, seq[:40])
        assert not re.search(r"(?:G{1,3}V){4,}", seq), (name, seq[:80])
