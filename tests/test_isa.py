"""The gfx950 code of the kernels, compiled here with the library's own flags
(no GPU needed): properties the parity and speed of the path rest on.

* The apply and pull kernels contain no packed-fp32 and no fused
  multiply-add instructions: every product and sum is rounded on its own
  (the binary32 reading of Eq. "gd"), and packed fp32 stays disabled.
* No kernel uses private (scratch) memory: registers hold every value.
* Launches of at most 8 gradients and 8 replicas take kernels over a compact
  argument block; the others a full one (64 pointers per array). With the
  runtime's implicit arguments the compact segments stay under 448 bytes and
  the full ones at 536 or more: the host enqueues a launch faster the smaller its
  argument segment.
* The fused applies of the VGG-16 shape (fp32 gradients, one group of 32)
  and of the Mixed shape (bf16 gradients, groups of 24) issue each group's
  gradient loads back to back, non-temporal, before waiting for the first:
  the loads a lane keeps in flight set the apply's bandwidth. The first group
  goes out together with the w/v loads. The remainder after the full groups
  is straight-line groups too (16, 8, then 7 loads together for a remainder
  of 7), not one load and one wait per gradient.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_1611_06213_amd import build as B

KERNELS = os.path.join(B.CSRC, "ps_kernels.hip")
VGG16_APPLY = "_ZN5gadei12_GLOBAL__N_19apply_vecILb1ELi0ELin1ELi4ELi32ENS_9ApplyArgsEEEvT4_"
MIXED_APPLY = "_ZN5gadei12_GLOBAL__N_19apply_vecILb1ELi1ELin1ELi8ELi24ENS_9ApplyArgsEEEvT4_"


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    if not os.path.exists(B.HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("hipcc not available")
    out = str(tmp_path_factory.mktemp("isa") / "ps_kernels.s")
    flags = [f for f in B.FLAGS if f not in ("-fPIC", "-shared")]
    r = subprocess.run([B.HIPCC, *flags, "--cuda-device-only", "-S", KERNELS, "-o", out],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(out) as f:
        return f.read()


def kernels(asm):
    """name -> (instruction lines of the kernel body, metadata block)."""
    names = re.findall(r"^\s*\.amdhsa_kernel (\S+)$", asm, re.M)
    out = {}
    for name in names:
        start = asm.index("\n" + name + ":")
        end = asm.index(".Lfunc_end", start)
        body = [l.split(";")[0].strip() for l in asm[start:end].splitlines()[1:]]
        meta_start = asm.index(".amdhsa_kernel " + name)
        meta = asm[meta_start:asm.index(".end_amdhsa_kernel", meta_start)]
        out[name] = ([l for l in body if l and not l.startswith(".")], meta)
    return out


def test_no_fused_or_packed_fp32_in_apply_and_pull(asm):
    ks = kernels(asm)
    checked = 0
    for name, (body, _) in ks.items():
        if not re.search(r"apply_vec|apply_scalar|pull_", name):
            continue
        checked += 1
        bad = [l for l in body if re.match(r"v_(pk_\w+|fma\w*|mac\w*|fmac\w*)\b", l)]
        assert not bad, (name, bad[:3])
    assert checked >= 60


def test_no_kernel_uses_scratch(asm):
    ks = kernels(asm)
    assert len(ks) >= 90
    for name, (_, meta) in ks.items():
        m = re.search(r"\.amdhsa_private_segment_fixed_size (\d+)", meta)
        assert m and int(m.group(1)) == 0, name


def test_compact_argument_blocks(asm):
    ks = kernels(asm)
    compact = full = 0
    for name, (_, meta) in ks.items():
        if not re.search(r"apply_vec|apply_scalar|pull_", name):
            continue
        size = int(re.search(r"\.amdhsa_kernarg_size (\d+)", meta).group(1))
        if "ArgsC" in name:
            compact += 1
            assert size <= 448, (name, size)
        else:
            full += 1
            assert size >= 536, (name, size)
    assert compact >= 60 and full >= 60, (compact, full)


@pytest.mark.parametrize("name,group,wv", [(VGG16_APPLY, 32, 2), (MIXED_APPLY, 24, 4)],
                         ids=["vgg16-fp32", "mixed-bf16"])
def test_group_loads_issued_together(asm, name, group, wv):
    body, _ = kernels(asm)[name]
    runs, run = [], 0
    for l in body:
        if l.startswith("global_load_dwordx4"):
            assert re.search(r"\bnt\b", l), l
            run += 1
        elif l.startswith("s_waitcnt") and "vmcnt" in l:
            runs.append(run)
            run = 0
    runs.append(run)
    runs = [r for r in runs if r]
    # the first group with the w/v loads (w and v: 1 load each of 4 fp32, 2
    # each of 8), the loop's groups, then the groups of 16 and 8
    assert runs[0] == wv + group, runs
    assert group in runs[1:] and 16 in runs and 8 in runs, runs
    # remainder groups of 1..7 loads, each issued whole
    for size in range(2, 8):
        assert size in runs, (size, runs)
