"""Register and scratch budget of every kernel (CPU only: hipcc cross-compiles).

Each translation unit under csrc/ is compiled for gfx950 with the library's own
flags and ``-Rpass-analysis=kernel-resource-usage``; the remarks give every
kernel's scratch (spill) bytes per lane, VGPRs and LDS per block.  The chunked
kernels must not spill (scratch traffic would sit on the HBM-bound paths) and
must fit the 160 KiB of LDS per compute unit.  The token-serial exact kernels,
which run only for streams whose inputs hold a NaN or Inf, keep a d_k-vector of
the state gradient per value column and are allowed to spill at d_k = 128.
"""
import concurrent.futures as cf
import os
import re
import subprocess
import tempfile

import pytest

from paper_2608_12700_amd import build as Bld

LDS_BYTES = 160 * 1024
EXEMPT = ("k_exact_fwd", "k_exact_bwd", "k_cw_exact_fwd", "k_cw_exact_bwd")


def _short(mangled):
    """gdn::k_name<ints...>[ bf16] from an Itanium-mangled kernel name (c++filt
    does not know the bf16 type code)."""
    m = re.match(r"_ZN3gdn(\d+)", mangled)
    if not m:
        return mangled
    n = int(m.group(1))
    start = m.end()
    name = mangled[start:start + n]
    rest = mangled[start + n:]
    ints = re.findall(r"Li(\d+)E", rest.split("EEv")[0] if "EEv" in rest else rest)
    return f"{name}<{','.join(ints)}>" + (" bf16" if "DF16b" in rest.split("EEv")[0] else "")


def _remarks(src, outdir):
    obj = os.path.join(outdir, os.path.basename(src) + ".o")
    cmd = [Bld.HIPCC] + Bld.COMMON + ["--cuda-device-only", "-c", src, "-o", obj,
                                      "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    kernels = []
    for block in re.split(r"Function Name: ", r.stderr)[1:]:
        name = block.split()[0]
        get = lambda key: int(re.search(key + r": (\d+)", block).group(1))
        kernels.append((name, get(r"ScratchSize \[bytes/lane\]"), get(r"VGPRs"),
                        get(r"LDS Size \[bytes/block\]")))
    return kernels


@pytest.fixture(scope="module")
def usage():
    srcs = [os.path.join(Bld.CSRC, f) for f in sorted(os.listdir(Bld.CSRC)) if f.endswith(".hip")]
    with tempfile.TemporaryDirectory() as d, cf.ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
        per = list(ex.map(lambda s: _remarks(s, d), srcs))
    rows = [k for ks in per for k in ks]
    return [(_short(r[0]), r[1], r[2], r[3]) for r in rows]


def test_every_translation_unit_has_kernels(usage):
    assert len(usage) > 50
    assert any(n.startswith("k_grad_bf<128,128,") for n, *_ in usage)


def test_chunked_kernels_do_not_spill(usage):
    bad = [(n, s) for n, s, _, _ in usage if s > 0 and not any(e in n for e in EXEMPT)]
    assert not bad, f"kernels with scratch (bytes/lane): {bad}"


def test_kernels_fit_lds(usage):
    bad = [(n, l) for n, _, _, l in usage if l > LDS_BYTES]
    assert not bad, bad


def test_gradient_kernel_keeps_four_waves_per_simd(usage):
    # the one-slice gradient kernel runs 16 waves per block (four per SIMD):
    # at most 128 VGPRs per lane
    seen = 0
    for n, _, v, _ in usage:
        m = re.match(r"k_grad_bf<(\d+),(\d+),", n)
        if m and int(m.group(2)) <= 128:
            seen += 1
            assert v <= 128, (n, v)
    assert seen >= 6
