"""Register budget of every built SpMM kernel (host only: compiles to gfx950 assembly).

Each kernel instantiation is built for a number of resident wavefronts per
SIMD (its launch bound), and the host's configuration choice counts on that
residency. This test compiles every kernel translation unit to
assembly and checks, for every instantiation, that its VGPRs fit that many
wavefronts (512 per SIMD lane, in granules of 8; the kernels use no AGPRs,
so the VGPR count is the whole register budget) and that it needs no
scratch. The expected figures restate the kernel header's waves_per_simd
table. Kernels above 16 activation columns on rows in stored order carry no
launch bound, so their budget is the four wavefronts the table assumes. The
units are compiled with the library's flags, kernel-argument preloading
included, and every SpMM kernel is checked to take its leading arguments
preloaded.
"""
import concurrent.futures as cf
import os
import re
import subprocess
import tempfile

import pytest

from paper_2608_09291_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_09291_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
UNITS = ("us_dense", "us_spmm", "us_spmm_narrow", "us_spmm_perm", "us_spmm_w2", "us_spmm_wide", "us_spmm_wide8",
         "us_spmm_burst_plain", "us_spmm_burst_narrow", "us_spmm_burst_perm", "us_spmm_burst_w2")


def unit_flags(unit):
    # The library's own flags for the unit (build.py), device code only, as assembly.
    return [f for f in build.hip_flags(unit + ".hip") if f != "-fPIC"] + ["-I", CSRC, "--cuda-device-only", "-S"]



def waves_per_simd(wpg, nmax, ch, multi, ring, perm):
    if nmax > 16:
        return 4 if multi else (7 if wpg >= 4 else 6)
    if not multi:
        return 8 if wpg >= 4 else 6
    if ring:
        return 5 if nmax <= 4 else 4
    if nmax <= 4:
        return 6 if perm and ch > 11 else 7
    return 7 if ch <= 4 else 5 if ch <= 8 or (perm and ch <= 11) else 4


@pytest.fixture(scope="module")
def kernels():
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    tmp = tempfile.mkdtemp(prefix="us_res_")

    def compile_unit(u):
        out = os.path.join(tmp, u + ".s")
        r = subprocess.run([HIPCC, *unit_flags(u), os.path.join(CSRC, u + ".hip"), "-o", out], capture_output=True,
                           text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return open(out).read()

    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        texts = list(ex.map(compile_unit, UNITS))
    m0_lines = []
    for text in texts:
        lines = [ln.strip() for ln in text.splitlines()]
        for i, ln in enumerate(lines):
            if "m0" in ln and not ln.startswith(";") and not ln.startswith("."):
                m0_lines.append((ln, lines[i + 1] if i + 1 < len(lines) else "", lines[i + 2] if i + 2 < len(lines) else ""))
    found = []
    burst = []
    for text in texts:
        for m in re.finditer(r"\.amdhsa_kernel (\S+)(.*?)\.end_amdhsa_kernel", text, re.S):
            b = re.search(r"us_spmm_burst_kernelILi(\d+)ELi(\d+)ELi(\d+)ELb(\d)ELi(\d)ELi(\d+)E", m.group(1))
            if b:
                wpg, nmax, ch, perm, bits, win = (int(v) for v in b.groups())
                burst.append(dict(wpg=wpg, nmax=nmax, ch=ch, perm=bool(perm), bits=bits, win=win,
                                  vgpr=int(re.search(r"\.amdhsa_next_free_vgpr (\d+)", m.group(2)).group(1)),
                                  scratch=int(re.search(r"\.amdhsa_private_segment_fixed_size (\d+)",
                                                        m.group(2)).group(1))))
                continue
            g = re.search(r"us_spmm_kernelILi(\d+)ELi(\d+)ELi(\d+)ELb(\d)ELb(\d)ELb(\d)ELi(\d)E", m.group(1))
            if not g:
                continue
            wpg, nmax, ch, multi, ring, perm, bits = (int(v) for v in g.groups())
            vgpr = int(re.search(r"\.amdhsa_next_free_vgpr (\d+)", m.group(2)).group(1))
            scratch = int(re.search(r"\.amdhsa_private_segment_fixed_size (\d+)", m.group(2)).group(1))
            preload = int(re.search(r"\.amdhsa_user_sgpr_kernarg_preload_length (\d+)", m.group(2)).group(1))
            found.append(dict(wpg=wpg, nmax=nmax, ch=ch, multi=bool(multi), ring=bool(ring), perm=bool(perm),
                              bits=bits, vgpr=vgpr, scratch=scratch, preload=preload))
    return found, m0_lines, burst


@pytest.fixture(scope="module")
def kernel_list(kernels):
    return kernels[0]


def burst_waves_per_simd(wpg, nmax):
    return (6 if wpg >= 4 else 5) if nmax > 4 else (7 if wpg >= 4 else 6)


def test_m0_is_only_the_direct_payload_loads(kernels):
    # The direct-to-LDS loads (the SpMM kernels' and the copy probe's) set
    # M0 in assembly and list it as clobbered; that is only sound while the
    # compiler itself keeps nothing in M0. The
    # LDS base must come from a scalar register: a vector register there
    # (a value the compiler did not prove wave-uniform) would not be a valid
    # M0 source, so every write is checked to name an SGPR.
    m0 = kernels[1]
    assert m0, "no direct payload loads found"
    for ln, nxt, nxt2 in m0:
        assert re.fullmatch(r"s_mov_b32 m0, s\d+", ln), ln
        assert nxt == "s_nop 0" and re.match(r"buffer_load_dword(x4)? v\d+, s\[\d+:\d+\], (s\d+|0) offen", nxt2) \
            and nxt2.endswith(" lds"), (ln, nxt, nxt2)


def test_single_pass_kernels_fit_their_residency(kernels):
    burst = kernels[2]
    assert len(burst) >= 4 * 5 * 6, len(burst)       # 4 families x 5 WPG x 6 slice lengths
    over = [k for k in burst if k["vgpr"] > (512 // burst_waves_per_simd(k["wpg"], k["nmax"])) // 8 * 8]
    assert not over, over[:5]
    assert not [k for k in burst if k["scratch"]]


def test_every_configuration_is_built(kernel_list):
    # 5 WPG x (4 linear + 2 ring chunk lengths) x single/multi for the N <= 4
    # and N <= 16 tiers, 5 x 2 x 2 for N <= 32, per translation unit.
    assert len(kernel_list) >= 4 * 5 * 2 * 2
    assert {k["nmax"] for k in kernel_list} == {4, 16, 32}


def test_registers_fit_the_residency_the_host_assumes(kernel_list):
    over = []
    for k in kernel_list:
        w = waves_per_simd(k["wpg"], k["nmax"], k["ch"], k["multi"], k["ring"], k["perm"])
        budget = (512 // w) // 8 * 8
        if k["vgpr"] > budget:
            over.append((k, budget))
    assert not over, over[:5]


def test_no_kernel_needs_scratch(kernel_list):
    spills = [k for k in kernel_list if k["scratch"]]
    assert not spills, spills[:5]


def test_leading_arguments_are_preloaded(kernel_list):
    # Built as the library is, every SpMM kernel takes its first 14 argument
    # dwords (the inputs' addresses and sizes its first loads need, through
    # the scale pointer) preloaded in scalar registers.
    short = [k for k in kernel_list if k["preload"] < 14]
    assert not short, short[:5]
