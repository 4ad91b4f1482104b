"""Host address check of the grouped bf16 GEMM kernel (csrc/gemm2.hpp).

The kernel's source is compiled for the CPU under AddressSanitizer, with a stand-in for
the HIP runtime header (tests/hostcheck/hip/hip_runtime.h), and every thread of every
block of each launch is run one after another (tests/hostcheck/gemm_bounds.cpp).  Global
buffers and the LDS are allocated at their exact sizes, so a tile, a stage or an epilogue
that reads or writes past them stops the run with the faulting access and its stack.
What the kernel computes is checked on the GPU by the parity tests; this test checks only
where it reads and writes, for every tile-shape family the layer launches, on ragged
routings (an empty expert, a heavy one, row counts around the tile boundaries, partial
column tiles).

The few statements that only make sense on the GPU are replaced in a copy of the source:
the direct-to-LDS load becomes a 16-byte copy to the lane's LDS slot, the barrier and the
LDS wait become nothing, and address-space casts are dropped.  Each replacement must match
the source exactly once or more, so a change to those statements fails this test instead
of silently checking something else.  The tile shapes are taken from the launch helpers
(csrc/grouped.hpp), so the check follows them.  CPU only."""
import os
import re
import subprocess

import pytest

from paper_2002_04013_amd import build as B

HERE = os.path.dirname(os.path.abspath(__file__))
CLANG = "/opt/rocm/llvm/bin/clang++"
CONFIGS = ("G2Fat", "G2Skinny", "G2DW", "G2DWShort")

# (pattern, replacement, regex): each must match the source at least once
SUBST = {
    "gemm2.hpp": [
        (r"template <int LOFF>\n__device__ __forceinline__ void g2l_16_at\(.*?\n}\n",
         "void hostcheck_g2l(const void* g, char* l);\n"
         "template <int LOFF>\n__device__ __forceinline__ void g2l_16_at(const bf16* base, uint32_t off_bytes, "
         "char* lds_base) {\n  hostcheck_g2l(reinterpret_cast<const char*>(base) + off_bytes, "
         "lds_base + LOFF + 16 * (threadIdx.x & 63));\n}\n", True),
        (r"__device__ __forceinline__ void block_sync_lds\(\) \{\n.*?\n}\n",
         "__device__ __forceinline__ void block_sync_lds() {}\n", True),
        ('asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");', "", False),
        ("extern __shared__ __align__(1024) char smem[];", "char* smem = hostcheck_smem;", False),
        ("__attribute__((address_space(3)))", "", False),
        ("__attribute__((address_space(4)))", "", False),
        ("namespace dmoe {", "extern thread_local char* hostcheck_smem;\nnamespace dmoe {", False),
    ],
}


def _patch(name, text):
    for pat, rep, is_re in SUBST.get(name, []):
        if is_re:
            text, n = re.subn(pat, lambda _m: rep, text, count=1, flags=re.S)
        else:
            n = text.count(pat)
            text = text.replace(pat, rep)
        assert n >= 1, f"{name}: the statement replaced for the host build is gone: {pat[:60]!r}"
    return text


def _configs():
    """The bf16 tile-shape structs of the launch helpers, as C++ text."""
    with open(os.path.join(B.CSRC, "grouped.hpp")) as f:
        src = f.read()
    out = []
    for name in CONFIGS:
        m = re.search(r"struct %s\s*\{.*?\};" % name, src, flags=re.S)
        assert m, f"tile shape {name} not found in grouped.hpp"
        out.append(m.group(0))
    return "#pragma once\nnamespace dmoe {\n" + "\n".join(out) + "\n}  // namespace dmoe\n"


@pytest.mark.skipif(not os.path.exists(CLANG), reason="clang++ not installed")
def test_grouped_gemm_addresses_stay_in_bounds(tmp_path):
    src = tmp_path / "src"
    src.mkdir()
    for name in ("common.hpp", "gemm.hpp", "gemm2.hpp"):
        with open(os.path.join(B.CSRC, name)) as f:
            text = f.read()
        (src / name).write_text(_patch(name, text))
    (src / "g2cfg.hpp").write_text(_configs())
    exe = tmp_path / "gemm_bounds"
    cmd = [CLANG, "-std=c++17", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer",
           "-I", os.path.join(HERE, "hostcheck"), "-I", str(src), "-I", os.path.join(B.ROOT, "include"),
           "-Wno-everything", os.path.join(HERE, "hostcheck", "gemm_bounds.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.stdout[-1000:] + r.stderr[-4000:])
    assert "launches checked" in r.stdout
    # the check itself: a weight-gradient buffer 8 elements short is reported, in the
    # staged store of the weight-gradient tile
    r = subprocess.run([str(exe), "short"], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr, r.stderr[-2000:]
    assert "grouped_gemm2<1, true, true" in r.stderr, r.stderr[-2000:]
