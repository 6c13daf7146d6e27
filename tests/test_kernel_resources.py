"""Register budgets of the kernels the planner picks, read from the metadata
of the built library's gfx950 code objects (no GPU needed).

A kernel that spills to scratch, or whose registers cost it a resident
wavefront, can lose half its speed with no change in its results, so parity
tests cannot see it (the 64 x 256 fp32 tile beside an element-wise gather
once spilled 176 bytes per lane and ran twice as long).  For each workload
and a few Appendix A contractions whose kernels sit at their register caps,
the kernel of the model's plan must not spill (the stream-K tail kernel,
whose piece loop carries more state, within a small budget), the one-box
fp64 tile's macro-kernels must stay within 128 VGPRs (four wavefronts per
SIMD), and the direct-load kernels, persistent or not, within 256 (two)."""
import json
import os
import re
import shutil
import struct
import subprocess
import tempfile

import pytest

import paper_1607_00145_amd as g
import workloads as wl
from workloads import appendix_a as ap

LLVM = "/opt/rocm/llvm/bin"
MODES = {"row-vector": 0, "k-vector": 1, "scalar": 2, "row-vector-strided": 3,
         "k-vector-strided": 4}
BUNDLE = b"__CLANG_OFFLOAD_BUNDLE__"
NAME = re.compile(r"_ZN4gett17gett_macro_kernelI([fd])((?:Li\d+E)+)EEv")
DIRECT = re.compile(r"_ZN4gett18gett_direct_kernelI([fd])((?:Li\d+E)+)Lb([01])EEEv")
DSTREAM = re.compile(r"_ZN4gett25gett_direct_stream_kernelI([fd])((?:Li\d+E)+)Lb([01])EEEv")
TAIL_SCRATCH_BUDGET = 64   # bytes per lane


def code_objects(lib):
    """The gfx950 code objects of every offload bundle in the library's
    .hip_fatbin section (one bundle per translation unit)."""
    tmp = tempfile.mkdtemp()
    try:
        fat = os.path.join(tmp, "fat.bin")
        subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fat}", lib,
                        os.path.join(tmp, "stripped.so")], check=True, capture_output=True)
        data = open(fat, "rb").read()
    finally:
        shutil.rmtree(tmp)
    out, pos = [], 0
    while (i := data.find(BUNDLE, pos)) >= 0:
        (n,) = struct.unpack_from("<Q", data, i + len(BUNDLE))
        p = i + len(BUNDLE) + 8
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", data, p)
            triple = data[p + 24:p + 24 + tlen].decode()
            p += 24 + tlen
            if "gfx950" in triple and size:
                out.append(data[i + off:i + off + size])
        pos = i + len(BUNDLE)
    return out


@pytest.fixture(scope="module")
def kernels():
    """(type, template integer arguments) -> (scratch bytes per lane, VGPRs)
    for every gett_macro_kernel instantiation in the library; ("direct" or
    "dstream", type, arguments + (WHOLE,)) for the direct-load kernels."""
    if not os.path.exists(f"{LLVM}/llvm-readelf"):
        pytest.skip("llvm-readelf not found")
    res = {}
    tmp = tempfile.mkdtemp()
    try:
        for k, co in enumerate(code_objects(g.LIB_PATH)):
            path = os.path.join(tmp, f"{k}.co")
            open(path, "wb").write(co)
            notes = subprocess.run([f"{LLVM}/llvm-readelf", "--notes", path], check=True,
                                   capture_output=True, text=True).stdout
            for blk in notes.split("\n  - ")[1:]:
                m, kind = NAME.search(blk), "macro"
                if not m:
                    m, kind = DIRECT.search(blk), "direct"
                if not m:
                    m, kind = DSTREAM.search(blk), "dstream"
                if not m:
                    continue
                field = lambda key: int(re.search(rf"\.{key}:\s+(\d+)", blk).group(1))
                args = tuple(int(x) for x in re.findall(r"Li(\d+)E", m.group(2)))
                key = ((m.group(1), args) if kind == "macro" else
                       (kind, m.group(1), args + (int(m.group(3)),)))
                res[key] = (field("private_segment_fixed_size"), field("vgpr_count"))
    finally:
        shutil.rmtree(tmp)
    assert len(res) > 100, "too few kernels found in the library's code objects"
    return res


def plan_kernel(w, kernels):
    """The resources of the kernel the model's plan for workload w launches.
    Template integer arguments of the macro-kernel: MT NT KT WM WN RX RY WPE
    PF NBUF XMODE YMODE ONEBOX CORDER TAIL SLICED; of the direct-load kernel:
    MT NT KT WM WN RX RY XMODE YMODE and WHOLE (both variants: which one runs
    is decided per call); all given by the plan's description."""
    code = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
    st, h = g.gett_plan(code, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None,
                        w.modes_B, w.shape("B"), None, 0)
    assert st == 0
    try:
        d = json.loads(g.gett_plan_describe(h))
    finally:
        g.gett_destroy(h)
    t = d["tile"]
    T = "f" if w.dtype == "f32" else "d"
    if d["kernel"] in ("direct", "direct-stream"):
        kind = "direct" if d["kernel"] == "direct" else "dstream"
        args = (t["mt"], t["nt"], t["kt"], t["waves"][0], t["waves"][1], t["reads"][0],
                t["reads"][1], MODES[d["gather_x"]], MODES[d["gather_y"]])
        both = [kernels.get((kind, T, args + (whole,))) for whole in (0, 1)]
        assert all(both), (w.name, args)
        return d, args, (max(v[0] for v in both), max(v[1] for v in both))
    want = {0: t["mt"], 1: t["nt"], 2: t["kt"], 3: t["waves"][0], 4: t["waves"][1],
            5: t["reads"][0], 6: t["reads"][1], 7: t["waves_per_simd"], 8: t["prefetch"],
            9: t["lds_buffers"], 10: MODES[d["gather_x"]], 11: MODES[d["gather_y"]],
            12: int(t["one_box"]), 13: int(t["c_order_epilogue"]),
            14: int(d["kernel"] == "tail"), 15: int(d["kslices"] > 1)}
    hits = [(a, v) for key, v in kernels.items() if len(key) == 2
            for (tt, a) in [key] if tt == T and all(a[i] == x for i, x in want.items())]
    assert len(hits) == 1, (w.name, d["tile"], d["kernel"], hits)
    return d, hits[0][0], hits[0][1]


def appendix(prefix, dtype):
    return next(w for w in ap.appendix_workloads(dtype) if w.name.startswith(prefix))


CASES = [(w.name, w) for w in wl.WORKLOADS] + [
    (p + dt, appendix(p, dt)) for p, dt in
    (("appA31_", "f32"), ("appA13_", "f32"), ("appA12_", "f64"), ("appA23_", "f32"),
     ("appA23_", "f64"), ("appA40_", "f64"))]


@pytest.mark.parametrize("name,w", CASES, ids=[c[0] for c in CASES])
def test_model_kernel_does_not_spill(kernels, name, w):
    d, args, (scratch, vgprs) = plan_kernel(w, kernels)
    budget = TAIL_SCRATCH_BUDGET if d["kernel"] == "tail" else 0
    assert scratch <= budget, f"{name}: kernel {args} spills {scratch} bytes per lane"


def test_direct_kernels_keep_two_wavefronts_per_simd(kernels):
    """Every direct-load kernel, persistent or not: no spills, at most 256
    VGPRs (two wavefronts per SIMD: the 256 x 128 and 128 x 256 tiles' eight,
    or two workgroups of four)."""
    direct = {k: v for k, v in kernels.items() if k[0] == "direct"}
    assert len(direct) >= 24, "the direct-load kernels of the fp32 tiles, both variants"
    dstream = {k: v for k, v in kernels.items() if k[0] == "dstream"}
    assert len(dstream) >= 8, "the persistent kernels of the fp64 one-box tile, both variants"
    direct.update(dstream)
    for key, (scratch, vgprs) in direct.items():
        assert scratch == 0 and vgprs <= 256, (key, scratch, vgprs)


def test_compute_bound_fp32_workload_runs_direct(kernels):
    d, args, (scratch, vgprs) = plan_kernel(wl.BY_NAME["gemm4_fp32"], kernels)
    assert d["kernel"] == "direct" and args[0] * args[1] == 256 * 128


def test_one_box_tile_keeps_four_wavefronts_per_simd(kernels):
    """ccsdt6's tile runs the persistent direct-load kernel (two workgroups
    per CU: at most 256 VGPRs); its one-box macro-kernel, which runs the calls
    that kernel does not take, keeps four workgroups per CU (<= 128 VGPRs)."""
    d, args, (scratch, vgprs) = plan_kernel(wl.BY_NAME["ccsdt6_fp64"], kernels)
    assert d["kernel"] == "direct-stream" and args[:3] == (64, 128, 24)
    assert vgprs <= 256 and scratch == 0, (args, vgprs, scratch)
    modes = (MODES[d["gather_x"]], MODES[d["gather_y"]])
    onebox = {k: v for k, v in kernels.items()
              if len(k) == 2 and k[0] == "d" and k[1][:3] == (64, 128, 24) and k[1][12] == 1
              and k[1][10:12] == modes and k[1][14:] == (0, 0)}
    assert onebox, "the one-box macro-kernels of the 64 x 128 x 24 fp64 tile"
    for key, (scratch, vgprs) in onebox.items():
        assert vgprs <= 128 and scratch == 0, (key, vgprs, scratch)
