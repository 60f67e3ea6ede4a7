"""Host-side checks of the C ABI that need no GPU.

* the library builds for gfx950 and exports every function include/qlayer.h declares;
* invalid arguments are rejected on the host, before anything is launched;
* workspace-size queries and status strings;
* the division-by-invariant helper the kernels use for index arithmetic.
"""
import ctypes
import os
import re
import subprocess
import sys

import pytest

import paper_2204_01701_amd as ql
from paper_2204_01701_amd import build as qbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qlayer.h")
NET_HEADER = os.path.join(ROOT, "include", "qnet.h")

QL_OK, QL_EINVAL, QL_EUNSUPPORTED, QL_EWORKSPACE, QL_EHIP = range(5)


@pytest.fixture(scope="module")
def L():
    if qbuild.is_stale():
        qbuild.build()
    return ql.lib()


def _declared_functions():
    txt = open(HEADER).read() + open(NET_HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b((?:qlayer|qnet)_\w+)\s*\(", txt)))


def test_header_declares_the_five_entry_points():
    names = _declared_functions()
    for f in ("qlayer_conv2d_fwd", "qlayer_conv2d_bwd_data", "qlayer_conv2d_bwd_weight",
              "qlayer_linear_fwd", "qlayer_linear_bwd"):
        assert f in names


def test_library_exports_every_declared_symbol(L):
    out = subprocess.run(["nm", "-D", "--defined-only", ql.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT ((?:qlayer|qnet)_\w+)", out))
    missing = [f for f in _declared_functions() if f not in exported]
    assert not missing, missing
    for f in _declared_functions():
        assert getattr(L, f) is not None


def test_status_strings_and_version(L):
    assert ql.qlayer_status_string(QL_OK) == "ok"
    assert "invalid" in ql.qlayer_status_string(QL_EINVAL)
    assert "workspace" in ql.qlayer_status_string(QL_EWORKSPACE)
    assert ql.qlayer_version() >= 100


FAKE = 1 << 20  # a 16-byte aligned fake device address; never dereferenced by these calls


def _fwd(L, d, x=FAKE, wa=FAKE, wb=FAKE, wc=FAKE, y=FAKE, ta=None, tb=None, ws=None, wsb=0):
    return L.qlayer_conv2d_fwd(ctypes.byref(d), x, wa, wb, wc, None, None, None, y, ta, tb, ws, wsb, None)


def test_conv_descriptor_validation(L):
    good = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32)
    bad = [
        ql.conv_desc(0, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32),       # n = 0
        ql.conv_desc(2, 16, 8, 8, -1, 3, 3, 1, 1, ql.QL_F32),       # o < 0
        ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 0, 1, ql.QL_F32),       # stride 0
        ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, -1, ql.QL_F32),      # pad < 0
        ql.conv_desc(2, 16, 2, 2, 16, 5, 5, 1, 0, ql.QL_F32),       # empty output
        ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, 7),               # unknown dtype
    ]
    for d in bad:
        assert _fwd(L, d) == QL_EINVAL
        assert L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(d)) == 0
    assert L.qlayer_conv2d_fwd(None, FAKE, FAKE, FAKE, FAKE, None, None, None, FAKE, None, None, None, 0,
                               None) == QL_EINVAL
    # required pointers
    assert _fwd(L, good, x=None) == QL_EINVAL
    assert _fwd(L, good, wb=None) == QL_EINVAL
    assert _fwd(L, good, y=None) == QL_EINVAL                      # no Y and no terms
    assert _fwd(L, good, y=None, ta=FAKE) == QL_EINVAL             # recompute needs both terms
    assert _fwd(L, good, x=FAKE + 4) == QL_EINVAL                  # misaligned
    # oversize: more than 2^31 - 1 elements in one tensor
    huge = ql.conv_desc(1 << 12, 1 << 10, 32, 32, 16, 3, 3, 1, 1, ql.QL_BF16)
    assert _fwd(L, huge) == QL_EUNSUPPORTED


def test_backward_validation(L):
    d = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32)
    ws = L.qlayer_conv2d_bwd_data_workspace_size(ctypes.byref(d))
    assert ws >= 3 * 16 * 9 * 16 * 4                                  # holds the transposed weights
    args = [FAKE] * 7
    assert L.qlayer_conv2d_bwd_data(ctypes.byref(d), *args, FAKE, ws - 1, None) == QL_EWORKSPACE
    assert L.qlayer_conv2d_bwd_data(ctypes.byref(d), *args, None, ws, None) == QL_EWORKSPACE
    args[1] = None                                                    # T_a missing
    assert L.qlayer_conv2d_bwd_data(ctypes.byref(d), *args, FAKE, ws, None) == QL_EINVAL
    # weight gradients: biases all or none
    w = [FAKE] * 7
    assert L.qlayer_conv2d_bwd_weight(ctypes.byref(d), *w, FAKE, None, None, FAKE, 1 << 30, None) == QL_EINVAL
    assert L.qlayer_conv2d_bwd_weight(ctypes.byref(d), FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, None, None,
                                      None, FAKE, 1 << 30, None) == QL_EINVAL
    # dense backward: at least one output, dW all-or-none, db needs dW
    dl = ql.linear_desc(64, 32, 48, ql.QL_BF16)
    base = [FAKE] * 7
    assert L.qlayer_linear_bwd(ctypes.byref(dl), *base, None, None, None, None, None, None, None,
                               FAKE, 1 << 30, None) == QL_EINVAL
    assert L.qlayer_linear_bwd(ctypes.byref(dl), *base, FAKE, FAKE, None, None, None, None, None,
                               FAKE, 1 << 30, None) == QL_EINVAL
    assert L.qlayer_linear_bwd(ctypes.byref(dl), *base, FAKE, None, None, None, FAKE, FAKE, FAKE,
                               FAKE, 1 << 30, None) == QL_EINVAL


def test_workspace_queries_are_consistent(L):
    # split-K partials only where the output tiles cannot fill the GPU and each
    # wave's K range is long (the 512-channel 4 x 4 layer); the 2 x 2 layer's
    # waves split K within the workgroup and need no workspace
    big = ql.conv_desc(64, 256, 56, 56, 256, 3, 3, 1, 1, ql.QL_BF16)
    small = ql.conv_desc(128, 512, 4, 4, 512, 3, 3, 1, 1, ql.QL_BF16)
    tiny = ql.conv_desc(128, 512, 2, 2, 512, 3, 3, 1, 1, ql.QL_BF16)
    assert L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(big)) == 0
    assert L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(small)) > 0
    assert L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(tiny)) == 0
    assert L.qlayer_conv2d_bwd_weight_workspace_size(ctypes.byref(big)) > 0
    # bf16 reads the weights untransposed; fp32 stages a transposed copy in the workspace
    dl = ql.linear_desc(8192, 4096, 4096, ql.QL_BF16)
    assert L.qlayer_linear_bwd_workspace_size(ctypes.byref(dl)) % 256 == 0
    dl32 = ql.linear_desc(8192, 4096, 4096, ql.QL_F32)
    assert L.qlayer_linear_bwd_workspace_size(ctypes.byref(dl32)) >= 3 * 4096 * 4096 * 4
    for f in ("conv2d_fwd", "conv2d_bwd_data", "conv2d_bwd_weight"):
        assert getattr(L, f"qlayer_{f}_workspace_size")(ctypes.byref(big)) % 256 == 0


def test_fastdiv_host_formula(tmp_path):
    """The multiply-shift division used for index arithmetic is exact (checked on the host)."""
    src = tmp_path / "fd.cpp"
    src.write_text(r'''
#include "qfastdiv.h"
#include <cstdio>
#include <cstdint>
int main() {
    const uint32_t ds[] = {1, 2, 3, 5, 7, 9, 16, 27, 56, 64, 100, 576, 1000, 3136, 4096, 12544,
                           200704, 262144, 1u << 20, 65537, 2147483647u};
    uint64_t x = 88172645463325252ull;
    for (uint32_t d : ds) {
        ql::FastDiv f = ql::make_fastdiv(d);
        for (int i = 0; i < 200000; ++i) {
            x ^= x << 13; x ^= x >> 7; x ^= x << 17;
            uint32_t n = (uint32_t)x;
            if (i % 3 == 0) n &= 0x7fffffffu;
            if (i < 4096) n = (uint32_t)i;
            if (ql::fdiv_host(n, f) != n / d) { std::printf("FAIL d=%u n=%u\n", d, n); return 1; }
        }
        const uint32_t edge[] = {d - 1, d, d + 1, 2 * d - 1, 0xffffffffu, 0x7fffffffu};
        for (uint32_t n : edge)
            if (ql::fdiv_host(n, f) != n / d) { std::printf("FAIL d=%u n=%u\n", d, n); return 1; }
    }
    std::printf("ok\n");
    return 0;
}
''')
    exe = tmp_path / "fd"
    subprocess.run(["g++", "-O2", "-std=c++17", "-I", os.path.join(ROOT, "paper_2204_01701_amd", "csrc"),
                    str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip() == "ok", out.stdout


def test_neuron_type_validation(L):
    # an unknown type, and the identity shortcut without C == O or with a changed map
    assert _fwd(L, ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32, 6)) == QL_EINVAL
    assert _fwd(L, ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32, -1)) == QL_EINVAL
    assert _fwd(L, ql.conv_desc(2, 16, 8, 8, 32, 3, 3, 1, 1, ql.QL_F32, ql.QL_NEURON_T4_IDENTITY)) == QL_EINVAL
    assert _fwd(L, ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 2, 1, ql.QL_F32, ql.QL_NEURON_T4_IDENTITY)) == QL_EINVAL
    assert _fwd(L, ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 0, ql.QL_F32, ql.QL_NEURON_T4_IDENTITY)) == QL_EINVAL
    # the weights a type has are required; recompute mode needs its saved maps; T2 saves none
    t4 = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32, ql.QL_NEURON_T4)
    assert _fwd(L, t4, wb=None) == QL_EINVAL
    assert _fwd(L, t4, y=None, ta=FAKE) == QL_EINVAL
    t3 = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32, ql.QL_NEURON_T3)
    assert _fwd(L, t3, wa=None) == QL_EINVAL
    assert _fwd(L, t3, y=None) == QL_EINVAL
    t2 = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32, ql.QL_NEURON_T2)
    assert _fwd(L, t2, y=None, ta=FAKE, tb=FAKE) == QL_EINVAL
    # backward: the saved maps of the type (T2's input gradient takes X in `ta`)
    ws = 1 << 30
    assert L.qlayer_conv2d_bwd_data(ctypes.byref(t3), FAKE, None, None, FAKE, None, None, FAKE, FAKE, ws,
                                    None) == QL_EINVAL
    assert L.qlayer_conv2d_bwd_data(ctypes.byref(t4), FAKE, FAKE, None, FAKE, FAKE, None, FAKE, FAKE, ws,
                                    None) == QL_EINVAL
    assert L.qlayer_conv2d_bwd_weight(ctypes.byref(t4), FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, None,
                                      None, FAKE, ws, None) == QL_EINVAL          # dW_b missing
    assert L.qlayer_conv2d_bwd_weight(ctypes.byref(t4), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, None,
                                      None, FAKE, ws, None) == QL_EINVAL          # biases of some terms only
    # T2&4: its input gradient needs X (the _ex entry point); the depthwise kernels do not cover it
    t24 = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32, ql.QL_NEURON_T24)
    assert L.qlayer_conv2d_bwd_data(ctypes.byref(t24), *[FAKE] * 7, FAKE, ws, None) == QL_EINVAL
    assert L.qlayer_conv2d_bwd_data_ex(ctypes.byref(t24), *[FAKE] * 3, None, *[FAKE] * 4, FAKE, ws,
                                       None) == QL_EINVAL                          # no X
    assert L.qlayer_conv2d_bwd_data_ex(ctypes.byref(t24), *[FAKE] * 8, FAKE, 16, None) == QL_EWORKSPACE
    assert _fwd(L, t24, wc=None) == QL_EINVAL                                      # W_c required
    dw24 = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32, ql.QL_NEURON_T24, groups=16)
    assert _fwd(L, dw24) == QL_EUNSUPPORTED
    # the workspace queries accept every type
    for n in range(6):
        d = ql.conv_desc(4, 512, 4, 4, 512, 3, 3, 1, 1, ql.QL_BF16, n)
        assert L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(d)) > 0


def test_depthwise_validation(L):
    # groups: 1 (or 0) is dense, C with O == C is depthwise, anything else is not supported
    assert _fwd(L, ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32, 0, groups=2)) == QL_EUNSUPPORTED
    assert _fwd(L, ql.conv_desc(2, 16, 8, 8, 32, 3, 3, 1, 1, ql.QL_F32, 0, groups=16)) == QL_EINVAL
    # the filters of a channel slice are staged in 64 KiB of LDS: 15 x 15 is too large, 13 x 13 fits
    assert _fwd(L, ql.conv_desc(2, 16, 16, 16, 16, 15, 15, 1, 7, ql.QL_F32, 0, groups=16)) == QL_EUNSUPPORTED
    big = ql.conv_desc(2, 16, 16, 16, 16, 13, 13, 1, 6, ql.QL_F32, 0, groups=16)
    assert L.qlayer_conv2d_bwd_weight_workspace_size(ctypes.byref(big)) >= 0
    assert _fwd(L, big, wb=None) == QL_EINVAL  # the pointer checks of the dense path apply
    # the forward and input gradient need no workspace; the weight gradient's
    # split partials grow with the pixel count
    for n in range(5):
        d = ql.conv_desc(128, 64, 56, 56, 64, 3, 3, 1, 1, ql.QL_BF16, n, groups=64)
        assert L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(d)) == 0
        assert L.qlayer_conv2d_bwd_data_workspace_size(ctypes.byref(d)) == 0
        nt = ql.NEURON_TERMS[n]
        ws = L.qlayer_conv2d_bwd_weight_workspace_size(ctypes.byref(d))
        assert ws >= 2 * nt * 64 * (9 + 1) * 4
    tiny = ql.conv_desc(1, 8, 4, 4, 8, 3, 3, 1, 1, ql.QL_F32, 0, groups=8)
    assert L.qlayer_conv2d_bwd_weight_workspace_size(ctypes.byref(tiny)) == 0  # one split writes dW directly
    # a depthwise weight gradient with too small a workspace
    assert L.qlayer_conv2d_bwd_weight(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None,
                                      None, FAKE, 16, None) == QL_EWORKSPACE


def test_epilogue_validation(L):
    d = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32)
    ld = ql.linear_desc(32, 64, 64, ql.QL_BF16)

    def fwd_ex(epi, y=FAKE, ta=None, tb=None, ws=FAKE, wsb=1 << 30):
        return L.qlayer_conv2d_fwd_ex(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None, None, None, y, ta, tb,
                                      ctypes.byref(epi) if epi is not None else None, ws, wsb, None)

    # recompute mode (no Y) with an epilogue that does anything; half of the statistics pair
    assert fwd_ex(ql.Epilogue(None, None, 1, None, None), y=None, ta=FAKE, tb=FAKE) == QL_EINVAL
    assert fwd_ex(ql.Epilogue(None, None, 0, FAKE, FAKE), y=None, ta=FAKE, tb=FAKE) == QL_EINVAL
    assert fwd_ex(ql.Epilogue(None, None, 0, FAKE, None)) == QL_EINVAL
    assert fwd_ex(ql.Epilogue(None, None, 0, None, FAKE)) == QL_EINVAL
    assert fwd_ex(ql.Epilogue(FAKE + 4, None, 0, None, None)) == QL_EINVAL  # 16-byte alignment
    # the statistics need partial sums in the workspace; the affine and ReLU alone need none
    relu = ql.Epilogue(FAKE, FAKE, 1, None, None)
    stats = ql.Epilogue(None, None, 0, FAKE, FAKE)
    plain = L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(d))
    assert L.qlayer_conv2d_fwd_ex_workspace_size(ctypes.byref(d), None) == plain
    assert L.qlayer_conv2d_fwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(relu)) == plain
    # (128 rows: at most one part of 2 x 16 sums per 16 rows)
    assert L.qlayer_conv2d_fwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(stats)) <= plain + 8 * 2 * 16 * 4
    d = ql.conv_desc(8, 64, 32, 32, 64, 3, 3, 1, 1, ql.QL_BF16)
    plain = L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(d))
    need = L.qlayer_conv2d_fwd_ex_workspace_size(ctypes.byref(d), ctypes.byref(stats))
    assert need >= plain + 2 * 64 * 4
    assert fwd_ex(stats, ws=FAKE, wsb=need - 1) == QL_EWORKSPACE
    ld = ql.linear_desc(8192, 64, 64, ql.QL_BF16)
    assert L.qlayer_linear_fwd_ex_workspace_size(ctypes.byref(ld), ctypes.byref(stats)) >= \
        L.qlayer_linear_fwd_workspace_size(ctypes.byref(ld)) + 2 * 64 * 4
    # depthwise: no workspace but the statistics' partial sums
    dd = ql.conv_desc(8, 32, 32, 32, 32, 3, 3, 1, 1, ql.QL_BF16, 0, groups=32)
    assert L.qlayer_conv2d_fwd_ex_workspace_size(ctypes.byref(dd), ctypes.byref(relu)) == 0
    assert L.qlayer_conv2d_fwd_ex_workspace_size(ctypes.byref(dd), ctypes.byref(stats)) >= 2 * 32 * 4


def test_few_channel_paths_need_no_workspace(L, monkeypatch):
    """The few-input-channel forward (no zero-padded copies) and the fused input
    gradient at stride 1 (partial sums in LDS) ask for no workspace; forced off,
    the padded forward and the two-kernel input gradient ask for their buffers."""
    for dt in (ql.QL_BF16, ql.QL_F32):
        stem = ql.conv_desc(128, 3, 32, 32, 64, 3, 3, 1, 1, dt)
        assert L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(stem)) == 0
        assert L.qlayer_conv2d_bwd_data_workspace_size(ctypes.byref(stem)) == 0
        strided = ql.conv_desc(128, 3, 32, 32, 64, 3, 3, 2, 1, dt)
        assert L.qlayer_conv2d_bwd_data_workspace_size(ctypes.byref(strided)) >= 128 * 16 * 16 * 27 * 4
    monkeypatch.setenv("QLAYER_FWD_SMALLC", "0")
    monkeypatch.setenv("QLAYER_BWD_DATA_FUSED_RB", "0")
    stem = ql.conv_desc(128, 3, 32, 32, 64, 3, 3, 1, 1, ql.QL_BF16)
    assert L.qlayer_conv2d_fwd_workspace_size(ctypes.byref(stem)) >= 128 * 32 * 32 * 8 * 2   # X padded to 8
    assert L.qlayer_conv2d_bwd_data_workspace_size(ctypes.byref(stem)) >= 128 * 32 * 32 * 27 * 4


def test_valid_call_without_a_device_returns_ehip():
    """A valid call in a process that sees no GPU reports QL_EHIP (the launch
    or the device query fails) and returns normally: no abort, no crash.  Run
    in a child process so that a crash would show as its exit status.  Only
    where no GPU is present (the fake pointers must never reach a kernel)."""
    if os.path.exists("/dev/kfd"):
        pytest.skip("a GPU device node is present")
    code = (
        "import ctypes, paper_2204_01701_amd as ql\n"
        "L = ql.lib()\n"
        "F = 1 << 20\n"
        "d = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32)\n"
        "r1 = L.qlayer_conv2d_fwd(ctypes.byref(d), F, F, F, F, None, None, None, F, None, None, None, 0, None)\n"
        "dl = ql.linear_desc(64, 32, 48, ql.QL_F32)\n"
        "r2 = L.qlayer_linear_fwd(ctypes.byref(dl), F, F, F, F, None, None, None, F, None, None, None, 0, None)\n"
        "print(r1, r2)\n"
    )
    env = dict(os.environ, HIP_VISIBLE_DEVICES="", ROCR_VISIBLE_DEVICES="")
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=ROOT, env=env,
                         timeout=120)
    assert res.returncode == 0, res.stderr[-2000:]
    assert res.stdout.split()[-2:] == [str(QL_EHIP), str(QL_EHIP)], res.stdout


def test_binding_rejects_host_and_mis_sized_tensors_before_any_call():
    """The Python binding checks device, element count and dtype of every tensor
    against the descriptor and raises before the C ABI is reached."""
    import torch
    d = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_F32)
    x = torch.zeros(2, 8, 8, 16)
    w = [torch.zeros(16, 3, 3, 16) for _ in range(3)]
    y = torch.zeros(2, 8, 8, 16)
    with pytest.raises(ValueError, match="CUDA"):
        ql.qlayer_conv2d_fwd(d, x, *w, None, None, None, y)
    dl = ql.linear_desc(64, 32, 48, ql.QL_F32)
    with pytest.raises(ValueError, match="CUDA"):
        ql.qlayer_linear_fwd(dl, torch.zeros(64, 32), *[torch.zeros(48, 32)] * 3, y=torch.zeros(64, 48))
    # sizes and dtypes are checked the same way (the device check fires first on the host)
    with pytest.raises(ValueError):
        ql._expect("w", torch.zeros(10), 11, None, None)


def test_noalloc_weight_gradient_rejects_a_layer_beyond_its_scratch(L):
    """The no-allocation entry point plans for its fixed scratch array: a
    few-channel bf16 layer whose zero-padded copy of X alone exceeds it is
    refused with QL_EWORKSPACE before anything is launched."""
    d = ql.conv_desc(1024, 3, 64, 64, 64, 3, 3, 1, 1, ql.QL_BF16)
    assert 1024 * 64 * 64 * 8 * 2 > ql.NOALLOC_SCRATCH_BYTES
    assert L.qlayer_conv2d_bwd_weight_noalloc(ctypes.byref(d), *[FAKE] * 10, None) == QL_EWORKSPACE
    assert L.qlayer_conv2d_bwd_weight_noalloc(ctypes.byref(d), *[FAKE] * 4, None, *[FAKE] * 5,
                                              None) == QL_EINVAL                   # dW_a missing


def test_relu_backward_validation(L):
    """The backward behind the fused ReLU: y' required, at least one gradient,
    a workspace of at least the query's size (which holds G before the larger
    of the two passes' workspaces)."""
    d = ql.conv_desc(2, 16, 8, 8, 16, 3, 3, 1, 1, ql.QL_BF16)
    need = L.qlayer_conv2d_bwd_relu_workspace_size(ctypes.byref(d))
    g_bytes = 2 * 8 * 8 * 16 * 2
    assert need >= g_bytes and need % 256 == 0
    assert need >= (g_bytes + 255) // 256 * 256 + max(L.qlayer_conv2d_bwd_data_workspace_size(ctypes.byref(d)),
                                                      L.qlayer_conv2d_bwd_weight_workspace_size(ctypes.byref(d)))
    full = [FAKE] * 9 + [FAKE] * 6   # x gy y' ta tb wa wb wc dx | dw x3, db x3
    fn = L.qlayer_conv2d_bwd_relu
    assert fn(ctypes.byref(d), *full, FAKE, need - 1, None) == QL_EWORKSPACE
    assert fn(ctypes.byref(d), *full, None, need, None) == QL_EWORKSPACE
    no_y = list(full)
    no_y[2] = None
    assert fn(ctypes.byref(d), *no_y, FAKE, need, None) == QL_EINVAL
    none_wanted = full[:8] + [None] * 7
    assert fn(ctypes.byref(d), *none_wanted, FAKE, need, None) == QL_EINVAL
    db_without_dw = full[:9] + [None] * 3 + [FAKE] * 3
    assert fn(ctypes.byref(d), *db_without_dw, FAKE, need, None) == QL_EINVAL
    dl = ql.linear_desc(64, 32, 48, ql.QL_F32)
    needl = L.qlayer_linear_bwd_relu_workspace_size(ctypes.byref(dl))
    assert needl >= 64 * 48 * 4
    assert L.qlayer_linear_bwd_relu(ctypes.byref(dl), *no_y, FAKE, needl, None) == QL_EINVAL
