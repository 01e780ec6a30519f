"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/mea.h, sizes workspaces, and rejects bad arguments before
launching anything (every case below fails validation, so no kernel runs)."""
import ctypes
import os
import re

import pytest

from paper_2112_05682_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mea.h")

FAKE = 0x10000  # aligned non-null address; only used where validation must fail first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mea_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert ctypes.cast(getattr(lib, name), ctypes.c_void_p).value


def test_status_strings():
    for s in range(6):
        assert _lib.status_string(s)
    assert _lib.status_string(99) == "unknown status"


def prob(**kw):
    base = dict(batch=1, heads=2, n_q=100, n_k=100, d=64, dtype=_lib.MEA_BF16, causal=0,
                scale=0.125, out_f32=0)
    base.update(kw)
    # built directly (no normalisation) so that invalid fields reach the library
    return _lib.MeaProblem(base["batch"], base["heads"], base["n_q"], base["n_k"], base["d"],
                           base["dtype"], base["causal"], base["scale"], base["out_f32"])


def ws_status(p):
    out = ctypes.c_size_t(0)
    return _lib.load().mea_attention_fwd_workspace_size(ctypes.byref(p), ctypes.byref(out)), out


def test_workspace_sizes():
    # One query tile per head and a long key sequence: keys are split, and the
    # per-split summaries (d + 2 floats per row and split) need workspace.
    p = prob(heads=1, n_q=256, n_k=1 << 20)
    ws = _lib.fwd_workspace_size(p)
    assert ws >= 2 * 256 * (64 + 2) * 4
    # Many query tiles: no split, no forward workspace.
    assert _lib.fwd_workspace_size(prob(heads=16, n_q=16384, n_k=16384)) == 0
    # Backward: D_i, one float per query row.
    assert _lib.bwd_workspace_size(prob(heads=16, n_q=16384, n_k=16384)) >= 16 * 16384 * 4


@pytest.mark.parametrize("kw,status", [
    (dict(d=32), _lib.MEA_ERR_UNSUPPORTED),
    (dict(d=96), _lib.MEA_ERR_UNSUPPORTED),
    (dict(dtype=7), _lib.MEA_ERR_UNSUPPORTED),
    (dict(n_q=0), _lib.MEA_ERR_INVALID_ARG),
    (dict(n_k=0), _lib.MEA_ERR_INVALID_ARG),
    (dict(batch=0), _lib.MEA_ERR_INVALID_ARG),
    (dict(heads=-1), _lib.MEA_ERR_INVALID_ARG),
    (dict(scale=0.0), _lib.MEA_ERR_INVALID_ARG),
    (dict(scale=-1.0), _lib.MEA_ERR_INVALID_ARG),
    (dict(scale=float("nan")), _lib.MEA_ERR_INVALID_ARG),
    (dict(scale=float("inf")), _lib.MEA_ERR_INVALID_ARG),
    (dict(causal=2), _lib.MEA_ERR_INVALID_ARG),
    (dict(out_f32=3), _lib.MEA_ERR_INVALID_ARG),
    (dict(n_q=1 << 31), _lib.MEA_ERR_INVALID_ARG),
    (dict(batch=1 << 40, heads=1 << 40), _lib.MEA_ERR_INVALID_ARG),
])
def test_problem_validation(kw, status):
    p = prob(**kw)
    st, _ = ws_status(p)
    assert st == status
    lib = _lib.load()
    out = ctypes.c_size_t(0)
    assert lib.mea_attention_bwd_workspace_size(ctypes.byref(p), ctypes.byref(out)) == status
    assert _lib.fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 30, None) == status
    assert _lib.bwd(p, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30,
                    None) == status


def test_null_problem_and_null_size_pointer():
    lib = _lib.load()
    out = ctypes.c_size_t(0)
    assert lib.mea_attention_fwd_workspace_size(None, ctypes.byref(out)) == _lib.MEA_ERR_INVALID_ARG
    p = prob()
    assert lib.mea_attention_fwd_workspace_size(ctypes.byref(p), None) == _lib.MEA_ERR_INVALID_ARG


@pytest.mark.parametrize("which", range(4))
def test_fwd_rejects_null_or_misaligned_pointers(which):
    p = prob()
    for bad in (None, FAKE + 2):
        ptrs = [FAKE] * 4
        ptrs[which] = bad
        assert _lib.fwd(p, *ptrs, None, None, None, 0, None) == _lib.MEA_ERR_INVALID_ARG
    # misaligned lse
    assert _lib.fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE + 4, None, None, 0, None) == _lib.MEA_ERR_INVALID_ARG


@pytest.mark.parametrize("which", [0, 1, 2, 3, 5, 6])
def test_bwd_rejects_null_inputs(which):
    # q, k, v, o, (o_lo: optional), do, lse, dq, dk, dv
    p = prob()
    ptrs = [FAKE] * 10
    ptrs[which] = None
    assert _lib.bwd(p, *ptrs, FAKE, 1 << 30, None) == _lib.MEA_ERR_INVALID_ARG


@pytest.mark.parametrize("grads", [(None, None, None), (FAKE, FAKE, None), (FAKE, None, FAKE),
                                   (None, FAKE, None), (FAKE + 8, FAKE, FAKE)])
def test_bwd_rejects_bad_gradient_pointer_sets(grads):
    # dq optional; dk and dv both or neither; at least one group; 16 B aligned.
    p = prob()
    assert _lib.bwd(p, *([FAKE] * 7), *grads, FAKE, 1 << 30, None) == _lib.MEA_ERR_INVALID_ARG


def test_workspace_too_small_is_rejected_before_launch():
    p = prob(heads=1, n_q=256, n_k=1 << 20)
    need = _lib.fwd_workspace_size(p)
    assert need > 0
    assert _lib.fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == _lib.MEA_ERR_WORKSPACE
    assert _lib.fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, need - 1, None) == _lib.MEA_ERR_WORKSPACE
    need_b = _lib.bwd_workspace_size(p)
    assert _lib.bwd(p, *([FAKE] * 10), None, 0, None) == _lib.MEA_ERR_WORKSPACE
    assert _lib.bwd(p, *([FAKE] * 10), FAKE, need_b - 1, None) == _lib.MEA_ERR_WORKSPACE


def test_problem_struct_layout_matches_the_header(tmp_path):
    # Compile a probe against include/mea.h with the host C compiler and compare
    # the struct layout with the ctypes mirror used by the binding.
    import shutil
    import subprocess
    if not shutil.which("gcc") or not os.path.isdir("/opt/rocm/include"):
        pytest.skip("needs gcc and the ROCm headers")
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "mea.h"\n'
        'int main(void) { printf("%zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu\\n", '
        'sizeof(mea_problem), '
        'offsetof(mea_problem, batch), offsetof(mea_problem, heads), offsetof(mea_problem, n_q), '
        'offsetof(mea_problem, n_k), offsetof(mea_problem, d), offsetof(mea_problem, dtype), '
        'offsetof(mea_problem, causal), offsetof(mea_problem, scale), '
        'offsetof(mea_problem, out_f32), offsetof(mea_problem, strides), '
        'offsetof(mea_problem, kv_len), offsetof(mea_problem, d_v), '
        'sizeof(mea_strides), offsetof(mea_strides, d_o), offsetof(mea_strides, dv)); return 0; }\n')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"),
                    "-I/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    got = [int(t) for t in subprocess.run([str(exe)], check=True, capture_output=True,
                                          text=True).stdout.split()]
    M, S = _lib.MeaProblem, _lib.MeaStrides
    want = [ctypes.sizeof(M)] + [getattr(M, f).offset for f, _ in M._fields_] + [
        ctypes.sizeof(S), S.d_o.offset, S.dv.offset]
    assert got == want


def _strided_prob(**over):
    # bf16, B=2, H=4, n_q=100, n_k=300, d=64 in the [B, n, H, d] layout, with
    # one tensor's strides replaced by `over`.
    B, H, nq, nk, d = 2, 4, 100, 300, 64
    st = {"q": (nq * H * d, d, H * d), "k": (nk * H * d, d, H * d), "v": (nk * H * d, d, H * d),
          "o": (nq * H * d, d, H * d), "d_o": (nq * H * d, d, H * d), "dq": (nq * H * d, d, H * d),
          "dk": (nk * H * d, d, H * d), "dv": (nk * H * d, d, H * d)}
    st.update(over)
    return _lib.problem(B, H, nq, nk, d, _lib.MEA_BF16, False, 0.125, strides=st)


@pytest.mark.parametrize("bad", [
    {"q": (100 * 256, 64, 32)},        # row stride below d
    {"k": (300 * 256, 64, 1 << 24)},   # row stride beyond the 32-bit copy offsets
    {"v": (300 * 256, 60, 256)},       # head stride not a multiple of 16 bytes
    {"o": (100 * 256, 0, 256)},        # output rows shared by every head
    {"q": (-1, 64, 256)},              # negative stride
])
def test_fwd_rejects_bad_strides(bad):
    # Validation fails before anything is launched (the pointers are fake).
    assert _lib.fwd(_strided_prob(**bad), FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == \
        _lib.MEA_ERR_INVALID_ARG


@pytest.mark.parametrize("bad", [{"dq": (100 * 256, 0, 256)}, {"dk": (300 * 256, 64, 8)},
                                 {"d_o": (100 * 256, 64, 36)}])
def test_bwd_rejects_bad_strides(bad):
    p = _strided_prob(**bad)
    assert _lib.bwd(p, *([FAKE] * 10), FAKE, 1 << 30, None) == _lib.MEA_ERR_INVALID_ARG


def test_shared_key_heads_are_valid_input_strides():
    # Head stride 0 for k and v (one key head for all query heads) is allowed
    # for inputs; for dk and dv it would make heads overwrite each other.
    ok = _strided_prob(k=(300 * 64, 0, 64), v=(300 * 64, 0, 64))
    assert ok.strides.contents.k.head == 0
    bad = _strided_prob(dk=(300 * 64, 0, 64))
    assert _lib.bwd(bad, *([FAKE] * 10), FAKE, 1 << 30, None) == _lib.MEA_ERR_INVALID_ARG


def test_rejects_misaligned_kv_len():
    # kv_len is an int32 device array: a pointer that is not 4-byte aligned is
    # rejected before anything is launched (the tensor pointers are fake).
    p = _lib.problem(1, 2, 100, 100, 64, _lib.MEA_BF16, False, 0.125, kv_len=FAKE + 2)
    assert _lib.fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == _lib.MEA_ERR_INVALID_ARG
    assert _lib.bwd(p, *([FAKE] * 10), FAKE, 1 << 30, None) == _lib.MEA_ERR_INVALID_ARG
    ok = _lib.problem(1, 2, 100, 100, 64, _lib.MEA_BF16, False, 0.125, kv_len=FAKE)
    assert ok.kv_len == FAKE


@pytest.mark.parametrize("d,d_v,status", [(64, 128, None), (128, 64, None), (64, 96, "unsupported"),
                                          (64, -64, "invalid")])
def test_value_head_dimension_validation(d, d_v, status):
    # d_v = 0 means d; 64 and 128 are supported in any combination with d.
    p = _lib.problem(1, 2, 100, 100, d, _lib.MEA_BF16, False, 0.125, d_v=d_v)
    st, _ = ws_status(p)
    want = {None: _lib.MEA_OK, "unsupported": _lib.MEA_ERR_UNSUPPORTED,
            "invalid": _lib.MEA_ERR_INVALID_ARG}[status]
    assert st == want


def test_value_head_dimension_sets_default_strides():
    # Contiguous strides of v, o, do and dv follow d_v; those of q, k, dq, dk d.
    p = _lib.problem(2, 3, 10, 20, 64, _lib.MEA_BF16, False, 0.125, d_v=128,
                     strides={"q": (3 * 10 * 64, 10 * 64, 64)})
    st = p.strides.contents
    assert (st.v.batch, st.v.head, st.v.row) == (3 * 20 * 128, 20 * 128, 128)
    assert (st.o.batch, st.o.head, st.o.row) == (3 * 10 * 128, 10 * 128, 128)
    assert (st.k.batch, st.k.head, st.k.row) == (3 * 20 * 64, 20 * 64, 64)
    # A value row stride below d_v is rejected before any launch.
    bad = _lib.problem(1, 1, 10, 20, 64, _lib.MEA_BF16, False, 0.125, d_v=128,
                       strides={"v": (20 * 128, 20 * 128, 64)})
    assert _lib.fwd(bad, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == _lib.MEA_ERR_INVALID_ARG


@pytest.mark.parametrize("dtype,out_f32", [(_lib.MEA_F32, False), (_lib.MEA_BF16, True)])
def test_residual_is_rejected_for_a_float32_output(dtype, out_f32):
    # o_lo exists only for a 16-bit o: with a float32 o it must be NULL.
    p = _lib.problem(1, 2, 100, 100, 64, dtype, False, 0.125, out_f32=out_f32)
    assert _lib.fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0, None) == _lib.MEA_ERR_INVALID_ARG
    assert _lib.bwd(p, *([FAKE] * 10), FAKE, 1 << 30, None) == _lib.MEA_ERR_INVALID_ARG


def test_residual_must_be_aligned():
    p = _lib.problem(1, 2, 100, 100, 64, _lib.MEA_BF16, False, 0.125)
    assert _lib.fwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 8, None, 0, None) == _lib.MEA_ERR_INVALID_ARG
    ptrs = [FAKE] * 10
    ptrs[4] = FAKE + 8
    assert _lib.bwd(p, *ptrs, FAKE, 1 << 30, None) == _lib.MEA_ERR_INVALID_ARG
