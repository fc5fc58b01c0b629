"""The C-ABI library loads, exports every entry point of include/bsa.h, and validates
its arguments on the host (no kernel is launched by these tests)."""
import ctypes as C
import os
import re

import pytest

from paper_2506_12541_amd import _lib
from paper_2506_12541_amd.bsa import Params

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2506_12541_amd.build import build
        build()
    return _lib.load()


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "bsa.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bsa_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_symbols()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(_lib._SIGS), "binding and header disagree"


def _sizes(lib, p):
    a, b, c = C.c_size_t(), C.c_size_t(), C.c_size_t()
    cp = p.c()
    return lib.bsa_sizes(C.byref(cp), C.byref(a), C.byref(b), C.byref(c)), a.value, c.value


def base(**kw):
    d = dict(batch=1, n=1024, heads=4, head_dim=32, ball_size=64, cmp_block=8, slc_block=16, topk=4, group_size=8)
    d.update(kw)
    return Params(**d)


def test_valid_params(lib):
    st, ws, saved = _sizes(lib, base())
    assert st == _lib.BSA_OK and ws > 0 and saved > 0


@pytest.mark.parametrize("kw,code", [
    (dict(n=1000), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(head_dim=48), _lib.BSA_ERR_UNSUPPORTED),
    (dict(ball_size=96), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(ball_size=2048), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(cmp_block=8, cmp_stride=4), _lib.BSA_ERR_UNSUPPORTED),
    (dict(slc_block=24), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(slc_block=64, cmp_block=8), _lib.BSA_ERR_UNSUPPORTED),
    (dict(group_size=12), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(group_size=4), _lib.BSA_ERR_UNSUPPORTED),        # 1 (per token) or >= 8
    (dict(group_size=1, dtype=_lib.BSA_F32), _lib.BSA_ERR_UNSUPPORTED),   # per token: bf16 only
    (dict(topk=0), _lib.BSA_ERR_UNSUPPORTED),
    (dict(topk=17), _lib.BSA_ERR_UNSUPPORTED),
    (dict(store_lse=2), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(dtype=7), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(softmax_scale=-1.0), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(q_coarsen=2), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(group_compression=2), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(group_size=16, q_coarsen=_lib.BSA_QC_MLP), _lib.BSA_ERR_INVALID_ARGUMENT),   # needs g == l
    (dict(group_size=16, group_compression=1), _lib.BSA_ERR_INVALID_ARGUMENT),
    (dict(n=256, group_compression=1), _lib.BSA_ERR_UNSUPPORTED),                       # n / l < 64
])
def test_invalid_params(lib, kw, code):
    st, _, _ = _sizes(lib, base(**kw))
    assert st == code
    assert lib.bsa_last_error().decode() != ""


def test_null_params(lib):
    assert lib.bsa_sizes(None, None, None, None) == _lib.BSA_ERR_INVALID_ARGUMENT


def test_forward_rejects_before_launch(lib):
    p = base()
    cp = p.c()
    saved = _lib.bsa_saved_t()
    # NULL q: rejected on the host, nothing launched
    st = lib.bsa_forward(C.byref(cp), None, None, None, None, None, None, None, None, None, C.byref(saved), None, 0,
                         None)
    assert st == _lib.BSA_ERR_INVALID_ARGUMENT


def test_variant_params_and_sizes(lib):
    # group compression and MLP query coarsening (Eq. 13-15) with g == l are accepted, and
    # they need more workspace than the regular layer (coarse queries, coarse outputs)
    st0, ws0, sv0 = _sizes(lib, base())
    st1, ws1, sv1 = _sizes(lib, base(q_coarsen=_lib.BSA_QC_MLP, group_compression=1))
    assert st0 == st1 == _lib.BSA_OK
    assert ws1 > ws0 and sv1 > sv0


def test_per_token_selection_sizes(lib):
    # g = 1 (Eq. 6-8 without grouping) is accepted for bf16 and needs the pair buffers
    st0, ws0, _ = _sizes(lib, base(dtype=_lib.BSA_BF16))
    st1, ws1, _ = _sizes(lib, base(dtype=_lib.BSA_BF16, group_size=1))
    assert st0 == st1 == _lib.BSA_OK and ws1 > ws0


def test_variant_forward_needs_phi_q(lib):
    p = base(q_coarsen=_lib.BSA_QC_MLP)
    cp = p.c()
    saved = _lib.bsa_saved_t()
    fake = C.c_void_p(256)
    for f in ("sel_idx", "lse", "o_branch", "kcmp", "vcmp", "hid_k", "hid_v", "cvalid", "qcmp", "hid_q", "ocmp",
              "o_cmp"):
        setattr(saved, f, 256)
    m = _lib.bsa_mlp_t(256, 256, 256, 256)
    # phi_q missing: rejected on the host before any launch
    st = lib.bsa_forward(C.byref(cp), fake, fake, fake, None, fake, C.byref(m), C.byref(m), None, fake,
                         C.byref(saved), fake, 1 << 40, None)
    assert st == _lib.BSA_ERR_INVALID_ARGUMENT
    assert "phi_q" in lib.bsa_last_error().decode()


def test_tree_argument_errors(lib):
    assert lib.bsa_ball_tree_workspace_bytes(100, 96, 3, 1) == 0
    assert lib.bsa_ball_tree_workspace_bytes(100, 128, 3, 1) > 0
    fake = C.c_void_p(16)
    assert lib.bsa_build_ball_tree(None, 10, 3, 16, 1, fake, fake, 1 << 20, None) == _lib.BSA_ERR_INVALID_ARGUMENT
    assert lib.bsa_build_ball_tree(fake, 10, 4, 16, 1, fake, fake, 1 << 20, None) == _lib.BSA_ERR_UNSUPPORTED
    assert lib.bsa_build_ball_tree(fake, 20, 3, 16, 1, fake, fake, 1 << 20, None) == _lib.BSA_ERR_INVALID_ARGUMENT
    assert lib.bsa_build_ball_tree(fake, 10, 3, 16, 1, fake, fake, 1, None) == _lib.BSA_ERR_WORKSPACE_TOO_SMALL


def test_set_streams_validates(lib):
    assert lib.bsa_set_streams(3) == _lib.BSA_ERR_INVALID_ARGUMENT
    assert lib.bsa_set_streams(-1) == _lib.BSA_ERR_INVALID_ARGUMENT
    assert lib.bsa_set_streams(0) == _lib.BSA_OK
    assert lib.bsa_set_streams(2) == _lib.BSA_OK


def _block_sizes(lib, p, ffn):
    a, b, c = C.c_size_t(), C.c_size_t(), C.c_size_t()
    cp = p.c()
    return lib.bsa_block_sizes(C.byref(cp), ffn, C.byref(a), C.byref(b), C.byref(c)), a.value, b.value, c.value


def test_block_sizes_and_validation(lib):
    bf = dict(dtype=_lib.BSA_BF16)
    st, wf, wb, sv = _block_sizes(lib, base(**bf), 512)        # C = 4 * 32 = 128
    assert st == _lib.BSA_OK and wf > 0 and wb > wf and sv > 0
    # the block's saved set holds the layer's
    st_l, _, sv_l = _sizes(lib, base(**bf))
    assert sv > sv_l
    assert _block_sizes(lib, base(dtype=_lib.BSA_F32), 512)[0] == _lib.BSA_ERR_UNSUPPORTED  # float32 layer
    assert _block_sizes(lib, base(heads=2, **bf), 512)[0] == _lib.BSA_ERR_UNSUPPORTED  # C = 64
    assert _block_sizes(lib, base(**bf), 100)[0] == _lib.BSA_ERR_UNSUPPORTED           # F not a multiple of 128
    assert _block_sizes(lib, base(**bf), 0)[0] == _lib.BSA_ERR_UNSUPPORTED


def test_block_struct_layout_matches_header(tmp_path):
    # the ctypes structs of the binding have the sizes the C compiler gives the header's
    src = tmp_path / "sz.c"
    src.write_text('#include "bsa.h"\n#include <stdio.h>\nint main(void) { printf("%zu %zu %zu %zu\\n", '
                   'sizeof(bsa_params_t), sizeof(bsa_saved_t), sizeof(bsa_block_weights_t), '
                   'sizeof(bsa_block_saved_t)); return 0; }\n')
    exe = tmp_path / "sz"
    import subprocess
    subprocess.run(["gcc", f"-I{os.path.join(ROOT, 'include')}", str(src), "-o", str(exe)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()]
    assert got == [C.sizeof(_lib.bsa_params_t), C.sizeof(_lib.bsa_saved_t), C.sizeof(_lib.bsa_block_weights_t),
                   C.sizeof(_lib.bsa_block_saved_t)]


def test_block_forward_rejects_before_launch(lib):
    p = base(dtype=_lib.BSA_BF16)
    cp = p.c()
    saved = _lib.bsa_block_saved_t()
    w = _lib.bsa_block_weights_t()
    fake = C.c_void_p(256)
    st = lib.bsa_block_forward(C.byref(cp), 512, C.byref(w), fake, None, C.c_void_p(512), C.byref(saved), fake,
                               1 << 40, None)
    assert st == _lib.BSA_ERR_INVALID_ARGUMENT and "weight" in lib.bsa_last_error().decode()
    st = lib.bsa_block_forward(C.byref(cp), 512, None, fake, None, fake, C.byref(saved), fake, 1 << 40, None)
    assert st == _lib.BSA_ERR_INVALID_ARGUMENT
