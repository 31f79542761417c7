"""The C ABI on the CPU: the library loads, exports every declared symbol and
rejects bad arguments before touching the GPU.  No kernel is launched here:
every call below fails validation or is an empty problem."""
import ctypes
import glob
import os
import re
import subprocess

import pytest

from conftest import ROOT
from paper_2402_09900_amd import binding as mb

HEADER = os.path.join(ROOT, "include", "memoroid.h")
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def declared_functions():
    names = set()
    for h in HEADERS:
        src = open(h).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(memoroid_\w+)\s*\(", src))
    return sorted(names)


def test_header_compiles_as_c_and_cxx(tmp_path):
    assert HEADER in HEADERS
    for h in HEADERS:
        for lang, comp in (("c", "gcc"), ("c++", "g++")):
            subprocess.run([comp, "-x", lang, "-fsyntax-only", "-Wall", "-Werror", h], check=True)


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert "memoroid_scan_diag" in names and "memoroid_scan_linattn" in names
    assert "memoroid_workspace_bytes" in names and "memoroid_scan_diag_prepared" in names
    assert "memoroid_testing_set_fallback_polls" in names
    lib = ctypes.CDLL(mb.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    for n in names:
        assert hasattr(mb, n), "binding lacks " + n


def test_version_and_status_strings():
    assert mb.memoroid_abi_version() == 4
    for s in (mb.OK, mb.EINVAL, mb.EUNSUPPORTED, mb.EWORKSPACE, mb.EHIP, mb.ETIMEOUT, mb.EMISMATCH):
        assert mb.status_string(s) and mb.status_string(s) != "unknown status"
    assert mb.status_string(12345) == "unknown status"


def test_workspace_prepare_validation():
    # argument errors are found before any HIP call
    assert mb.memoroid_workspace_prepare(None, 4096, None) == mb.EINVAL
    assert mb.memoroid_workspace_prepare(W, 255, None) == mb.EINVAL        # smaller than the header
    assert mb.memoroid_workspace_prepare(W + 8, 4096, None) == mb.EINVAL   # not 16-byte aligned
    assert mb.memoroid_workspace_status(None, 4096, None) == mb.EINVAL


def test_prepared_workspaces_hold_two_banks():
    """The prepared entry points keep two banks of descriptor words, so their
    workspaces grow with the tile count roughly twice as fast as one bank
    would."""
    small = mb.memoroid_scan_diag_workspace_bytes(1, 1 << 16, 256, mb.C64, mb.C64)
    large = mb.memoroid_scan_diag_workspace_bytes(1, 1 << 20, 256, mb.C64, mb.C64)
    # 16x the tiles: 16 (tiles per chain) * 16 chains * 16 features * 24 bytes per bank
    per_tile_pair = (large - small) / ((1 << 20) - (1 << 16)) * 512
    assert per_tile_pair >= 2 * 16 * 16 * 24 * 0.99


def test_generic_workspace_query():
    """memoroid_workspace_bytes(op, ...) covers every dtype and flag
    combination of the entry point at those sizes."""
    q = mb.memoroid_workspace_bytes
    B, T, d = 2, 70000, 96
    assert q(mb.OP_DIAG, B, T, d, 0, 0, 0) == max(mb.memoroid_scan_diag_workspace_bytes(B, T, d, i, o) for i, o in
                                                 ((mb.F32, mb.F32), (mb.BF16, mb.BF16), (mb.BF16, mb.F32),
                                                  (mb.C64, mb.C64)))
    assert q(mb.OP_DIAG_BWD, B, T, d, 0, 0, 0) == max(mb.memoroid_scan_diag_bwd_workspace_bytes(B, T, d, dt, s)
                                                     for dt in (mb.F32, mb.C64) for s in (0, d))
    assert q(mb.OP_LINATTN, 1, 32768, 4, 64, 64, 64) == mb.memoroid_scan_linattn_workspace_bytes(32768, 4, 64, 64, 64)
    assert q(mb.OP_LINATTN_BWD, 7, 32768, 4, 64, 64, 64) == \
        mb.memoroid_scan_linattn_bwd_workspace_bytes(32768, 4, 64, 64, 64)
    assert q(mb.OP_LINATTN, 1, 32768, 4, 32, 64, 64) == 0
    assert q(mb.OP_FFM, 1, 1 << 18, 32, 8, 0, 0) == mb.memoroid_scan_ffm_workspace_bytes(1, 1 << 18, 32, 8)
    assert q(mb.OP_FFM_BWD, 1, 1 << 18, 32, 8, 0, 0) == mb.memoroid_scan_ffm_bwd_workspace_bytes(1, 1 << 18, 32, 8)
    assert q(mb.OP_RETURN, 3, 1 << 20, 0, 0, 0, 0) == mb.memoroid_discount_workspace_bytes(3, 1 << 20)
    assert q(mb.OP_GAE, 3, 1 << 20, 0, 0, 0, 0) == mb.memoroid_discount_workspace_bytes(3, 1 << 20)
    assert q(mb.OP_TBB_BEGIN_INDICES, 0, 1 << 24, 0, 0, 0, 0) == mb.memoroid_tbb_begin_indices_workspace_bytes(1 << 24)
    assert q(mb.OP_TBB_SAMPLE, 1 << 20, 1 << 20, 0, 0, 0, 0) == mb.memoroid_tbb_sample_workspace_bytes(1 << 20, 1 << 20)
    assert q(mb.OP_DIAG, -1, T, d, 0, 0, 0) == 0 and q(mb.OP_DIAG, B, 0, d, 0, 0, 0) == 0
    assert q(99, B, T, d, 0, 0, 0) == 0
    for op in range(10):
        assert q(op, 1, 4096, 64, 64, 64, 64) > 0


def test_prepared_variants_validate_like_the_defaults():
    """The *_prepared entry points reject the same bad arguments (before any
    HIP call) as the self-initialising ones."""
    for entry in (mb.memoroid_scan_diag, mb.memoroid_scan_diag_prepared):
        def call(**kw):
            args = dict(a=A, a_stride_t=8, x=X, start=S, h=H, episode_idx=None, B=2, T=100, d=8,
                        in_dtype=mb.F32, out_dtype=mb.F32, workspace=W, workspace_bytes=1 << 30, stream=None)
            args.update(kw)
            return entry(*args.values())
        assert call(B=-1) == mb.EINVAL and call(T=0) == mb.OK
        assert call(in_dtype=mb.F32, out_dtype=mb.BF16) == mb.EUNSUPPORTED
        assert call(h=X) == mb.EINVAL and call(workspace=None) == mb.EWORKSPACE
    assert mb.memoroid_scan_diag_bwd_prepared(A, 8, S, H, X, X, None, 1, 50, 8, mb.F32, W, 1 << 30, None) == mb.EINVAL
    assert mb.memoroid_scan_ffm_prepared(A, X, S, H + 0x100, I + 4, None, 2, 100, 4, 3, W, 1 << 30, None) == mb.EINVAL
    assert mb.memoroid_scan_ffm_bwd_prepared(A, X, S, H, I, 0x90000, None, None, 1, 100, 4, 3, W, 1 << 30,
                                             None) == mb.EUNSUPPORTED
    assert mb.memoroid_discounted_return_prepared(A, S, 1.5, H, 2, 100, W, 1 << 30, None) == mb.EINVAL
    assert mb.memoroid_gae_prepared(A, X, None, None, S, 0.99, 0.95, H, I, 2, 100, None, 0, None) == mb.EWORKSPACE
    assert mb.memoroid_tbb_begin_indices_prepared(S, -1, 0, I, A, W, 1 << 30, None) == mb.EINVAL
    assert mb.memoroid_tbb_sample_prepared(A, 1000, 0, X, 10, S, 100, 500, H, I, None, None, W, 1 << 30,
                                           None) == mb.EINVAL


def test_fallback_control_round_trips():
    old = mb.memoroid_testing_set_fallback_polls(0)
    assert old == 4096
    assert mb.memoroid_testing_set_fallback_polls(17) == 0
    assert mb.memoroid_testing_set_fallback_polls(-1) == 17
    assert mb.memoroid_testing_set_fallback_polls(-1) == 4096


def test_workspace_queries():
    f = mb.memoroid_scan_diag_workspace_bytes
    assert f(1, 1 << 20, 256, mb.F32, mb.F32) > 0
    assert f(64, 16384, 512, mb.BF16, mb.BF16) > 0
    assert f(1, 65536, 256, mb.C64, mb.C64) > 0
    assert f(1, 100, 8, mb.F32, mb.BF16) == 0          # unsupported pair
    assert f(1, 100, 8, mb.C64, mb.F32) == 0
    assert f(-1, 100, 8, mb.F32, mb.F32) == 0
    assert f(0, 100, 8, mb.F32, mb.F32) == 0            # empty problem needs nothing
    g = mb.memoroid_scan_diag_bwd_workspace_bytes
    assert g(1, 65536, 256, mb.C64, 0) > 0 and g(1, 65536, 256, mb.C64, 256) > 0
    assert g(4, 65536, 256, mb.C64, 0) > 4 * g(1, 65536, 256, mb.C64, 0) // 2   # da partial rows per tape
    assert g(1, 100, 8, mb.BF16, 8) == 0
    h = mb.memoroid_scan_linattn_workspace_bytes
    assert h(32768, 4, 64, 64, 64) > 0
    assert h(32768, 4, 32, 64, 64) == 0
    # descriptor storage grows linearly in T
    assert f(1, 1 << 21, 256, mb.F32, mb.F32) < 2.2 * f(1, 1 << 20, 256, mb.F32, mb.F32)


# fake, well-aligned device addresses: validation must reject the call before
# any of them is dereferenced or any HIP call is made
A, X, S, H, W, I = 0x10000, 0x20000, 0x30000, 0x40000, 0x50000, 0x60000


def diag(**kw):
    args = dict(a=A, a_stride_t=8, x=X, start=S, h=H, episode_idx=None, B=2, T=100, d=8,
                in_dtype=mb.F32, out_dtype=mb.F32, workspace=W, workspace_bytes=1 << 30, stream=None)
    args.update(kw)
    return mb.memoroid_scan_diag(*args.values())


def test_diag_validation():
    assert diag(B=-1) == mb.EINVAL
    assert diag(T=-5) == mb.EINVAL
    assert diag(B=0) == mb.OK and diag(T=0) == mb.OK and diag(d=0) == mb.OK
    assert diag(in_dtype=mb.F32, out_dtype=mb.BF16) == mb.EUNSUPPORTED
    assert diag(in_dtype=7) == mb.EUNSUPPORTED
    assert diag(x=None) == mb.EINVAL
    assert diag(a=None) == mb.EINVAL
    assert diag(start=None) == mb.EINVAL
    assert diag(h=None) == mb.EINVAL
    assert diag(a_stride_t=3) == mb.EINVAL
    assert diag(x=X + 2) == mb.EINVAL                   # misaligned f32
    assert diag(h=X) == mb.EINVAL                       # output aliases input
    assert diag(episode_idx=H) == mb.EINVAL
    assert diag(workspace=None) == mb.EWORKSPACE
    need = mb.memoroid_scan_diag_workspace_bytes(2, 100, 8, mb.F32, mb.F32)
    assert diag(workspace_bytes=need - 1) == mb.EWORKSPACE
    assert diag(B=1 << 40, T=1 << 40) == mb.EINVAL      # extent overflow
    assert diag(in_dtype=mb.C64, out_dtype=mb.C64, x=X + 4) == mb.EINVAL


def test_diag_bwd_validation():
    def bwd(**kw):
        args = dict(a=A, a_stride_t=8, start=S, h=H, grad_h=X, grad_x=I, grad_a=W + 0x1000, B=1, T=50,
                    d=8, dtype=mb.F32, workspace=W, workspace_bytes=1 << 30, stream=None)
        args.update(kw)
        return mb.memoroid_scan_diag_bwd(*args.values())
    assert bwd(dtype=mb.BF16) == mb.EUNSUPPORTED
    assert bwd(T=0) == mb.OK
    assert bwd(grad_x=X) == mb.EINVAL                   # aliases grad_h
    assert bwd(h=None) == mb.EINVAL                     # grad_a needs h
    assert bwd(a_stride_t=2) == mb.EINVAL
    assert bwd(workspace=None) == mb.EWORKSPACE
    assert bwd(workspace_bytes=16) == mb.EWORKSPACE


def test_linattn_validation():
    def la(**kw):
        args = dict(q=A, k=X, v=S, start=H + 0x100, out=I, episode_idx=None, T=1000, H=4, dk=64, dv=64,
                    chunk=64, workspace=W, workspace_bytes=1 << 30, stream=None)
        args.update(kw)
        return mb.memoroid_scan_linattn(*args.values())
    assert la(dk=32) == mb.EUNSUPPORTED
    assert la(chunk=128) == mb.EUNSUPPORTED
    assert la(T=0) == mb.OK
    assert la(out=A) == mb.EINVAL
    assert la(q=A + 4) == mb.EINVAL
    assert la(workspace=None) == mb.EWORKSPACE
    assert la(workspace_bytes=1000) == mb.EWORKSPACE


def test_linattn_bwd_validation():
    def lb(**kw):
        args = dict(q=A, k=X, v=S, start=H + 0x100, out=I, grad_out=W + 0x100000, grad_q=0x90000, grad_k=0xA0000,
                    grad_v=0xB0000, T=1000, H=4, dk=64, dv=64, chunk=64, workspace=W, workspace_bytes=1 << 30,
                    stream=None)
        args.update(kw)
        return mb.memoroid_scan_linattn_bwd(*args.values())
    assert mb.memoroid_scan_linattn_bwd_workspace_bytes(32768, 4, 64, 64, 64) > \
        mb.memoroid_scan_linattn_workspace_bytes(32768, 4, 64, 64, 64)
    assert lb(dk=32) == mb.EUNSUPPORTED and lb(chunk=32) == mb.EUNSUPPORTED
    assert lb(T=0) == mb.OK and lb(T=-1) == mb.EINVAL
    assert lb(q=None) == mb.EINVAL and lb(grad_out=None) == mb.EINVAL and lb(grad_v=None) == mb.EINVAL
    assert lb(grad_q=A) == mb.EINVAL and lb(grad_k=0x90000) == mb.EINVAL     # aliasing
    assert lb(q=A + 4) == mb.EINVAL
    assert lb(workspace=None) == mb.EWORKSPACE and lb(workspace_bytes=4096) == mb.EWORKSPACE


def test_ffm_validation():
    def ffm(**kw):
        args = dict(alpha=A, omega=X, x=S, start=H + 0x100, S=I, episode_idx=None, B=2, T=100, m=4, c=3,
                    workspace=W, workspace_bytes=1 << 30, stream=None)
        args.update(kw)
        return mb.memoroid_scan_ffm(*args.values())
    assert mb.memoroid_scan_ffm_workspace_bytes(1, 1 << 18, 32, 8) > 0
    assert mb.memoroid_scan_ffm_workspace_bytes(1, 100, 0, 8) == 0
    assert ffm(B=-1) == mb.EINVAL
    assert ffm(T=0) == mb.OK and ffm(m=0) == mb.OK and ffm(c=0) == mb.OK
    assert ffm(alpha=None) == mb.EINVAL and ffm(omega=None) == mb.EINVAL and ffm(x=None) == mb.EINVAL
    assert ffm(S=None) == mb.EINVAL and ffm(start=None) == mb.EINVAL
    assert ffm(S=I + 4) == mb.EINVAL                    # complex64 needs 8-byte alignment
    assert ffm(x=S + 2) == mb.EINVAL
    assert ffm(S=S) == mb.EINVAL                        # output aliases x
    assert ffm(workspace=None) == mb.EWORKSPACE
    assert ffm(workspace_bytes=100) == mb.EWORKSPACE
    assert ffm(m=1 << 30, c=1 << 30) == mb.EINVAL       # extent overflow


def test_tbb_validation():
    def bi(**kw):
        args = dict(start=S, n=1000, offset=0, indices=I, count=A, workspace=W, workspace_bytes=1 << 30,
                    stream=None)
        args.update(kw)
        return mb.memoroid_tbb_begin_indices(*args.values())

    def sm(**kw):
        args = dict(D=A, n_D=1000, row_bytes=64, I=X, n_I=10, draws=S, n_draws=100, batch=500, out=H,
                    out_start=I, out_src=None, filled=None, workspace=W, workspace_bytes=1 << 30, stream=None)
        args.update(kw)
        return mb.memoroid_tbb_sample(*args.values())
    assert mb.memoroid_tbb_begin_indices_workspace_bytes(1 << 24) > 256
    assert mb.memoroid_tbb_sample_workspace_bytes(0, 10) > 0 and mb.memoroid_tbb_sample_workspace_bytes(-1, 10) == 0
    assert mb.memoroid_tbb_sample_workspace_bytes(10, -1) == 0 and mb.memoroid_tbb_sample_workspace_bytes(10, 1 << 47) == 0
    assert mb.memoroid_tbb_sample_workspace_bytes(1 << 20, 1 << 20) >= (1 << 20) * 16
    assert bi(n=-1) == mb.EINVAL and bi(n=1 << 31) == mb.EUNSUPPORTED
    assert bi(count=None) == mb.EINVAL and bi(start=None) == mb.EINVAL and bi(indices=None) == mb.EINVAL
    assert bi(count=A + 4) == mb.EINVAL and bi(indices=S) == mb.EINVAL
    assert bi(workspace=None) == mb.EWORKSPACE and bi(workspace_bytes=16) == mb.EWORKSPACE
    assert sm(row_bytes=0) == mb.EINVAL and sm(batch=-1) == mb.EINVAL and sm(n_draws=-1) == mb.EINVAL
    assert sm(n_draws=(1 << 24) + 1) == mb.EUNSUPPORTED
    assert sm(I=None) == mb.EINVAL and sm(draws=None) == mb.EINVAL and sm(n_I=0) == mb.EINVAL
    assert sm(out=None) == mb.EINVAL and sm(out_start=None) == mb.EINVAL
    assert sm(out=A) == mb.EINVAL                       # batch aliases D
    assert sm(I=X + 4) == mb.EINVAL
    assert sm(workspace=None) == mb.EWORKSPACE and sm(workspace_bytes=8) == mb.EWORKSPACE
    assert sm(batch=1 << 62) == mb.EINVAL               # batch * row_bytes overflows
    assert sm(batch=1 << 47, row_bytes=1) == mb.EUNSUPPORTED and sm(n_D=1 << 47, row_bytes=1) == mb.EUNSUPPORTED
    assert sm(workspace_bytes=mb.memoroid_tbb_sample_workspace_bytes(100, 500) - 1) == mb.EWORKSPACE


def test_ffm_bwd_validation():
    def fb(**kw):
        args = dict(alpha=A, omega=X, start=S, S=H, grad_S=I, grad_x=0x90000, grad_alpha=0xA0000,
                    grad_omega=0xB0000, B=1, T=100, m=4, c=4, workspace=W, workspace_bytes=1 << 30, stream=None)
        args.update(kw)
        return mb.memoroid_scan_ffm_bwd(*args.values())
    assert mb.memoroid_scan_ffm_bwd_workspace_bytes(1, 1 << 18, 32, 8) > 0
    assert fb(T=0) == mb.OK and fb(B=-1) == mb.EINVAL
    assert fb(c=3) == mb.EUNSUPPORTED and fb(c=32) == mb.EUNSUPPORTED
    assert fb(S=None) == mb.EINVAL                           # parameter grads need S
    assert fb(grad_x=None) == mb.EINVAL and fb(grad_S=None) == mb.EINVAL
    assert fb(grad_x=I) == mb.EINVAL and fb(grad_alpha=0x90000) == mb.EINVAL   # aliasing
    assert fb(grad_S=I + 4) == mb.EINVAL
    assert fb(workspace=None) == mb.EWORKSPACE and fb(workspace_bytes=64) == mb.EWORKSPACE


def test_discount_validation():
    def ret(**kw):
        args = dict(r=A, start=S, gamma=0.99, G=H, B=2, T=100, workspace=W, workspace_bytes=1 << 30, stream=None)
        args.update(kw)
        return mb.memoroid_discounted_return(*args.values())

    def gae(**kw):
        args = dict(r=A, value=X, value_next=None, done=None, start=S, gamma=0.99, lam=0.95, adv=H, target=I,
                    B=2, T=100, workspace=W, workspace_bytes=1 << 30, stream=None)
        args.update(kw)
        return mb.memoroid_gae(*args.values())
    assert mb.memoroid_discount_workspace_bytes(1, 1 << 24) > mb.memoroid_discount_workspace_bytes(1, 4096) > 0
    assert mb.memoroid_discount_workspace_bytes(0, 10) == 0
    for f in (ret, gae):
        assert f(B=-1) == mb.EINVAL
        assert f(B=0) == mb.OK and f(T=0) == mb.OK
        assert f(gamma=1.5) == mb.EINVAL and f(gamma=-0.1) == mb.EINVAL and f(gamma=float("nan")) == mb.EINVAL
        assert f(r=None) == mb.EINVAL and f(start=None) == mb.EINVAL
        assert f(r=A + 2) == mb.EINVAL                 # misaligned f32
        assert f(workspace=None) == mb.EWORKSPACE
        assert f(workspace_bytes=64) == mb.EWORKSPACE
        assert f(B=1 << 40, T=1 << 40) == mb.EINVAL
    assert ret(G=A) == mb.EINVAL                       # output aliases input
    assert ret(G=None) == mb.EINVAL
    assert gae(lam=2.0) == mb.EINVAL
    assert gae(value=None) == mb.EINVAL and gae(adv=None) == mb.EINVAL
    assert gae(adv=X) == mb.EINVAL and gae(target=A) == mb.EINVAL and gae(target=H) == mb.EINVAL
    assert gae(value_next=0x70000, done=0x80000, target=None, B=0) == mb.OK


def test_torch_layer_rejects_cpu_tensors():
    torch = pytest.importorskip("torch")
    a = torch.rand(4, 8)
    with pytest.raises(ValueError):
        mb.scan_diag(a, torch.rand(4, 8), torch.zeros(4, dtype=torch.uint8))


def test_noalloc_rejects_before_any_hip_call():
    """memoroid_scan_diag_noalloc validates like memoroid_scan_diag and
    rejects a tiling larger than its fixed scratch array with EWORKSPACE,
    all before touching the GPU."""
    def na(**kw):
        args = dict(a=A, a_stride_t=8, x=X, start=S, h=H, episode_idx=None, B=2, T=100, d=8,
                    in_dtype=mb.F32, out_dtype=mb.F32, stream=None)
        args.update(kw)
        return mb.memoroid_scan_diag_noalloc(*args.values())
    assert na(B=-1) == mb.EINVAL and na(T=0) == mb.OK and na(d=0) == mb.OK
    assert na(in_dtype=mb.F32, out_dtype=mb.BF16) == mb.EUNSUPPORTED
    assert na(h=X) == mb.EINVAL and na(x=None) == mb.EINVAL and na(a_stride_t=3) == mb.EINVAL
    # 64 tapes x 65536 steps x 512 bf16 features: about 4 x 48 MiB of tiles' words
    assert na(B=64, T=65536, d=512, a_stride_t=512, in_dtype=mb.BF16, out_dtype=mb.BF16) == mb.EWORKSPACE
    assert na(B=1, T=1 << 24, d=256, a_stride_t=256) == mb.EWORKSPACE
    assert mb.memoroid_scan_diag_workspace_bytes(1, 1 << 20, 256, mb.F32, mb.F32) <= mb.NOALLOC_SCRATCH_BYTES
    m = re.search(r"#define MEMOROID_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == mb.NOALLOC_SCRATCH_BYTES
