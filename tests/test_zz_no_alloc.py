"""memoroid_scan_diag_noalloc: the forward scan on the library's static
scratch array, through the C ABI, against memoroid_scan_diag (the same scan
on a caller's workspace) and the fp64 oracle: two calls in a row, the second
on a smaller problem (the array keeps the first call's contents), plus a
bf16 batch of the size class of the 64-tape workload on the vectorised
kernels.  Floats within the parity tolerance (conditioned relative error,
1e-4 fp32, 2e-2 bf16 inputs), episode indices bit-exact."""
import numpy as np
import pytest

import oracle
from conftest import announce, cond_err
from paper_2402_09900_amd import tapes

torch = pytest.importorskip("torch")
from paper_2402_09900_amd import binding as mb  # noqa: E402

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
CODE = {"f32": mb.F32, "bf16": mb.BF16, "c64": mb.C64}
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "c64": torch.complex64}
TOL = {"f32": 1e-4, "c64": 1e-4, "bf16": 2e-2}


def to_dev(arr, kind):
    arr = np.ascontiguousarray(arr)
    if kind == "bf16":
        return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(arr).to(DEV)


def host(t):
    if t.dtype == torch.bfloat16:
        return tapes.bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return t.cpu().numpy()


def run(w, noalloc):
    """One forward scan through the C ABI; returns (h, episode_idx) on the host."""
    a, x, s = to_dev(w.a, w.dtype), to_dev(w.x, w.dtype), to_dev(w.start, "u8")
    h = torch.full((w.B, w.T, w.d), 5.0, dtype=TORCH[w.out_dtype], device=DEV)
    idx = torch.full((w.B, w.T), -7, dtype=torch.int32, device=DEV)
    stream = torch.cuda.current_stream().cuda_stream
    stride = 0 if w.a_invariant else w.d
    if noalloc:
        st = mb.memoroid_scan_diag_noalloc(a.data_ptr(), stride, x.data_ptr(), s.data_ptr(), h.data_ptr(),
                                           idx.data_ptr(), w.B, w.T, w.d, CODE[w.dtype], CODE[w.out_dtype], stream)
    else:
        nb = mb.memoroid_scan_diag_workspace_bytes(w.B, w.T, w.d, CODE[w.dtype], CODE[w.out_dtype])
        ws = torch.empty(max(nb, 256), dtype=torch.uint8, device=DEV)
        st = mb.memoroid_scan_diag(a.data_ptr(), stride, x.data_ptr(), s.data_ptr(), h.data_ptr(), idx.data_ptr(),
                                   w.B, w.T, w.d, CODE[w.dtype], CODE[w.out_dtype], ws.data_ptr(), ws.numel(),
                                   stream)
    assert st == mb.OK, mb.status_string(st)
    torch.cuda.synchronize()
    return host(h), idx.cpu().numpy()


def check_against_default(w, label):
    announce("noalloc %s B=%d T=%d d=%d %s" % (label, w.B, w.T, w.d, w.dtype))
    h_na, i_na = run(w, noalloc=True)
    h_df, i_df = run(w, noalloc=False)
    np.testing.assert_array_equal(i_na, i_df)
    np.testing.assert_array_equal(i_na, oracle.episode_idx(w.start))
    tol = TOL["bf16" if w.out_dtype == "bf16" else w.dtype]
    for b in range(w.B):
        ref, mag = oracle.diag_fwd(w.decoded("a") if w.a_invariant else w.decoded("a")[b:b + 1],
                                   w.decoded("x")[b:b + 1], w.start[b:b + 1])
        # against the existing entry point, on the oracle's scale; and against the oracle
        assert cond_err(h_na[b:b + 1], h_df[b:b + 1].astype(ref.dtype), mag) <= tol, (label, b)
        assert cond_err(h_na[b:b + 1], ref, mag) <= tol, (label, b)


def test_two_calls_second_smaller():
    big = tapes.make_custom_diag("f32", 2, 120000, 256, False, seed=4101, with_grad=False)
    check_against_default(big, "first call")
    small = tapes.make_custom_diag("c64", 1, 3001, 40, True, seed=4102, with_grad=False)
    check_against_default(small, "second call, smaller")


def test_bf16_batch_on_the_vectorised_kernels():
    w = tapes.make_diag(4, B=8, seed=4103)
    assert mb.memoroid_scan_diag_workspace_bytes(8, w.T, w.d, mb.BF16, mb.BF16) > 0
    check_against_default(w, "bf16 batch")
