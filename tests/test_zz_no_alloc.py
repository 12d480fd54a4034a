"""gs_compress_noalloc (no allocation: the library's static scratch array)
against gs_compress with a caller workspace, through the C ABI.

Two calls in a row on the same GPU, the second with a smaller codebook, so
the second runs on scratch memory the first left behind: both must return
what the workspace entry returns for the same codebook, bit for bit (the same
kernels run in the same order on the same inputs), including rank and kept
rows.
"""
import ctypes

import pytest
import torch

from paper_2608_01528_amd import gramspace as gsm
from paper_2608_01528_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gsm.lib()


def codebook(M, D, seed, dup):
    C = wl.bipolar_codebook(M, D, seed)
    if dup:
        C, _, _ = wl.duplicate_rows(C, dup, seed)
    return C


def outputs(M, D, dt):
    """Full-capacity outputs, pre-filled with NaN / -7 so that every element
    the call must write is seen to be written."""
    Q = gsm.alloc_rows(M, D, dt, "cuda")
    R = gsm.alloc_rows(M, M, dt, "cuda")
    Q.fill_(float("nan"))
    R.fill_(float("nan"))
    kept = torch.full((M,), -7, dtype=torch.int32, device="cuda")
    cnorm = torch.full((M,), float("nan"), dtype=torch.float32, device="cuda")
    return Q, R, kept, cnorm


def via_c_abi(C, dt):
    """gs_compress_noalloc called directly through the C ABI."""
    M, D = C.shape
    Q, R, kept, cnorm = outputs(M, D, dt)
    rank = ctypes.c_int32(-1)
    L = gsm.lib()
    st = L.gs_compress_noalloc(ctypes.c_void_p(C.data_ptr()), gsm.GS_F32, M, D, C.stride(0), 1e-10,
                               ctypes.c_void_p(Q.data_ptr()), gsm._DT[dt], Q.stride(0),
                               ctypes.c_void_p(R.data_ptr()), gsm._DT[dt], R.stride(0),
                               ctypes.c_void_p(kept.data_ptr()), ctypes.c_void_p(cnorm.data_ptr()),
                               ctypes.byref(rank), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == gsm.GS_OK, L.gs_last_error().decode()
    return Q, R, rank.value, kept, cnorm


def with_workspace(C, dt):
    M, D = C.shape
    Q, R, kept, cnorm = outputs(M, D, dt)
    need = gsm.compress_workspace_bytes(M, D)
    ws = torch.full((need + 256,), 0xAB, dtype=torch.uint8, device="cuda")   # not zeroed on purpose
    base = ws.data_ptr()
    off = (-base) % 256
    rank = ctypes.c_int32(-1)
    L = gsm.lib()
    st = L.gs_compress(ctypes.c_void_p(C.data_ptr()), gsm.GS_F32, M, D, C.stride(0), 1e-10,
                       ctypes.c_void_p(Q.data_ptr()), gsm._DT[dt], Q.stride(0),
                       ctypes.c_void_p(R.data_ptr()), gsm._DT[dt], R.stride(0),
                       ctypes.c_void_p(kept.data_ptr()), ctypes.c_void_p(cnorm.data_ptr()),
                       ctypes.byref(rank), ctypes.c_void_p(base + off), need,
                       ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == gsm.GS_OK, L.gs_last_error().decode()
    return Q, R, rank.value, kept, cnorm


def same(a, b):
    """Bit-identical tensors (NaN where both hold NaN counts as equal)."""
    if a.dtype == torch.int32:
        return torch.equal(a, b)
    return torch.equal(a.view(torch.int16 if a.element_size() == 2 else
                              (torch.int32 if a.element_size() == 4 else torch.int64)),
                       b.view(torch.int16 if b.element_size() == 2 else
                              (torch.int32 if b.element_size() == 4 else torch.int64)))


@pytest.mark.parametrize("dt", [torch.float64, torch.float32, torch.bfloat16],
                         ids=["f64", "f32", "bf16"])
def test_noalloc_matches_workspace_entry_twice(dt):
    cases = [(700, 4096, 81, 0.1), (40, 1024, 82, 0.0)]     # second call smaller than the first
    for M, D, seed, dup in cases:
        print("noalloc", M, D, dup, dt, flush=True)
        C = torch.from_numpy(codebook(M, D, seed, dup)).cuda()
        got = via_c_abi(C, dt)
        ref = with_workspace(C, dt)
        torch.cuda.synchronize()
        Qg, Rg, rg, kg, cg = got
        Qr, Rr, rr, kr, cr = ref
        assert rg == rr == M - int(round(dup * M))
        assert same(kg, kr) and same(cg, cr)
        assert same(Qg, Qr) and same(Rg, Rr)
        # every capacity element was written (rows / columns past the rank are zero-filled)
        assert not torch.isnan(Qg.float()).any() and not torch.isnan(Rg.float()).any()
        assert torch.all(kg[rg:] == -1) and torch.all(kg[:rg] >= 0)
