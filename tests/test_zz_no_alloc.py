"""The allocation-free GEMM entry point (clover_op_linear_noalloc) against clover_op_linear:
the same kernels, with the split-K partials in the library's own device array instead of a
caller scratch buffer.  Two calls in a row, the second on a smaller shape (the array keeps
the first call's partials), must each equal the scratch-buffer entry point bit for bit; a
shape whose partials exceed the array is refused before anything runs."""
import pytest
import torch

from tests.gpu_util import need_gpu, note, seeded

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_noalloc_linear_equals_op_linear_on_two_calls(dt):
    P = need_gpu()
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    shapes = [(64, 4096, 4096), (13, 1024, 512)] if dt == "bf16" else [(41, 768, 256), (5, 256, 256)]
    for M, N, K in shapes:
        note(f"noalloc linear {dt} M={M} N={N} K={K}")
        assert P.lib().clover_op_scratch_bytes(1 if dt == "bf16" else 0, M, N, K) <= \
            P.lib().clover_op_linear_noalloc_max_bytes()
        X = seeded((M, K), 3000 + M, 1.0, tdt)
        W = seeded((N, K), 4000 + N, 0.02, tdt)
        Wp = P.pack_matrix(W)
        ref = P.op_linear(X, Wp, N)
        got = P.op_linear_noalloc(X, Wp, N)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), float((got - ref).abs().max())


def test_noalloc_linear_refuses_partials_beyond_its_array():
    P = need_gpu()
    note("noalloc linear capacity check")
    M, N, K = 2048, 8192, 8192
    assert P.lib().clover_op_scratch_bytes(1, M, N, K) > P.lib().clover_op_linear_noalloc_max_bytes()
    X = torch.zeros(M, K, dtype=torch.bfloat16, device="cuda")
    Wp = torch.zeros(N * K * 2, dtype=torch.uint8, device="cuda")
    with pytest.raises(P.CloverError) as e:
        P.op_linear_noalloc(X, Wp, N)
    assert e.value.status == 2
