"""The no-allocation GEMM entry point (chimera_gemm_static) against the
allocating test hook it mirrors (chimera_debug_gemm): identical bits on two
calls in a row, the second with a smaller input, through the C ABI; and a
shape beyond the static scratch is refused before any launch."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _case(dtype, M, N, K, seed):
    import torch
    from paper_2402_15758_amd import binding as B
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(M, K, generator=g)
    w = torch.randn(K, N, generator=g) * 0.05
    if dtype == "bf16":
        x, w, code = x.to(torch.bfloat16), w.to(torch.bfloat16), B.CHIMERA_BF16
        xh, wh = x.view(torch.int16).numpy(), w.view(torch.int16).numpy()
    else:
        code = B.CHIMERA_F32
        xh, wh = x.numpy(), w.numpy()
    y_ref = np.zeros((M, N), dtype=np.float32)
    B.chimera_debug_gemm(code, xh.ctypes.data, wh.ctypes.data, M, N, K, y_ref.ctypes.data)
    xd, wd = x.cuda(), w.cuda()
    yd = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    B.chimera_gemm_static(code, xd.data_ptr(), wd.data_ptr(), M, N, K, yd.data_ptr(),
                          torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    y = yd.cpu().numpy()
    assert np.array_equal(y.view(np.uint32), y_ref.view(np.uint32)), f"{dtype} {M}x{N}x{K}"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_gemm_static_matches_the_allocating_hook(dtype):
    print(f"gemm_static {dtype}: 64x1024x2048 then 17x512x1024", flush=True)
    _case(dtype, 64, 1024, 2048, 1)   # reduction split 2 ways: partials in the scratch
    _case(dtype, 17, 512, 1024, 2)    # smaller, after the first call's contents


def test_gemm_static_refuses_shapes_beyond_the_scratch():
    from paper_2402_15758_amd import binding as B
    with pytest.raises(B.ChimeraError) as e:
        # a 4096 x 4096 bf16 weight alone fills the 32 MiB scratch; refused on
        # the host before anything is read or launched
        B.chimera_gemm_static(B.CHIMERA_BF16, 1, 1, 64, 4096, 4096, 1, 0)
    assert e.value.status == B.CHIMERA_ENOMEM
