"""GPU parity of molt_dense_gemm (the decoder's dense projections and LM head) against a
float64 product of the same bf16/f32 operands: |C - ref| <= 1e-4 * sqrt(K) * max|a||b|
(f32 accumulation), at the verify step's shapes and ragged row/column counts, with and
without split-K, on the LDS-tiled kernel (also at the fp8 layer's 2304 rows) and on the
big-tile one (the LM head)."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,N,K,dt,acc", [
    (320, 5120, 2048, torch.bfloat16, False),   # QKV at 64 x 5 tokens: 128-row tiles, ragged tail
    (640, 2048, 4096, torch.bfloat16, True),    # O projection into the residual
    (77, 128, 2048, torch.bfloat16, False),     # router, 64-row tiles
    (25, 256, 2048, torch.bfloat16, False),     # 32-row tiles
    (640, 151936, 2048, torch.bfloat16, False), # LM head
    (128, 151936, 2048, torch.bfloat16, False), # the draft head's LM head: weight-streaming kernel
    (100, 16384, 512, torch.bfloat16, False),   # streaming kernel, ragged last row block
    (20, 8192, 1024, torch.bfloat16, False),    # streaming kernel, 32-row tile
    (2304, 5120, 2048, torch.bfloat16, False),  # QKV at 2304 rows: 128-row tiles
    (2304, 2048, 4096, torch.bfloat16, True),   # O at 2304 rows, accumulate
    (1100, 2048, 4096, torch.bfloat16, True),   # ragged rows, accumulate
    (1024, 1024, 1024, torch.bfloat16, False),
    (200, 131195, 512, torch.bfloat16, True),   # many columns: ragged rows and columns, accumulate
    (130, 131104, 192, torch.bfloat16, False),  # odd slice count
    (33, 200, 128, torch.bfloat16, False),      # N not a multiple of 128
    (16, 768, 256, torch.float32, True),        # f32 model
])
def test_dense_gemm(molt_lib, M, N, K, dt, acc):
    print(f"case M={M} N={N} K={K} {dt} acc={acc}", flush=True)
    g = torch.Generator().manual_seed(M * 7 + N)
    A = torch.randn(M, K, generator=g).to(dt)
    B = (torch.randn(N, K, generator=g) * 0.02).to(dt)
    C0 = torch.randn(M, N, generator=g)
    C = molt_lib.dense_gemm(A.cuda(), B.cuda(), C0.clone().cuda() if acc else None, accumulate=acc)
    torch.cuda.synchronize()
    ref = A.double() @ B.double().T + (C0.double() if acc else 0)
    err = (C.cpu().double() - ref).abs().max().item()
    bound = 1e-4 * np.sqrt(K) * float(A.float().abs().max() * B.float().abs().max()) * 4
    print(f"max err {err:.3e} (bound {bound:.3e})", flush=True)
    assert err <= bound
