"""The allocation-free projection entry point (vla_gemm_noalloc) against the
allocating one (vla_debug_gemm): same kernels, same K ranges, so the same
bits; two calls in a row on the shared static scratch, the second smaller,
and K-split plans whose partials do not fit the scratch rejected before any
work is enqueued."""
import ctypes

import numpy as np
import pytest

from paper_2609_12075_amd import vla


def test_noalloc_rejects_plans_beyond_the_scratch():
    """Checked on the host: a K-split plan needing 24 MiB of partials."""
    fake = ctypes.c_void_p(4096)
    st = vla.lib().vla_gemm_noalloc(1536, 2048, 16384, fake, 16384, 1, fake, 16384, 1, None, 0, fake, 2048, None)
    assert st == vla.VLA_EINVAL
    msg = vla.lib().vla_last_error().decode()
    assert "25165824 bytes of split-K partials" in msg and "16777216" in msg


# pairs of calls: a larger projection, then a smaller one on the same scratch
PAIRS = [
    ((256, 1024, 8192, "bf16"), (64, 512, 1024, "bf16")),      # long K (K ranges), then a short one
    ((800, 720, 1920, "bf16"), (100, 256, 512, "bf16")),       # action-stage-sized, then ragged-free small
    ((200, 2048, 4096, "f32"), (33, 72, 136, "bf16")),         # fp32 activations, then ragged M/N/K
]


@pytest.mark.gpu
@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: f"{p[0][:3]}->{p[1][:3]}")
def test_noalloc_matches_allocating_entry_point(pair):
    import torch
    g = torch.Generator(device="cpu").manual_seed(11)
    for (M, N, K, at) in pair:
        A = torch.randn(M, K, generator=g).to("cuda")
        A = A.to(torch.bfloat16) if at == "bf16" else A
        Wt = (torch.randn(N, K, generator=g) * 0.05).to(torch.bfloat16).cuda()
        bias = torch.randn(N, generator=g).cuda()
        for act in (0, 2):
            ref = vla.debug_gemm(A, Wt, bias=bias, act=act)
            got = torch.full_like(ref, float("nan"))
            vla.gemm_noalloc(A, Wt, bias=bias, act=act, out=got)
            torch.cuda.synchronize()
            print(f"[noalloc] M={M} N={N} K={K} A={at} act={act}", flush=True)
            assert torch.equal(got, ref), (M, N, K, at, act)
