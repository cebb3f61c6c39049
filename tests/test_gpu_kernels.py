"""Per-kernel parity on the GPU (through the C ABI's test hooks): the
projection kernel and the prefix-KV attention kernel against numpy fp64 on
the same (bf16-representable) inputs, at the shapes of the VLA stages plus
ragged edges; and the placement of work on CU-masked streams."""
import numpy as np
import pytest

from oracle import vla as O
from tests.gpu_util import log

pytestmark = pytest.mark.gpu

RNG = np.random.default_rng(2024)


def _bf16(a):
    return O.bf16_round(np.asarray(a, np.float32))


GEMM_SHAPES = [
    # (M, N, K): stage shapes and ragged edges
    (1, 16, 8), (17, 32, 592), (50, 720, 720), (130, 200, 64), (300, 1000, 264), (4, 6144, 1024),
    (800, 3840, 720), (3840, 960, 960), (240, 1600, 960), (37, 33, 40),
    # multi-stage kernel tiles: 256x128 with a K tail, 128x128 with a K tail,
    # 256x128 with ragged M, N and K
    (2048, 4096, 592), (2048, 2048, 4304), (4000, 5000, 200),
    # small-M kernel: one and two weight-row subtiles, K tails, several K
    # rounds, ragged N; 1024-1535 weight rows with K <= 1024 (ragged)
    (50, 3840, 720), (17, 1600, 1000), (63, 1537, 3000), (64, 8192, 1024), (17, 1024, 1024), (60, 1200, 1000),
    # K ranges of the LDS-staged kernel (partial + ordered reduce), ragged
    (800, 720, 1920), (600, 1000, 1544),
    # register-pipelined 64 x 32 tiles with K ranges
    (100, 1024, 4096), (200, 720, 1920),
    # large-tile kernel (K >= 2048): 224-row tiles (2600 rows: 12 row tiles
    # fill one round as 11 of 256 rows would) with ragged M, N and K, and
    # 256-row tiles (3584 rows: 224-row tiles would need a second round)
    (2600, 4100, 2056), (3584, 4600, 2056),
    # staged 64 x 64 tiles (short K, mid-sized M), ragged
    (800, 1600, 720), (431, 2500, 1000),
    # two wave groups per K-step of 128: 128 x 128 tiles, ragged M, N and K;
    # 64 x 64 tiles with two and four K ranges (two and three stages), ragged
    (777, 3000, 1000), (390, 1000, 4000), (130, 700, 1800), (300, 700, 1800),
    # a few hundred rows with K past 4096: LDS-staged tiles with K ranges
    # (the GR00T-like LLM MLP down and ViT MLP down at batch 1), ragged M
    (296, 2048, 16384), (256, 1152, 4304), (65, 1000, 8200),
]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("a_fp32", [False, True])
def test_gemm_bf16(M, N, K, a_fp32):
    import torch
    from paper_2609_12075_amd import vla
    log(f"[gemm bf16] M={M} N={N} K={K} a_fp32={a_fp32}")
    A = RNG.standard_normal((M, K)).astype(np.float32)
    W = _bf16(RNG.standard_normal((N, K)) * 0.05)
    bias = RNG.standard_normal(N).astype(np.float32)
    Ab = _bf16(A)
    ref = Ab.astype(np.float64) @ W.astype(np.float64).T + bias
    At = torch.from_numpy(A).cuda() if a_fp32 else torch.from_numpy(Ab).to(torch.bfloat16).cuda()
    Wt = torch.from_numpy(W).to(torch.bfloat16).cuda()
    out = vla.debug_gemm(At, Wt, bias=torch.from_numpy(bias).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    scale = np.sqrt(K) * 0.05 * 1.0 + 1.0
    np.testing.assert_allclose(got, ref, rtol=1e-4, atol=1e-5 * scale)


@pytest.mark.parametrize("act", [1, 2])
@pytest.mark.parametrize("amp", [1.0, 40.0])
def test_gemm_activations(act, amp):
    """SiLU and tanh-form GELU epilogues against fp64; amp = 40 drives the
    pre-activations to about +-100, where e^-x (SiLU) and e^-2u (GELU)
    overflow to +inf or vanish: outputs must stay finite and tend to -0 / x."""
    import torch
    from paper_2609_12075_amd import vla
    M, N, K = 70, 96, 128
    A = _bf16(RNG.standard_normal((M, K)) * amp)
    W = _bf16(RNG.standard_normal((N, K)) * 0.2)
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    ref = O.silu(ref) if act == 1 else O.gelu_tanh(ref)
    out = vla.debug_gemm(torch.from_numpy(A).to(torch.bfloat16).cuda(), torch.from_numpy(W).to(torch.bfloat16).cuda(),
                         act=act)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.isfinite(got).all()
    np.testing.assert_allclose(got, ref, rtol=2e-4, atol=2e-5 * amp)


@pytest.mark.parametrize("M,N,K", [
    # large-tile kernel, epilogue from registers: 224-row tiles with ragged M,
    # K and a last weight tile holding one 16-column group; 256-row tiles
    (2600, 4112, 2056), (3584, 4608, 2048),
    # large-tile kernel through LDS (N % 16 != 0)
    (3584, 4600, 2048),
    # large tiles below K = 2048 (full rounds of tiles, output from registers)
    (16384, 3072, 768),
    # staged 128 x 128 and 128 x 64 tiles from registers, ragged N; through LDS
    (4000, 1616, 640), (1500, 1616, 640), (4000, 1608, 640),
    # small-M kernel (LDS epilogue)
    (50, 8192, 1024),
])
@pytest.mark.parametrize("glu,act", [(1, 0), (0, 2), (0, 0)])
def test_gemm_bf16_out(M, N, K, glu, act):
    """bf16-output projections, gated-GELU (interleaved gate/up rows) or a
    plain store with or without an activation, against fp64 on sampled rows;
    every element of the default output bit-equal to a run whose output rows
    are only 4-byte aligned (the per-element epilogue), and nothing written
    outside the output view."""
    _check_bf16_out(M, N, K, glu, act, rms=False)


@pytest.mark.parametrize("M,N,K,glu", [
    # folded RMSNorm: staged 128 x 64 tiles from registers (the action
    # stage's gate/up at batch 16), ragged N; 64 x 64 tiles with two wave
    # groups and the small-M kernel through LDS
    (800, 3840, 720, 1), (1500, 1616, 640, 1), (1500, 1616, 640, 0), (400, 3840, 720, 1), (50, 3840, 720, 1),
])
def test_gemm_bf16_out_rms(M, N, K, glu):
    """The same with the RMSNorm of the input rows folded into the product
    (rows of different scales and one all-zero row)."""
    _check_bf16_out(M, N, K, glu, 0, rms=True)


def _check_bf16_out(M, N, K, glu, act, rms):
    import torch
    from paper_2609_12075_amd import vla
    log(f"[gemm bf16 out] M={M} N={N} K={K} glu={glu} act={act} rms={rms}")
    A = RNG.standard_normal((M, K))
    if rms:
        A = A * np.exp(RNG.uniform(-2, 2, (M, 1)))
        A[M // 2] = 0.0
    A = _bf16(A)
    W = _bf16(RNG.standard_normal((N, K)) * 0.05)
    bias = (RNG.standard_normal(N) * 0.3).astype(np.float32)
    At = torch.from_numpy(A).to(torch.bfloat16).cuda()
    Wt = torch.from_numpy(W).to(torch.bfloat16).cuda()
    bt = torch.from_numpy(bias).cuda()
    No = N // 2 if glu else N
    eps = 1e-6
    out = vla.debug_gemm_bf16(At, Wt, bt, glu=glu, act=act, rms=rms, eps=eps)
    wide = torch.full((M, No + 8), float("nan"), dtype=torch.bfloat16, device="cuda")
    vla.debug_gemm_bf16(At, Wt, bt, glu=glu, act=act, rms=rms, eps=eps, out=wide[:, 2:2 + No])
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    assert torch.equal(out.view(torch.int16), wide[:, 2:2 + No].view(torch.int16))
    assert torch.isnan(wide[:, :2].float()).all() and torch.isnan(wide[:, 2 + No:].float()).all()
    rows = np.unique(np.concatenate([np.arange(min(M, 24)), RNG.integers(0, M, 40), np.arange(max(0, M - 24), M)]))
    A64 = A[rows].astype(np.float64)
    D = A64 @ W.astype(np.float64).T
    if rms:
        D = D / np.sqrt((A64 * A64).mean(axis=1, keepdims=True) + eps)
    D = D + bias
    if glu:
        ref = O.gelu_tanh(D[:, 0::2]) * D[:, 1::2]
    else:
        ref = O.gelu_tanh(D) if act == 2 else D
    scale = np.abs(ref).max()
    np.testing.assert_allclose(got[rows], ref, rtol=8e-3, atol=2e-3 * scale)


@pytest.mark.parametrize("M,N,K", [(8, 7, 128), (80, 768, 256), (5, 128, 7), (65, 130, 1024), (17, 1024, 1024)])
def test_gemm_f32(M, N, K):
    import torch
    from paper_2609_12075_amd import vla
    A = RNG.standard_normal((M, K)).astype(np.float32)
    W = RNG.standard_normal((N, K)).astype(np.float32)
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    out = vla.debug_gemm(torch.from_numpy(A).cuda(), torch.from_numpy(W).cuda())
    torch.cuda.synchronize()
    np.testing.assert_allclose(out.cpu().numpy(), ref, rtol=1e-5, atol=1e-5 * np.sqrt(K))


@pytest.mark.parametrize("M,N,K,kind", [(50, 720, 960, 0), (50, 720, 1920, 0), (800, 720, 1920, 0),
                                          (17, 1024, 4096, 2), (200, 1024, 2048, 1), (3840, 960, 960, 0),
                                          (7, 36, 72, 1), (400, 720, 1920, 2), (296, 2048, 16384, 0),
                                          (256, 1152, 4304, 1), (768, 1152, 4304, 0)])
def test_resid_norm(M, N, K, kind):
    """Residual projection + row norm (fused into the split-K reduce when
    the projection splits K) against fp64."""
    import torch
    from paper_2609_12075_amd import vla
    log(f"[resid_norm] M={M} N={N} K={K} kind={kind}")
    A = _bf16(RNG.standard_normal((M, K)))
    W = _bf16(RNG.standard_normal((N, K)) * 0.05)
    x0 = RNG.standard_normal((M, N)).astype(np.float32)
    bias = RNG.standard_normal(N).astype(np.float32) * 0.1
    gate = (1 + 0.1 * RNG.standard_normal(N)).astype(np.float32) if kind == 2 else None
    g = (1 + 0.1 * RNG.standard_normal(N)).astype(np.float32) if kind != 1 else None
    b = (0.1 * RNG.standard_normal(N)).astype(np.float32) if kind == 2 else None
    y = A.astype(np.float64) @ W.astype(np.float64).T + bias
    if gate is not None:
        y = y * gate
    x_ref = x0.astype(np.float64) + y
    if kind == 0:
        z_ref = O.rmsnorm(x_ref, g.astype(np.float64), 1e-6)
    else:
        z_ref = O.layernorm(x_ref, None, None, 1e-6)
        if kind == 2:
            z_ref = z_ref * (1 + g) + b
    t = lambda a: None if a is None else torch.from_numpy(a).cuda()
    x = t(x0)
    z = vla.debug_resid_norm(torch.from_numpy(A).to(torch.bfloat16).cuda(), torch.from_numpy(W).to(torch.bfloat16).cuda(),
                             x, kind, g=t(g), b=t(b), bias=t(bias), gate=t(gate))
    torch.cuda.synchronize()
    np.testing.assert_allclose(x.cpu().numpy(), x_ref, rtol=1e-4, atol=1e-4)
    zg = z.float().cpu().numpy()
    assert np.abs(zg - z_ref).max() < 2e-2 * np.abs(z_ref).max(), np.abs(zg - z_ref).max()


RMS_SHAPES = [
    # small-M kernel, ragged; 64 x 64 tiles with three and two stages; 128 x 128
    # tiles with two wave groups, ragged; 128 x 64 and 128 x 128 tiles with
    # K-steps of 64; shapes whose unfolded plan would split K or take the
    # register-pipelined or large-tile kernel
    (50, 3840, 720), (17, 1600, 1000), (100, 1600, 720), (400, 3840, 720), (777, 3000, 1000),
    (800, 3840, 720), (1600, 3840, 720), (37, 33, 40), (200, 720, 1920), (2600, 4100, 2056),
]


@pytest.mark.parametrize("M,N,K", RMS_SHAPES)
def test_gemm_rms(M, N, K):
    """Projection with the RMSNorm of its input rows folded in, against fp64:
    rows of different scales, one all-zero row (its scale is 1/sqrt(eps))."""
    import torch
    from paper_2609_12075_amd import vla
    log(f"[gemm rms] M={M} N={N} K={K}")
    eps = 1e-6
    A = RNG.standard_normal((M, K)) * np.exp(RNG.uniform(-2, 2, (M, 1)))
    A[M // 2] = 0.0
    A = _bf16(A)
    W = _bf16(RNG.standard_normal((N, K)) * 0.05)
    bias = RNG.standard_normal(N).astype(np.float32)
    A64 = A.astype(np.float64)
    r = 1.0 / np.sqrt((A64 * A64).mean(axis=1) + eps)
    ref = r[:, None] * (A64 @ W.astype(np.float64).T) + bias
    out = vla.debug_gemm_rms(torch.from_numpy(A).to(torch.bfloat16).cuda(), torch.from_numpy(W).to(torch.bfloat16).cuda(),
                             bias=torch.from_numpy(bias).cuda(), eps=eps)
    torch.cuda.synchronize()
    scale = np.sqrt(K) * 0.05 + 1.0
    np.testing.assert_allclose(out.cpu().numpy(), ref, rtol=1e-4, atol=1e-5 * scale)


@pytest.mark.parametrize("M,N,K", [
    # register-pipelined kernel; 64 x 64 tiles with two wave groups (the
    # residual update from registers); ragged, per-element epilogue
    (50, 720, 1920), (800, 720, 1920), (800, 720, 960), (37, 33, 40), (130, 202, 64),
    # staged 128 x 64 and 128 x 128 tiles (LDS-staged update), ragged
    (3840, 960, 960), (2000, 1156, 1000), (4000, 1156, 640),
    # 128 x 128 tiles with two wave groups and K-steps of 128 (update from registers)
    (777, 3000, 1000),
])
def test_resid_copy(M, N, K):
    """Residual projection with the bf16 copy of the updated rows: x against
    fp64, the copy bit-identical to x rounded to bf16; x and the copy
    bit-identical to a run on rows that are not 16-byte aligned (the
    per-element epilogue), nothing written outside the rows."""
    import torch
    from paper_2609_12075_amd import vla
    log(f"[resid copy] M={M} N={N} K={K}")
    A = _bf16(RNG.standard_normal((M, K)))
    W = _bf16(RNG.standard_normal((N, K)) * 0.05)
    x0 = RNG.standard_normal((M, N)).astype(np.float32)
    bias = RNG.standard_normal(N).astype(np.float32) * 0.1
    gate = (1 + 0.1 * RNG.standard_normal(N)).astype(np.float32)
    x_ref = x0.astype(np.float64) + (A.astype(np.float64) @ W.astype(np.float64).T + bias) * gate
    At = torch.from_numpy(A).to(torch.bfloat16).cuda()
    Wt = torch.from_numpy(W).to(torch.bfloat16).cuda()
    bt, gt = torch.from_numpy(bias).cuda(), torch.from_numpy(gate).cuda()
    x = torch.from_numpy(x0).cuda()
    xb = vla.debug_resid_copy(At, Wt, x, bias=bt, gate=gt)
    # the same update on rows 4-byte aligned only (x and its copy)
    xw = torch.full((M, N + 5), float("nan"), dtype=torch.float32, device="cuda")
    xw[:, 1:1 + N] = torch.from_numpy(x0).cuda()
    xbw = torch.full((M, N + 3), float("nan"), dtype=torch.bfloat16, device="cuda")
    vla.debug_resid_copy(At, Wt, xw[:, 1:1 + N], bias=bt, gate=gt, xb=xbw[:, 1:1 + N])
    torch.cuda.synchronize()
    np.testing.assert_allclose(x.cpu().numpy(), x_ref, rtol=1e-4, atol=1e-4)
    assert torch.equal(xb.cpu(), x.cpu().to(torch.bfloat16))
    assert torch.equal(x.view(torch.int32), xw[:, 1:1 + N].contiguous().view(torch.int32))
    assert torch.equal(xb.view(torch.int16), xbw[:, 1:1 + N].contiguous().view(torch.int16))
    assert torch.isnan(xw[:, 0]).all() and torch.isnan(xw[:, 1 + N:]).all()
    assert torch.isnan(xbw[:, 0].float()).all() and torch.isnan(xbw[:, 1 + N:].float()).all()


ATTN_SHAPES = [
    # (B, Hq, Hkv, Lq, hd, len0, len1)
    (2, 8, 1, 50, 256, 816, 50),     # pi0-shaped action decode
    (1, 8, 1, 100, 256, 100, 0),     # pi0-shaped prefill (short prefix)
    (1, 15, 5, 240, 64, 240, 0),     # SmolVLA-shaped prefill
    (2, 15, 5, 50, 64, 240, 50),     # SmolVLA-shaped action decode
    (3, 16, 16, 256, 72, 256, 0),    # ViT per image, head dim 72
    (2, 32, 32, 17, 32, 17, 0),      # DiT self-attention
    (2, 32, 32, 17, 32, 296, 0),     # DiT cross-attention
    (1, 4, 2, 7, 64, 5, 3),          # ragged, tiny
    (1, 2, 1, 1, 8, 1, 0),           # single key
    # many blocks (one key group per block): prefill-sized grids
    (8, 15, 5, 240, 64, 240, 0),
    (24, 8, 1, 100, 256, 150, 7),
    (70, 4, 1, 64, 128, 70, 0),
    # head dim 128 with key groups, two segments
    (2, 4, 2, 40, 128, 200, 10),
]


def _attn_ref(q, k0, v0, k1, v1):
    B, Hq, Lq, hd = q.shape
    out = np.zeros((B, Lq, Hq * hd))
    for b in range(B):
        k = k0[b] if k1 is None else np.concatenate([k0[b], k1[b]], axis=1)
        v = v0[b] if v1 is None else np.concatenate([v0[b], v1[b]], axis=1)
        out[b] = O.merge(O.attention(q[b].astype(np.float64), k.astype(np.float64), v.astype(np.float64)))
    return out


@pytest.mark.parametrize("B,Hq,Hkv,Lq,hd,len0,len1", ATTN_SHAPES)
def test_attention_bf16(B, Hq, Hkv, Lq, hd, len0, len1):
    import torch
    from paper_2609_12075_amd import vla
    log(f"[attn bf16] B={B} Hq={Hq} Hkv={Hkv} Lq={Lq} hd={hd} len0={len0} len1={len1}")
    q = _bf16(RNG.standard_normal((B, Hq, Lq, hd)))
    k0 = _bf16(RNG.standard_normal((B, Hkv, len0, hd)))
    v0 = _bf16(RNG.standard_normal((B, Hkv, len0, hd)))
    k1 = _bf16(RNG.standard_normal((B, Hkv, len1, hd))) if len1 else None
    v1 = _bf16(RNG.standard_normal((B, Hkv, len1, hd))) if len1 else None
    ref = _attn_ref(q, k0, v0, k1, v1)
    t = lambda a: None if a is None else torch.from_numpy(a).to(torch.bfloat16).cuda()
    o = vla.debug_attention(t(q), t(k0), t(v0), t(k1), t(v1))
    torch.cuda.synchronize()
    got = o.float().cpu().numpy()
    # bf16 output and bf16 probabilities: ~2^-8 relative per element
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert rel < 1e-2, rel
    assert np.abs(got - ref).max() < 0.05 * np.abs(ref).max() + 1e-3


@pytest.mark.parametrize("B,Hq,Hkv,Lq,hd,len0,len1", [(1, 4, 4, 8, 64, 80, 8), (2, 4, 2, 80, 64, 80, 0), (1, 2, 1, 3, 136, 70, 2)])
def test_attention_f32(B, Hq, Hkv, Lq, hd, len0, len1):
    import torch
    from paper_2609_12075_amd import vla
    q = RNG.standard_normal((B, Hq, Lq, hd)).astype(np.float32)
    k0 = RNG.standard_normal((B, Hkv, len0, hd)).astype(np.float32)
    v0 = RNG.standard_normal((B, Hkv, len0, hd)).astype(np.float32)
    k1 = RNG.standard_normal((B, Hkv, len1, hd)).astype(np.float32) if len1 else None
    v1 = RNG.standard_normal((B, Hkv, len1, hd)).astype(np.float32) if len1 else None
    ref = _attn_ref(q, k0, v0, k1, v1)
    t = lambda a: None if a is None else torch.from_numpy(a).cuda()
    o = vla.debug_attention(t(q), t(k0), t(v0), t(k1), t(v1))
    torch.cuda.synchronize()
    np.testing.assert_allclose(o.cpu().numpy(), ref, rtol=1e-4, atol=1e-5)


def _placements(words):
    w = words.cpu().numpy().astype(np.uint32).reshape(-1, 2)
    hw, xcc = w[:, 0], w[:, 1] & 0xF
    cu, sh, se = (hw >> 8) & 0xF, (hw >> 12) & 0x1, (hw >> 13) & 0x7
    return set(zip(xcc.tolist(), se.tolist(), sh.tolist(), cu.tolist()))


def test_cu_masked_streams_confine_work():
    import torch
    from paper_2609_12075_amd import vla
    full = _placements(vla.debug_cu_probe(256, 4096, spin=50))
    torch.cuda.synchronize()
    log(f"[cu probe] unrestricted: {len(full)} distinct CUs, XCCs {sorted({p[0] for p in full})}")
    assert len(full) > 200
    for k in (64, 128):
        got = _placements(vla.debug_cu_probe(k, 4096, spin=50))
        top = _placements(vla.debug_cu_probe(256 - k, 4096, spin=50, from_top=True))
        torch.cuda.synchronize()
        per_xcc = {}
        for p in got:
            per_xcc[p[0]] = per_xcc.get(p[0], 0) + 1
        log(f"[cu probe] mask {k}: {len(got)} CUs, per XCC {per_xcc}; top {256 - k}: {len(top)} CUs, "
            f"overlap {len(got & top)}")
        assert len(got) <= k
        assert len(top) <= 256 - k
        assert not (got & top), "low and high masks must be disjoint"


def test_cu_masked_streams_confine_graph_replays():
    """The stages reach the restricted streams as graph replays (captured on an
    unrestricted stream): the mask of the stream the graph is launched on
    still confines the work, and the low and high masks stay disjoint."""
    import torch
    from paper_2609_12075_amd import vla
    for k in (64, 128, 192):
        got = _placements(vla.debug_cu_probe(k, 4096, spin=50, via_graph=True))
        top = _placements(vla.debug_cu_probe(256 - k, 4096, spin=50, from_top=True, via_graph=True))
        direct = _placements(vla.debug_cu_probe(k, 4096, spin=50))
        torch.cuda.synchronize()
        log(f"[cu probe] graph replay, mask {k}: {len(got)} CUs (direct launch {len(direct)}); top {256 - k}: "
            f"{len(top)} CUs, overlap {len(got & top)}")
        assert len(got) <= k and len(top) <= 256 - k
        assert not (got & top)
        assert len(got) >= k // 2, "a replayed graph spreads over the stream's CUs"
        if len(direct) == k:          # the direct launch reached every CU of the mask
            assert got <= direct


def test_sync_probe_barriers_hand_off_data():
    """The grid-barrier probe: every block arrives at every barrier (the
    counter ends at iters x grid, no poll overruns) and each block's reads
    after a barrier see the other block's writes of that round."""
    import torch
    from paper_2609_12075_amd import vla
    grid, iters, words = 64, 12, 1000
    buf = torch.zeros(2 * grid * words, dtype=torch.float32, device="cuda:0")
    sink = torch.zeros(grid * 256, dtype=torch.float32, device="cuda:0")
    ctr = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    err = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    log(f"[sync probe] grid={grid} iters={iters} words={words}")
    vla.debug_sync_probe(2, grid, iters, words, buf=buf, ctr=ctr, err=err, sink=sink)
    torch.cuda.synchronize()
    assert int(ctr.item()) == grid * iters
    assert int(err.item()) == 0
    # thread t of every block sums (i + it) over its strided i < words, it < iters
    t = np.arange(256)
    want = np.array([sum(i + it for it in range(iters) for i in range(tt, words, 256)) for tt in t], dtype=np.float64)
    got = sink.view(grid, 256).cpu().numpy().astype(np.float64)
    assert np.array_equal(got, np.broadcast_to(want, got.shape))
