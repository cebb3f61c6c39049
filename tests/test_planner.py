"""The projection planner (host logic, no GPU): plans of the model's
projection shapes that were chosen by measurement, and invariants every plan
must satisfy (K covered by non-empty ranges, the split workspace respected,
each kernel kind within the shapes it serves)."""
import itertools

import pytest

from paper_2609_12075_amd import vla

STORE, RESID, GEGLU, QKV, EULER = 0, 1, 2, 3, 4
SPLIT_FLOATS = 16 << 20          # the split-K workspace of a model's stage (floats)


def plan(M, N, K, mode=STORE, **kw):
    return vla.gemm_plan(M, N, K, mode, **kw)


def test_few_rows_long_k_take_k_ranges_on_staged_tiles():
    """The GR00T-like LLM MLP down at batch 1 (296 rows, K = 16384): LDS-staged
    tiles with K ranges, not the register tiles with one K loop per tile."""
    p = plan(296, 2048, 16384, RESID, norm_follows=True)
    assert p["kind"] == 1 and p["splits"] >= 2, p


@pytest.mark.parametrize("M", [256, 512, 768])
def test_vit_mlp_down_two_group_tiles_with_k_ranges(M):
    """The ViT MLP down (K = 4304) at 256-768 rows: two-group K-steps of 128
    with two K ranges."""
    p = plan(M, 1152, 4304, RESID, norm_follows=True)
    assert (p["kind"], p["splits"], p["bk"], p["kg"]) == (4, 2, 128, 2), p


def test_k_past_4096_needs_k_ranges_on_two_group_tiles():
    """At 1024 rows the same product would take one 34-step range on the
    two-group tiles (measured slower): it stays on the staged tiles."""
    p = plan(1024, 1152, 4304, RESID, norm_follows=True)
    assert p["kind"] != 4, p


def test_small_m_kernel_for_one_action_chunk():
    p = plan(50, 8192, 1024, GEGLU, out_bf16=True, rms=True)
    assert p["kind"] == 2 and p["splits"] == 1, p


def test_large_tiles_for_the_pi0_gate_up_at_batch_8():
    p = plan(6528, 32768, 2048, GEGLU, out_bf16=True)
    assert (p["kind"], p["tile_n"], p["tile_m"], p["splits"]) == (3, 256, 256, 1), p


@pytest.mark.parametrize("M,N,K", [(800, 3840, 720), (50, 2560, 1024), (400, 2560, 1024), (3000, 5120, 960)])
def test_folded_norm_never_splits_k(M, N, K):
    p = plan(M, N, K, GEGLU if N % 2 == 0 else STORE, out_bf16=True, rms=True)
    assert p["splits"] == 1 and p["kind"] in (1, 2, 4), p


MS = [1, 17, 50, 64, 65, 100, 256, 296, 512, 768, 1024, 1632, 4096, 6528]
NS = [16, 720, 1152, 2048, 3840, 8192, 32768]
KS = [64, 720, 1152, 2048, 4304, 8192, 16384]


@pytest.mark.parametrize("mode", [STORE, RESID])
def test_plan_invariants(mode):
    for M, N, K in itertools.product(MS, NS, KS):
        p = plan(M, N, K, mode, norm_follows=mode == RESID)
        s, ks, kind = p["splits"], p["ksplit"], p["kind"]
        where = (M, N, K, mode, p)
        assert kind in (0, 1, 2, 3, 4), where
        assert 1 <= s <= 16 and ks > 0, where
        assert s * ks >= K and (s - 1) * ks < K, where            # K covered, no empty range
        if s > 1:
            assert ks % p["bk"] == 0, where                        # ranges end on K-step boundaries
            assert s * M * ((N + 3) & ~3) <= SPLIT_FLOATS, where   # partials fit the workspace
        if kind == 2:
            assert M <= 64 and s == 1, where
        if kind == 3:
            assert s == 1 and p["tile_n"] == 256 and p["tile_m"] in (224, 256) and M >= 256 and K >= 512, where
        if kind == 4:
            assert M <= 1024 and p["bk"] == 128 and p["kg"] == 2, where
            assert K <= 4096 or s > 1, where


def test_bad_arguments_are_rejected():
    assert vla.lib().vla_debug_gemm_plan(0, 16, 64, 0, 0, 0, 0, (vla.ctypes.c_int * 8)()) == vla.VLA_EINVAL
    assert vla.lib().vla_debug_gemm_plan(16, 15, 64, GEGLU, 1, 0, 0, (vla.ctypes.c_int * 8)()) == vla.VLA_EINVAL
    assert vla.lib().vla_debug_gemm_plan(16, 16, 60, 0, 0, 0, 0, (vla.ctypes.c_int * 8)()) == vla.VLA_EINVAL
    assert vla.lib().vla_debug_gemm_plan(16, 16, 64, RESID, 0, 1, 0, (vla.ctypes.c_int * 8)()) == vla.VLA_EINVAL
