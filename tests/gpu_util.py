"""Helpers for the GPU tests: build models, run the library's stages on seeded
inputs, and evaluate the oracle on the same inputs."""
import functools
import sys

import numpy as np

from oracle import vla as O
from paper_2609_12075_amd import synth

_models = {}
_weights = {}


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def weights(cfg):
    if cfg not in _weights:
        _weights[cfg] = synth.make_weights(cfg)
    return _weights[cfg]


def model(cfg):
    from paper_2609_12075_amd import vla
    if cfg not in _models:
        log(f"[gpu] creating model {cfg.name}")
        _models[cfg] = vla.Model(cfg, weights(cfg), device=0)
    return _models[cfg]


@functools.lru_cache(maxsize=8)
def oracle_params(cfg):
    return O.params(cfg, weights(cfg))


def to_dev(inputs):
    import torch
    return {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in inputs.items()}


def run(cfg, inputs, steps=None, graphs=True, m=None):
    """Prefill + denoise on the GPU. Returns (actions np [B,H,A], kv bytes tensor)."""
    import torch
    steps = cfg.steps if steps is None else steps
    m = model(cfg) if m is None else m
    m.set_graphs(graphs)
    d = to_dev(inputs)
    B = inputs["noise"].shape[0]
    kv = m.alloc_kv(B)
    act = torch.empty_like(d["noise"])
    log(f"[gpu] {cfg.name} B={B} steps={steps} graphs={graphs}")
    m.prefill(B, d["pixels"], d["text_ids"], kv, state=d.get("state"))
    m.denoise(B, kv, d["noise"], steps, act)
    torch.cuda.synchronize()
    return act.cpu().numpy(), kv


def kv_arrays(cfg, kv, B):
    """Decode the library's KV bundle (documented layout) into numpy fp64."""
    import torch
    dt = torch.bfloat16 if cfg.dtype == synth.DTYPE_BF16 else torch.float32
    flat = kv.view(dt).float().cpu().numpy().astype(np.float64)
    P = cfg.prefix_len
    if cfg.head_kind == synth.HEAD_JOINT:
        return flat.reshape(cfg.llm_layers, 2, B, cfg.n_kv, P, cfg.head_dim)
    n = B * P * cfg.act_layers * 2 * cfg.act_d
    return flat[:n].reshape(B, P, cfg.act_layers, 2, cfg.act_d), flat[n:].reshape(B, cfg.act_d)


def rel_l2(a, b):
    return float(np.linalg.norm(np.asarray(a, np.float64) - b) / np.linalg.norm(b))


def oracle_run(cfg, inputs, steps=None, rows=None):
    return O.run(cfg, oracle_params(cfg), inputs, steps=steps, rows=rows)


def check_chunk(got, ref, noise, tol, what=""):
    """Assert the parity bounds on action chunks [.., H, A]:
    rel-L2 of the actions and of the displacement (actions - noise; the
    noise itself is exact and would dilute errors) within tol, and no element
    off by more than 5*tol times the RMS of the reference displacement.
    Returns (actions rel-L2, displacement rel-L2, max element error / RMS)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    noise = np.asarray(noise, np.float64)
    assert np.isfinite(got).all(), what
    r = rel_l2(got, ref)
    rd = rel_l2(got - noise, ref - noise)
    rms = float(np.sqrt(np.mean((ref - noise) ** 2)))
    me = float(np.abs(got - ref).max()) / rms
    log(f"[parity] {what}: actions rel-L2 {r:.3e}, displacement rel-L2 {rd:.3e}, max elem err / rms {me:.3e}")
    assert r <= tol, (what, r)
    assert rd <= tol, (what, rd)
    assert me <= 5 * tol, (what, me)
    return r, rd, me


def drop_model(cfg):
    """Destroy a cached model (and forget its parameters) to free memory."""
    m = _models.pop(cfg, None)
    if m is not None:
        m.close()
    _weights.pop(cfg, None)
