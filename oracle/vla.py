"""CPU oracle for one batched VLA inference step (test infrastructure).

This is the plain, slow reference that the GPU library is checked against.
Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
it; the product path never imports it.

What is computed (paper Section 2.1 and Fig. 1 describe the two stages; the
paper gives no layer mathematics, so every formula below is the reading
stated in its docstring):

* VLM stage (``prefill``): camera images are cut into patches and embedded
  (optionally through a pre-LN ViT), text ids are embedded, and the
  concatenated prefix runs through a Gemma-style LLM. Each layer's
  post-RoPE keys and values are the per-layer prefix KV cache handed to the
  action stage (Section 2.1: the VLM passes either hidden states or a
  per-layer KV cache to the action model).
* Action stage (``denoise``): a flow-matching Euler loop of N steps
  (Section 2.1: 5-10 diffusion steps, a chunk of 10-50 actions). For the
  joint action expert every layer's action tokens attend over
  [prefix K,V of LLM layer l ; their own K,V]; for the DiT head the action
  tokens use adaLN-modulated self-attention and cross-attention to the
  projected VLM features.

Arithmetic is numpy in fp64 (``dtype`` may be set to float32 for the
self-consistency check). For bf16 models every parameter is first rounded
to bf16 (round to nearest even) and then upcast, so the comparison measures
the GPU kernels' arithmetic, not parameter quantisation. Batch rows are
independent: the oracle loops over rows.

Parity pins for every function live in tests/test_oracle_pins.py.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional

import numpy as np

F64 = np.float64


# ---------------------------------------------------------------------------
# number formats
# ---------------------------------------------------------------------------
def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32.

    bf16 keeps the top 16 bits of the IEEE-754 binary32 pattern. Adding
    0x7FFF plus the lowest kept bit before truncation is round-to-nearest
    with ties to the even neighbour. Inputs here are finite.
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def params(cfg, flat: np.ndarray, dtype=F64) -> Dict[str, np.ndarray]:
    """Name -> parameter tensor in the oracle's precision. bf16 models see
    bf16-rounded parameters."""
    from paper_2609_12075_amd.synth import weight_views, DTYPE_BF16
    src = bf16_round(flat) if cfg.dtype == DTYPE_BF16 else np.asarray(flat, np.float32)
    return {k: v.astype(dtype) for k, v in weight_views(cfg, src).items()}


# ---------------------------------------------------------------------------
# building blocks
# ---------------------------------------------------------------------------
def rmsnorm(x, g, eps):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def layernorm(x, g=None, b=None, eps=1e-6):
    """(x - mean) / sqrt(var + eps), then optional gain and bias."""
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    y = (x - mu) / np.sqrt(var + eps)
    if g is not None:
        y = y * g
    if b is not None:
        y = y + b
    return y


def gelu_tanh(x):
    """tanh approximation of GELU: 0.5 x (1 + tanh(sqrt(2/pi)(x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def silu(x):
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def rope(x, pos, base):
    """Rotary position embedding, half-split form: dimension i is paired with
    i + hd/2 and rotated by angle pos * base^(-2i/hd). x: [..., L, hd]."""
    hd = x.shape[-1]
    half = hd // 2
    inv = base ** (-(2.0 * np.arange(half, dtype=F64)) / hd)
    ang = np.asarray(pos, dtype=F64)[:, None] * inv[None, :]
    c, s = np.cos(ang).astype(x.dtype), np.sin(ang).astype(x.dtype)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q, k, v, scale=None):
    """softmax(q k^T * scale) v with grouped KV heads.

    q: [Hq, Lq, hd]; k, v: [Hkv, Lk, hd]; query head h uses KV head
    floor(h * Hkv / Hq) (contiguous groups). No mask: every query sees every
    key it is given."""
    hq, hkv = q.shape[0], k.shape[0]
    hd = q.shape[-1]
    scale = 1.0 / math.sqrt(hd) if scale is None else scale
    out = np.empty(q.shape[:2] + (v.shape[-1],), dtype=q.dtype)
    for h in range(hq):
        g = (h * hkv) // hq
        s = (q[h] @ k[g].T) * scale
        s = s - s.max(axis=-1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=-1, keepdims=True)
        out[h] = p @ v[g]
    return out


def timestep_embedding(t, dim):
    """[sin(1000 t w_i) ; cos(1000 t w_i)], w_i = 10000^(-i/(dim/2)), i < dim/2."""
    half = dim // 2
    w = 10000.0 ** (-np.arange(half, dtype=F64) / half)
    a = 1000.0 * float(t) * w
    return np.concatenate([np.sin(a), np.cos(a)])


def time_grid(n):
    """Flow time at the start of each Euler step (noise at t = 1, data at
    t = 0): t_k = 1 - k/N, with step dt = -1/N."""
    return [1.0 - k / n for k in range(n)], -1.0 / n


def euler(x0, velocity, n):
    """Explicit Euler integration of dx/dt = velocity(x, t) from t = 1 to 0
    in n uniform steps."""
    ts, dt = time_grid(n)
    x = x0
    for t in ts:
        x = x + dt * velocity(x, t)
    return x


def patchify(img, p):
    """img [3, H, W] -> [(H/p)*(W/p), 3*p*p]: patches in raster order, each
    flattened channel-major then row then column (c, dy, dx)."""
    c, h, w = img.shape
    t = img.reshape(c, h // p, p, w // p, p)          # c, py, dy, px, dx
    return t.transpose(1, 3, 0, 2, 4).reshape((h // p) * (w // p), c * p * p)


def pixel_shuffle(x, g, s):
    """Merge s x s blocks of a g x g token grid (tokens in raster order,
    x [g*g, d]) into (g/s)^2 tokens of width s*s*d: output token I*(g/s) + J
    (raster order over the blocks) concatenates the block's tokens
    (s*I + di, s*J + dj) in row-major (di, dj) order, channels innermost."""
    d = x.shape[-1]
    t = x.reshape(g // s, s, g // s, s, d)            # I, di, J, dj, c
    return t.transpose(0, 2, 1, 3, 4).reshape((g // s) ** 2, s * s * d)


def heads(x, n, hd):
    """[L, n*hd] -> [n, L, hd]."""
    return x.reshape(x.shape[0], n, hd).transpose(1, 0, 2)


def merge(x):
    """[n, L, hd] -> [L, n*hd]."""
    return x.transpose(1, 0, 2).reshape(x.shape[1], -1)


# ---------------------------------------------------------------------------
# VLM stage
# ---------------------------------------------------------------------------
def vit_layer(cfg, W, l, x):
    """Pre-LN ViT block with biases: x += MHA(LN(x)); x += MLP_gelu(LN(x))."""
    p = f"vit.{l}."
    d, nh = cfg.vit_d, cfg.vit_heads
    hd = d // nh
    z = layernorm(x, W[p + "ln1.g"], W[p + "ln1.b"], cfg.norm_eps)
    q = heads(z @ W[p + "wq"] + W[p + "bq"], nh, hd)
    k = heads(z @ W[p + "wk"] + W[p + "bk"], nh, hd)
    v = heads(z @ W[p + "wv"] + W[p + "bv"], nh, hd)
    x = x + merge(attention(q, k, v)) @ W[p + "wo"] + W[p + "bo"]
    z = layernorm(x, W[p + "ln2.g"], W[p + "ln2.b"], cfg.norm_eps)
    return x + gelu_tanh(z @ W[p + "w1"] + W[p + "b1"]) @ W[p + "w2"] + W[p + "b2"]


def image_tokens(cfg, W, pixels_row):
    """pixels [n_img, 3, H, W] -> image tokens [n_img*T, llm_d]: per image,
    patch embedding + position table, the ViT blocks, the final LayerNorm,
    the s x s token merge when the model has one, and the projection to the
    LLM width."""
    dt = W["patch.w"].dtype
    toks = []
    for i in range(cfg.n_img):
        x = patchify(pixels_row[i].astype(dt), cfg.patch) @ W["patch.w"] + W["patch.b"] + W["patch.pos"]
        if cfg.vit_layers > 0:
            for l in range(cfg.vit_layers):
                x = vit_layer(cfg, W, l, x)
            x = layernorm(x, W["vit.lnf.g"], W["vit.lnf.b"], cfg.norm_eps)
            if cfg.pix_shuffle > 1:
                x = pixel_shuffle(x, cfg.patch_grid, cfg.pix_shuffle)
            x = x @ W["vit.proj.w"] + W["vit.proj.b"]
        toks.append(x)
    return np.concatenate(toks, axis=0)


def llm_layer(cfg, W, l, h, pos, need_out=True):
    """Gemma-style block. Returns (h_next, K_l, V_l) with K post-RoPE."""
    p = f"llm.{l}."
    hd = cfg.head_dim
    z = rmsnorm(h, W[p + "ln1.g"], cfg.norm_eps)
    q = rope(heads(z @ W[p + "wq"], cfg.n_q, hd), pos, cfg.rope_base)
    k = rope(heads(z @ W[p + "wk"], cfg.n_kv, hd), pos, cfg.rope_base)
    v = heads(z @ W[p + "wv"], cfg.n_kv, hd)
    if not need_out:
        return None, k, v
    h = h + merge(attention(q, k, v)) @ W[p + "wo"]
    z = rmsnorm(h, W[p + "ln2.g"], cfg.norm_eps)
    h = h + (gelu_tanh(z @ W[p + "wg"]) * (z @ W[p + "wu"])) @ W[p + "wd"]
    return h, k, v


def prefill_row(cfg, W, pixels_row, ids_row, state_row=None):
    """One request through the VLM stage.

    Joint head: returns {"k": [L][n_kv, P, hd], "v": [...]} (the prefix KV of
    every LLM layer). The last layer's attention output and MLP feed nothing
    and are not evaluated.
    DiT head: returns {"kc": [L_dit][P, d_a], "vc": [...], "state": [d_a]}
    (cross-attention K/V of the projected final hidden states, and the
    embedded robot state)."""
    from paper_2609_12075_amd.synth import HEAD_DIT
    h = np.concatenate([image_tokens(cfg, W, pixels_row), W["embed"][np.asarray(ids_row)]], axis=0)
    pos = np.arange(h.shape[0])
    ks, vs = [], []
    dit = cfg.head_kind == HEAD_DIT
    for l in range(cfg.llm_layers):
        last = l == cfg.llm_layers - 1
        h2, k, v = llm_layer(cfg, W, l, h, pos, need_out=dit or not last)
        ks.append(k); vs.append(v)
        h = h2
    if not dit:
        return {"k": ks, "v": vs}
    f = rmsnorm(h, W["llm.lnf.g"], cfg.norm_eps) @ W["vp.w"] + W["vp.b"]
    kc = [f @ W[f"xkv.{l}.wk"] + W[f"xkv.{l}.bk"] for l in range(cfg.act_layers)]
    vc = [f @ W[f"xkv.{l}.wv"] + W[f"xkv.{l}.bv"] for l in range(cfg.act_layers)]
    st = np.zeros(cfg.state_dim, W["state.w"].dtype) if state_row is None else np.asarray(state_row, W["state.w"].dtype)
    return {"kc": kc, "vc": vc, "state": st @ W["state.w"] + W["state.b"]}


# ---------------------------------------------------------------------------
# Action stage
# ---------------------------------------------------------------------------
def joint_velocity(cfg, W, pre, x, t):
    """Velocity of the joint action expert for one request.

    x [H, A] -> v [H, A]. Action tokens get a time-conditioned embedding
    (concat MLP over [action embedding ; sinusoid(t)]), then each layer l
    attends over [prefix K_l, V_l ; own K, V] with RoPE positions P..P+H-1
    in the LLM's head layout."""
    P = pre["k"][0].shape[1]
    hd = cfg.head_dim
    e = x @ W["act.in.w"] + W["act.in.b"]
    phi = timestep_embedding(t, cfg.tdim).astype(e.dtype)
    h = silu(e @ W["act.t1a.w"] + phi @ W["act.t1t.w"] + W["act.t1.b"]) @ W["act.t2.w"] + W["act.t2.b"]
    pos = P + np.arange(cfg.horizon)
    for l in range(cfg.act_layers):
        p = f"act.{l}."
        z = rmsnorm(h, W[p + "ln1.g"], cfg.norm_eps)
        q = rope(heads(z @ W[p + "wq"], cfg.n_q, hd), pos, cfg.rope_base)
        k = rope(heads(z @ W[p + "wk"], cfg.n_kv, hd), pos, cfg.rope_base)
        v = heads(z @ W[p + "wv"], cfg.n_kv, hd)
        kk = np.concatenate([pre["k"][l], k], axis=1)
        vv = np.concatenate([pre["v"][l], v], axis=1)
        h = h + merge(attention(q, kk, vv)) @ W[p + "wo"]
        z = rmsnorm(h, W[p + "ln2.g"], cfg.norm_eps)
        h = h + (gelu_tanh(z @ W[p + "wg"]) * (z @ W[p + "wu"])) @ W[p + "wd"]
    return rmsnorm(h, W["act.lnf.g"], cfg.norm_eps) @ W["act.out.w"] + W["act.out.b"]


def dit_velocity(cfg, W, pre, x, t):
    """Velocity of the DiT action head for one request.

    Tokens [state ; action embeddings] + learned positions; per layer the
    time conditioning c gives (shift, scale, gate) pairs that modulate a
    non-affine LayerNorm before self-attention and before the MLP (adaLN),
    and plain LayerNorm feeds cross-attention to the VLM features."""
    d, nh = cfg.act_d, cfg.act_heads
    hd = d // nh
    eps = cfg.norm_eps
    phi = timestep_embedding(t, cfg.tdim).astype(x.dtype)
    c = silu(phi @ W["dit.t1.w"] + W["dit.t1.b"]) @ W["dit.t2.w"] + W["dit.t2.b"]
    sc = silu(c)
    X = np.concatenate([pre["state"][None, :], x @ W["dit.ain.w"] + W["dit.ain.b"]], axis=0) + W["dit.pos"]
    for l in range(cfg.act_layers):
        p = f"dit.{l}."
        mod = sc @ W[p + "mod.w"] + W[p + "mod.b"]
        sh1, s1, g1, sh2, s2, g2 = np.split(mod, 6)
        z = layernorm(X, eps=eps) * (1.0 + s1) + sh1
        q = heads(z @ W[p + "wq"] + W[p + "bq"], nh, hd)
        k = heads(z @ W[p + "wk"] + W[p + "bk"], nh, hd)
        v = heads(z @ W[p + "wv"] + W[p + "bv"], nh, hd)
        X = X + g1 * (merge(attention(q, k, v)) @ W[p + "wo"] + W[p + "bo"])
        z = layernorm(X, eps=eps)
        q = heads(z @ W[p + "cq.w"] + W[p + "cq.b"], nh, hd)
        o = attention(q, heads(pre["kc"][l], nh, hd), heads(pre["vc"][l], nh, hd))
        X = X + merge(o) @ W[p + "co.w"] + W[p + "co.b"]
        z = layernorm(X, eps=eps) * (1.0 + s2) + sh2
        X = X + g2 * (gelu_tanh(z @ W[p + "w1"] + W[p + "b1"]) @ W[p + "w2"] + W[p + "b2"])
    modf = sc @ W["dit.modf.w"] + W["dit.modf.b"]
    shf, sf = np.split(modf, 2)
    z = layernorm(X, eps=eps) * (1.0 + sf) + shf
    return z[1:] @ W["dit.out.w"] + W["dit.out.b"]


def velocity_fn(cfg):
    from paper_2609_12075_amd.synth import HEAD_DIT
    return dit_velocity if cfg.head_kind == HEAD_DIT else joint_velocity


def denoise_row(cfg, W, pre, noise_row, steps):
    """Euler loop from the noise (t = 1) to the action chunk (t = 0)."""
    vf = velocity_fn(cfg)
    return euler(np.asarray(noise_row, dtype=W["act.out.w" if "act.out.w" in W else "dit.out.w"].dtype),
                 lambda x, t: vf(cfg, W, pre, x, t), steps)


# ---------------------------------------------------------------------------
# batched entry points (loops over independent rows)
# ---------------------------------------------------------------------------
def prefill(cfg, W, pixels, text_ids, state=None) -> List[dict]:
    return [prefill_row(cfg, W, pixels[b], text_ids[b], None if state is None else state[b])
            for b in range(pixels.shape[0])]


def denoise(cfg, W, pre: List[dict], noise, steps) -> np.ndarray:
    return np.stack([denoise_row(cfg, W, pre[b], noise[b], steps) for b in range(noise.shape[0])])


def run(cfg, W, inputs: dict, steps: Optional[int] = None, rows=None):
    """Prefill + denoise for the given rows (default: all). Returns
    (actions [B, H, A], prefix list)."""
    steps = cfg.steps if steps is None else steps
    rows = range(inputs["noise"].shape[0]) if rows is None else rows
    st = inputs.get("state")
    pre = [prefill_row(cfg, W, inputs["pixels"][b], inputs["text_ids"][b], None if st is None else st[b])
           for b in rows]
    act = np.stack([denoise_row(cfg, W, pre[i], inputs["noise"][b], steps) for i, b in enumerate(rows)])
    return act, pre
